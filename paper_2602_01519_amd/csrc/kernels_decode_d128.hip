// bf16 GQA link attention for decode-shaped requests on gfx950, head dim 128.
//
// Decode reads every linked key once per query token (a generated token is a
// query token, Sec. 4), so the work is a stream over the request's
// concatenated chunk KV (Sec. 4.2) bounded by HBM bandwidth, not by math.
// Each wave owns one work item (request, kv head, key split) and streams its
// key range in 32-key tiles straight from HBM into registers, already in the
// operand layout of v_mfma_f32_16x16x32_bf16:
//   S^T[32 keys][16 cols] = K . Q^T    2 key blocks x 4 d steps  (8 MFMAs)
//   O^T[128][16 cols]    += V^T . P^T  8 value blocks x 1 step   (8 MFMAs)
// The 16 columns are the work item's rows (query token x GQA head, at most
// 16; unused columns are zero). The next tile's 16 x 16-byte loads per lane
// are in flight while the current tile is computed (register double
// buffering, loop unrolled by two), so each wave keeps 16 KB in flight.
//
// Row permutation: M index m of key block b reads key row 8*(m/4) + 4*b +
// m%4, so after QK^T lane l holds the scores of keys 8*(l/16) + 0..7 (four
// per block) for column l%16 -- exactly the 8 keys its PV operand needs, and
// the matching V^T operand is one 16-byte load of those 8 keys.
//
// Softmax: log2 domain, exact running max per tile (column max over the 4
// lane groups by two lane swaps), unnormalised partial (o, m, l) written per
// split and merged by the log-sum-exp combine (or normalised here when the
// range is not split).
#include "pic_internal.hpp"

namespace pic {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kD = 128;
constexpr int kT = 32;            // keys per decode tile
constexpr int kCols = 16;         // MFMA N: rows of a work item
constexpr int kWaves = 4;

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ const char *uni(const void *p) {
  const uint64_t u = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
  return (const char *)(((uint64_t)hi << 32) | lo);
}

// Reduction over the 4 lane groups (l, l^16, l^32, l^48) of a column.
__device__ __forceinline__ float col_max(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float col_sum(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// One tile's operands as loaded: K rows for the 2 key blocks x 4 d steps,
// V^T rows for the 8 value blocks.
struct Tile {
  uint4 k[8];
  uint4 v[8];
};

// Uniform facts of the tile being loaded / computed.
struct TileInfo {
  const char *k;    // first K row of the tile, kv head applied (bytes)
  const char *v;    // the tile's V^T panel, kv head applied
  int lp;           // padded tokens of the link
  int nvalid;       // valid keys in the tile
  int j0;           // key index of the tile's first key within its link
  int own;          // own-KV tile (causal mask)
};

struct Cursor {
  const LinkEntry *links;  // the request's links
  int li;                  // current link
  int kvh;
  int doc_tiles32;         // 32-key tiles over the documents
};

// Tile t (32-key units, t only grows) of the request.
__device__ __forceinline__ TileInfo tile_info(Cursor &c, int t) {
  for (;;) {
    const LinkEntry &e = c.links[c.li];
    const int tile0 = uni(e.tile0) * (kTile / kT), lp = uni(e.lp);
    if (t < tile0 + (uni(e.len) + kTile - 1) / kTile * (kTile / kT)) {
      const int tt = t - tile0;
      TileInfo r;
      r.lp = lp;
      r.nvalid = min(kT, uni(e.len) - tt * kT);
      r.j0 = tt * kT;
      r.own = t >= c.doc_tiles32;
      r.k = uni(e.k) + ((int64_t)c.kvh * lp + tt * kT) * kD * 2;
      r.v = uni(e.v) + ((int64_t)c.kvh * kD * lp + tt * kT * kD) * 2;   // the tile's V^T panel
      return r;
    }
    ++c.li;
  }
}

// Per-lane byte offsets of the tile's loads: K block b, step s: key row
// krow_b, d = 32 s + 8 (l/16); V block b: value row 16 b + l%16 of the
// tile's 32-key panel, keys 8 (l/16) .. +7 (two lanes of a 16-lane group
// read one 128-byte line).
// The keys are read once per call: the loads carry the nontemporal hint
// (streaming, measured 11% faster on a plain read stream).
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) const u32x4 *global_u32x4;
__device__ __forceinline__ uint4 load_nt(const char *p) {
  const u32x4 w = __builtin_nontemporal_load((global_u32x4)p);
  return make_uint4(w.x, w.y, w.z, w.w);
}

__device__ __forceinline__ void load_tile(const TileInfo &r, int lane, Tile &x) {
  const int grp = lane >> 4, m = lane & 15;
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int krow = 8 * (m >> 2) + 4 * b + (m & 3);
#pragma unroll
    for (int s = 0; s < 4; ++s)
      x.k[b * 4 + s] = load_nt(r.k + (uint32_t)((krow * kD + 32 * s + 8 * grp) * 2));
  }
#pragma unroll
  for (int b = 0; b < 8; ++b) x.v[b] = load_nt(r.v + (uint32_t)((16 * b + m) * kT * 2 + 16 * grp));
}

struct State {
  f32x4 o[8];       // O^T blocks: value rows 16 b + 4 (l/16) + i, column l%16
  float m, l;       // running max (log2 domain, per column) and this lane's partial sum
};

__device__ __forceinline__ void compute_tile(const Tile &x, const TileInfo &r,
                                             const bf16x8 (&qf)[4], State &st, int lane,
                                             int lim, float sc) {
  f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(x.k[s]), qf[s], s0, 0, 0, 0);
    s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(x.k[4 + s]), qf[s], s1, 0, 0, 0);
  }
  // s0[i]: key 8 (l/16) + i, s1[i]: key 8 (l/16) + 4 + i, column l%16
  const int kbase = 8 * (lane >> 4);
  if (r.own || r.nvalid < kT) {
    const int kl = (r.own ? min(lim - r.j0, r.nvalid - 1) : r.nvalid - 1) - kbase;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (i > kl) s0[i] = -INFINITY;
      if (4 + i > kl) s1[i] = -INFINITY;
    }
  }
  float tmax = fmaxf(fmaxf(fmaxf(s0[0], s0[1]), fmaxf(s0[2], s0[3])),
                     fmaxf(fmaxf(s1[0], s1[1]), fmaxf(s1[2], s1[3])));
  tmax = col_max(tmax);
  const float mnew = fmaxf(st.m, tmax * sc);
  if (mnew > st.m) {             // per lane: rescale this column's state
    const float alpha = __builtin_amdgcn_exp2f(st.m - mnew);   // 0 when st.m = -inf
    st.l *= alpha;
#pragma unroll
    for (int b = 0; b < 8; ++b) st.o[b] *= alpha;
    st.m = mnew;
  }
  const float neg_m = st.m == -INFINITY ? 0.f : -st.m;
  bf16x8 pf;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    pf[i] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s0[i], sc, neg_m));
    pf[4 + i] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s1[i], sc, neg_m));
  }
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
  for (int i = 0; i < 8; i += 2) {
    const bf16x2 pp = {pf[i], pf[i + 1]};
    st.l = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, st.l, false);
  }
#pragma unroll
  for (int b = 0; b < 8; ++b)
    st.o[b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(x.v[b]), pf, st.o[b], 0, 0, 0);
}

__global__ __launch_bounds__(256, 2) void link_decode_d128_kernel(LinkParams p) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // work item: (group = request x kv head, split); waves of a block take
  // consecutive splits of one group
  const int item = blockIdx.x * kWaves + wave;
  const int S = p.num_splits;
  const int grp = item / S, split = item % S;
  if (grp >= p.batch * p.n_kv_heads) return;
  const int req_i = p.order[grp / p.n_kv_heads];
  const int kvh = grp % p.n_kv_heads;
  const ReqEntry R = p.reqs[req_i];
  const int group = p.group;
  const int nrows = R.lq * group;                 // <= kCols (checked by the planner)
  const int tiles = R.tiles * (kTile / kT);
  const int t_begin = (int)((int64_t)tiles * split / S);
  const int t_end = (int)((int64_t)tiles * (split + 1) / S);

  Cursor cur;
  cur.links = p.links + R.link0;
  cur.li = 0;
  cur.kvh = kvh;
  cur.doc_tiles32 = R.doc_tiles * (kTile / kT);

  // This lane's column (row of the work item).
  const int col = lane & 15;
  const bool cvalid = col < nrows;
  const int qi = cvalid ? col / group : 0;
  const int qh = kvh * group + (cvalid ? col % group : 0);
  const int lim = cvalid ? qi + R.ls - R.lq : -1;
  const int64_t orow = (int64_t)(R.q0 + qi) * p.n_q_heads + qh;

  Tile ta, tb;
  TileInfo ia{}, ib{};
  if (t_begin < t_end) {
    ia = tile_info(cur, t_begin);
    load_tile(ia, lane, ta);
  }
  // Q operand: Q^T[d = 32 s + 8 (l/16) + 0..7][col]
  bf16x8 qf[4];
  {
    const uint4 *qrow = (const uint4 *)((const uint16_t *)p.q + orow * kD);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (cvalid) v = qrow[4 * s + (lane >> 4)];
      qf[s] = as_bf16x8(v);
    }
  }
  State st;
#pragma unroll
  for (int b = 0; b < 8; ++b) st.o[b] = f32x4{0.f, 0.f, 0.f, 0.f};
  st.m = -INFINITY;
  st.l = 0.f;
  const float sc = p.scale_log2;

  for (int t = t_begin; t < t_end; t += 2) {
    if (t + 1 < t_end) {
      ib = tile_info(cur, t + 1);
      load_tile(ib, lane, tb);
    }
    compute_tile(ta, ia, qf, st, lane, lim, sc);
    if (t + 1 >= t_end) break;
    if (t + 2 < t_end) {
      ia = tile_info(cur, t + 2);
      load_tile(ia, lane, ta);
    }
    compute_tile(tb, ib, qf, st, lane, lim, sc);
  }

  const float ltot = col_sum(st.l);
  if (!cvalid) return;
  // lane l holds value rows 16 b + 4 (l/16) + i of column l%16
  const int r4 = 4 * (lane >> 4);
  const int total_rows = p.total_q * p.n_q_heads;
  if (S == 1) {
    const float inv = ltot > 0.f ? 1.f / ltot : 0.f;
    uint16_t *out = (uint16_t *)p.out + orow * kD;
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      __bf16 v4[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) v4[i] = (__bf16)(st.o[b][i] * inv);
      *(uint2 *)(out + 16 * b + r4) = __builtin_bit_cast(uint2, v4);
    }
    if (p.lse && lane < 16)
      p.lse[orow] = ltot > 0.f ? (st.m + log2f(ltot)) * 0.69314718055994531f : -INFINITY;
  } else {
    const int64_t prow = (int64_t)split * total_rows + orow;
    float *po = p.part_o + prow * kD;
#pragma unroll
    for (int b = 0; b < 8; ++b)
      *(float4 *)(po + 16 * b + r4) = make_float4(st.o[b][0], st.o[b][1], st.o[b][2], st.o[b][3]);
    if (lane < 16) {
      p.part_m[prow] = ltot > 0.f ? st.m : -INFINITY;
      p.part_l[prow] = ltot;
    }
  }
}

}  // namespace

int decode_d128_max_rows() { return kCols; }

hipError_t launch_link_decode_d128(const LinkParams &p, hipStream_t st, const char **name) {
  *name = "link_decode_d128_kernel";
  const int64_t items = (int64_t)p.batch * p.n_kv_heads * p.num_splits;
  dim3 grid((unsigned)((items + kWaves - 1) / kWaves));
  hipLaunchKernelGGL(link_decode_d128_kernel, grid, dim3(64 * kWaves), 0, st, p);
  return hipGetLastError();
}

}  // namespace pic
