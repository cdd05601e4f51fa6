// bf16 GQA link attention on gfx950 matrix cores, head dim 128.
//
// Workgroup: 4 waves x 32 rows = 128 rows of one (request, kv head), where a
// row is (query token, query head of the GQA group): the group's query heads
// share every K/V byte the workgroup stages. Keys are walked in 64-key tiles:
// the request's linked chunks in link order (Sec. 4.2: concatenated along
// the document axis, no mask), then its own KV (Sec. 4.1: causal mask,
// bottom-right aligned).
//
// Per tile and wave:
//   S^T[64 keys][32 rows] = K . Q^T        16 x v_mfma_f32_32x32x16_bf16
//   online softmax on S^T (each lane holds one row's 32 scores)
//   O^T[128][32 rows]    += V^T . P^T      16 x v_mfma_f32_32x32x16_bf16
// K and V^T tiles are staged in LDS, double-buffered, with 16-byte chunks
// XOR-swizzled so the fragment reads are bank-conflict free. The store keeps
// V transposed per chunk, so a V^T tile is 128 rows of 128 contiguous bytes.
// The M index of the QK^T product is permuted (key row pi(m) feeds M index m)
// so that the scores a lane receives for a 16-key PV step are 8 consecutive
// keys: P^T then feeds the PV product straight from registers, and the V^T
// fragment for those keys is one 16-byte LDS read.
//
// Softmax: log2 domain (scale * log2 e applied by FMA), row max through one
// cross-half lane swap, and a lazy rescale: the running max used for the
// exponentials is only moved when a row's max grows by more than 8 (p stays
// <= 2^8), which skips the accumulator rescale on almost every tile. The row
// sums are kept per lane half and added once at the end.
#include "pic_internal.hpp"

namespace pic {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kD = 128;
constexpr int kWaves = 4;
constexpr int kRowsPerWave = 32;
constexpr int kRows = kWaves * kRowsPerWave;
constexpr float kLazy = 8.0f;

struct Smem {
  uint4 k[2][kTile * 16];   // [buf][key][16 chunks of 8 d], chunk c at c ^ (key & 15)
  uint4 vt[2][kD * 8];      // [buf][dv][8 chunks of 8 keys], chunk c at c ^ (dv & 7)
};

__device__ __forceinline__ int k_slot(int key, int c) { return key * 16 + (c ^ (key & 15)); }
__device__ __forceinline__ int v_slot(int dv, int c) { return dv * 8 + (c ^ (dv & 7)); }

// Key row that feeds M index m of the QK^T product (see the file comment).
__device__ __forceinline__ int key_of_m(int m) {
  const int a = m >> 3, gg = (m >> 2) & 1, c = m & 3;
  return (a >> 1) * 16 + gg * 8 + (a & 1) * 4 + c;
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) {
  return __builtin_bit_cast(bf16x8, u);
}

// One tile's worth of global loads, held in registers between the load and
// the LDS store so the loads overlap the previous tile's math.
struct TileRegs {
  uint4 k[4];
  uint4 v[4];
};

struct TileSrc {
  bool own;
  int nvalid;     // valid keys in the tile
  int j0;         // own-key index of the tile's first key (own tiles)
  const uint16_t *kbase;   // doc: first K row of the tile; own: k_self row 0 of the request
  const uint16_t *vbase;   // doc: V^T row 0 at the tile's first key; own: v_self row 0
  int64_t vstride;         // doc: elements between V^T rows (= lp); own: unused
};

__device__ __forceinline__ TileSrc resolve_tile(const LinkParams &p, const ReqEntry &R, int kvh,
                                                int t, int &li) {
  TileSrc s;
  const uint16_t *pool = (const uint16_t *)p.pool;
  if (t < R.doc_tiles) {
    while (p.links[R.link0 + li].tile0 + p.links[R.link0 + li].lp / kTile <= t) ++li;
    const LinkEntry E = p.links[R.link0 + li];
    const int tt = t - E.tile0;
    s.own = false;
    s.nvalid = min(kTile, E.len - tt * kTile);
    s.j0 = 0;
    s.kbase = pool + E.k_off + ((int64_t)kvh * E.lp + tt * kTile) * kD;
    s.vbase = pool + E.v_off + (int64_t)kvh * kD * E.lp + tt * kTile;
    s.vstride = E.lp;
  } else {
    s.own = true;
    s.j0 = (t - R.doc_tiles) * kTile;
    s.nvalid = min(kTile, R.ls - s.j0);
    s.kbase = (const uint16_t *)p.k_self + ((int64_t)R.s0 * p.n_kv_heads + kvh) * kD;
    s.vbase = (const uint16_t *)p.v_self + ((int64_t)R.s0 * p.n_kv_heads + kvh) * kD;
    s.vstride = 0;
  }
  return s;
}

__device__ __forceinline__ void load_tile(const TileSrc &s, int n_kv_heads, TileRegs &r) {
  const int tid = threadIdx.x;
  if (!s.own) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + 256 * u;          // 1024 chunks: key = idx/16, c = idx%16
      r.k[u] = ((const uint4 *)s.kbase)[idx];
      const int e = idx >> 3, c = idx & 7;    // 1024 chunks: dv = idx/8, keys c*8..
      r.v[u] = *(const uint4 *)(s.vbase + (int64_t)e * s.vstride + c * 8);
    }
  } else {
    const int64_t rs = (int64_t)n_kv_heads * kD;   // elements between own rows
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + 256 * u;
      const int key = idx >> 4, c = idx & 15;
      uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
      if (key < s.nvalid) {
        kv = *(const uint4 *)(s.kbase + (int64_t)(s.j0 + key) * rs + c * 8);
        vv = *(const uint4 *)(s.vbase + (int64_t)(s.j0 + key) * rs + c * 8);
      }
      r.k[u] = kv;
      r.v[u] = vv;       // 8 value dims (c*8 ..) of one key
    }
  }
}

__device__ __forceinline__ void store_tile(const TileSrc &s, const TileRegs &r, Smem &sm, int buf) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int idx = tid + 256 * u;
    sm.k[buf][k_slot(idx >> 4, idx & 15)] = r.k[u];
  }
  if (!s.own) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + 256 * u;
      sm.vt[buf][v_slot(idx >> 3, idx & 7)] = r.v[u];
    }
  } else {
    // token-major own values: scatter the 8 dims of one key into V^T
    uint16_t *vt16 = (uint16_t *)sm.vt[buf];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = tid + 256 * u;
      const int key = idx >> 4, c = idx & 15;
      const uint16_t *vals = (const uint16_t *)&r.v[u];
#pragma unroll
      for (int x = 0; x < 8; ++x) {
        const int dv = c * 8 + x;
        vt16[v_slot(dv, key >> 3) * 8 + (key & 7)] = vals[x];
      }
    }
  }
}

__global__ __launch_bounds__(256, 1) void link_mfma_d128_kernel(LinkParams p) {
  __shared__ Smem sm;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 31, g = lane >> 5;

  // XCD-aware work mapping: consecutive blocks go round-robin to the 8 XCDs;
  // all row blocks of one (request, kv head) land on the same XCD (same L2)
  // and are dispatched back to back. Heaviest requests first.
  const int lin = blockIdx.x;
  const int xcd = lin & 7, j = lin >> 3;
  const int grp = xcd + 8 * (j / p.nrb);
  const int rb = j % p.nrb;
  const int split = blockIdx.y;
  if (grp >= p.batch * p.n_kv_heads) return;
  const int req_i = p.order[grp / p.n_kv_heads];
  const int kvh = grp % p.n_kv_heads;
  const ReqEntry R = p.reqs[req_i];
  const int group = p.group;
  const int nrows = R.lq * group;
  const int row0 = rb * kRows;
  if (row0 >= nrows) return;
  const int t_begin = (int)((int64_t)R.tiles * split / p.num_splits);
  const int t_end = (int)((int64_t)R.tiles * (split + 1) / p.num_splits);

  // This lane's row.
  const int row = row0 + wave * kRowsPerWave + n;
  const bool rvalid = row < nrows;
  const int qi = rvalid ? row / group : 0;
  const int qh = kvh * group + (rvalid ? row % group : 0);
  const int lim = rvalid ? qi + R.ls - R.lq : -1;     // last visible own key
  const int64_t orow = (int64_t)(R.q0 + qi) * p.n_q_heads + qh;

  // Q fragments: d = step*16 + g*8 + (0..7)
  bf16x8 qf[8];
  {
    const uint4 *qrow = (const uint4 *)((const uint16_t *)p.q + orow * kD);
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (rvalid) v = qrow[s * 2 + g];
      qf[s] = as_bf16x8(v);
    }
  }

  f32x16 o[4];
#pragma unroll
  for (int d = 0; d < 4; ++d)
#pragma unroll
    for (int x = 0; x < 16; ++x) o[d][x] = 0.f;
  float m_used = -INFINITY, lsum = 0.f;
  const float c = p.scale_log2;

  int li = 0;
  TileRegs regs;
  TileSrc cur = resolve_tile(p, R, kvh, t_begin < t_end ? t_begin : 0, li);
  if (t_begin < t_end) {
    load_tile(cur, p.n_kv_heads, regs);
    store_tile(cur, regs, sm, 0);
  }
  __syncthreads();

  const int krow0 = key_of_m(n);      // key row feeding this lane's M index, block 0
  for (int t = t_begin; t < t_end; ++t) {
    const int buf = (t - t_begin) & 1;
    TileSrc nxt;
    const bool more = t + 1 < t_end;
    if (more) {
      nxt = resolve_tile(p, R, kvh, t + 1, li);
      load_tile(nxt, p.n_kv_heads, regs);
    }

    // ---- S^T = K Q^T : two 32-key blocks
    f32x16 s[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
#pragma unroll
      for (int x = 0; x < 16; ++x) s[b][x] = 0.f;
      const int krow = b * 32 + krow0;
#pragma unroll
      for (int st = 0; st < 8; ++st) {
        const bf16x8 kf = as_bf16x8(sm.k[buf][k_slot(krow, st * 2 + g)]);
        s[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[st], s[b], 0, 0, 0);
      }
    }

    // ---- masking (only on ragged or own tiles)
    // s[b][x] is the score of key b*32 + (x>>3)*16 + g*8 + (x&7) for this row
    if (cur.own || cur.nvalid < kTile) {
      const int kl = cur.own ? lim - cur.j0 : kTile;     // visible iff key <= kl
      const int kv = cur.nvalid;
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int x = 0; x < 16; ++x) {
          const int key = b * 32 + (x >> 3) * 16 + g * 8 + (x & 7);
          if (key >= kv || key > kl) s[b][x] = -INFINITY;
        }
    }

    // ---- online softmax (log2 domain, lazy rescale)
    float tmax = -INFINITY;
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int x = 0; x < 16; x += 2) tmax = fmaxf(fmaxf(tmax, s[b][x]), s[b][x + 1]);
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
    const float mnew = fmaxf(m_used, tmax * c);
    if (__any(mnew > m_used + kLazy)) {
      const float alpha = mnew == m_used ? 1.f : __builtin_amdgcn_exp2f(m_used - mnew);
      m_used = mnew;
      lsum *= alpha;
#pragma unroll
      for (int d = 0; d < 4; ++d)
#pragma unroll
        for (int x = 0; x < 16; ++x) o[d][x] *= alpha;
    }
    const float neg_m = m_used == -INFINITY ? 0.f : -m_used;
    bf16x8 pf[4];
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2)
#pragma unroll
        for (int x = 0; x < 8; ++x) {
          const float pv = __builtin_amdgcn_exp2f(__builtin_fmaf(s[b][h2 * 8 + x], c, neg_m));
          lsum += pv;
          pf[b * 2 + h2][x] = (__bf16)pv;
        }

    // ---- O^T += V^T P^T : 4 value blocks x 4 key steps
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        const bf16x8 vf = as_bf16x8(sm.vt[buf][v_slot(d * 32 + n, ks * 2 + g)]);
        o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[ks], o[d], 0, 0, 0);
      }
    }

    if (more) {
      store_tile(nxt, regs, sm, buf ^ 1);
      cur = nxt;
    }
    __syncthreads();
  }

  // ---- epilogue: O^T[dv][row] with dv = d*32 + (x>>2)*8 + g*4 + (x&3)
  const float ltot = lsum + __shfl_xor(lsum, 32);
  if (!rvalid) return;
  const int total_rows = p.total_q * p.n_q_heads;
  if (p.num_splits == 1) {
    const float inv = ltot > 0.f ? 1.f / ltot : 0.f;
    uint16_t *out = (uint16_t *)p.out + orow * kD;
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int dv = d * 32 + jj * 8 + g * 4;
        __bf16 v4[4];
#pragma unroll
        for (int x = 0; x < 4; ++x) v4[x] = (__bf16)(o[d][jj * 4 + x] * inv);
        *(uint2 *)(out + dv) = __builtin_bit_cast(uint2, v4);
      }
    if (p.lse && g == 0)
      p.lse[orow] = ltot > 0.f ? (m_used + log2f(ltot)) * 0.69314718055994531f : -INFINITY;
  } else {
    const int64_t prow = (int64_t)split * total_rows + orow;
    float *po = p.part_o + prow * kD;
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int dv = d * 32 + jj * 8 + g * 4;
        *(float4 *)(po + dv) =
            make_float4(o[d][jj * 4], o[d][jj * 4 + 1], o[d][jj * 4 + 2], o[d][jj * 4 + 3]);
      }
    if (g == 0) {
      p.part_m[prow] = ltot > 0.f ? m_used : -INFINITY;
      p.part_l[prow] = ltot;
    }
  }
}

}  // namespace

int mfma_d128_rows_per_block() { return kRows; }

hipError_t launch_link_mfma_d128(const LinkParams &p, hipStream_t st, const char **name) {
  *name = "link_mfma_d128_kernel";
  dim3 grid(p.n_groups * p.nrb, p.num_splits);
  hipLaunchKernelGGL(link_mfma_d128_kernel, grid, dim3(256), 0, st, p);
  return hipGetLastError();
}

}  // namespace pic
