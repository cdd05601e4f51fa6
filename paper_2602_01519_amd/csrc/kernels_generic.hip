// Store layout transforms, the gather test hook, the generic vector-ALU link
// attention and the split-K log-sum-exp combine. gfx950 only.
#include "pic_internal.hpp"

#include <cmath>
#include <type_traits>

namespace pic {
namespace {

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// fp32 -> bf16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint16_t bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ uint16_t from_f32<uint16_t>(float x) { return bf16_rne(x); }

// ---------------------------------------------------------------------------
// Store layout transforms (the compile-side put; not on the link path).

// src token-major [n][heads][width] -> dst [heads][lp][width], rows >= n zero.
// width * esz is a multiple of 16, so every row is a whole number of uint4.
__global__ void put_rows_kernel(const uint4 *__restrict__ src, uint4 *__restrict__ dst,
                                int64_t n, int32_t lp, int32_t heads, int32_t vpr) {
  const int64_t total = (int64_t)heads * lp * vpr;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t h = idx / ((int64_t)lp * vpr);
    const int64_t rem = idx - h * lp * vpr;
    const int64_t t = rem / vpr;
    const int64_t c = rem - t * vpr;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (t < n) v = src[(t * heads + h) * vpr + c];
    dst[idx] = v;
  }
}

// src token-major [n][heads][width] -> dst [heads][lp / 32][width][32]
// (32-token panels, tokens contiguous), columns >= n zero. 64x64 tiles
// through LDS so both the read and the write are coalesced.
template <typename E>
__global__ void put_transposed_kernel(const E *__restrict__ src, E *__restrict__ dst, int64_t n,
                                      int32_t lp, int32_t heads, int32_t width) {
  __shared__ E tile[64][65];
  const int64_t t0 = (int64_t)blockIdx.x * 64;
  const int e0 = blockIdx.y * 64;
  const int h = blockIdx.z;
  for (int i = threadIdx.x; i < 64 * 64; i += blockDim.x) {
    const int tl = i >> 6, el = i & 63;
    const int64_t t = t0 + tl;
    const int e = e0 + el;
    E v = E(0);
    if (t < n && e < width) v = src[(t * heads + h) * width + e];
    tile[tl][el] = v;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < 64 * 64; i += blockDim.x) {
    const int el = i >> 6, tl = i & 63;
    const int64_t t = t0 + tl;
    const int e = e0 + el;
    if (e < width && t < lp) dst[vt_offset(h, e, t, lp, width)] = tile[tl][el];
  }
}

// ---------------------------------------------------------------------------
// Address resolution shared by the gather hook and the attention kernels.

// Link holding document token j of a request (links sorted by tok0).
__device__ __forceinline__ int find_link(const LinkEntry *links, int n, int64_t j) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (links[mid].tok0 <= j) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Key row `row` of head `head` in a slot (GQA head-major K; MLA has one head).
template <typename E>
__device__ __forceinline__ const E *key_row(const LinkEntry &e, int head, int row, int d_k) {
  return (const E *)e.k + ((int64_t)head * e.lp + row) * d_k;
}
// Value dim `dim` of token `row` of head `head` (GQA transposed V block).
template <typename E>
__device__ __forceinline__ const E *value_at(const LinkEntry &e, int head, int dim, int row,
                                             int d_v) {
  return (const E *)e.v + vt_offset(head, dim, row, e.lp, d_v);
}

template <typename E>
__global__ void gather_kernel(const LinkEntry *__restrict__ links, int32_t n_links, int64_t total,
                              int32_t heads, int32_t d_k, int32_t d_v, int32_t mla,
                              E *__restrict__ k_out, E *__restrict__ v_out) {
  const int64_t nk = total * heads * d_k;
  const int64_t nv = mla ? 0 : total * heads * d_v;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < nk + nv;
       idx += (int64_t)gridDim.x * blockDim.x) {
    if (idx < nk) {
      const int64_t j = idx / ((int64_t)heads * d_k);
      const int h = (int)((idx / d_k) % heads);
      const int c = (int)(idx % d_k);
      const LinkEntry e = links[find_link(links, n_links, j)];
      k_out[idx] = key_row<E>(e, mla ? 0 : h, (int)(j - e.tok0), d_k)[c];
    } else {
      const int64_t x = idx - nk;
      const int64_t j = x / ((int64_t)heads * d_v);
      const int h = (int)((x / d_v) % heads);
      const int c = (int)(x % d_v);
      const LinkEntry e = links[find_link(links, n_links, j)];
      v_out[x] = *value_at<E>(e, h, c, (int)(j - e.tok0), d_v);
    }
  }
}

// Rows written into chunk slots (rows recomputed at link time): row i of the
// token-major sources goes to dst[i], K into its head-major row, V into its
// transposed column. Off the link path.
template <typename E>
__global__ void write_rows_kernel(const RowDst *__restrict__ dst, int32_t n,
                                  const E *__restrict__ src_k, const E *__restrict__ src_v,
                                  int32_t heads, int32_t d_k, int32_t d_v, int32_t mla) {
  const int i = blockIdx.x;
  if (i >= n) return;
  const RowDst d = dst[i];
  for (int x = threadIdx.x; x < heads * d_k; x += blockDim.x) {
    const int h = x / d_k, c = x - h * d_k;
    ((E *)d.k)[(int64_t)h * d.lp * d_k + c] = src_k[(int64_t)i * heads * d_k + x];
  }
  if (!mla)
    for (int x = threadIdx.x; x < heads * d_v; x += blockDim.x) {
      const int h = x / d_v, e = x - h * d_v;
      ((E *)d.v)[(int64_t)h * d_v * d.lp + e * kPanel] = src_v[(int64_t)i * heads * d_v + x];
    }
}

// ---------------------------------------------------------------------------
// Own KV of a request laid out like a chunk slot (at its last link): K rows
// head-major, V transposed, zero padding up to lp. One launch per call:
// blockIdx.z = request; the first rows_blocks blocks copy K rows, the others
// transpose 64x64 tiles of V.

struct PrepParams {
  const ReqEntry *reqs;       // the call's tables: in the host-mapped staging buffer
  const LinkEntry *links;     // while the copy slice moves them, else on the device
  const void *k_self, *v_self;
  int32_t heads, d_k, d_v, mla, esz;
  int32_t rows_blocks;        // blocks per request doing K rows
  int32_t prep_z;             // z slices preparing own KV (one per request, or 0)
  const uint4 *copy_src;      // table copy (z slice prep_z), n16 = 0: none
  uint4 *copy_dst;
  int64_t copy_n16;
  int32_t has_own;            // own[] holds every request's own rows and slot
  char *work;                 // workspace the slots are in
  OwnArg own[kOwnArgs];
};

// One 64-token x 64-value tile of own V, transposed into the slot's V block.
// 16-byte global loads of 8 values of one token, an LDS tile with padded rows,
// then 16-byte global stores of 8 tokens of one value dim.
template <typename E>
__device__ __forceinline__ void prep_transposed_tile(const ReqEntry &R, const LinkEntry &L,
                                                     const E *__restrict__ src, int heads,
                                                     int width, int tile) {
  constexpr int EPV = 16 / sizeof(E);          // elements per 16 bytes
  constexpr int ROW = 64 + EPV;                // padded LDS row (elements)
  __shared__ __attribute__((aligned(16))) E tile_s[64 * ROW];
  const int eblocks = (width + 63) / 64;
  const int per_h = (L.lp / 64) * eblocks;
  const int h = tile / per_h, rem = tile - h * per_h;
  const int64_t t0 = (int64_t)(rem / eblocks) * 64;
  const int e0 = (rem % eblocks) * 64;
  E *dst = (E *)L.v;
  for (int i = threadIdx.x; i < 64 * (64 / EPV); i += blockDim.x) {
    const int tl = i / (64 / EPV), ec = i % (64 / EPV);
    const int64_t t = t0 + tl;
    const int e = e0 + ec * EPV;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (t < R.ls && e < width) v = *(const uint4 *)(src + ((R.s0 + t) * heads + h) * width + e);
    *(uint4 *)(tile_s + tl * ROW + ec * EPV) = v;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < 64 * (64 / EPV); i += blockDim.x) {
    const int el = i / (64 / EPV), tc = i % (64 / EPV);
    const int e = e0 + el;
    if (e >= width) continue;
    union {
      uint4 u;
      E e[EPV];
    } vals;
#pragma unroll
    for (int x = 0; x < EPV; ++x) vals.e[x] = tile_s[(tc * EPV + x) * ROW + el];
    // EPV tokens (4 or 8) never straddle a 32-token panel
    *(uint4 *)(dst + vt_offset(h, e, t0 + tc * EPV, L.lp, width)) = vals.u;
  }
}

// The call's prologue. z slices 0 .. prep_z-1 lay out request z's own KV
// like a chunk slot; the last slice, if any, copies the call's link and
// request tables from the host-mapped staging buffer to the device (read
// over PCIe, latency-bound). The prep slices take their request's own rows
// and slot from the kernel arguments (batches of up to kOwnArgs requests),
// else read their two table entries where they are (the staging buffer, or
// a plan's device tables), so neither part waits for the other.
__global__ void prep_own_kernel(PrepParams pp) {
  if ((int)blockIdx.z == pp.prep_z) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < pp.copy_n16;
         i += (int64_t)gridDim.x * blockDim.x)
      pp.copy_dst[i] = pp.copy_src[i];
    return;
  }
  ReqEntry R;
  LinkEntry L;
  if (pp.has_own) {     // from the kernel arguments: no table read
    const OwnArg o = pp.own[blockIdx.z];
    R.s0 = o.s0;
    R.ls = o.ls;
    L.lp = (o.ls + kTile - 1) / kTile * kTile;
    L.k = pp.work + o.off;
    L.v = pp.work + o.off + (int64_t)L.lp * pp.heads * pp.d_k * pp.esz;
  } else {
    R = pp.reqs[blockIdx.z];
    if (R.ls > 0) L = pp.links[R.link0 + R.nlinks - 1];
  }
  if (R.ls == 0) return;
  if ((int)blockIdx.x < pp.rows_blocks) {
    // K rows: dst [heads][lp][vpr] from src [token][heads][vpr] in 16-byte
    // units (zeros past the own rows)
    const int vpr = pp.d_k * pp.esz / 16;
    const uint4 *src = (const uint4 *)pp.k_self;
    uint4 *dst = (uint4 *)L.k;
    const int64_t total = (int64_t)pp.heads * L.lp * vpr;
    if (total < (int64_t)1 << 31) {
      // 32-bit index math, and four units per thread loaded before any is
      // stored, so their latencies overlap
      const int per_h = L.lp * vpr, n = (int)total;
      const int stride = pp.rows_blocks * blockDim.x;
      for (int base = blockIdx.x * blockDim.x + threadIdx.x; base < n; base += 4 * stride) {
        uint4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int idx = min(base + u * stride, n - 1);
          const int h = idx / per_h, rem = idx - h * per_h, t = rem / vpr, c = rem - t * vpr;
          v[u] = t < R.ls ? src[((int64_t)(R.s0 + t) * pp.heads + h) * vpr + c]
                          : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (base + u * stride < n) dst[base + u * stride] = make_uint4(v[u].x, v[u].y, v[u].z, v[u].w);
      }
      return;
    }
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)pp.rows_blocks * blockDim.x) {
      const int64_t h = idx / ((int64_t)L.lp * vpr);
      const int64_t rem = idx - h * L.lp * vpr;
      const int64_t t = rem / vpr;
      const int64_t c = rem - t * vpr;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (t < R.ls) v = src[((R.s0 + t) * pp.heads + h) * vpr + c];
      dst[idx] = v;
    }
    return;
  }
  if (pp.mla) return;
  const int tile = blockIdx.x - pp.rows_blocks;
  const int tiles = pp.heads * (L.lp / 64) * ((pp.d_v + 63) / 64);
  if (tile >= tiles) return;
  if (pp.esz == 2)
    prep_transposed_tile<uint16_t>(R, L, (const uint16_t *)pp.v_self, pp.heads, pp.d_v, tile);
  else
    prep_transposed_tile<uint32_t>(R, L, (const uint32_t *)pp.v_self, pp.heads, pp.d_v, tile);
}

// ---------------------------------------------------------------------------
// Generic link attention on the vector ALU.
//
// One workgroup = 4 waves = 16 rows of one (request, kv head); a row is a
// (query token, query head of the group) pair. Keys are walked tile by tile:
// the request's linked chunks in link order (no mask), then its own KV
// (bottom-right causal). Per tile the K rows (and the value tile, transposed
// so lanes index the value dim) are staged in LDS; lane = key for the scores,
// lane = value dim for the P.V update. Online softmax in the log2 domain
// (scale folded with log2 e into the staged queries).

constexpr int kValuRows = 16;

// All-lane max / sum of a wave without LDS round trips: DPP moves inside
// each 16-lane row (lane ^ 1, lane ^ 2 by quad permutes, then the mirrors
// of each 8-lane half and of the row), then lanes l ^ 16 and l ^ 32 by the
// permlane swaps. Every lane ends with the wave's result.
template <int kCtrl>
__device__ __forceinline__ float dpp_mov(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), kCtrl, 0xF, 0xF, false));
}
__device__ __forceinline__ float wave_max(float x) {
  x = fmaxf(x, dpp_mov<0xB1>(x));    // quad_perm [1,0,3,2]
  x = fmaxf(x, dpp_mov<0x4E>(x));    // quad_perm [2,3,0,1]
  x = fmaxf(x, dpp_mov<0x141>(x));   // row_half_mirror
  x = fmaxf(x, dpp_mov<0x140>(x));   // row_mirror
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float wave_sum(float x) {
  x += dpp_mov<0xB1>(x);
  x += dpp_mov<0x4E>(x);
  x += dpp_mov<0x141>(x);
  x += dpp_mov<0x140>(x);
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Copies rows of 16-byte units from global memory into LDS rows of 4-byte
// words (row r, unit c at dst[r * stride + 4 c ..]): each thread issues 4
// loads before storing any, so the loads' latencies overlap (a plain loop
// waits for each load before its store). Past the end a thread reloads the
// last unit and stores nothing, which keeps the loads free of branches.
__device__ __forceinline__ void copy_rows_lds(const char *src, int64_t src_row_bytes, int rows,
                                              int units, uint32_t *dst, int stride) {
  const int n = rows * units;
  for (int base = threadIdx.x; base < n; base += 4 * blockDim.x) {
    uint4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = min(base + u * (int)blockDim.x, n - 1);
      const int r = i / units, c = i - r * units;
      v[u] = *(const uint4 *)(src + r * src_row_bytes + 16 * c);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = base + u * blockDim.x;
      if (i < n) {
        const int r = i / units, c = i - r * units;
        uint32_t *d = dst + r * stride + 4 * c;
        d[0] = v[u].x;
        d[1] = v[u].y;
        d[2] = v[u].z;
        d[3] = v[u].w;
      }
    }
  }
}

// kSmall: the call's tables come by value in `t` (a kernel argument) rather
// than from device memory, and own-KV tiles are read straight from the
// caller's token-major k_self / v_self: no prologue kernel before.
// Transposes token-major value rows into LDS: element e of row r (src +
// r * src_stride + e) lands at dst[e * dst_stride + r], for rows 0 .. rows-1
// and e < d_v. Each thread loads the 16-byte units of 4 (row, unit) pairs
// before storing any, as copy_rows_lds does.
template <typename T>
__device__ __forceinline__ void gather_vt_lds(const T *src, int64_t src_stride, int rows, int d_v,
                                              T *dst, int dst_stride) {
  constexpr int kPer = 16 / sizeof(T);
  const int units = d_v / kPer;
  const int n = rows * units;
  for (int base = threadIdx.x; base < n; base += 4 * blockDim.x) {
    uint4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = min(base + u * (int)blockDim.x, n - 1);
      const int r = i / units, c = i - r * units;
      v[u] = *(const uint4 *)(src + r * src_stride + c * kPer);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i = base + u * blockDim.x;
      if (i < n) {
        const int r = i / units, c = i - r * units;
        T x[kPer];
        __builtin_memcpy(x, &v[u], 16);
#pragma unroll
        for (int k = 0; k < kPer; ++k) dst[(c * kPer + k) * dst_stride + r] = x[k];
      }
    }
  }
}

// kPf: the tile's K and V units go out as one batch of register loads (at
// most kPfUnits 16-byte units per thread each, unit counts powers of two),
// stored to LDS after one wait, and the next tile's batch is issued before
// the current tile is computed; the first tile's batch goes out beside the
// query loads. Without it, K rows and each V panel were a memory round trip
// of their own (tiny_f32: three per tile, ≈ 7 us per tile per workgroup).
constexpr int kPfUnits = 8;

struct PfTile {                 // the tile whose loads are in flight
  LinkEntry E;
  int tt, nvalid, j0, tok;
  bool own;
};

template <typename T, bool MLA, bool kSmall, bool kPf>
__device__ __forceinline__ void valu_body(const LinkParams &p, const SmallTabs &t) {
  extern __shared__ float smem[];
  const int d_k = p.d_k, d_v = p.d_v, group = p.group;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  auto link = [&](int i) -> LinkEntry { return kSmall ? t.links[i] : p.links[i]; };

  const int g = blockIdx.x / p.nrb, rb = blockIdx.x % p.nrb;
  const int split = blockIdx.y;
  const int req_i = kSmall ? t.order[g / p.n_kv_heads] : p.order[g / p.n_kv_heads];
  const int kvh = g % p.n_kv_heads;
  const ReqEntry R = kSmall ? t.reqs[req_i] : p.reqs[req_i];
  const int nrows = R.lq * group;
  const int row0 = rb * kValuRows;
  if (row0 >= nrows) return;
  // the block's key range ends at the last own key its last row sees
  const int vis = visible_tiles(R, min(nrows - 1, row0 + kValuRows - 1) / group);
  const int t_begin = (int)((int64_t)vis * split / p.num_splits);
  const int t_end = (int)((int64_t)vis * (split + 1) / p.num_splits);

  const T *__restrict__ q = (const T *)p.q;

  constexpr int EPW = 4 / sizeof(T);          // elements per 32-bit word
  const int kwords = d_k / EPW;                // words per K row
  const int kstride = kwords + 1;              // odd stride: conflict-free lane = key reads
  const int vwords = kTile / EPW;              // words per value row (64 keys)
  const int vstride = vwords + 1;
  float *qs = smem;                                          // [16][d_k]
  uint32_t *ks = (uint32_t *)(qs + kValuRows * d_k);         // [64][kstride]
  uint32_t *vts = ks + kTile * kstride;                      // [d_v][vstride] (GQA)
  float4 *pb = (float4 *)(vts + (MLA ? 0 : d_v * vstride));  // [4][64]
  const T *ks_e = (const T *)ks;
  const T *vts_e = (const T *)vts;

  int li = 0;
  auto tile_info = [&](int tl) -> PfTile {
    while (link(R.link0 + li).tile0 + (link(R.link0 + li).len + kTile - 1) / kTile <= tl) ++li;
    PfTile x;
    x.E = link(R.link0 + li);
    x.tt = tl - x.E.tile0;
    x.nvalid = min(kTile, x.E.len - x.tt * kTile);
    x.j0 = x.tt * kTile;        // key index within the link (own: within the own KV)
    x.tok = x.E.tok0 + x.j0;    // ... within the request's linked rows
    x.own = tl >= R.doc_tiles;
    return x;
  };
  // kPf unit coordinates of this thread (unit i = tid + 256 u): K unit c of
  // row r; slot V unit c of panel row (panel, dv) = vr (panels [2][d_v][32]
  // are contiguous, so panel row vr starts at vr * 32 elements); own V
  // (token-major, small calls) unit c of key row r.
  const int tid = threadIdx.x;
  const int ku = d_k * (int)sizeof(T) / 16, lku = 31 - __clz(ku);
  const int kc = tid & (ku - 1), kr0 = tid >> lku, krs = 256 >> lku;
  const int n_k = kTile * ku;
  constexpr int pu = kPanel * (int)sizeof(T) / 16;
  constexpr int lpu = pu == 8 ? 3 : 2;
  const int vc = tid & (pu - 1), vr0 = tid >> lpu, vrs = 256 >> lpu;
  const int vu = d_v * (int)sizeof(T) / 16, lvu = 31 - __clz(vu), ldv = 31 - __clz(d_v);
  const int oc = tid & (vu - 1), or0 = tid >> lvu, ors = 256 >> lvu;
  const int n_v = MLA ? 0 : kTile * vu;
  const int kv_heads = MLA ? 1 : p.n_kv_heads;
  uint4 rk[kPfUnits], rv[kPfUnits];
  auto pf_load = [&](const PfTile &x) {
    const bool in_place = kSmall && x.own;   // own rows straight from k_self / v_self
    const char *kb = in_place
        ? (const char *)((const T *)p.k_self + ((int64_t)(R.s0 + x.j0) * kv_heads + kvh) * d_k)
        : (const char *)key_row<T>(x.E, MLA ? 0 : kvh, x.j0, d_k);
    const int64_t krow_b = (int64_t)(in_place ? kv_heads : 1) * d_k * sizeof(T);
#pragma unroll
    for (int u = 0; u < kPfUnits; ++u)
      if (tid + 256 * u < n_k) {
        const int r = kr0 + u * krs;
        rk[u] = *(const uint4 *)(kb + (in_place ? min(r, x.nvalid - 1) : r) * krow_b + 16 * kc);
      }
    if (MLA) return;
    if (in_place) {
      const char *vb =
          (const char *)((const T *)p.v_self + ((int64_t)(R.s0 + x.j0) * kv_heads + kvh) * d_v);
      const int64_t vrow_b = (int64_t)kv_heads * d_v * sizeof(T);
#pragma unroll
      for (int u = 0; u < kPfUnits; ++u)
        if (tid + 256 * u < n_v)
          rv[u] = *(const uint4 *)(vb + min(or0 + u * ors, x.nvalid - 1) * vrow_b + 16 * oc);
    } else {
      const char *vb = (const char *)value_at<T>(x.E, kvh, 0, x.j0, d_v);
#pragma unroll
      for (int u = 0; u < kPfUnits; ++u)
        if (tid + 256 * u < n_v)
          rv[u] = *(const uint4 *)(vb + (int64_t)(vr0 + u * vrs) * kPanel * sizeof(T) + 16 * vc);
    }
  };
  auto pf_store = [&](const PfTile &x) {
#pragma unroll
    for (int u = 0; u < kPfUnits; ++u)
      if (tid + 256 * u < n_k) {
        uint32_t *d = ks + (kr0 + u * krs) * kstride + 4 * kc;
        d[0] = rk[u].x;
        d[1] = rk[u].y;
        d[2] = rk[u].z;
        d[3] = rk[u].w;
      }
    if (MLA) return;
    if (kSmall && x.own) {
      constexpr int kPer = 16 / sizeof(T);
      T *vt = (T *)vts;
#pragma unroll
      for (int u = 0; u < kPfUnits; ++u)
        if (tid + 256 * u < n_v) {
          T e[kPer];
          __builtin_memcpy(e, &rv[u], 16);
#pragma unroll
          for (int k = 0; k < kPer; ++k) vt[(oc * kPer + k) * (vstride * EPW) + or0 + u * ors] = e[k];
        }
    } else {
#pragma unroll
      for (int u = 0; u < kPfUnits; ++u)
        if (tid + 256 * u < n_v) {
          const int vr = vr0 + u * vrs, dv = vr & (d_v - 1), hp = vr >> ldv;
          uint32_t *d = vts + dv * vstride + hp * (kPanel / EPW) + 4 * vc;
          d[0] = rv[u].x;
          d[1] = rv[u].y;
          d[2] = rv[u].z;
          d[3] = rv[u].w;
        }
    }
  };
  PfTile cur{};
  if (kPf && t_begin < t_end) {
    cur = tile_info(t_begin);
    pf_load(cur);
  }

  // the block's query rows, scaled; 4 loads per thread in flight at once
  for (int base = threadIdx.x; base < kValuRows * d_k; base += 4 * blockDim.x) {
    float v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      // rows past the request read its last row (stored as zero below)
      const int x = min(base + u * (int)blockDim.x, kValuRows * d_k - 1);
      const int rl = x / d_k, c = x - rl * d_k;
      const int row = min(row0 + rl, nrows - 1);
      const int i = row / group, h = kvh * group + row % group;
      v[u] = to_f32(q[((int64_t)(R.q0 + i) * p.n_q_heads + h) * d_k + c]);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int x = base + u * blockDim.x;
      if (x < kValuRows * d_k) qs[x] = row0 + x / d_k < nrows ? v[u] * p.scale_log2 : 0.f;
    }
  }

  int lim[4];          // last visible own key per row (-1: none)
  int dl[4];           // linked rows visible to the row
  bool rvalid[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int row = row0 + wave * 4 + r;
    rvalid[r] = row < nrows;
    lim[r] = rvalid[r] ? row / group + R.ls - R.lq : -1;
    dl[r] = p.doc_lim && rvalid[r] ? p.doc_lim[R.q0 + row / group] : kNoLimit;
  }
  float m[4], l[4], acc[4][8];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    m[r] = -INFINITY;
    l[r] = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[r][j] = 0.f;
  }
  const int nvj = (d_v + 63) / 64;

  for (int t = t_begin; t < t_end; ++t) {
    __syncthreads();
    PfTile x;
    if constexpr (kPf) {
      // tile t's loads have landed (the stores wait for them); tile t+1's
      // go out now and run under this tile's arithmetic
      pf_store(cur);
      x = cur;
      if (t + 1 < t_end) {
        cur = tile_info(t + 1);
        pf_load(cur);
      }
    } else {
      x = tile_info(t);
      if (kSmall && x.own) {
        // own keys j0 .. j0 + nvalid - 1 from the caller's token-major rows
        // (rows past nvalid stay unread: they are masked below)
        const T *krow0 = (const T *)p.k_self + ((int64_t)(R.s0 + x.j0) * kv_heads + kvh) * d_k;
        copy_rows_lds((const char *)krow0, (int64_t)kv_heads * d_k * sizeof(T), x.nvalid,
                      kwords / 4, ks, kstride);
        if (!MLA)
          gather_vt_lds<T>((const T *)p.v_self + ((int64_t)(R.s0 + x.j0) * kv_heads + kvh) * d_v,
                           (int64_t)kv_heads * d_v, x.nvalid, d_v, (T *)vts, vstride * EPW);
      } else {
        // 64 consecutive key rows (the slot's padding rows are zeros)
        // K rows (d_k elements, whole 16-byte units) and V^T rows (64 keys)
        copy_rows_lds((const char *)key_row<T>(x.E, MLA ? 0 : kvh, x.j0, d_k),
                      (int64_t)d_k * sizeof(T), kTile, kwords / 4, ks, kstride);
        // V^T: the tile's two 32-token panels, each d_v rows of 32 keys
        if (!MLA)
#pragma unroll
          for (int hp = 0; hp < kTile / kPanel; ++hp)
            copy_rows_lds((const char *)value_at<T>(x.E, kvh, 0, x.j0 + hp * kPanel, d_v),
                          (int64_t)kPanel * sizeof(T), d_v, kPanel * (int)sizeof(T) / 16,
                          vts + hp * (kPanel / EPW), vstride);
      }
    }
    const bool own = x.own;
    const int nvalid = x.nvalid, j0 = x.j0, tok = x.tok;
    __syncthreads();

    // scores: lane = key
    float s[4] = {0.f, 0.f, 0.f, 0.f};
    const uint32_t *krow = ks + lane * kstride;
    const float *qw = qs + (wave * 4) * d_k;
    for (int w = 0; w < kwords; ++w) {
      const uint32_t kw = krow[w];
      if (EPW == 2) {
        const float k0 = __uint_as_float(kw << 16), k1 = __uint_as_float(kw & 0xffff0000u);
#pragma unroll
        for (int r = 0; r < 4; ++r) s[r] += qw[r * d_k + 2 * w] * k0 + qw[r * d_k + 2 * w + 1] * k1;
      } else {
        const float k0 = __uint_as_float(kw);
#pragma unroll
        for (int r = 0; r < 4; ++r) s[r] += qw[r * d_k + w] * k0;
      }
    }
    float pr[4], alpha[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      bool vis = rvalid[r] && lane < nvalid && (own ? j0 + lane <= lim[r] : tok + lane < dl[r]);
      float sv = vis ? s[r] : -INFINITY;
      const float mx = wave_max(sv);
      const float mnew = fmaxf(m[r], mx);
      float pv = 0.f;
      alpha[r] = 1.f;
      if (mnew != -INFINITY) {
        pv = vis ? exp2f(sv - mnew) : 0.f;
        alpha[r] = exp2f(m[r] - mnew);
      }
      const float sum = wave_sum(pv);
      l[r] = l[r] * alpha[r] + sum;
      m[r] = mnew;
      pr[r] = pv;
    }
    pb[wave * 64 + lane] = make_float4(pr[0], pr[1], pr[2], pr[3]);
    __syncthreads();

#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[r][j] *= alpha[r];
    // O += P V: per 64-dim value chunk j, keys four at a time with their
    // probability and value reads issued together (one load at a time per
    // key made every step wait for the LDS round trip). A lane past d_v
    // reads a valid column; its sums are not stored.
    const int kmax = nvalid;
    const float4 *pw = pb + wave * 64;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (j >= nvj) break;
      const int e = min(lane + 64 * j, d_v - 1);
      const T *vc = MLA ? ks_e + e : vts_e + e * vstride * EPW;
      const int kst = MLA ? kstride * EPW : 1;
      float a0 = acc[0][j], a1 = acc[1][j], a2 = acc[2][j], a3 = acc[3][j];
      int k = 0;
      for (; k + 4 <= kmax; k += 4) {
        float4 pp[4];
        float vv[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          pp[u] = pw[k + u];
          vv[u] = to_f32(vc[(k + u) * kst]);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          a0 += pp[u].x * vv[u];
          a1 += pp[u].y * vv[u];
          a2 += pp[u].z * vv[u];
          a3 += pp[u].w * vv[u];
        }
      }
      for (; k < kmax; ++k) {
        const float4 p4 = pw[k];
        const float v = to_f32(vc[k * kst]);
        a0 += p4.x * v;
        a1 += p4.y * v;
        a2 += p4.z * v;
        a3 += p4.w * v;
      }
      acc[0][j] = a0;
      acc[1][j] = a1;
      acc[2][j] = a2;
      acc[3][j] = a3;
    }
  }

  const int total_rows = p.total_q * p.n_q_heads;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    if (!rvalid[r]) continue;
    const int row = row0 + wave * 4 + r;
    const int i = row / group, h = kvh * group + row % group;
    const int64_t orow = (int64_t)(R.q0 + i) * p.n_q_heads + h;
    if (p.num_splits == 1) {
      const float inv = l[r] > 0.f ? 1.f / l[r] : 0.f;
      T *out = (T *)p.out + orow * d_v;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int e = lane + 64 * j;
        if (j < nvj && e < d_v) out[e] = from_f32<T>(acc[r][j] * inv);
      }
      if (p.lse && lane == 0)
        p.lse[orow] = l[r] > 0.f ? (m[r] + log2f(l[r])) * 0.69314718055994531f : -INFINITY;
    } else {
      const int64_t prow = (int64_t)split * total_rows + orow;
      float *po = p.part_o + prow * d_v;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int e = lane + 64 * j;
        if (j < nvj && e < d_v) po[e] = acc[r][j];
      }
      if (lane == 0) {
        p.part_m[prow] = m[r];
        p.part_l[prow] = l[r];
      }
    }
  }
}

template <typename T, bool MLA, bool kPf>
__global__ __launch_bounds__(256) void link_valu_kernel(LinkParams p) {
  valu_body<T, MLA, false, kPf>(p, SmallTabs{});
}

template <typename T, bool MLA, bool kPf>
__global__ __launch_bounds__(256) void link_small_kernel(LinkParams p, SmallTabs t) {
  valu_body<T, MLA, true, kPf>(p, t);
}

// ---------------------------------------------------------------------------
// Split-K combine: one wave per output row, lane j covering value dims
// 2j, 2j+1 of each of the row's kChunks 128-wide chunks (8-byte loads: a
// row's partial of one split is one coalesced 512-byte read per chunk).
// One pass over the splits, kB at a time: their maxima and sums (wave-
// uniform, read through the scalar cache) and partial outputs are loaded
// together, and the running merge is rescaled when the maximum grows, as in
// the online softmax -- a row with up to kB splits costs one memory round
// trip and no cross-lane reduction. Every (split, row) partial is written by
// the attention kernels (zeros with m = -inf for an empty split).
template <typename T>
__device__ __forceinline__ void store_pair(T *out, int e, float x, float y);
template <>
__device__ __forceinline__ void store_pair<float>(float *out, int e, float x, float y) {
  *(float2 *)(out + e) = make_float2(x, y);
}
template <>
__device__ __forceinline__ void store_pair<uint16_t>(uint16_t *out, int e, float x, float y) {
  *(uint32_t *)(out + e) = (uint32_t)bf16_rne(x) | ((uint32_t)bf16_rne(y) << 16);
}

template <typename T, int kChunks>
__global__ __launch_bounds__(256) void combine_kernel(LinkParams p) {
  typedef __attribute__((address_space(4))) const float *const_floats;
  constexpr int kB = 4;
  // the wave index read as a uniform value, so the row's split loads are
  // scalar loads
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int64_t rows = (int64_t)p.total_q * p.n_q_heads;
  const int64_t orow = (int64_t)blockIdx.x * 4 + wave;
  if (orow >= rows) return;
  const int S = p.num_splits, dv = p.d_v;
  const int e0 = 2 * lane;
  const const_floats pm = (const_floats)p.part_m + orow;
  const const_floats pl = (const_floats)p.part_l + orow;
  float M = -INFINITY, L = 0.f;
  float2 acc[kChunks];
#pragma unroll
  for (int c = 0; c < kChunks; ++c) acc[c] = make_float2(0.f, 0.f);
  for (int s0 = 0; s0 < S; s0 += kB) {
    float mb[kB], lb[kB];
    float2 vb[kB][kChunks];
#pragma unroll
    for (int i = 0; i < kB; ++i) {
      const int sc = min(s0 + i, S - 1);      // past the last split: reread it, weight 0
      mb[i] = pm[(int64_t)sc * rows];
      lb[i] = pl[(int64_t)sc * rows];
      const float *po = p.part_o + ((int64_t)sc * rows + orow) * dv;
#pragma unroll
      for (int c = 0; c < kChunks; ++c) {
        const int e = 128 * c + e0;
        vb[i][c] = e < dv ? *(const float2 *)(po + e) : make_float2(0.f, 0.f);
      }
      if (s0 + i >= S) mb[i] = -INFINITY;
    }
    float bm = M;
#pragma unroll
    for (int i = 0; i < kB; ++i) bm = fmaxf(bm, mb[i]);
    if (bm == -INFINITY) continue;
    const float r = M == -INFINITY ? 0.f : exp2f(M - bm);
    L *= r;
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      acc[c].x *= r;
      acc[c].y *= r;
    }
#pragma unroll
    for (int i = 0; i < kB; ++i) {
      const float w = mb[i] == -INFINITY ? 0.f : exp2f(mb[i] - bm);
      L += w * lb[i];
#pragma unroll
      for (int c = 0; c < kChunks; ++c) {
        acc[c].x += w * vb[i][c].x;
        acc[c].y += w * vb[i][c].y;
      }
    }
    M = bm;
  }
  T *out = (T *)p.out + orow * dv;
  const float inv = M == -INFINITY ? 0.f : 1.f / L;
#pragma unroll
  for (int c = 0; c < kChunks; ++c) {
    const int e = 128 * c + e0;
    if (e < dv) store_pair<T>(out, e, acc[c].x * inv, acc[c].y * inv);
  }
  if (p.lse && lane == 0)
    p.lse[orow] = M == -INFINITY ? -INFINITY : (M + log2f(L)) * 0.69314718055994531f;
}

size_t valu_lds_bytes(int esz, int mla, int d_k, int d_v) {
  const int epw = 4 / esz;
  const size_t kstride = d_k / epw + 1, vstride = kTile / epw + 1;
  return sizeof(float) * kValuRows * d_k + 4 * kTile * kstride +
         (mla ? 0 : 4 * d_v * vstride) + sizeof(float4) * 4 * 64;
}

// Shapes the register-prefetch tile path (kPf) takes: 16-byte unit counts
// per K and V row that are powers of two (and d_v one too), at most
// kPfUnits units per thread for each of a tile's K and V.
bool valu_prefetch_ok(int esz, bool mla, int d_k, int d_v) {
  auto pow2 = [](int x) { return x > 0 && (x & (x - 1)) == 0; };
  const int ku = d_k * esz / 16, vu = d_v * esz / 16;
  if (d_k * esz % 16 || !pow2(ku) || kTile * ku > kPfUnits * 256) return false;
  if (!mla && (d_v * esz % 16 || !pow2(vu) || !pow2(d_v) || kTile * vu > kPfUnits * 256))
    return false;
  return true;
}

template <typename T, bool MLA, bool kPf>
hipError_t launch_valu_tp(const LinkParams &p, hipStream_t st) {
  const size_t lds = valu_lds_bytes(sizeof(T), MLA, p.d_k, p.d_v);
  hipError_t e = hipFuncSetAttribute((const void *)link_valu_kernel<T, MLA, kPf>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  dim3 grid(p.n_groups * p.nrb, p.num_splits);
  hipLaunchKernelGGL((link_valu_kernel<T, MLA, kPf>), grid, dim3(256), lds, st, p);
  return hipGetLastError();
}

template <typename T, bool MLA>
hipError_t launch_valu_t(const LinkParams &p, hipStream_t st) {
  return valu_prefetch_ok(sizeof(T), MLA, p.d_k, p.d_v) ? launch_valu_tp<T, MLA, true>(p, st)
                                                        : launch_valu_tp<T, MLA, false>(p, st);
}

template <typename T, bool MLA, bool kPf>
hipError_t launch_small_tp(const LinkParams &p, const SmallTabs &t, hipStream_t st) {
  const size_t lds = valu_lds_bytes(sizeof(T), MLA, p.d_k, p.d_v);
  hipError_t e = hipFuncSetAttribute((const void *)link_small_kernel<T, MLA, kPf>,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  dim3 grid(p.n_groups * p.nrb, p.num_splits);
  hipLaunchKernelGGL((link_small_kernel<T, MLA, kPf>), grid, dim3(256), lds, st, p, t);
  return hipGetLastError();
}

template <typename T, bool MLA>
hipError_t launch_small_t(const LinkParams &p, const SmallTabs &t, hipStream_t st) {
  return valu_prefetch_ok(sizeof(T), MLA, p.d_k, p.d_v) ? launch_small_tp<T, MLA, true>(p, t, st)
                                                        : launch_small_tp<T, MLA, false>(p, t, st);
}

// ---------------------------------------------------------------------------
// Lean small-call kernel (GQA, d_k = d_v = D fixed at compile time, power-of-
// two query group): the computation of link_small_kernel for calls that are
// latency-bound, 16 rows per workgroup. A wave alone on its SIMD issues at
// most one instruction every four cycles, so such a call's time is its
// per-wave instruction count plus its memory round trips; this kernel keeps
// both low. The grid carries (row block, split, request x kv head); every
// tile's link comes from the host's tile map; each 16-byte unit of a tile is
// one load and one LDS store, and the next tile's loads run under the
// current tile's arithmetic. Products run on 16x16 matrix-core instructions
// (fp32: v_mfma_f32_16x16x4_f32, bf16: v_mfma_f32_16x16x16_bf16): wave w
// takes keys 16w .. 16w+15 of every tile for all 16 rows and keeps its own
// online softmax, as S^T = K Q^T and O^T += V^T P^T, so each lane's
// probabilities are exactly its operand of the value product and never leave
// its registers; the four waves' (m, l, O) are merged through LDS at the end.
// Queries stay in registers for the whole call.
//
// 16x16 operand layouts (lane l): A[m = l & 15][k-slot group l >> 4],
// B[k-slot group l >> 4][n = l & 15], C register j: [m = 4 (l >> 4) + j][n = l & 15].
// For S^T the key of lane l's row of K is 16w + (l & 15) and its k-slot group
// reads head dims [D/4 (l >> 4), D/4 (l >> 4 + 1)) of that row and of the
// query row l & 15; C register j then holds key 16w + 4 (l >> 4) + j, row l & 15.

template <typename T, int D>
struct LeanShape {
  static constexpr int E = 16 / (int)sizeof(T);        // elements per 16-byte unit
  static constexpr int KU = D / E;                      // units per K row
  static constexpr int KSW = D * (int)sizeof(T) / 4 + 4;    // K row stride in LDS (words)
  static constexpr int VSW = kTile * (int)sizeof(T) / 4 + 4; // V^T row stride (64 keys)
  static constexpr int PRU = kPanel / E;                // units per row of a 32-key panel
  static constexpr int NU = kTile * KU / 256;           // K (and V) units per thread
  static constexpr int SEG = D / 4;                     // head dims per k-slot group
  static constexpr int SEGU = SEG / E;                  // their 16-byte units
  static constexpr int NB = D / 16;                     // 16-wide value-dim blocks
  static constexpr int OSW = D + 1;                     // merge buffer row stride (floats)
  static constexpr int TILE_WORDS = kTile * KSW + D * VSW;
  static constexpr int MERGE_WORDS = 4 * kValuRows * OSW;
  static constexpr int ML_OFF = TILE_WORDS > MERGE_WORDS ? TILE_WORDS : MERGE_WORDS;
  static constexpr int WORDS = ML_OFF + 2 * 4 * kValuRows;   // + per-wave m and l
  static_assert(NU >= 1 && kTile * KU % 256 == 0, "whole units per thread");
  static_assert(SEGU >= 1 && SEG % E == 0, "whole units per k-slot group");
};

typedef float lean_f4 __attribute__((ext_vector_type(4)));
typedef short lean_s4 __attribute__((ext_vector_type(4)));

// max / sum over the four lanes l & 15 + 16 g (one row of a 16x16 C tile)
__device__ __forceinline__ float quad_rows_max(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float quad_rows_sum(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <typename T, int D>
__global__ __launch_bounds__(256) void link_lean_kernel(LinkParams p, LeanTabs t) {
  using S = LeanShape<T, D>;
  constexpr int E = S::E;
  constexpr bool F32 = sizeof(T) == 4;
  __shared__ __attribute__((aligned(16))) uint32_t lds[S::WORDS];
  uint32_t *ks = lds, *vts = lds + kTile * S::KSW;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int lr = lane & 15, lg4 = lane >> 4;
  const int rb = blockIdx.x, split = blockIdx.y;
  const int pos = blockIdx.z / p.n_kv_heads, kvh = blockIdx.z - pos * p.n_kv_heads;
  const ReqEntry R = t.reqs[pos];
  const int lg = __builtin_ctz(p.group);
  const int nrows = R.lq << lg;
  const int row0 = rb * kValuRows;
  if (row0 >= nrows) return;
  const int vis = visible_tiles(R, min(nrows - 1, row0 + kValuRows - 1) >> lg);
  const int t_begin = vis * split / p.num_splits, t_end = vis * (split + 1) / p.num_splits;
  const int kvn = p.n_kv_heads;

  // the loads of one tile into registers: K units (key, c) and V^T units
  // (panel, value dim, key unit) in slot order; own tiles from the caller's
  // token-major rows (rows past the tile's valid keys reread its last one)
  struct Tile {
    const T *kb, *vb;
    int nvalid, j0;
    bool own;
  };
  auto tile_at = [&](int tl) {
    const LinkEntry L = t.links[R.link0 + t.tile_link[t.tile_base[pos] + tl]];
    Tile x;
    x.j0 = (tl - L.tile0) * kTile;
    x.nvalid = min(kTile, L.len - x.j0);
    x.own = tl >= R.doc_tiles;
    if (x.own) {
      x.kb = (const T *)p.k_self + ((int64_t)(R.s0 + x.j0) * kvn + kvh) * D;
      x.vb = (const T *)p.v_self + ((int64_t)(R.s0 + x.j0) * kvn + kvh) * D;
    } else {
      x.kb = (const T *)L.k + ((int64_t)kvh * L.lp + x.j0) * D;
      x.vb = (const T *)L.v + vt_offset(kvh, 0, x.j0, L.lp, D);
    }
    return x;
  };
  uint4 rk[S::NU], rv[S::NU];
  auto issue = [&](const Tile &x) {
#pragma unroll
    for (int u = 0; u < S::NU; ++u) {
      const int i = tid + 256 * u, key = i / S::KU, c = i % S::KU;
      if (x.own) {
        const int64_t r = (int64_t)min(key, x.nvalid - 1) * kvn * D;
        rk[u] = *(const uint4 *)(x.kb + r + c * E);
        rv[u] = *(const uint4 *)(x.vb + r + c * E);
      } else {
        rk[u] = *(const uint4 *)(x.kb + (int64_t)i * E);
        rv[u] = *(const uint4 *)(x.vb + (int64_t)i * E);
      }
    }
  };
  auto land = [&](const Tile &x) {
#pragma unroll
    for (int u = 0; u < S::NU; ++u) {
      const int i = tid + 256 * u, key = i / S::KU, c = i % S::KU;
      // (whole-struct copies of array elements put the arrays in scratch)
      *(uint4 *)(ks + key * S::KSW + 4 * c) = make_uint4(rk[u].x, rk[u].y, rk[u].z, rk[u].w);
      if (x.own) {
        // token-major: the unit holds value dims c*E .. c*E+E-1 of one key
        using U = std::conditional_t<F32, uint32_t, uint16_t>;   // T's bits
        const uint32_t w[4] = {rv[u].x, rv[u].y, rv[u].z, rv[u].w};
        U *vt = (U *)vts + key;
        constexpr int VSE = S::VSW * 4 / (int)sizeof(T);    // V^T row stride (elements)
#pragma unroll
        for (int k = 0; k < E; ++k) {
          const uint32_t wk = w[k * (int)sizeof(T) / 4];
          vt[(c * E + k) * VSE] = (U)(F32 ? wk : k & 1 ? wk >> 16 : wk & 0xffffu);
        }
      } else {
        // slot V^T: panel, value dim, unit of 32-key panel row
        const int pan = i / (D * S::PRU), dv = (i / S::PRU) % D, kc = i % S::PRU;
        *(uint4 *)(vts + dv * S::VSW + pan * (kPanel * (int)sizeof(T) / 4) + 4 * kc) =
            make_uint4(rv[u].x, rv[u].y, rv[u].z, rv[u].w);
      }
    }
  };

  Tile cur{};
  if (t_begin < t_end) {
    cur = tile_at(t_begin);
    issue(cur);
  }
  // query row lr of the block, head dims [SEG lg4, SEG (lg4 + 1)), as the
  // B operand of S^T = K Q^T (rows past the request: zeros)
  const int qrow = row0 + lr;
  const bool qvalid = qrow < nrows;
  uint4 qu[S::SEGU];
  {
    const int row = min(qrow, nrows - 1);
    const T *qp = (const T *)p.q +
                  ((int64_t)(R.q0 + (row >> lg)) * p.n_q_heads + kvh * p.group + (row & (p.group - 1))) * D +
                  S::SEG * lg4;
#pragma unroll
    for (int u = 0; u < S::SEGU; ++u) {
      const uint4 v = *(const uint4 *)(qp + u * E);
      qu[u] = qvalid ? make_uint4(v.x, v.y, v.z, v.w) : make_uint4(0u, 0u, 0u, 0u);
    }
  }
  const int lim = ((min(qrow, nrows - 1)) >> lg) + R.ls - R.lq;   // last own key row lr sees
  float m = -INFINITY, l = 0.f;
  lean_f4 oacc[S::NB];
#pragma unroll
  for (int c = 0; c < S::NB; ++c) oacc[c] = lean_f4{0.f, 0.f, 0.f, 0.f};

  for (int tl = t_begin; tl < t_end; ++tl) {
    __syncthreads();              // the previous tile's reads are done
    land(cur);
    const Tile x = cur;
    if (tl + 1 < t_end) {
      cur = tile_at(tl + 1);
      issue(cur);
    }
    __syncthreads();

    // S^T block: keys 16 wave .. +15 of the tile x rows 0..15
    lean_f4 sacc = {0.f, 0.f, 0.f, 0.f};
    const uint4 *krow = (const uint4 *)(ks + (16 * wave + lr) * S::KSW) + S::SEGU * lg4;
#pragma unroll
    for (int u = 0; u < S::SEGU; ++u) {
      const uint4 kk = krow[u];
      const uint4 qq = qu[u];
      if constexpr (F32) {
        sacc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kk.x), __uint_as_float(qq.x), sacc, 0, 0, 0);
        sacc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kk.y), __uint_as_float(qq.y), sacc, 0, 0, 0);
        sacc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kk.z), __uint_as_float(qq.z), sacc, 0, 0, 0);
        sacc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(kk.w), __uint_as_float(qq.w), sacc, 0, 0, 0);
      } else {
        const lean_s4 a0 = {(short)(kk.x & 0xffff), (short)(kk.x >> 16), (short)(kk.y & 0xffff), (short)(kk.y >> 16)};
        const lean_s4 b0 = {(short)(qq.x & 0xffff), (short)(qq.x >> 16), (short)(qq.y & 0xffff), (short)(qq.y >> 16)};
        const lean_s4 a1 = {(short)(kk.z & 0xffff), (short)(kk.z >> 16), (short)(kk.w & 0xffff), (short)(kk.w >> 16)};
        const lean_s4 b1 = {(short)(qq.z & 0xffff), (short)(qq.z >> 16), (short)(qq.w & 0xffff), (short)(qq.w >> 16)};
        sacc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a0, b0, sacc, 0, 0, 0);
        sacc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a1, b1, sacc, 0, 0, 0);
      }
    }
    // online softmax of row lr over this wave's 16 keys (register j: key
    // 16 wave + 4 lg4 + j of the tile)
    float sv[4];
    float mx = -INFINITY;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int kt = 16 * wave + 4 * lg4 + j;
      const bool vk = qvalid && kt < x.nvalid && (!x.own || x.j0 + kt <= lim);
      sv[j] = vk ? sacc[j] * p.scale_log2 : -INFINITY;
      mx = fmaxf(mx, sv[j]);
    }
    const float mnew = fmaxf(m, quad_rows_max(mx));
    float pj[4], alpha = 1.f, rs = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      pj[j] = mnew == -INFINITY ? 0.f : exp2f(sv[j] - mnew);
      rs += pj[j];
    }
    if (mnew != -INFINITY) alpha = exp2f(m - mnew);
    l = l * alpha + quad_rows_sum(rs);
    m = mnew;

    // O^T += V^T P^T: value dims 16 c + lr, this wave's 16 keys
    const uint32_t *vrow = vts + lr * S::VSW + (16 * wave + 4 * lg4) * (int)sizeof(T) / 4;
#pragma unroll
    for (int c = 0; c < S::NB; ++c) {
      oacc[c] *= alpha;
      if constexpr (F32) {
        const uint4 vv = *(const uint4 *)(vrow + 16 * c * S::VSW);
        oacc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(vv.x), pj[0], oacc[c], 0, 0, 0);
        oacc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(vv.y), pj[1], oacc[c], 0, 0, 0);
        oacc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(vv.z), pj[2], oacc[c], 0, 0, 0);
        oacc[c] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(vv.w), pj[3], oacc[c], 0, 0, 0);
      } else {
        const uint2 vv = *(const uint2 *)(vrow + 16 * c * S::VSW);
        const lean_s4 a = {(short)(vv.x & 0xffff), (short)(vv.x >> 16), (short)(vv.y & 0xffff), (short)(vv.y >> 16)};
        const lean_s4 b = {(short)bf16_rne(pj[0]), (short)bf16_rne(pj[1]), (short)bf16_rne(pj[2]),
                           (short)bf16_rne(pj[3])};
        oacc[c] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, oacc[c], 0, 0, 0);
      }
    }
  }

  // merge the four waves' (m, l, O) of each row; O^T register j of block c
  // is value dim 16 c + 4 lg4 + j of row lr
  __syncthreads();                // the last tile's reads are done
  constexpr int NW = 4;                                   // waves with a partial
  float *ob = (float *)lds;                               // [wave][row][OSW]
  float *mb = (float *)(lds + S::ML_OFF), *lb = mb + NW * kValuRows;
#pragma unroll
  for (int c = 0; c < S::NB; ++c)
#pragma unroll
    for (int j = 0; j < 4; ++j) ob[(wave * kValuRows + lr) * S::OSW + 16 * c + 4 * lg4 + j] = oacc[c][j];
  if (lg4 == 0) {
    mb[wave * kValuRows + lr] = m;
    lb[wave * kValuRows + lr] = l;
  }
  __syncthreads();
  // thread i: outputs (row, dv) = divmod(i + 256 k, D)
  const int64_t total_rows = (int64_t)p.total_q * p.n_q_heads;
  for (int idx = tid; idx < kValuRows * D; idx += 256) {
    const int row = idx / D, dv = idx % D;
    if (row0 + row >= nrows) break;       // later indices are later rows
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, mb[w * kValuRows + row]);
    float L = 0.f, o = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float mw = mb[w * kValuRows + row];
      const float wt = M == -INFINITY || mw == -INFINITY ? 0.f : exp2f(mw - M);
      L += wt * lb[w * kValuRows + row];
      o += wt * ob[(w * kValuRows + row) * S::OSW + dv];
    }
    const int grow = row0 + row;
    const int64_t orow =
        (int64_t)(R.q0 + (grow >> lg)) * p.n_q_heads + kvh * p.group + (grow & (p.group - 1));
    if (p.num_splits == 1) {
      ((T *)p.out)[orow * D + dv] = from_f32<T>(L > 0.f ? o / L : 0.f);
      if (dv == 0 && p.lse) p.lse[orow] = L > 0.f ? (M + log2f(L)) * 0.69314718055994531f : -INFINITY;
    } else {
      const int64_t prow = split * total_rows + orow;
      p.part_o[prow * D + dv] = o;
      if (dv == 0) {
        p.part_m[prow] = M;
        p.part_l[prow] = L;
      }
    }
  }
}

template <typename T, int D>
hipError_t launch_lean_t(const LinkParams &p, const LeanTabs &t, hipStream_t st) {
  dim3 grid(p.nrb, p.num_splits, p.batch * p.n_kv_heads);
  hipLaunchKernelGGL((link_lean_kernel<T, D>), grid, dim3(256), 0, st, p, t);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_link_small(const LinkParams &p, const SmallTabs &t, int dtype, int mla,
                             hipStream_t st, const char **name) {
  if (dtype == 0) {
    *name = mla ? "link_small_kernel<float,MLA>" : "link_small_kernel<float,GQA>";
    return mla ? launch_small_t<float, true>(p, t, st) : launch_small_t<float, false>(p, t, st);
  }
  *name = mla ? "link_small_kernel<bf16,MLA>" : "link_small_kernel<bf16,GQA>";
  return mla ? launch_small_t<uint16_t, true>(p, t, st) : launch_small_t<uint16_t, false>(p, t, st);
}

bool lean_supported(int dtype, int d_k, int d_v, int group) {
  if (d_k != d_v || group < 1 || (group & (group - 1))) return false;
  return d_k == 32 || d_k == 64 || (d_k == 128 && dtype == 0);
}

hipError_t launch_link_lean(const LinkParams &p, const LeanTabs &t, int dtype, hipStream_t st,
                            const char **name) {
  if (dtype == 0) {
    *name = "link_lean_kernel<float>";
    if (p.d_k == 32) return launch_lean_t<float, 32>(p, t, st);
    if (p.d_k == 64) return launch_lean_t<float, 64>(p, t, st);
    return launch_lean_t<float, 128>(p, t, st);
  }
  *name = "link_lean_kernel<bf16>";
  if (p.d_k == 32) return launch_lean_t<uint16_t, 32>(p, t, st);
  return launch_lean_t<uint16_t, 64>(p, t, st);
}

int valu_rows_per_block() { return kValuRows; }

size_t valu_lds_bytes_for(int esz, int mla, int d_k, int d_v) {
  return valu_lds_bytes(esz, mla, d_k, d_v);
}

hipError_t launch_link_valu(const LinkParams &p, int dtype, int mla, hipStream_t st,
                            const char **name) {
  if (dtype == 0) {
    *name = mla ? "link_valu_kernel<float,MLA>" : "link_valu_kernel<float,GQA>";
    return mla ? launch_valu_t<float, true>(p, st) : launch_valu_t<float, false>(p, st);
  }
  *name = mla ? "link_valu_kernel<bf16,MLA>" : "link_valu_kernel<bf16,GQA>";
  return mla ? launch_valu_t<uint16_t, true>(p, st) : launch_valu_t<uint16_t, false>(p, st);
}

hipError_t launch_combine(const LinkParams &p, int dtype, hipStream_t st) {
  const int64_t rows = (int64_t)p.total_q * p.n_q_heads;
  if (rows == 0) return hipSuccess;
  dim3 grid((unsigned)((rows + 3) / 4));
  const int chunks = (p.d_v + 127) / 128;     // 1 .. 8 (d_v <= 1024)
  auto go = [&](auto kc) {
    constexpr int kC = decltype(kc)::value;
    if (dtype == 0)
      hipLaunchKernelGGL((combine_kernel<float, kC>), grid, dim3(256), 0, st, p);
    else
      hipLaunchKernelGGL((combine_kernel<uint16_t, kC>), grid, dim3(256), 0, st, p);
  };
  if (chunks == 1)
    go(std::integral_constant<int, 1>());
  else if (chunks <= 4)
    go(std::integral_constant<int, 4>());
  else
    go(std::integral_constant<int, 8>());
  return hipGetLastError();
}

// Per-call table upload: the host-mapped staging buffer is read over PCIe
// by one kernel. (A host-to-device hipMemcpyAsync of a table above a few KB
// goes through the SDMA engine, about 20 us per call against 4 us here.)
__global__ __launch_bounds__(256) void table_copy_kernel(const uint4 *src, uint4 *dst,
                                                         int64_t n16) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16;
       i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

hipError_t launch_table_copy(const void *src, void *dst, int64_t bytes, hipStream_t st) {
  const int64_t n16 = bytes / 16;
  const unsigned blocks = (unsigned)std::max<int64_t>(1, std::min<int64_t>((n16 + 255) / 256, 64));
  hipLaunchKernelGGL(table_copy_kernel, dim3(blocks), dim3(256), 0, st, (const uint4 *)src,
                     (uint4 *)dst, n16);
  return hipGetLastError();
}

hipError_t launch_put_rows(const void *src, void *dst, int64_t n_tokens, int32_t lp,
                           int32_t heads, int32_t width, int32_t esz, hipStream_t st) {
  const int32_t vpr = width * esz / 16;
  const int64_t total = (int64_t)heads * lp * vpr;
  const unsigned blocks = (unsigned)std::min<int64_t>((total + 255) / 256, 65536);
  hipLaunchKernelGGL(put_rows_kernel, dim3(blocks), dim3(256), 0, st, (const uint4 *)src,
                     (uint4 *)dst, n_tokens, lp, heads, vpr);
  return hipGetLastError();
}

hipError_t launch_put_transposed(const void *src, void *dst, int64_t n_tokens, int32_t lp,
                                 int32_t heads, int32_t width, int32_t esz, hipStream_t st) {
  dim3 grid(lp / 64, (width + 63) / 64, heads);
  if (esz == 2)
    hipLaunchKernelGGL(put_transposed_kernel<uint16_t>, grid, dim3(256), 0, st,
                       (const uint16_t *)src, (uint16_t *)dst, n_tokens, lp, heads, width);
  else
    hipLaunchKernelGGL(put_transposed_kernel<uint32_t>, grid, dim3(256), 0, st,
                       (const uint32_t *)src, (uint32_t *)dst, n_tokens, lp, heads, width);
  return hipGetLastError();
}

hipError_t launch_write_rows(const RowDst *dst, int32_t n, const void *src_k, const void *src_v,
                             int32_t heads, int32_t d_k, int32_t d_v, int32_t mla, int32_t esz,
                             hipStream_t st) {
  if (n <= 0) return hipSuccess;
  if (esz == 2)
    hipLaunchKernelGGL(write_rows_kernel<uint16_t>, dim3(n), dim3(256), 0, st, dst, n,
                       (const uint16_t *)src_k, (const uint16_t *)src_v, heads, d_k, d_v, mla);
  else
    hipLaunchKernelGGL(write_rows_kernel<uint32_t>, dim3(n), dim3(256), 0, st, dst, n,
                       (const uint32_t *)src_k, (const uint32_t *)src_v, heads, d_k, d_v, mla);
  return hipGetLastError();
}

hipError_t launch_gather(const LinkEntry *links, int32_t n_links, int64_t total_tokens,
                         int32_t heads, int32_t d_k, int32_t d_v, int32_t mla, int32_t esz,
                         void *k_out, void *v_out, hipStream_t st) {
  const int64_t n = total_tokens * heads * (d_k + (mla ? 0 : d_v));
  if (n == 0) return hipSuccess;
  const unsigned blocks = (unsigned)std::min<int64_t>((n + 255) / 256, 65536);
  if (esz == 2)
    hipLaunchKernelGGL(gather_kernel<uint16_t>, dim3(blocks), dim3(256), 0, st, links, n_links,
                       total_tokens, heads, d_k, d_v, mla, (uint16_t *)k_out, (uint16_t *)v_out);
  else
    hipLaunchKernelGGL(gather_kernel<uint32_t>, dim3(blocks), dim3(256), 0, st, links, n_links,
                       total_tokens, heads, d_k, d_v, mla, (uint32_t *)k_out, (uint32_t *)v_out);
  return hipGetLastError();
}

hipError_t launch_prologue(const LinkParams &p, const LinkEntry *links, const ReqEntry *reqs,
                           int32_t mla, int32_t esz, int32_t max_own_lp, const OwnArg *own,
                           const void *work, const void *copy_src, void *copy_dst,
                           int64_t copy_bytes, hipStream_t st) {
  if (p.batch == 0) return hipSuccess;
  PrepParams pp;
  pp.has_own = own != nullptr && p.batch <= kOwnArgs;
  pp.work = (char *)work;
  if (pp.has_own)
    for (int32_t r = 0; r < p.batch; ++r) pp.own[r] = own[r];
  pp.reqs = reqs;
  pp.links = links;
  pp.copy_src = (const uint4 *)copy_src;
  pp.copy_dst = (uint4 *)copy_dst;
  pp.copy_n16 = copy_bytes / 16;
  pp.prep_z = max_own_lp > 0 ? p.batch : 0;
  pp.k_self = p.k_self;
  pp.v_self = p.v_self;
  pp.heads = p.n_kv_heads;
  pp.d_k = p.d_k;
  pp.d_v = p.d_v;
  pp.mla = mla;
  pp.esz = esz;
  const int64_t rows_vec = (int64_t)p.n_kv_heads * max_own_lp * (p.d_k * esz / 16);
  pp.rows_blocks = (int32_t)std::max<int64_t>(1, std::min<int64_t>((rows_vec + 1023) / 1024, 256));
  const int64_t tblocks = mla ? 0 : (int64_t)p.n_kv_heads * (max_own_lp / 64) * ((p.d_v + 63) / 64);
  const int64_t copy_blocks = std::min<int64_t>((pp.copy_n16 + 255) / 256, 64);
  const int64_t gx = std::max<int64_t>(pp.prep_z ? pp.rows_blocks + tblocks : 0, copy_blocks);
  const int gz = pp.prep_z + (pp.copy_n16 > 0 ? 1 : 0);
  if (gx == 0 || gz == 0) return hipSuccess;
  hipLaunchKernelGGL(prep_own_kernel, dim3((unsigned)gx, 1, (unsigned)gz), dim3(256), 0, st, pp);
  return hipGetLastError();
}

}  // namespace pic
