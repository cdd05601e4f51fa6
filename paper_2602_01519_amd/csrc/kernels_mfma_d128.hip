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

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }

typedef __attribute__((address_space(3))) void *lds_ptr;

// Starts the copy of key tile tt of link E (kv head kvh) into LDS buffers
// kdst / vdst with direct global->LDS loads: lane i of a load lands at slot
// base + i, so each lane fetches the global chunk that belongs at that slot
// of the swizzled layout. 4 K loads + 4 V loads per lane, 16 bytes each.
__device__ __forceinline__ void issue_tile(const LinkEntry &E, int kvh, int tt, uint4 *kdst,
                                           uint4 *vdst, int wave, int lane) {
  const uint16_t *kb = (const uint16_t *)E.k + ((int64_t)kvh * E.lp + tt * kTile) * kD;
  const uint16_t *vb = (const uint16_t *)E.v + (int64_t)kvh * kD * E.lp + tt * kTile;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int base = (u * kWaves + wave) * 64;
    const int s = base + lane;
    const int key = s >> 4, kc = (s & 15) ^ (key & 15);
    __builtin_amdgcn_global_load_lds(kb + key * kD + kc * 8, (lds_ptr)(kdst + base), 16, 0, 0);
    const int dv = s >> 3, vc = (s & 7) ^ (dv & 7);
    __builtin_amdgcn_global_load_lds(vb + (int64_t)dv * E.lp + vc * 8, (lds_ptr)(vdst + base), 16,
                                     0, 0);
  }
}

// Sum / max of a value over lanes i and i ^ 32 (the two key halves of a row).
__device__ __forceinline__ float half_swap_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float half_swap_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// The request's link table is read through a window of kWin entries staged
// in LDS, so walking tiles costs LDS reads instead of dependent global loads.
constexpr int kWin = 32;

struct LinkCursor {
  int li = 0;       // current link (index within the request)
  int wb = 0;       // first link held in the window
};

__device__ __forceinline__ void load_window(const LinkParams &p, const ReqEntry &R, LinkEntry *win,
                                            int wb) {
  const int n = min(kWin, R.nlinks - wb);
  for (int i = threadIdx.x; i < n; i += blockDim.x) win[i] = p.links[R.link0 + wb + i];
}

// Moves the cursor to the link holding tile t (t only grows) and returns it.
// Uniform across the workgroup: it may reload the window between barriers.
__device__ __forceinline__ LinkEntry advance(const LinkParams &p, const ReqEntry &R,
                                             LinkEntry *win, LinkCursor &cur, int t) {
  for (;;) {
    if (cur.li - cur.wb >= kWin) {
      __syncthreads();
      cur.wb += kWin;
      load_window(p, R, win, cur.wb);
      __syncthreads();
    }
    const LinkEntry e = win[cur.li - cur.wb];
    if (t < e.tile0 + e.lp / kTile) return e;
    ++cur.li;
  }
}

__global__ __launch_bounds__(256, 2) void link_mfma_d128_kernel(LinkParams p) {
  __shared__ Smem sm;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
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

  __shared__ LinkEntry win[kWin];
  LinkCursor cur;
  load_window(p, R, win, 0);
  __syncthreads();
  // masking facts of the tile being computed: valid keys, own-KV key offset
  int nvalid_cur = kTile, j0_cur = 0;
  if (t_begin < t_end) {
    const LinkEntry E = advance(p, R, win, cur, t_begin);
    const int tt = t_begin - E.tile0;
    issue_tile(E, kvh, tt, sm.k[0], sm.vt[0], wave, lane);
    nvalid_cur = min(kTile, E.len - tt * kTile);
    j0_cur = tt * kTile;
  }

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
  const int krow0 = key_of_m(n);      // key row feeding this lane's M index, block 0
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  for (int t = t_begin; t < t_end; ++t) {
    const int buf = (t - t_begin) & 1;
    const int nvalid = nvalid_cur, j0 = j0_cur;
    const bool own = t >= R.doc_tiles;
    if (t + 1 < t_end) {
      const LinkEntry E = advance(p, R, win, cur, t + 1);
      const int tt = t + 1 - E.tile0;
      issue_tile(E, kvh, tt, sm.k[buf ^ 1], sm.vt[buf ^ 1], wave, lane);
      nvalid_cur = min(kTile, E.len - tt * kTile);
      j0_cur = tt * kTile;
    }

    // ---- S^T = K Q^T : two 32-key blocks
    const uint4 *kt = sm.k[buf];
    bf16x8 ka[8], kb[8];
#pragma unroll
    for (int st = 0; st < 8; ++st) {
      ka[st] = as_bf16x8(kt[k_slot(krow0, st * 2 + g)]);
      kb[st] = as_bf16x8(kt[k_slot(32 + krow0, st * 2 + g)]);
    }
    f32x16 s0, s1;
#pragma unroll
    for (int x = 0; x < 16; ++x) { s0[x] = 0.f; s1[x] = 0.f; }
#pragma unroll
    for (int st = 0; st < 8; ++st) {
      s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[st], qf[st], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kb[st], qf[st], s1, 0, 0, 0);
    }

    // ---- masking (only on ragged or own tiles)
    // s_b[x] is the score of key b*32 + (x>>3)*16 + g*8 + (x&7) for this row
    if (own || nvalid < kTile) {
      const int kl = own ? lim - j0 : kTile;     // visible iff key <= kl
#pragma unroll
      for (int x = 0; x < 16; ++x) {
        const int key = (x >> 3) * 16 + g * 8 + (x & 7);
        if (key >= nvalid || key > kl) s0[x] = -INFINITY;
        if (key + 32 >= nvalid || key + 32 > kl) s1[x] = -INFINITY;
      }
    }

    // ---- online softmax (log2 domain, lazy rescale)
    float tmax = -INFINITY;
#pragma unroll
    for (int x = 0; x < 16; x += 2) {
      tmax = fmaxf(fmaxf(tmax, s0[x]), s0[x + 1]);
      tmax = fmaxf(fmaxf(tmax, s1[x]), s1[x + 1]);
    }
    tmax = half_swap_max(tmax);
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
    for (int x = 0; x < 8; ++x) {
      pf[0][x] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s0[x], c, neg_m));
      pf[1][x] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s0[8 + x], c, neg_m));
      pf[2][x] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s1[x], c, neg_m));
      pf[3][x] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s1[8 + x], c, neg_m));
    }
    // row sum of the rounded probabilities (the values the PV product uses)
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int x = 0; x < 8; x += 2) {
        const bf16x2 pp = {pf[ks][x], pf[ks][x + 1]};
        lsum = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, lsum, false);
      }

    // ---- O^T += V^T P^T : 4 value blocks x 4 key steps
    const uint4 *vt = sm.vt[buf];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      bf16x8 vf[4];
#pragma unroll
      for (int d = 0; d < 4; ++d) vf[d] = as_bf16x8(vt[v_slot(d * 32 + n, ks * 2 + g)]);
#pragma unroll
      for (int d = 0; d < 4; ++d)
        o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[d], pf[ks], o[d], 0, 0, 0);
    }

    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  }

  // ---- epilogue: O^T[dv][row] with dv = d*32 + (x>>2)*8 + g*4 + (x&3)
  const float ltot = half_swap_sum(lsum);
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
