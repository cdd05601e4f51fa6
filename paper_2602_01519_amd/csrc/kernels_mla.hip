// bf16 MLA link attention (absorbed latent form) on gfx950 matrix cores:
// one latent KV "head" of width 576 (512 latent + 64 rope), value = the first
// 512 entries of each row, every query head reads the same latent rows
// (the DeepSeek-V2-Lite backbone of Sec. 5.1). Keys are walked as in the GQA
// kernels: linked chunks in link order (Sec. 4.2, no mask), then own KV
// (Sec. 4.1, causal, bottom-right aligned).
//
// Workgroup: 4 waves, 64 rows (two row blocks of 32; a row is (query token,
// head)), 64-key tiles of the latent rows staged in LDS (72 KB per tile,
// double-buffered with load-to-LDS copies). Per tile:
//   1. wave (rb, kb) computes S^T[32 keys kb][32 rows rb] = K Q^T over the 576
//      latent dims (36 x v_mfma_f32_32x32x16_bf16, Q held in registers);
//   2. the four waves exchange per-row tile maxima through LDS, update the
//      shared running max (lazy rescale, identical in every wave), turn their
//      scores into bf16 probabilities and publish them in LDS;
//   3. wave w owns value dims [128 w, 128 w + 128) of all 64 rows and adds
//      O^T += V^T P^T (32 MFMAs): V^T fragments are read straight out of the
//      key tile with transposing LDS reads (ds_read_b64_tr_b16), so the
//      latent rows are stored once, row-major, and serve as K and as V.
// K tile layout: row r (1152 bytes = 72 chunks of 16 B) keeps chunk c at
// c ^ f(r), f(r) = ((r >> 1) & 1) << 2 | ((r >> 2) & 3), which makes both the
// 16-byte QK fragment reads and the 8-byte transposing PV reads bank-conflict
// free (64 banks).
#include "pic_internal.hpp"

namespace pic {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void *lds_ptr;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int kDK = 576;                 // key / query width
constexpr int kDV = 512;                 // value width (latent part)
constexpr int kChunks = kDK * 2 / 16;    // 72 chunks of 16 B per key row
constexpr int kSteps = kDK / 16;         // 36 QK steps of 16 dims
constexpr int kRowsMla = 64;             // rows per workgroup
constexpr float kLazy = 8.0f;
constexpr int kWin = 32;                 // link-table entries staged in LDS
constexpr int kTileChunks = kTile * kChunks;   // 4608 chunks per key tile
constexpr int kDmaPerLane = kTileChunks / 256; // 18 load-to-LDS per lane per tile
constexpr int kAhead = 6;                // K fragment read lead in the QK loop

__device__ __forceinline__ int swz(int r) { return (((r >> 1) & 1) << 2) | ((r >> 2) & 3); }
__device__ __forceinline__ int kpos(int r, int c) { return r * kChunks + (c ^ swz(r)); }

__device__ __forceinline__ int key_of_m(int m) {
  const int a = m >> 3, gg = (m >> 2) & 1, c = m & 3;
  return (a >> 1) * 16 + gg * 8 + (a & 1) * 4 + c;
}
__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ const char *uni(const void *p) {
  const uint64_t u = (uint64_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
  return (const char *)(((uint64_t)hi << 32) | lo);
}
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

struct MlaSmem {
  uint4 k[2][kTileChunks];                 // two 72 KB key tiles
  uint4 p[2][2][2][64];                    // probabilities [rb][kb][h][lane]
  float xm[4][32];                         // per-wave row maxima / row sums
  LinkEntry win[kWin];
};

struct TileRef {
  const char *k;    // first latent row of the tile (bytes)
  int nvalid, j0, own;
};

struct Cursor {
  const LinkParams *p;
  ReqEntry R;
  LinkEntry *win;
  int li, wb;
};

__device__ __forceinline__ void load_window(Cursor &c) {
  const int n = min(kWin, c.R.nlinks - c.wb);
  for (int i = threadIdx.x; i < n; i += blockDim.x) c.win[i] = c.p->links[c.R.link0 + c.wb + i];
}

__device__ __forceinline__ TileRef tile_ref(Cursor &c, int t) {
  for (;;) {
    if (c.li - c.wb >= kWin) {
      __syncthreads();
      c.wb += kWin;
      load_window(c);
      __syncthreads();
    }
    const LinkEntry &e = c.win[c.li - c.wb];
    const int tile0 = uni(e.tile0), lp = uni(e.lp);
    if (t < tile0 + lp / kTile) {
      const int tt = t - tile0;
      TileRef r;
      r.nvalid = min(kTile, uni(e.len) - tt * kTile);
      r.j0 = tt * kTile;
      r.own = t >= c.R.doc_tiles;
      r.k = uni(e.k) + (int64_t)tt * kTile * kDK * 2;
      return r;
    }
    ++c.li;
  }
}

// Copy of one 64-key tile (64 rows x 1152 B) into an LDS buffer: load u of a
// lane fills slot (u * 256 + tid), which holds chunk (slot % 72) ^ f(row).
__device__ __forceinline__ void issue_tile(const TileRef &r, const uint32_t (&goff)[kDmaPerLane],
                                           uint4 *dst, int wave) {
#pragma unroll
  for (int u = 0; u < kDmaPerLane; ++u)
    __builtin_amdgcn_global_load_lds(r.k + goff[u], (lds_ptr)(dst + u * 256 + wave * 64), 16, 0,
                                     0);
}

__global__ __launch_bounds__(256, 1) void link_mla_kernel(LinkParams p) {
  __shared__ MlaSmem sm;
  const int lane = threadIdx.x & 63;
  const int wave = uni(threadIdx.x >> 6);
  const int n = lane & 31, g = lane >> 5;
  const int rb_s = wave >> 1, kb_s = wave & 1;      // this wave's score tile

  const int nrb = p.nrb;
  const int grp = blockIdx.x / nrb, rblk = blockIdx.x % nrb;
  const int split = blockIdx.y;
  if (grp >= p.batch) return;
  Cursor cur;
  cur.p = &p;
  cur.R = p.reqs[p.order[grp]];
  const ReqEntry &R = cur.R;
  const int group = p.group;           // query heads (one latent kv head)
  const int nrows = R.lq * group;
  const int row0 = rblk * kRowsMla;
  if (row0 >= nrows) return;
  const int t_begin = (int)((int64_t)R.tiles * split / p.num_splits);
  const int t_end = (int)((int64_t)R.tiles * (split + 1) / p.num_splits);

  // Rows: this lane's row in block rb is row0 + 32 rb + n.
  int lim[2];
  bool rvalid[2];
  int64_t orow[2];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const int row = row0 + 32 * rb + n;
    rvalid[rb] = row < nrows;
    const int qi = rvalid[rb] ? row / group : 0;
    const int qh = rvalid[rb] ? row % group : 0;
    lim[rb] = rvalid[rb] ? qi + R.ls - R.lq : -1;
    orow[rb] = (int64_t)(R.q0 + qi) * p.n_q_heads + qh;
  }

  // Per-lane byte offsets of the tile copy.
  uint32_t goff[kDmaPerLane];
#pragma unroll
  for (int u = 0; u < kDmaPerLane; ++u) {
    const int s = u * 256 + wave * 64 + lane;
    const int r = s / kChunks, q = s - r * kChunks;
    goff[u] = (uint32_t)(r * kDK * 2 + (q ^ swz(r)) * 16);
  }

  cur.win = sm.win;
  cur.li = 0;
  cur.wb = 0;
  load_window(cur);
  __syncthreads();

  TileRef ref0{}, ref1{};
  if (t_begin < t_end) {
    ref0 = tile_ref(cur, t_begin);
    issue_tile(ref0, goff, sm.k[0], wave);
  }

  // Q of the score tile's row block: d = 16 st + 8 g + (0..7)
  bf16x8 qf[kSteps];
  {
    const uint4 *qrow = (const uint4 *)((const uint16_t *)p.q + orow[rb_s] * kDK);
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (rvalid[rb_s]) v = qrow[2 * st + g];
      qf[st] = as_bf16x8(v);
    }
  }

  f32x16 o[4][2];                // O^T[dv block][row block], dv = 128 wave + 32 db + ...
#pragma unroll
  for (int db = 0; db < 4; ++db)
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int x = 0; x < 16; ++x) o[db][rb][x] = 0.f;
  float m_used[2] = {-INFINITY, -INFINITY};
  float lsum = 0.f;             // partial row sum of the score tile (rb_s, kb_s)
  const float sc = p.scale_log2;
  // QK fragment addresses (16-byte units): chunk 2 st + g of key row krow sits
  // at krow * 72 + ((2 st + g) ^ f(krow)) = kq[st % 4] + 8 (st / 4).
  const int krow = 32 * kb_s + key_of_m(n);
  int kq[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) kq[b] = krow * kChunks + ((2 * b + g) ^ swz(krow));
  // Transposing-read byte offsets: in read t, lane (q = lane/16, s = lane%16)
  // points at key row 8 (q/2) + 4 t + s/4 (+16 ks) and value dims
  // 128 wave + 32 db + 16 (q%2) + 4 (s%4) .. +3; with db = 2 a + b the
  // offset is tr_off[t][b] + 128 a (+ ks * 16 rows).
  int tr_off[2][2];
  {
    const int q4 = lane >> 4, s4 = lane & 15;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int row = 8 * (q4 >> 1) + 4 * t + (s4 >> 2);
        const int dv = 128 * wave + 32 * b + 16 * (q4 & 1) + 4 * (s4 & 3);
        tr_off[t][b] = kpos(row, dv >> 3) * 16 + ((dv & 7) >> 2) * 8;
      }
  }

  auto compute = [&](const uint4 *kt, const TileRef &ref) {
    // 1. scores
    f32x16 s;
#pragma unroll
    for (int x = 0; x < 16; ++x) s[x] = 0.f;
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
      // chunk 2 st + g of key row krow: (2 st + g) ^ f keeps 8 (st / 4) intact
      const bf16x8 kf = as_bf16x8(kt[kq[st & 3] + 8 * (st >> 2)]);
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[st], s, 0, 0, 0);
    }
    // K fragment reads run kAhead steps ahead of their MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, kAhead, 0);
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if (st + kAhead < kSteps) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    // s[x]: key 32 kb_s + (x>>3)*16 + g*8 + (x&7) of row 32 rb_s + n
    if (ref.own || ref.nvalid < kTile) {
      const int kl = (ref.own ? min(lim[rb_s] - ref.j0, ref.nvalid - 1) : ref.nvalid - 1) -
                     32 * kb_s - g * 8;
#pragma unroll
      for (int x = 0; x < 16; ++x)
        if ((x >> 3) * 16 + (x & 7) > kl) s[x] = -INFINITY;
    }
    float tmax = -INFINITY;
#pragma unroll
    for (int x = 0; x < 16; x += 2) tmax = fmaxf(fmaxf(tmax, s[x]), s[x + 1]);
    tmax = half_swap_max(tmax);
    if (g == 0) sm.xm[wave][n] = tmax;
    __syncthreads();
    // 2. shared running max of both row blocks (same arithmetic in every wave)
    float mnew[2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
      mnew[rb] = fmaxf(m_used[rb], fmaxf(sm.xm[2 * rb][n], sm.xm[2 * rb + 1][n]) * sc);
    if (__any(mnew[0] > m_used[0] + kLazy || mnew[1] > m_used[1] + kLazy)) {
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        const float alpha =
            mnew[rb] == m_used[rb] ? 1.f : __builtin_amdgcn_exp2f(m_used[rb] - mnew[rb]);
        m_used[rb] = mnew[rb];
        if (rb == rb_s) lsum *= alpha;
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
          for (int x = 0; x < 16; ++x) o[db][rb][x] *= alpha;
      }
    }
    const float mu = rb_s ? m_used[1] : m_used[0];
    const float neg_m = mu == -INFINITY ? 0.f : -mu;
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      bf16x8 pf;
#pragma unroll
      for (int x = 0; x < 8; ++x)
        pf[x] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s[8 * h + x], sc, neg_m));
#pragma unroll
      for (int x = 0; x < 8; x += 2) {
        const bf16x2 pp = {pf[x], pf[x + 1]};
        lsum = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, lsum, false);
      }
      sm.p[rb_s][kb_s][h][lane] = __builtin_bit_cast(uint4, pf);
    }
    __syncthreads();
    // 3. O^T += V^T P^T for this wave's 128 value dims
    const char *kbytes = (const char *)kt;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const bf16x8 pb0 = as_bf16x8(sm.p[0][ks >> 1][ks & 1][lane]);
      const bf16x8 pb1 = as_bf16x8(sm.p[1][ks >> 1][ks & 1][lane]);
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        // transposing reads (see tr_off): key rows 16 ks + .., value block db
        i16x4 part[2];
#pragma unroll
        for (int t = 0; t < 2; ++t)
          part[t] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (lds_i16x4 *)(kbytes + tr_off[t][db & 1] + ks * 16 * kChunks * 16 + (db >> 1) * 128));
        const bf16x8 vf = __builtin_bit_cast(
            bf16x8, (uint4){(uint32_t)(uint16_t)part[0][0] | ((uint32_t)(uint16_t)part[0][1] << 16),
                            (uint32_t)(uint16_t)part[0][2] | ((uint32_t)(uint16_t)part[0][3] << 16),
                            (uint32_t)(uint16_t)part[1][0] | ((uint32_t)(uint16_t)part[1][1] << 16),
                            (uint32_t)(uint16_t)part[1][2] | ((uint32_t)(uint16_t)part[1][3] << 16)});
        o[db][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb0, o[db][0], 0, 0, 0);
        o[db][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb1, o[db][1], 0, 0, 0);
      }
    }
    // per (ks, db): 2 transposing reads (+2 probability reads per ks) then 2 MFMAs
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      }
    }
  };

  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  for (int t = t_begin; t < t_end; t += 2) {
    if (t + 1 < t_end) {
      ref1 = tile_ref(cur, t + 1);
      issue_tile(ref1, goff, sm.k[1], wave);
    }
    compute(sm.k[0], ref0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (t + 1 >= t_end) break;
    if (t + 2 < t_end) {
      ref0 = tile_ref(cur, t + 2);
      issue_tile(ref0, goff, sm.k[0], wave);
    }
    compute(sm.k[1], ref1);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  }

  // Row sums: the two score waves of a row block hold halves of it.
  const float lhalf = half_swap_sum(lsum);
  if (g == 0) sm.xm[wave][n] = lhalf;
  __syncthreads();
  float ltot[2];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) ltot[rb] = sm.xm[2 * rb][n] + sm.xm[2 * rb + 1][n];

  const int total_rows = p.total_q * p.n_q_heads;
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    if (!rvalid[rb]) continue;
    if (p.num_splits == 1) {
      const float inv = ltot[rb] > 0.f ? 1.f / ltot[rb] : 0.f;
      uint16_t *out = (uint16_t *)p.out + orow[rb] * kDV;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const int dv = 128 * wave + 32 * db + jj * 8 + g * 4;
          __bf16 v4[4];
#pragma unroll
          for (int x = 0; x < 4; ++x) v4[x] = (__bf16)(o[db][rb][jj * 4 + x] * inv);
          *(uint2 *)(out + dv) = __builtin_bit_cast(uint2, v4);
        }
      if (p.lse && wave == 0 && g == 0)
        p.lse[orow[rb]] =
            ltot[rb] > 0.f ? (m_used[rb] + log2f(ltot[rb])) * 0.69314718055994531f : -INFINITY;
    } else {
      const int64_t prow = (int64_t)split * total_rows + orow[rb];
      float *po = p.part_o + prow * kDV;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          const int dv = 128 * wave + 32 * db + jj * 8 + g * 4;
          *(float4 *)(po + dv) = make_float4(o[db][rb][jj * 4], o[db][rb][jj * 4 + 1],
                                             o[db][rb][jj * 4 + 2], o[db][rb][jj * 4 + 3]);
        }
      if (wave == 0 && g == 0) {
        p.part_m[prow] = ltot[rb] > 0.f ? m_used[rb] : -INFINITY;
        p.part_l[prow] = ltot[rb];
      }
    }
  }
}

}  // namespace

int mla_rows_per_block() { return kRowsMla; }

hipError_t launch_link_mla(const LinkParams &p, hipStream_t st, const char **name) {
  *name = "link_mla_kernel";
  dim3 grid(p.batch * p.nrb, p.num_splits);
  hipLaunchKernelGGL(link_mla_kernel, grid, dim3(256), 0, st, p);
  return hipGetLastError();
}

}  // namespace pic
