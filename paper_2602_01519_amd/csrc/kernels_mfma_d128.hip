// bf16 GQA link attention on gfx950 matrix cores, head dim 128.
//
// Workgroup: 8 waves x 32 rows = 256 rows of one (request, kv head), where a
// row is (query token, query head of the GQA group): the group's query heads
// share every K/V byte the workgroup stages. One workgroup per CU (2 waves
// per SIMD); against two 4-wave workgroups per CU this halves the tile
// copies and L2 reads per FLOP (measured: 4.5% faster on llama_prefill). Keys are walked in 64-key tiles:
// the request's linked chunks in link order (Sec. 4.2: concatenated along
// the document axis, no mask), then its own KV (Sec. 4.1: causal mask,
// bottom-right aligned).
//
// Per tile and wave:
//   S^T[64 keys][32 rows] = K . Q^T        16 x v_mfma_f32_32x32x16_bf16
//   online softmax on S^T (each lane holds one row's 32 scores)
//   O^T[128][32 rows]    += V^T . P^T      16 x v_mfma_f32_32x32x16_bf16
// K and V^T tiles are copied global -> LDS by the load-to-LDS path
// (buffer_load_dwordx4 ... lds, no register staging), double-buffered in four
// distinct LDS arrays; the tile loop is unrolled by two so every access names
// its buffer statically, which lets the compiler see that a tile's reads and
// the next tile's copy never alias (no wait on the copy before the reads).
// The next tile's copies (4 per lane) are spread over the current tile's QK
// loop rather than issued as one burst: a burst from all 8 waves of a CU at
// once stalls every wave at issue until the copy path drains.
// Calls whose (request, kv head) row counts do not fill a workgroup (short
// questions) have few busy waves and short tiles, and one tile in flight
// per CU does not cover the copies' latency: they run a three-stage loop
// (three buffer pairs, 96 KB; the copy of tile t+2 is issued while tile t+1
// is in flight), measured 13.5% faster on the skinny-question workload and
// about 1% slower where every wave is busy.
// The store keeps V transposed per chunk in panels of 32 tokens, so a V^T
// tile is two contiguous 8 KB panels of 128 rows of 64 bytes. The M index of the QK^T product is permuted (key row
// pi(m) feeds M index m) so that the scores a lane receives for a 16-key PV
// step are 8 consecutive keys: P^T feeds the PV product straight from
// registers and the V^T fragment for those keys is one 16-byte LDS read.
//
// Softmax: log2 domain (scale * log2 e applied by FMA). Probabilities are
// formed against the running max as it stands; only when a lane's share of
// the tile's row sum exceeds 2^64 (or a row with a visible key has no
// running max yet, i.e. on its first such tile) does the wave form the
// tile's row max (one cross-half lane swap), rescale O and the sums, and
// redo the tile. fp32 and bf16 keep their relative precision at any such
// magnitude, so almost every tile skips both the max and the rescale. Row
// sums are kept per lane half (bf16 dot products of the rounded
// probabilities, i.e. the weights the PV product uses) and added at the end.
#include "pic_internal.hpp"

namespace pic {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) void *lds_ptr;

constexpr int kD = 128;
constexpr int kWaves = 8;                       // waves (32 rows each) per workgroup
constexpr int kCopySets = 16 / kWaves;          // 64-chunk copies per lane per K (or V) tile
constexpr int kRowsPerWave = 32;
constexpr int kRows = kWaves * kRowsPerWave;
constexpr float kJumpSum = 18446744073709551616.0f;   // 2^64: redo a tile past it
constexpr int kQkAhead = 5;    // K-fragment read lead, in QK steps
constexpr int kPvAhead = 8;    // V-fragment read lead, in PV MFMAs

// LDS tiles, 16-byte chunks XOR-swizzled within each row. The swizzles keep
// every fragment read conflict-free whether a 16-byte-per-lane read is served
// 8 or 16 lanes at a time: the 8 (16) lanes of a group read 8 (16) distinct
// chunk positions of the bank row.
//   K   [key][16 chunks of 8 d]:   chunk c at c ^ hk(key), hk swaps bits 2 and 3
//       of key & 15 (a lane group reads keys {0-3, 8-11} or {4-7, 12-15}).
//   V^T [dv][8 chunks of 8 keys]:  chunk c at c ^ hv(dv & 31) with
//       hv(x) = (x ^ (x >> 3)) & 7 (two 128-byte rows share a 256-byte bank
//       row; depending on dv & 31 only, the 4 value blocks of a lane share
//       one address register).
__device__ __forceinline__ int hk(int key) {
  return (key & 3) | ((key & 8) >> 1) | ((key & 4) << 1);
}
__device__ __forceinline__ int hv(int x) { return (x ^ (x >> 3)) & 7; }
__device__ __forceinline__ int k_slot(int key, int c) { return key * 16 + (c ^ hk(key & 15)); }
__device__ __forceinline__ int v_slot(int dv, int c) { return dv * 8 + (c ^ hv(dv & 31)); }

// Key row that feeds M index m of the QK^T product (see the file comment).
__device__ __forceinline__ int key_of_m(int m) {
  const int a = m >> 3, gg = (m >> 2) & 1, c = m & 3;
  return (a >> 1) * 16 + gg * 8 + (a & 1) * 4 + c;
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }

__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Max / sum of a value over lanes i and i ^ 32 (the two key halves of a row).
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

// A key tile: workgroup-uniform facts.
struct TileRef {
  const char *k;     // first K row of the tile (kv head applied), bytes
  const char *v;     // V^T row 0 at the tile's first key (kv head applied)
  int lp;            // padded tokens of the link
  int nvalid;        // valid keys in the tile
  int j0;            // key index of the tile's first key within its link
  int tok;           // ... within the request's linked rows (document tiles)
  int own;           // the tile belongs to the request's own KV (causal mask)
};

// The link and request tables are read through the constant address space:
// every lookup is a scalar load and the link cursor lives in scalar
// registers (no LDS, no barrier).
typedef __attribute__((address_space(4))) const LinkEntry *const_links;
typedef __attribute__((address_space(4))) const ReqEntry *const_reqs;
typedef __attribute__((address_space(4))) const int32_t *const_ints;

struct Ctx {
  ReqEntry R;
  int kvh, wave, lane, n, g;
  const_links links;           // the request's links
  int li;                      // cursor: current link
  const char *lk, *lv;         // its K / V^T blocks
  int llen, llp, ltile0, lend; // its tokens, padded tokens, first tile, tile after its last
  int ltok0;                   // its first row within the request's linked rows
  uint32_t koff[kCopySets];    // byte offsets of this lane's K chunks within a tile
  uint32_t voff[kCopySets];    // byte offsets of its V^T chunks within a tile's two panels
};

__device__ __forceinline__ void cursor_load(Ctx &c) {
  c.lk = (const char *)c.links[c.li].k;
  c.lv = (const char *)c.links[c.li].v;
  c.llen = c.links[c.li].len;
  c.llp = c.links[c.li].lp;
  c.ltile0 = c.links[c.li].tile0;
  c.ltok0 = c.links[c.li].tok0;
  c.lend = c.ltile0 + (c.llen + kTile - 1) / kTile;
}

// Tile t of the request (t only grows across calls).
__device__ __forceinline__ TileRef tile_ref(Ctx &c, int t) {
  while (t >= c.lend) {
    ++c.li;
    cursor_load(c);
  }
  const int tt = t - c.ltile0;
  TileRef r;
  r.lp = c.llp;
  r.nvalid = min(kTile, c.llen - tt * kTile);
  r.j0 = tt * kTile;
  r.tok = c.ltok0 + tt * kTile;
  r.own = t >= c.R.doc_tiles;
  r.k = c.lk + ((int64_t)c.kvh * c.llp + tt * kTile) * kD * 2;
  r.v = c.lv + ((int64_t)c.kvh * kD * c.llp + tt * kTile * kD) * 2;   // the tile's two panels
  return r;
}

// Copies of a tile into LDS: lane i of a load-to-LDS lands at slot base + i,
// so each lane fetches the global chunk that belongs at that slot of the
// swizzled layout (uniform base address + per-lane 32-bit offset).
// Copy i (0 .. 2 kCopySets - 1) of a tile: i < kCopySets is K chunk set i,
// the rest V^T chunk set i - kCopySets.
// The copies go through a buffer resource (MUBUF load-to-LDS) rather than a
// global (FLAT-encoded) one: the compiler counts a FLAT load-to-LDS as a
// possible LDS access in flight, which turns every wait for an LDS fragment
// read into a wait for all of them; with buffer copies it keeps precise
// counts and the fragment reads stay ahead of their MFMAs.
// kAux: the copies' cache policy; kNonTemporal for calls in which every K/V
// byte is read by one workgroup only (short questions: the key range is
// split, not shared by row blocks), so it need not stay in the caches.
constexpr int kNonTemporal = 2;
template <int kAux>
__device__ __forceinline__ void lds_dma16(const void *base, uint32_t voff, uint4 *dst) {
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, -1, 0x00020000);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr)dst, 16, voff, 0, 0, kAux);
}

template <int kAux>
__device__ __forceinline__ void tile_copy(const Ctx &c, int i, const TileRef &r, uint4 *kdst,
                                          uint4 *vdst) {
  if (i < kCopySets) {
    lds_dma16<kAux>(r.k, c.koff[i], kdst + (i * kWaves + c.wave) * 64);
  } else {
    const int u = i - kCopySets;
    lds_dma16<kAux>(r.v, c.voff[u], vdst + (u * kWaves + c.wave) * 64);
  }
}
template <int kAux>
__device__ __forceinline__ void issue_tile(const Ctx &c, const TileRef &r, uint4 *kdst,
                                           uint4 *vdst) {
#pragma unroll
  for (int i = 0; i < 2 * kCopySets; ++i) tile_copy<kAux>(c, i, r, kdst, vdst);
}

// Workgroup barrier of the tile loop, without the memory fence of
// __syncthreads (whose release half waits for every copy in flight): the
// wait for the copies that must have landed is explicit before it, LDS reads
// of the tile are done, and the empty asm statements keep the compiler from
// moving memory accesses across it.
__device__ __forceinline__ void tile_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

struct Acc {
  f32x16 o[4];
  float m_used, lsum;
};

// Per-row limit on the visible linked rows: dl for this lane's row, wmin
// its minimum over the wave (both far above any row count without limits).
struct DocLim {
  int dl, wmin;
};

// Masks keys past the tile's valid end, in own tiles keys after the row's
// causal limit, and in document tiles rows at or past the row's limit.
// s0[x] / s1[x] hold key (x>>3)*16 + g*8 + (x&7) (+32).
// kLim: the call carries per-row limits (a separate instantiation, so that
// calls without them run no limit code).
template <bool kLim>
__device__ __forceinline__ void mask_tile(const Ctx &c, f32x16 &s0, f32x16 &s1, const TileRef &r,
                                          int lim, const DocLim &dlm) {
  const int nvalid = r.nvalid;
  if (r.own || nvalid < kTile || (kLim && r.tok + kTile > dlm.wmin)) {
    // visible iff key <= kl; compared as (key - g*8) against kl - g*8 so the
    // left side is a compile-time constant per element
    const int kl = (r.own   ? min(lim - r.j0, nvalid - 1)
                    : kLim ? min(dlm.dl - r.tok, nvalid) - 1
                           : nvalid - 1) -
                   c.g * 8;
#pragma unroll
    for (int x = 0; x < 16; ++x) {
      const int key = (x >> 3) * 16 + (x & 7);
      if (key > kl) s0[x] = -INFINITY;
      if (key + 32 > kl) s1[x] = -INFINITY;
    }
  }
}

// One tile: S = K Q^T from kt, mask, online softmax (log2 domain, against
// the running max as it stands), O += V^T P^T from vt. In both matrix sections the LDS fragment
// reads are issued a few MFMAs ahead of their use (scheduling groups), so an
// MFMA does not wait on the read issued right before it.
template <bool kLim, int kAux>
__device__ __forceinline__ void compute_tile(const Ctx &c, const uint4 *kt, const uint4 *vt,
                                             const bf16x8 (&qf)[8], Acc &a, const TileRef &ref,
                                             int lim, const DocLim &dlm, float sc,
                                             const TileRef &nref, uint4 *nk, uint4 *nv) {
  const int krow0 = key_of_m(c.n);
  f32x16 s0, s1;
#pragma unroll
  for (int x = 0; x < 16; ++x) {
    s0[x] = 0.f;
    s1[x] = 0.f;
  }
  // QK, pipelined by hand: K reads kQkAhead steps ahead of their MFMAs, one
  // copy of the next tile per step; sched_barrier keeps that order.
  bf16x8 ka[8], kb[8];
#pragma unroll
  for (int st = 0; st < kQkAhead; ++st) {
    ka[st] = as_bf16x8(kt[k_slot(krow0, st * 2 + c.g)]);
    kb[st] = as_bf16x8(kt[k_slot(32 + krow0, st * 2 + c.g)]);
  }
#pragma unroll
  for (int st = 0; st < 8; ++st) {
    if (st + kQkAhead < 8) {
      ka[st + kQkAhead] = as_bf16x8(kt[k_slot(krow0, (st + kQkAhead) * 2 + c.g)]);
      kb[st + kQkAhead] = as_bf16x8(kt[k_slot(32 + krow0, (st + kQkAhead) * 2 + c.g)]);
    }
    constexpr int kEvery = 8 / (2 * kCopySets);   // QK steps per copy
    if (st % kEvery == 0) tile_copy<kAux>(c, st / kEvery, nref, nk, nv);
    s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[st], qf[st], s0, 0, 0, 0);
    s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kb[st], qf[st], s1, 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
  mask_tile<kLim>(c, s0, s1, ref, lim, dlm);

  // Probabilities against the running max as it stands, and this lane's
  // (bf16-rounded) sum of them. The tile's own max is only computed when
  // some lane's sum exceeds 2^64 (a probability could then overflow in a
  // later sum) or a row with a visible key has no running max yet; the tile
  // is then redone against the new max.
  bf16x8 pf[4];
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  auto probs = [&]() {
    const float neg_m = a.m_used == -INFINITY ? 0.f : -a.m_used;
#pragma unroll
    for (int x = 0; x < 8; ++x) {
      pf[0][x] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s0[x], sc, neg_m));
      pf[1][x] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s0[8 + x], sc, neg_m));
      pf[2][x] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s1[x], sc, neg_m));
      pf[3][x] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s1[8 + x], sc, neg_m));
    }
    float ts = 0.f;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int x = 0; x < 8; x += 2) {
        const bf16x2 pp = {pf[ks][x], pf[ks][x + 1]};
        ts = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, ts, false);
      }
    return ts;
  };
  float ts = probs();
  if (__any(!(ts <= kJumpSum) || (a.m_used == -INFINITY && ts > 0.f))) {
    float tmax = -INFINITY;
#pragma unroll
    for (int x = 0; x < 16; x += 2) {
      tmax = fmaxf(fmaxf(tmax, s0[x]), s0[x + 1]);
      tmax = fmaxf(fmaxf(tmax, s1[x]), s1[x + 1]);
    }
    tmax = half_swap_max(tmax);
    const float mnew = fmaxf(a.m_used, tmax * sc);
    const float alpha = mnew == a.m_used ? 1.f : __builtin_amdgcn_exp2f(a.m_used - mnew);
    a.m_used = mnew;
    a.lsum *= alpha;
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int x = 0; x < 16; ++x) a.o[d][x] *= alpha;
    ts = probs();
  }
  a.lsum += ts;

#pragma unroll
  for (int ks = 0; ks < 4; ++ks)
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      const bf16x8 vf = as_bf16x8(vt[v_slot(d * 32 + c.n, ks * 2 + c.g)]);
      a.o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[ks], a.o[d], 0, 0, 0);
    }
  // V reads run kPvAhead MFMAs ahead
  __builtin_amdgcn_sched_group_barrier(0x100, kPvAhead, 0);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if (i + kPvAhead < 16) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
}

// kStages: tile buffer pairs, 2 or 3 (see the tile loops).
template <bool kLim, int kStages>
__global__ __launch_bounds__(kWaves * 64, 8 / kWaves) void link_mfma_d128_kernel(LinkParams p) {
  __shared__ uint4 sk0[kTile * 16], sk1[kTile * 16];
  __shared__ uint4 sv0[kD * 8], sv1[kD * 8];
  __shared__ uint4 sk2[kStages == 3 ? kTile * 16 : 1], sv2[kStages == 3 ? kD * 8 : 1];

  constexpr int kAux = kStages == 3 ? kNonTemporal : 0;
  Ctx c;
  c.lane = threadIdx.x & 63;
  c.wave = uni(threadIdx.x >> 6);
  c.n = c.lane & 31;
  c.g = c.lane >> 5;

  // XCD-aware work mapping: consecutive blocks go round-robin to the XCDs;
  // all row blocks of one (request, kv head) land on the same XCD (same L2)
  // and are dispatched back to back. Heaviest requests first.
  const int lin = blockIdx.x;
  const int xcd = lin % p.n_xcd, j = lin / p.n_xcd;
  const int grp = xcd + p.n_xcd * (j / p.nrb);
  const int rb = j % p.nrb;
  const int split = blockIdx.y;
  if (grp >= p.batch * p.n_kv_heads) return;
  const int req_i = ((const_ints)p.order)[grp / p.n_kv_heads];
  c.kvh = grp % p.n_kv_heads;
  {
    const_reqs rq = (const_reqs)p.reqs + req_i;
    c.R.link0 = rq->link0;
    c.R.nlinks = rq->nlinks;
    c.R.q0 = rq->q0;
    c.R.lq = rq->lq;
    c.R.ls = rq->ls;
    c.R.doc_tiles = rq->doc_tiles;
    c.R.tiles = rq->tiles;
  }
  const ReqEntry &R = c.R;
  const int group = p.group;
  const int nrows = R.lq * group;
  const int row0 = rb * kRows;
  if (row0 >= nrows) return;
  // Own tiles past the causal limit of the block's last row hold no key any
  // of its rows sees: the block's key range ends at the last visible one.
  const int vis = visible_tiles(R, min(nrows - 1, row0 + kRows - 1) / group);
  const int t_begin = (int)((int64_t)vis * split / p.num_splits);
  const int t_end = (int)((int64_t)vis * (split + 1) / p.num_splits);

  // This lane's row. A wave whose 32 rows are all past the request's rows
  // (short questions: a 16-token question fills 64 of the 256 rows) only
  // copies its share of every tile and meets the barriers, leaving its SIMD
  // to the other workgroup on the CU.
  const bool active = row0 + c.wave * kRowsPerWave < nrows;
  const int row = row0 + c.wave * kRowsPerWave + c.n;
  const bool rvalid = row < nrows;
  const int qi = rvalid ? row / group : 0;
  const int qh = c.kvh * group + (rvalid ? row % group : 0);
  const int lim = rvalid ? qi + R.ls - R.lq : -1;     // last visible own key
  const int64_t orow = (int64_t)(R.q0 + qi) * p.n_q_heads + qh;
  DocLim dlm{kNoLimit, kNoLimit};
  if (kLim) {
    if (rvalid) dlm.dl = p.doc_lim[R.q0 + qi];
    int w = dlm.dl;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) w = min(w, __shfl_xor(w, o));
    dlm.wmin = uni(w);
  }

  // Per-lane load-to-LDS offsets (see issue_k / issue_v).
#pragma unroll
  for (int u = 0; u < kCopySets; ++u) {
    const int s = (u * kWaves + c.wave) * 64 + c.lane;
    const int key = s >> 4, kc = (s & 15) ^ hk(key & 15);
    c.koff[u] = (uint32_t)((key * kD + kc * 8) * 2);
    // V^T chunk cc (keys 8 cc .. 8 cc + 7) of value row dv: panel cc / 4,
    // row dv, 16-byte unit cc % 4
    const int dv = s >> 3, cc = (s & 7) ^ hv(dv & 31);
    c.voff[u] = (uint32_t)((cc >> 2) * kD * kPanel * 2 + dv * kPanel * 2 + (cc & 3) * 16);
  }

  c.links = (const_links)p.links + c.R.link0;
  c.li = 0;
  c.lk = c.lv = nullptr;
  c.llen = c.llp = c.ltile0 = c.lend = 0;
  if (c.R.nlinks > 0) cursor_load(c);

  // masking facts of the tile held in each buffer pair
  TileRef ref0{}, ref1{}, ref2{};
  if (t_begin < t_end) {
    ref0 = tile_ref(c, t_begin);
    issue_tile<kAux>(c, ref0, sk0, sv0);
  }

  // Q fragments: d = step*16 + g*8 + (0..7)
  bf16x8 qf[8];
  {
    const uint4 *qrow = (const uint4 *)((const uint16_t *)p.q + orow * kD);
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (rvalid) v = qrow[s * 2 + c.g];
      qf[s] = as_bf16x8(v);
    }
  }
  // three stages: the second tile is in flight while the first is computed
  // (a repeat of the first when there is no second, which keeps the wait
  // counts fixed)
  if (kStages == 3 && t_begin < t_end) {
    ref1 = t_begin + 1 < t_end ? tile_ref(c, t_begin + 1) : ref0;
    issue_tile<kAux>(c, ref1, sk1, sv1);
  }

  Acc a;
#pragma unroll
  for (int d = 0; d < 4; ++d)
#pragma unroll
    for (int x = 0; x < 16; ++x) a.o[d][x] = 0.f;
  a.m_used = -INFINITY;
  a.lsum = 0.f;
  const float sc = p.scale_log2;

  if constexpr (kStages == 3) {
    // the first tile and Q have landed; the second tile's copies (the last
    // 2 kCopySets issued) may still be in flight
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * kCopySets) : "memory");
    tile_barrier();

    // Three buffer pairs, unrolled by three so every access names its buffers
    // statically: tile t is computed while tile t+1 is in flight and the copy
    // of tile t+2 is issued (into the buffers tile t-1 used, free since the
    // last barrier). After each tile only tile t+1 has to have landed. Past
    // the last tile the copies repeat an earlier tile into buffers nobody
    // reads again.
    for (int t = t_begin; t < t_end; t += 3) {
      ref2 = t + 2 < t_end ? tile_ref(c, t + 2) : ref1;
      if (active)
        compute_tile<kLim, kAux>(c, sk0, sv0, qf, a, ref0, lim, dlm, sc, ref2, sk2, sv2);
      else
        issue_tile<kAux>(c, ref2, sk2, sv2);
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * kCopySets) : "memory");
      tile_barrier();
      if (t + 1 >= t_end) break;
      ref0 = t + 3 < t_end ? tile_ref(c, t + 3) : ref2;
      if (active)
        compute_tile<kLim, kAux>(c, sk1, sv1, qf, a, ref1, lim, dlm, sc, ref0, sk0, sv0);
      else
        issue_tile<kAux>(c, ref0, sk0, sv0);
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * kCopySets) : "memory");
      tile_barrier();
      if (t + 2 >= t_end) break;
      ref1 = t + 4 < t_end ? tile_ref(c, t + 4) : ref0;
      if (active)
        compute_tile<kLim, kAux>(c, sk2, sv2, qf, a, ref2, lim, dlm, sc, ref1, sk1, sv1);
      else
        issue_tile<kAux>(c, ref1, sk1, sv1);
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * kCopySets) : "memory");
      tile_barrier();
    }
    // no copy may still be writing LDS when the workgroup ends
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  } else {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();

    // Unrolled by two so every access names its buffers statically. The
    // copy of the next tile runs inside the current tile's QK loop; after the
    // last tile that copy repeats the current tile into the idle buffers,
    // which keeps the loop free of branches around it.
    for (int t = t_begin; t < t_end; t += 2) {
      // tile t in buffers 0; copy tile t+1 into buffers 1
      ref1 = t + 1 < t_end ? tile_ref(c, t + 1) : ref0;
      if (active)
        compute_tile<kLim, kAux>(c, sk0, sv0, qf, a, ref0, lim, dlm, sc, ref1, sk1, sv1);
      else
        issue_tile<kAux>(c, ref1, sk1, sv1);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
      if (t + 1 >= t_end) break;
      // tile t+1 in buffers 1; copy tile t+2 into buffers 0
      ref0 = t + 2 < t_end ? tile_ref(c, t + 2) : ref1;
      if (active)
        compute_tile<kLim, kAux>(c, sk1, sv1, qf, a, ref1, lim, dlm, sc, ref0, sk0, sv0);
      else
        issue_tile<kAux>(c, ref0, sk0, sv0);
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
    }
  }

  // ---- epilogue: O^T[dv][row] with dv = d*32 + (x>>2)*8 + g*4 + (x&3)
  const float ltot = half_swap_sum(a.lsum);
  if (!rvalid) return;
  const int total_rows = p.total_q * p.n_q_heads;
  if (p.num_splits == 1) {
    const float inv = ltot > 0.f ? 1.f / ltot : 0.f;
    uint16_t *out = (uint16_t *)p.out + orow * kD;
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int dv = d * 32 + jj * 8 + c.g * 4;
        __bf16 v4[4];
#pragma unroll
        for (int x = 0; x < 4; ++x) v4[x] = (__bf16)(a.o[d][jj * 4 + x] * inv);
        *(uint2 *)(out + dv) = __builtin_bit_cast(uint2, v4);
      }
    if (p.lse && c.g == 0)
      p.lse[orow] = ltot > 0.f ? (a.m_used + log2f(ltot)) * 0.69314718055994531f : -INFINITY;
  } else {
    const int64_t prow = (int64_t)split * total_rows + orow;
    float *po = p.part_o + prow * kD;
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int dv = d * 32 + jj * 8 + c.g * 4;
        *(float4 *)(po + dv) = make_float4(a.o[d][jj * 4], a.o[d][jj * 4 + 1],
                                           a.o[d][jj * 4 + 2], a.o[d][jj * 4 + 3]);
      }
    if (c.g == 0) {
      p.part_m[prow] = ltot > 0.f ? a.m_used : -INFINITY;
      p.part_l[prow] = ltot;
    }
  }
}

}  // namespace

int mfma_d128_rows_per_block() { return kRows; }
int mfma_d128_blocks_per_cu() { return 8 / kWaves; }

hipError_t launch_link_mfma_d128(const LinkParams &p, hipStream_t st, const char **name) {
  *name = "link_mfma_d128_kernel";
  dim3 grid(p.n_groups * p.nrb, p.num_splits);
  // Calls in which no (request, kv head) fills a workgroup's rows (short
  // questions: few busy waves, short tiles) are bound by the latency of the
  // tile copies and get the three-stage loop; the others the two-stage one.
  const dim3 block(kWaves * 64);
  if (p.max_rows < kRows) {
    if (p.doc_lim)
      hipLaunchKernelGGL((link_mfma_d128_kernel<true, 3>), grid, block, 0, st, p);
    else
      hipLaunchKernelGGL((link_mfma_d128_kernel<false, 3>), grid, block, 0, st, p);
  } else {
    if (p.doc_lim)
      hipLaunchKernelGGL((link_mfma_d128_kernel<true, 2>), grid, block, 0, st, p);
    else
      hipLaunchKernelGGL((link_mfma_d128_kernel<false, 2>), grid, block, 0, st, p);
  }
  return hipGetLastError();
}

}  // namespace pic
