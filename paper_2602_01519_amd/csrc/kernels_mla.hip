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
//      latent dims (36 x v_mfma_f32_32x32x16_bf16, Q held in registers) and
//      turns it into bf16 probabilities against the running max it already
//      holds, publishing them in LDS with one flag: some probability of the
//      wave may exceed 2^64 (its partial row sum does), or a row has no
//      running max yet;
//   2. one barrier; if any wave raised the flag (the first tile of every
//      row, and tiles whose max jumps by more than 2^64 over the running
//      max), all waves redo the tile: exact tile maxima through LDS, new
//      running max, rescaled accumulators, probabilities published again.
//      Otherwise the running max stays as it is: fp32 and bf16 keep their
//      relative precision at any magnitude, and probabilities stay <= 2^64,
//      so no per-tile rescale is needed;
//   3. wave w owns value dims [128 w, 128 w + 128) of all 64 rows and adds
//      O^T += V^T P^T (32 MFMAs): V^T fragments are read straight out of the
//      key tile with transposing LDS reads (ds_read_b64_tr_b16), so the
//      latent rows are stored once and serve as keys and as values;
//   4. one barrier ends the tile (buffer and probability reuse).
// Tile layout (16-byte chunks): latent part [64 rows][64 chunks], chunk c of
// row r at r*64 + (c ^ f(r)), f(r) = (r & 3) << 2 | (r >> 2) & 3; rope part
// [64 rows][8 chunks] after it, chunk c of row r at r*8 + (c ^ ((r >> 1) & 7)).
// Both the 16-byte score-operand reads and the 8-byte transposing reads are
// free of bank conflicts (64 banks), and a wave's tile copy needs only two
// lane offsets.
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
constexpr int kRowBytes = kDK * 2;       // 1152 bytes per latent row
constexpr int kLatChunks = 64;           // 16-byte chunks of the latent part
constexpr int kRopeChunks = 8;           // ... of the rope part
constexpr int kSteps = kDK / 16;         // 36 score steps of 16 dims
constexpr int kLatSteps = 32;            // of which over the latent part
constexpr int kRowsMla = 64;             // rows per workgroup
constexpr int kRopeBase = kTile * kLatChunks;                   // 4096 chunks
constexpr int kTileChunks = kTile * (kLatChunks + kRopeChunks); // 4608 chunks
constexpr float kJumpSum = 18446744073709551616.0f;  // 2^64: redo a tile past it
constexpr int kAhead = 6;                // K fragment read lead in the score loop
constexpr int kVLead = 3;                // value fragment read lead in the value loop

// Workgroup barrier for exchanges through LDS only (probabilities, flags,
// maxima inside a tile): it waits for this wave's LDS accesses but not for
// the next tile's copies in flight, which the memory fence of __syncthreads
// would wait for (forcing them to land before the value product). The empty
// asm statements keep the compiler from moving memory accesses across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

__device__ __forceinline__ int swz(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }
__device__ __forceinline__ int swr(int r) { return (r >> 1) & 7; }

__device__ __forceinline__ int key_of_m(int m) {
  const int a = m >> 3, gg = (m >> 2) & 1, c = m & 3;
  return (a >> 1) * 16 + gg * 8 + (a & 1) * 4 + c;
}
__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }
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

// The two 72 KB key tiles are separate __shared__ arrays: with one array the
// compiler cannot tell a tile's reads from the copy into the other tile and
// waits for that copy before every read.
__device__ __forceinline__ uint32_t lds_addr(const void *p) {
  return (uint32_t)(uintptr_t)(lds_ptr)p;
}

struct MlaSmem {
  uint4 p[2][2][2][64];                    // probabilities [rb][kb][h][lane]
  float xm[4][32];                         // per-wave row maxima of the tile / row sums
  int4 jump;                               // per wave: the tile must be redone
};

struct TileRef {
  const char *k;    // first latent row of the tile (bytes)
  int nvalid, j0, own;
  int tok;          // first key's row within the request's linked rows (document tiles)
};

// Walks a request's links in order. The tables are read through the
// constant address space, so every lookup is a scalar load and the cursor
// lives in scalar registers (no LDS, no barrier).
typedef __attribute__((address_space(4))) const LinkEntry *const_links;
typedef __attribute__((address_space(4))) const ReqEntry *const_reqs;
typedef __attribute__((address_space(4))) const int32_t *const_ints;

struct Cursor {
  const_links links;     // this request's links
  int li;                // current link
  const char *k;         // its first latent row
  int len, tile0, end;   // its tokens, first tile and the tile after its last
  int tok0;              // its first row within the request's linked rows
};

__device__ __forceinline__ void cursor_load(Cursor &c) {
  c.k = (const char *)c.links[c.li].k;
  c.len = c.links[c.li].len;
  c.tile0 = c.links[c.li].tile0;
  c.tok0 = c.links[c.li].tok0;
  c.end = c.tile0 + (c.len + kTile - 1) / kTile;
}

// Tile t of the request (tiles are visited in increasing order).
__device__ __forceinline__ TileRef tile_ref(Cursor &c, int t, int doc_tiles) {
  while (t >= c.end) {
    ++c.li;
    cursor_load(c);
  }
  const int tt = t - c.tile0;
  TileRef r;
  r.nvalid = min(kTile, c.len - tt * kTile);
  r.j0 = tt * kTile;
  r.tok = c.tok0 + tt * kTile;
  r.own = t >= doc_tiles;
  r.k = c.k + (int64_t)tt * kTile * kRowBytes;
  return r;
}

// Copy i (0..17) of one 64-key tile into an LDS buffer, 16 bytes per lane.
// Latent part, i < 16: wave w fills row r = 4i + w (64 lanes x 16 B),
// position j holding chunk j ^ f(r) = j ^ (w << 2) ^ (i & 3), so
// lat_off = 16 (lane ^ (w << 2)). Rope part, i = 16 + u: slot s = 256 u + tid
// holds chunk (s & 7) ^ ((s >> 4) & 7) of row s >> 3; rope_off is that offset
// for u = 0 (u = 1 adds 32 rows). The tile base is uniform, so each copy is
// a scalar base plus one 32-bit lane offset; dst is the LDS byte address of
// the buffer.
// Copies go through a buffer resource (MUBUF load-to-LDS, base = the tile,
// uniform part of the offset in soffset) rather than a global (FLAT-encoded)
// load-to-LDS: the compiler counts the latter as a possible LDS access in
// flight, which turns every wait for a fragment read into a wait for all
// of them.
__device__ __forceinline__ void tile_copy(int i, const char *k, uint32_t dst, int wave,
                                          uint32_t lat_off, uint32_t rope_off) {
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<char *>(k), (short)0, -1, 0x00020000);
  if (i < kTile / 4) {
    const int r = 4 * i + wave;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr)(uintptr_t)(dst + r * kLatChunks * 16),
                                             16, lat_off ^ (16u * (i & 3)), r * kRowBytes, 0, 0);
  } else {
    const int u = i - kTile / 4;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rs, (lds_ptr)(uintptr_t)(dst + (kRopeBase + u * 256 + wave * 64) * 16), 16, rope_off,
        u * 32 * kRowBytes, 0, 0);
  }
}
constexpr int kCopies = kTile / 4 + 2;   // 18 copies per lane per tile

// kLim: the call carries per-row limits on the linked rows (a separate
// instantiation, so that calls without them run no limit code).
template <bool kLim>
__global__ __launch_bounds__(256, 1) void link_mla_kernel(LinkParams p) {
  __shared__ MlaSmem sm;
  __shared__ uint4 sk0[kTileChunks], sk1[kTileChunks];
  const int lane = threadIdx.x & 63;
  const int wave = uni(threadIdx.x >> 6);
  const int n = lane & 31, g = lane >> 5;
  const int rb_s = wave >> 1, kb_s = wave & 1;      // this wave's score tile

  // Blocks are dealt to the XCDs round-robin; give each XCD a contiguous
  // run of row blocks so the row blocks of one request share an L2.
  int b = blockIdx.x;
  if (gridDim.x % p.n_xcd == 0)
    b = (b % p.n_xcd) * (gridDim.x / p.n_xcd) + b / p.n_xcd;
  const int nrb = p.nrb;
  const int grp = b / nrb, rblk = b % nrb;
  const int split = blockIdx.y;
  if (grp >= p.batch) return;
  ReqEntry R;
  {
    const int ri = ((const_ints)p.order)[grp];
    const_reqs rq = (const_reqs)p.reqs + ri;
    R.link0 = rq->link0;
    R.nlinks = rq->nlinks;
    R.q0 = rq->q0;
    R.lq = rq->lq;
    R.ls = rq->ls;
    R.doc_tiles = rq->doc_tiles;
    R.tiles = rq->tiles;
  }
  const int group = p.group;           // query heads (one latent kv head)
  const int nrows = R.lq * group;
  const int row0 = rblk * kRowsMla;
  if (row0 >= nrows) return;
  // the block's key range ends at the last own key its last row sees
  const int vis = visible_tiles(R, min(nrows - 1, row0 + kRowsMla - 1) / group);
  const int t_begin = (int)((int64_t)vis * split / p.num_splits);
  const int t_end = (int)((int64_t)vis * (split + 1) / p.num_splits);

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
  // Limit on the visible linked rows of this lane's score row (dl_s) and its
  // minimum over the wave (wmin_s).
  int dl_s = kNoLimit, wmin_s = kNoLimit;
  if (kLim) {
    if (rvalid[rb_s]) dl_s = p.doc_lim[R.q0 + (row0 + 32 * rb_s + n) / group];
    int w = dl_s;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) w = min(w, __shfl_xor(w, o));
    wmin_s = uni(w);
  }

  const uint32_t lat_off = 16u * (uint32_t)(lane ^ (wave << 2));
  const int tid = threadIdx.x;
  const uint32_t rope_off = (uint32_t)((tid >> 3) * kRowBytes + kLatChunks * 16 +
                                       16 * ((tid & 7) ^ ((tid >> 4) & 7)));

  Cursor cur;
  cur.links = (const_links)p.links + R.link0;
  cur.li = 0;
  cur.k = nullptr;
  cur.len = cur.tile0 = cur.end = 0;
  if (R.nlinks > 0) cursor_load(cur);

  // The first tile is copied up front; every later one during its
  // predecessor's score loop (the last tile re-copies itself into the idle
  // buffer, which keeps the loop free of branches).
  TileRef ref0{}, ref1{};
  if (t_begin < t_end) {
    ref0 = tile_ref(cur, t_begin, R.doc_tiles);
#pragma unroll
    for (int i = 0; i < kCopies; ++i)
      tile_copy(i, ref0.k, lds_addr(sk0), wave, lat_off, rope_off);
  }

  // Q^T operand of the score tile's row block: dims 16 st + 8 g + (0..7).
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
  // Running max (log2 domain) of both row blocks, identical in every wave.
  float m_used[2] = {-INFINITY, -INFINITY};
  float lsum = 0.f;             // partial row sum of the score tile (rb_s, kb_s)
  const float sc = p.scale_log2;
  // Score-operand addresses (16-byte units): lane (n, g) reads key row
  // kr = 32 kb + key_of_m(n), chunk 2 st + g.
  // Latent: kr*64 + ((2 st + g) ^ f(kr)) = kq[st % 8] + 16 (st / 8).
  // Rope:   4096 + kr*8 + ((2 st' + g) ^ f'(kr)) = kp[st'], st' = st - 32.
  // (f and f' do not depend on bit 5 of the row.)
  const int krow = 32 * kb_s + key_of_m(n);
  int kq[8], kp[4];
#pragma unroll
  for (int i = 0; i < 8; ++i) kq[i] = krow * kLatChunks + ((2 * i + g) ^ swz(krow));
#pragma unroll
  for (int i = 0; i < 4; ++i) kp[i] = kRopeBase + krow * kRopeChunks + ((2 * i + g) ^ swr(krow));
  // Transposing-read byte offsets: in read t, lane (q = lane/16, s = lane%16)
  // points at key row 16 ks + 8 (q/2) + 4 t + s/4 and value dims
  // 128 wave + 32 db + 16 (q%2) + 4 (s%4) .. +3; the offset is
  // tr_off[t][db] + 16384 ks (f does not depend on bits 4-5 of the row).
  int tr_off[2][4];
  {
    const int q4 = lane >> 4, s4 = lane & 15;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        const int r = 8 * (q4 >> 1) + 4 * t + (s4 >> 2);
        const int dv = 128 * wave + 32 * db + 16 * (q4 & 1) + 4 * (s4 & 3);
        tr_off[t][db] = (r * kLatChunks + ((dv >> 3) ^ swz(r))) * 16 + ((dv & 7) >> 2) * 8;
      }
  }
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

  // Probabilities of the score tile against max mu, published in LDS;
  // returns their (bf16-rounded) sum over this lane's keys.
  auto publish = [&](const f32x16 &s, float mu) {
    const float neg_m = mu == -INFINITY ? 0.f : -mu;
    float ts = 0.f;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      bf16x8 pf;
#pragma unroll
      for (int x = 0; x < 8; ++x)
        pf[x] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s[8 * h + x], sc, neg_m));
#pragma unroll
      for (int x = 0; x < 8; x += 2) {
        const bf16x2 pp = {pf[x], pf[x + 1]};
        ts = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, ts, false);
      }
      sm.p[rb_s][kb_s][h][lane] = __builtin_bit_cast(uint4, pf);
    }
    return ts;
  };
  // Moves the running max of both row blocks to mnew, rescaling O and lsum.
  auto rescale = [&](const float (&mnew)[2]) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const float alpha =
          mnew[rb] == m_used[rb] ? 1.f : __builtin_amdgcn_exp2f(m_used[rb] - mnew[rb]);
      m_used[rb] = mnew[rb];
      if (rb == rb_s) lsum *= alpha;
      // one accumulator at a time, so that at most 16 of them pass through
      // vector registers at once
#pragma unroll
      for (int db = 0; db < 4; ++db) {
#pragma unroll
        for (int x = 0; x < 16; ++x) o[db][rb][x] *= alpha;
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };

  // One tile: scores, softmax and value product on kt, while the copy of
  // the next tile (global nk -> LDS ndst) is spread over the score loop, one
  // copy every second MFMA, so its issue never stalls the wave for long.
  auto compute = [&](const uint4 *kt, const TileRef &ref, const char *nk, uint4 *ndst) {
    // Opaque copies of the copy addresses: otherwise the compiler hoists all
    // 36 LDS destinations and 18 source addresses out of the tile loop and
    // spills them.
    uint32_t lo = lat_off, ro = rope_off, nd = lds_addr(ndst);
    const char *nkb = nk;
    asm volatile("" : "+v"(lo), "+v"(ro), "+s"(nd), "+s"(nkb));
    // 1. scores
    // The loops are software-pipelined by hand (fragment reads kAhead steps
    // ahead of their MFMA) and sched_barrier keeps that order.
    f32x16 s;
#pragma unroll
    for (int x = 0; x < 16; ++x) s[x] = 0.f;
    bf16x8 kf[kSteps];
    auto kaddr = [&](int st) {
      return st < kLatSteps ? kq[st & 7] + 16 * (st >> 3) : kp[st - kLatSteps];
    };
#pragma unroll
    for (int st = 0; st < kAhead; ++st) kf[st] = as_bf16x8(kt[kaddr(st)]);
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
      if (st + kAhead < kSteps) kf[st + kAhead] = as_bf16x8(kt[kaddr(st + kAhead)]);
      if ((st & 1) == 0) tile_copy(st >> 1, nkb, nd, wave, lo, ro);
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[st], qf[st], s, 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    // s[x]: key 32 kb_s + (x>>3)*16 + g*8 + (x&7) of row 32 rb_s + n
    if (ref.own || ref.nvalid < kTile || (kLim && ref.tok + kTile > wmin_s)) {
      const int kl = (ref.own ? min(lim[rb_s] - ref.j0, ref.nvalid - 1)
                      : kLim  ? min(dl_s - ref.tok, ref.nvalid) - 1
                              : ref.nvalid - 1) -
                     32 * kb_s - g * 8;
#pragma unroll
      for (int x = 0; x < 16; ++x)
        if ((x >> 3) * 16 + (x & 7) > kl) s[x] = -INFINITY;
    }
    // 2. probabilities against the running max as it stands. A lane whose
    // partial sum stays <= 2^64 has every probability <= 2^64; the
    // tile's own max is only computed when some lane of the workgroup fails
    // that test (or has no running max yet).
    const float mu = rb_s ? m_used[1] : m_used[0];
    const float lsum0 = lsum;
    const float ts = publish(s, mu);
    lsum += ts;
    const bool jump = !(ts <= kJumpSum) || (mu == -INFINITY && ts > 0.f);
    const bool wjump = __any(jump);
    if (lane == 0) ((int *)&sm.jump)[wave] = wjump;
    lds_barrier();
    // 3. O^T += V^T P^T for this wave's 128 value dims
    // Fragment f = 4 ks + db: two transposing reads (key rows 16 ks ..,
    // value block db), issued kVLead fragments ahead of its two MFMAs; the
    // probability operands of step ks are read with fragment 4 ks.
    const char *kbytes = (const char *)kt;
    bf16x8 vf[16], pb[4][2];
    auto read_frag = [&](int f) {
      const int ks = f >> 2, db = f & 3;
      if (db == 0) {
        pb[ks][0] = as_bf16x8(sm.p[0][ks >> 1][ks & 1][lane]);
        pb[ks][1] = as_bf16x8(sm.p[1][ks >> 1][ks & 1][lane]);
      }
      i16x4 part[2];
#pragma unroll
      for (int t = 0; t < 2; ++t)
        part[t] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_i16x4 *)(kbytes + tr_off[t][db] + ks * 16384));
      vf[f] = __builtin_bit_cast(
          bf16x8, (uint4){(uint32_t)(uint16_t)part[0][0] | ((uint32_t)(uint16_t)part[0][1] << 16),
                          (uint32_t)(uint16_t)part[0][2] | ((uint32_t)(uint16_t)part[0][3] << 16),
                          (uint32_t)(uint16_t)part[1][0] | ((uint32_t)(uint16_t)part[1][1] << 16),
                          (uint32_t)(uint16_t)part[1][2] | ((uint32_t)(uint16_t)part[1][3] << 16)});
    };
    const int4 jf = sm.jump;
    if (jf.x | jf.y | jf.z | jf.w) {
      // redo the tile against the new running max (uniform over the workgroup)
      float tmax = -INFINITY;
#pragma unroll
      for (int x = 0; x < 16; x += 2) tmax = fmaxf(fmaxf(tmax, s[x]), s[x + 1]);
      tmax = half_swap_max(tmax) * sc;
      if (g == 0) sm.xm[wave][n] = tmax;
      lds_barrier();
      float mnew[2];
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
        mnew[rb] = fmaxf(m_used[rb], fmaxf(sm.xm[2 * rb][n], sm.xm[2 * rb + 1][n]));
      lsum = lsum0;
      rescale(mnew);
      lsum += publish(s, rb_s ? m_used[1] : m_used[0]);
      lds_barrier();
    }
#pragma unroll
    for (int f = 0; f < kVLead; ++f) read_frag(f);
#pragma unroll
    for (int f = 0; f < 16; ++f) {
      if (f + kVLead < 16) read_frag(f + kVLead);
      const int ks = f >> 2, db = f & 3;
      o[db][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[f], pb[ks][0], o[db][0], 0, 0, 0);
      o[db][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[f], pb[ks][1], o[db][1], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  // Two tiles per trip, one per buffer, with no branch in between (any
  // branch there makes the compiler copy all accumulators out of the
  // accumulation registers on every trip): an odd tile count ends with an
  // empty tile, whose keys are all masked.
  for (int t = t_begin; t < t_end; t += 2) {
    ref1 = t + 1 < t_end ? tile_ref(cur, t + 1, R.doc_tiles) : TileRef{ref0.k, 0, 0, 0};
    compute(sk0, ref0, ref1.k, sk1);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    ref0 = t + 2 < t_end ? tile_ref(cur, t + 2, R.doc_tiles) : ref1;
    compute(sk1, ref1, ref0.k, sk0);
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
  if (p.doc_lim)
    hipLaunchKernelGGL(link_mla_kernel<true>, grid, dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL(link_mla_kernel<false>, grid, dim3(256), 0, st, p);
  return hipGetLastError();
}

}  // namespace pic
