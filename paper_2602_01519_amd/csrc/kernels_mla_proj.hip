// Dense per-head projections around absorbed MLA link attention (the
// DeepSeek-V2-Lite backbone of Sec. 5.1, whose non-absorbed keys and values
// are k_nope = W_UK c and v = W_UV c of the latent row c):
//   absorb: q_out[t,h, 0:512]   = W_UK[h]^T q[t,h, 0:128]   (the query side of
//           q_nope . (W_UK c) = (W_UK^T q_nope) . c); q_out[t,h, 512:576] =
//           q[t,h, 128:192] (the rope part passes through)
//   up:     out[t,h, 0:128]     = W_UV[h] o[t,h, 0:512]     (sum_j p_j W_UV c_j
//           = W_UV sum_j p_j c_j)
// Both are C^T[n][t] = sum_k W[n][k] A[t][k] per head, with the weight stored
// [N][K] (K contiguous) and the activation rows strided by tokens, computed
// on v_mfma_f32_32x32x16_bf16 with fp32 accumulation and bf16 outputs
// (round to nearest even). Each of a workgroup's four waves holds a 128 (n)
// x 128 (k) slice of the head's weights in registers, read once, and the
// workgroup then walks its share of the 32-token blocks: with N = 512 the
// waves split n (one 128-wide range each, K = 128 in full), with K = 512
// they split k and add their partial tiles through LDS. Per block a wave
// loads its eight 16-byte activation fragments per lane and issues 32 MFMAs.
// These projections move more bytes than they compute (about 100 FLOP/B),
// so HBM bounds them; reading the weights from L2 for every block instead
// made them 2-3x slower.
#include "pic_internal.hpp"

#include <algorithm>

namespace pic {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }

typedef __attribute__((address_space(3))) void *lds_ptr;

// Load-to-LDS copy: 16 bytes per lane from base + voff (bytes) to LDS at
// dst + 16 * lane, through a buffer resource of `records` bytes (a lane past
// them reads zeros and touches no memory). The compiler tracks such copies
// per LDS array, so a read of one array does not wait for copies into
// another.
// base, records and dst must be uniform across the wave.
__device__ __forceinline__ void lds_copy16(const void *base, uint32_t records, uint32_t voff,
                                           void *dst) {
  // (the resource is scalar: make the uniformity explicit, or the compiler
  // loops over the distinct values it cannot rule out)
  const uint64_t b = (uint64_t)base;
  const uint64_t ub = (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)b) |
                      ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(b >> 32)) << 32);
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      (void *)ub, (short)0, __builtin_amdgcn_readfirstlane((int)records), 0x00020000);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr)dst, 16, voff, 0, 0, 0);
}

// Stores 16 bytes at base + off bytes with the sc1 (system coherence)
// cache policy; base must be uniform across the wave and off < 2^31. These
// kernels write more than they read (the absorption's 38 MB of outputs at
// 2048 tokens x 16 heads are more than the L2s hold): with the default
// policy the lines stayed dirty in L2 and their write-back at the end of
// the kernel held the next launch back; with sc1 they leave as the kernel
// runs (back to back, absorption 12.4 -> 10.1 us; the up-projection gained
// only once its stores wrote whole 256-byte rows, 11.0 -> 10.2 us).
__device__ __forceinline__ void store16_sc1(void *base, uint32_t off, uint4 v) {
  const uint64_t b = (uint64_t)base;
  const uint64_t ub = (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)b) |
                      ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(b >> 32)) << 32);
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc((void *)ub, (short)0, 0x7fffffff, 0x00020000);
  const u32x4 d = {v.x, v.y, v.z, v.w};
  __builtin_amdgcn_raw_buffer_store_b128(d, rs, (int)off, 0, 16 /* sc1 */);
}

// Workgroup barrier without the memory fence of __syncthreads (whose release
// half would wait for every copy and store in flight): this wave's LDS
// accesses are done, and the empty asm statements keep the compiler from
// moving memory accesses across it.
__device__ __forceinline__ void block_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

struct ProjArgs {
  const uint16_t *a;      // activation, row (t, h) at a + t * a_tok + h * a_head
  const uint16_t *w;      // weights [H][N][K]
  uint16_t *c;            // output, row (t, h) at c + t * c_tok + h * c_head
  int64_t a_tok, a_head, c_tok, c_head;
  int32_t n_tokens, n_heads;
  int32_t parts;          // workgroups per head
  int32_t n_xcd;          // XCDs of the device
};

// kRope: also copy a[.., 128:192] to c[.., 512:576] (the absorb projection).
// Workgroup (head h, part j) of `parts` per head walks token blocks j,
// j + parts, ... Consecutive workgroup ids go round-robin to the XCDs;
// when the head count allows, all parts of a head go to one XCD, so that
// its weights are fetched into one L2 only.
template <int K, int N, bool kRope>
__global__ __launch_bounds__(256, 1) void proj_kernel(ProjArgs p) {
  static_assert((K == 128 && N == 512) || (K == 512 && N == 128), "one 128 x 128 slice per wave");
  constexpr bool kSplitK = K > 128;
  // K = 512: the four waves' partial tiles, [wave][token][n] fp32 with rows
  // padded to 132 floats.
  // K = 128: each wave's bf16 output tile, [token][n] with rows padded to
  // 272 bytes, so that the stores go out as whole 256-byte row pieces.
  // K = 128 also keeps a ring of kRing token blocks in LDS (see below).
  constexpr int kOutRow = 136;                          // bf16 per padded row
  constexpr int kRedRow = 132;
  constexpr int kRing = 5;
  constexpr int kSlotBytes = 32 * 256 + 32 * 128;       // q[., 0:128] then q[., 128:192]
  constexpr int kAreaBytes = kSplitK ? 4 * 32 * kRedRow * 4 : 4 * 32 * kOutRow * 2;
  __shared__ __attribute__((aligned(16))) uint4 smem[kAreaBytes / 16];
  // the ring: one array per slot (see lds_copy16)
  constexpr int kSlotVec = kSplitK ? 1 : kSlotBytes / 16;
  __shared__ uint4 ring0[kSlotVec], ring1[kSlotVec], ring2[kSlotVec], ring3[kSlotVec],
      ring4[kSlotVec];
  static_assert(kRing == 5, "one array per slot");
  auto ring_slot = [&](int q) -> unsigned char * {
    return (unsigned char *)(q == 0 ? ring0 : q == 1 ? ring1 : q == 2 ? ring2 : q == 3 ? ring3 : ring4);
  };
  float *red = (float *)smem;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int parts = p.parts;
  int h, part;
  if (p.n_heads % p.n_xcd == 0) {
    const int xcd = blockIdx.x % p.n_xcd, j = blockIdx.x / p.n_xcd;
    h = xcd + p.n_xcd * (j / parts);
    part = j % parts;
  } else {
    h = blockIdx.x / parts;
    part = blockIdx.x % parts;
  }
  const int g = lane >> 5;
  const int n0 = kSplitK ? 0 : wave * 128;       // this wave's n range
  const int k0 = kSplitK ? wave * 128 : 0;       // this wave's k range
  const uint16_t *ah = p.a + (int64_t)h * p.a_head;
  uint16_t *ch = p.c + (int64_t)h * p.c_head;

  // weight fragments: w[nt][s] = W[n0 + nt*32 + (lane&31)][k0 + s*16 + g*8 .. +8]
  // In that layout one load instruction touches 32 rows (32 bytes of each),
  // which the L1 serves a line at a time. The slice is therefore read in
  // whole 128-byte lines instead (instruction i of row group nt: rows
  // nt*32 + 4i + lane/16, 16 bytes each of the 256-byte k range) and
  // rearranged through a wave-private LDS area, rows padded to 272 bytes so
  // that neither side conflicts on the banks. The area is the one the
  // per-block outputs use later.
  const int n_blocks = (p.n_tokens + 31) / 32;
  // No load or store depends on a branch: rows past the last token (and
  // blocks past the last block) read the last token's row instead. A token's
  // output column depends on its own activation row only, so those columns
  // reproduce the last token's outputs bit for bit, and storing them to the
  // last token's row rewrites it with the same bytes.
  const int last = p.n_tokens - 1;
  const int n_mine = (n_blocks - part + parts - 1) / parts;   // blocks of this workgroup

  constexpr int kRow = 136;                              // bf16 per padded LDS row
  static_assert(kAreaBytes >= 4 * 32 * kRow * 2, "transpose area");
  u32x4 raw[4][8];
  {
    const uint16_t *wh = p.w + (int64_t)h * N * K + (int64_t)(n0 + (lane >> 4)) * K + k0 +
                         (lane & 15) * 8;
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int i = 0; i < 8; ++i) raw[nt][i] = *(const u32x4 *)(wh + (nt * 32 + 4 * i) * K);
  }

  // K = 128: the activation blocks stream through a ring of kRing LDS slots
  // by load-to-LDS copies, kRing - 1 blocks ahead, shared by the four waves
  // (which all need the same 32 x 128 slice). A slot holds the block's
  // q[., 0:128] rows (256 bytes, the 16-byte chunk c of row r at position
  // c ^ (r & 15), so that the fragment reads below hit 16 distinct bank
  // groups) and its q[., 128:192] rope rows. Each wave copies its quarter
  // of a block with three 1 KB copies (whole 128-byte lines), so its vector
  // memory operations per block are fixed: 3 copies, then 1 + 8 stores.
  // The wait for block i's copies therefore counts the operations issued
  // after them: 3 (kRing - 2) + 9 min(i, kRing - 1). A refill past the last
  // block is still issued, with an empty buffer range (no memory touched),
  // to keep that count.
  auto issue_block = [&](int tb, unsigned char *dst) {
    const bool real = tb < n_blocks;
    const int row0 = min(tb, n_blocks - 1) * 32;
    const uint16_t *base = ah + (int64_t)row0 * p.a_tok;
    const uint32_t tok_bytes = (uint32_t)p.a_tok * 2;
    const uint32_t records = real ? 0xFFFFFFFFu : 0u;
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      const int j = 2 * wave + jj, r = 4 * j + (lane >> 4);
      const int c = (lane & 15) ^ (r & 15);
      lds_copy16(base, records, (uint32_t)(min(row0 + r, last) - row0) * tok_bytes + c * 16,
                 dst + j * 1024);
    }
    const int r = 8 * wave + (lane >> 3);
    lds_copy16(base, records,
               (uint32_t)(min(row0 + r, last) - row0) * tok_bytes + 256 + (lane & 7) * 16,
               dst + 8192 + wave * 1024);
  };
  if constexpr (!kSplitK) {
    asm volatile("" ::: "memory");
#pragma unroll
    for (int q = 0; q < kRing - 1; ++q) issue_block(part + q * parts, ring_slot(q));
    asm volatile("" ::: "memory");
  }
  // K = 512: the first two blocks' activation fragments (b[s] = A[t][k0 +
  // s*16 + g*8 .. +8]) are loaded beside the weights, not after them
  auto load_a = [&](int tb, uint4 (&b)[8]) {
    const int t = min(tb * 32 + (lane & 31), last);
    const uint16_t *arow = ah + (int64_t)t * p.a_tok + k0 + g * 8;
#pragma unroll
    for (int s = 0; s < 8; ++s) b[s] = *(const uint4 *)(arow + s * 16);
  };
  uint4 b0[8], b1[8];
  if constexpr (kSplitK) {
    load_a(part, b0);
    load_a(part + parts, b1);
  }

  // weight fragments: w[nt][s] = W[n0 + nt*32 + (lane&31)][k0 + s*16 + g*8 .. +8]
  // In that layout one load instruction touches 32 rows (32 bytes of each),
  // which the L1 serves a line at a time. The slice is therefore read in
  // whole 128-byte lines instead (instruction i of row group nt: rows
  // nt*32 + 4i + lane/16, 16 bytes each of the 256-byte k range, in raw) and
  // rearranged through a wave-private LDS area, rows padded to 272 bytes so
  // that neither side conflicts on the banks. The area is the one the
  // per-block outputs use later.
  bf16x8 w[4][8];
  {
    uint16_t *tw = (uint16_t *)red + wave * 32 * kRow;
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {
#pragma unroll
      for (int i = 0; i < 8; ++i)
        *(u32x4 *)(tw + (4 * i + (lane >> 4)) * kRow + (lane & 15) * 8) = raw[nt][i];
      // (a wave's LDS accesses complete in order: the reads see the writes,
      // and the next group's writes follow these reads)
#pragma unroll
      for (int st = 0; st < 8; ++st)
        w[nt][st] = as_bf16x8(*(const uint4 *)(tw + (lane & 31) * kRow + st * 16 + g * 8));
    }
  }
  // K = 512: the partial tiles of block 0 overlap other waves' areas
  if (kSplitK) __syncthreads();

  // The products of one block: C^T tile, lane holds token t and
  // n = nt*32 + jj*8 + g*4 + (0..3).
  auto products = [&](const uint4 (&b)[8], f32x16 (&acc)[4]) {
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int x = 0; x < 16; ++x) acc[nt][x] = 0.f;
#pragma unroll
    for (int s = 0; s < 8; ++s)
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
        acc[nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(w[nt][s], as_bf16x8(b[s]), acc[nt], 0,
                                                          0, 0);
  };

  if constexpr (!kSplitK) {
    // this wave's tile to LDS as bf16 [token][n], then out as row pieces
    // (16 bytes per lane, 256 bytes per row)
    uint16_t *mine = (uint16_t *)red + wave * 32 * kOutRow;
    auto step = [&](int i, const unsigned char *slot, unsigned char *refill) {
      const int tb = part + i * parts;
      switch (min(i, kRing - 1)) {       // block i's copies (this wave's) have landed
        case 0: asm volatile("s_waitcnt vmcnt(9)" ::: "memory"); break;
        case 1: asm volatile("s_waitcnt vmcnt(18)" ::: "memory"); break;
        case 2: asm volatile("s_waitcnt vmcnt(27)" ::: "memory"); break;
        case 3: asm volatile("s_waitcnt vmcnt(36)" ::: "memory"); break;
        default: asm volatile("s_waitcnt vmcnt(45)" ::: "memory"); break;
      }
      block_barrier();                   // every wave's copies landed; block i-1's slot is free
      issue_block(tb + (kRing - 1) * parts, refill);
      asm volatile("" ::: "memory");
      uint4 b[8];
      {
        const int t = lane & 31;
#pragma unroll
        for (int s = 0; s < 8; ++s)
          b[s] = *(const uint4 *)(slot + (t * 16 + ((2 * s + g) ^ (t & 15))) * 16);
      }
      // the block's output rows start at cb (offsets within a block stay far
      // below 2^31 bytes)
      uint16_t *cb = ch + (int64_t)min(tb * 32, last) * p.c_tok;
      const int brow0 = min(tb * 32, last);
      {
        const uint4 rope = *(const uint4 *)(slot + 8192 + threadIdx.x * 16);
        const int tt = min(tb * 32 + (int)(threadIdx.x >> 3), last);
        store16_sc1(cb, (uint32_t)(((int64_t)(tt - brow0) * p.c_tok + 512 + (threadIdx.x & 7) * 8) * 2),
                    rope);
      }
      f32x16 acc[4];
      products(b, acc);
#pragma unroll
      for (int nt = 0; nt < 4; ++nt)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          __bf16 v4[4];
#pragma unroll
          for (int x = 0; x < 4; ++x) v4[x] = (__bf16)acc[nt][jj * 4 + x];
          *(uint2 *)(mine + (lane & 31) * kOutRow + nt * 32 + jj * 8 + g * 4) =
              __builtin_bit_cast(uint2, v4);
        }
      // (a wave's LDS accesses complete in order: the reads see the writes)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int piece = lane + 64 * j, tok = piece >> 4, nb = (piece & 15) * 8;
        const uint4 v = *(const uint4 *)(mine + tok * kOutRow + nb);
        store16_sc1(cb, (uint32_t)(((int64_t)(min(tb * 32 + tok, last) - brow0) * p.c_tok + n0 + nb) * 2),
                    v);
      }
      __builtin_amdgcn_wave_barrier();   // reads done before the next block's writes
    };
    // unrolled by the ring size, so that every slot is a fixed array
    for (int i0 = 0; i0 < n_mine; i0 += kRing) {
      step(i0, ring_slot(0), ring_slot(4));
      if (i0 + 1 >= n_mine) break;
      step(i0 + 1, ring_slot(1), ring_slot(0));
      if (i0 + 2 >= n_mine) break;
      step(i0 + 2, ring_slot(2), ring_slot(1));
      if (i0 + 3 >= n_mine) break;
      step(i0 + 3, ring_slot(3), ring_slot(2));
      if (i0 + 4 >= n_mine) break;
      step(i0 + 4, ring_slot(4), ring_slot(3));
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // no copy outlives the workgroup
    return;
  }

  // K = 512: activation fragments in registers, two blocks in flight: the
  // fragments of blocks tb and tb + parts sit in b0 / b1 (two fixed register
  // sets, so that no copy waits on a load; the first two were issued beside
  // the weight loads); a set is refilled with the block after next once its
  // block's products are issued.
  auto process = [&](int tb, uint4 (&b)[8], int tb_next) {
    f32x16 acc[4];
    products(b, acc);
    load_a(tb_next, b);
    // partial tiles to LDS as [wave][token][n]; then every thread adds the
    // four partials of 8 consecutive n of one token (2 pieces per thread,
    // 16 consecutive lanes on one token's 256-byte output row, so each
    // store instruction writes whole rows)
    float *mine = red + wave * 32 * kRedRow;
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        *(float4 *)(mine + (lane & 31) * kRedRow + nt * 32 + jj * 8 + g * 4) =
            make_float4(acc[nt][jj * 4], acc[nt][jj * 4 + 1], acc[nt][jj * 4 + 2],
                        acc[nt][jj * 4 + 3]);
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int piece = threadIdx.x + 256 * j, tok = piece >> 4, nb = (piece & 15) * 8;
      float sum[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 a = *(const float4 *)(red + (q * 32 + tok) * kRedRow + nb);
        const float4 b = *(const float4 *)(red + (q * 32 + tok) * kRedRow + nb + 4);
        sum[0] += a.x, sum[1] += a.y, sum[2] += a.z, sum[3] += a.w;
        sum[4] += b.x, sum[5] += b.y, sum[6] += b.z, sum[7] += b.w;
      }
      __bf16 v8[8];
#pragma unroll
      for (int x = 0; x < 8; ++x) v8[x] = (__bf16)sum[x];
      const int brow0 = min(tb * 32, last);
      store16_sc1(ch + (int64_t)brow0 * p.c_tok,
                  (uint32_t)(((int64_t)(min(tb * 32 + tok, last) - brow0) * p.c_tok + nb) * 2),
                  __builtin_bit_cast(uint4, v8));
    }
    __syncthreads();      // before the next block overwrites the partials
  };
  int i = 0;
  for (; i + 1 < n_mine; i += 2) {
    const int tb = part + i * parts;
    process(tb, b0, tb + 2 * parts);
    process(tb + parts, b1, tb + 3 * parts);
  }
  if (i < n_mine) process(part + i * parts, b0, n_blocks);
}

// Workgroups per head: about one per CU over all heads, never more than
// the head's token blocks.
int proj_parts(int32_t n_tokens, int32_t n_heads, int32_t cus) {
  const int blocks = (n_tokens + 31) / 32;
  return std::max(1, std::min(blocks, (cus + n_heads - 1) / n_heads));
}

}  // namespace

hipError_t launch_mla_absorb_q(const void *q, const void *w_uk_t, void *q_out, int32_t n_tokens,
                               int32_t n_heads, const DevShape &ds, hipStream_t st) {
  ProjArgs p{(const uint16_t *)q, (const uint16_t *)w_uk_t, (uint16_t *)q_out,
             (int64_t)n_heads * 192, 192, (int64_t)n_heads * 576, 576, n_tokens, n_heads,
             proj_parts(n_tokens, n_heads, ds.cus), ds.xcds};
  hipLaunchKernelGGL((proj_kernel<128, 512, true>), dim3(p.parts * n_heads), dim3(256), 0, st, p);
  return hipGetLastError();
}

hipError_t launch_mla_up_v(const void *o_lat, const void *w_uv, void *out, int32_t n_tokens,
                           int32_t n_heads, const DevShape &ds, hipStream_t st) {
  ProjArgs p{(const uint16_t *)o_lat, (const uint16_t *)w_uv, (uint16_t *)out,
             (int64_t)n_heads * 512, 512, (int64_t)n_heads * 128, 128, n_tokens, n_heads,
             proj_parts(n_tokens, n_heads, ds.cus), ds.xcds};
  hipLaunchKernelGGL((proj_kernel<512, 128, false>), dim3(p.parts * n_heads), dim3(256), 0, st, p);
  return hipGetLastError();
}

}  // namespace pic
