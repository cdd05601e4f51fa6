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

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }

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
  constexpr int kOutRow = 136;                          // bf16 per padded row
  constexpr int kRedRow = 132;
  __shared__ __attribute__((aligned(16))) float red[kSplitK ? 4 * 32 * kRedRow : 4 * 32 * kOutRow / 2];
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
  bf16x8 w[4][8];
  {
    const uint16_t *wh = p.w + (int64_t)h * N * K + (int64_t)(n0 + (lane & 31)) * K + k0 + g * 8;
#pragma unroll
    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
      for (int s = 0; s < 8; ++s) w[nt][s] = as_bf16x8(*(const uint4 *)(wh + nt * 32 * K + s * 16));
  }

  const int n_blocks = (p.n_tokens + 31) / 32;
  // No load or store depends on a branch: rows past the last token (and
  // blocks past the last block) read the last token's row instead. A token's
  // output column depends on its own activation row only, so those columns
  // reproduce the last token's outputs bit for bit, and storing them to the
  // last token's row rewrites it with the same bytes.
  const int last = p.n_tokens - 1;
  // activation fragments of a block: b[s] = A[t][k0 + s*16 + g*8 .. +8]
  auto load_a = [&](int tb, uint4 (&b)[8]) {
    const int t = min(tb * 32 + (lane & 31), last);
    const uint16_t *arow = ah + (int64_t)t * p.a_tok + k0 + g * 8;
#pragma unroll
    for (int s = 0; s < 8; ++s) b[s] = *(const uint4 *)(arow + s * 16);
  };
  // rope piece of a block: 32 tokens x 128 bytes, one 16-byte piece per thread
  auto load_rope = [&](int tb, uint4 &r) {
    if (kRope) {
      const int tt = min(tb * 32 + (int)(threadIdx.x >> 3), last);
      r = *(const uint4 *)(ah + (int64_t)tt * p.a_tok + 128 + (threadIdx.x & 7) * 8);
    }
  };
  // Block tb from b / rope; once its products are issued, b / rope are
  // refilled with block tb_next.
  auto process = [&](int tb, uint4 (&b)[8], uint4 &rope, int tb_next) {
    if (kRope) {
      const int tt = min(tb * 32 + (int)(threadIdx.x >> 3), last);
      *(uint4 *)(ch + (int64_t)tt * p.c_tok + 512 + (threadIdx.x & 7) * 8) = rope;
    }
    f32x16 acc[4];
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
    load_a(tb_next, b);
    load_rope(tb_next, rope);

    // C^T tile: lane holds token t and n = nt*32 + jj*8 + g*4 + (0..3).
    // Stores: 16 bytes per lane.
    if (kSplitK) {
      // partial tiles to LDS as [wave][token][n]; then every thread adds the
      // four partials of 8 consecutive n of one token (2 pieces per thread,
      // consecutive lanes on consecutive tokens)
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
        const int piece = threadIdx.x + 256 * j, tok = piece & 31, nb = (piece >> 5) * 8;
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
        *(uint4 *)(ch + (int64_t)min(tb * 32 + tok, last) * p.c_tok + nb) =
            __builtin_bit_cast(uint4, v8);
      }
      __syncthreads();      // before the next block overwrites the partials
    } else {
      // this wave's tile to LDS as bf16 [token][n], then row pieces out
      uint16_t *mine = (uint16_t *)red + wave * 32 * kOutRow;
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
        *(uint4 *)(ch + (int64_t)min(tb * 32 + tok, last) * p.c_tok + n0 + nb) = v;
      }
      __builtin_amdgcn_wave_barrier();      // reads done before the next block's writes
    }
  };
  // Two blocks in flight: the fragments of blocks tb and tb + parts sit in
  // b0 / b1 (two fixed register sets, so that no copy waits on a load).
  uint4 b0[8], b1[8];
  uint4 r0 = make_uint4(0, 0, 0, 0), r1 = make_uint4(0, 0, 0, 0);
  load_a(part, b0);
  load_rope(part, r0);
  load_a(part + parts, b1);
  load_rope(part + parts, r1);
  const int n_mine = (n_blocks - part + parts - 1) / parts;   // blocks of this workgroup
  int i = 0;
  for (; i + 1 < n_mine; i += 2) {
    const int tb = part + i * parts;
    process(tb, b0, r0, tb + 2 * parts);
    process(tb + parts, b1, r1, tb + 3 * parts);
  }
  if (i < n_mine) process(part + i * parts, b0, r0, n_blocks);
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
