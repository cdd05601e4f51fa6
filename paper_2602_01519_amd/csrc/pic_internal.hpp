// Internal declarations shared by the host planner and the HIP kernels.
// Not part of the C ABI (include/pic.h is).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace pic {

// Keys per attention tile. Every chunk slot in the pool is padded to a
// multiple of it (zero rows), so a tile never straddles two chunks and the
// pool's rows stay 16-byte aligned.
constexpr int kTile = 64;

// Layout of one chunk slot with padded length lp (elements of the store's
// dtype):
//   GQA  K block  [n_kv_heads][lp][d_k]    (head-major, token rows)
//        V block  [n_kv_heads][lp / 32][d_v][32]
//                                          (transposed in panels of 32 tokens:
//                                          value dim = row of a panel, its 32
//                                          tokens contiguous)
//   MLA  K block  [lp][d_k]                (value = first d_v of each row)
// The transposed V lets a matrix-core operand read 8 consecutive keys of one
// value column with a single 16-byte load; the panels keep the rows of a
// 32-key tile together, so a 32-key tile reads whole 128-byte lines (two
// bf16 rows, or one fp32 row) and a 64-key tile is one contiguous block. A
// request's own KV is laid out the same way (in the call's workspace) before
// the attention kernel runs, so every key tile of a request -- document or
// own -- is read alike.
constexpr int kPanel = 32;

// Element offset of value dim e of token t (relative to the slot's first
// token) of head h in a V block with padded length lp.
__host__ __device__ __forceinline__ int64_t vt_offset(int64_t h, int64_t e, int64_t t, int64_t lp,
                                                     int64_t d_v) {
  return h * d_v * lp + (t / kPanel) * (d_v * kPanel) + e * kPanel + (t % kPanel);
}

// A per-row limit on the visible linked rows that no request reaches.
constexpr int kNoLimit = 1 << 30;

struct LinkEntry {        // one link of one request, in link order
  const void *k;          // K block of the slot
  const void *v;          // GQA: V block; MLA: same as k
  int32_t len;            // tokens; the link spans ceil(len / kTile) tiles
  int32_t lp;             // row stride of its K / V^T blocks in tokens (multiple of kTile)
  int32_t tile0;          // index of the link's first tile within the request
  int32_t tok0;           // index of the link's first token within the request
};

struct ReqEntry {
  int32_t link0, nlinks;  // links[link0 .. link0+nlinks); the own KV, if any, is the last
  int32_t q0, lq;         // query rows q0 .. q0+lq of q / out
  int32_t s0, ls;         // own rows s0 .. s0+ls of k_self / v_self (ls = 0: none)
  int32_t doc_tiles;      // tiles over the linked documents (own tiles follow)
  int32_t tiles;          // doc_tiles + ceil(ls / kTile)
};

// Tiles of a request that hold a key visible to query token q_last or any
// earlier one: every document tile, then the own tiles up to the one holding
// own key q_last + ls - lq (the causal limit, bottom-right aligned).
__host__ __device__ __forceinline__ int visible_tiles(const ReqEntry &r, int q_last) {
  const int own_last = q_last + r.ls - r.lq;
  return own_last >= 0 ? (r.doc_tiles + own_last / kTile + 1 < r.tiles
                              ? r.doc_tiles + own_last / kTile + 1
                              : r.tiles)
                       : r.doc_tiles;
}

struct LinkParams {
  const LinkEntry *links;
  const ReqEntry *reqs;
  const int32_t *order;   // requests, heaviest first
  const void *q;
  const void *k_self;
  const void *v_self;
  void *out;
  float *lse;
  float *part_o;          // split partials: [split][Tq*H_q][d_v] unnormalised
  float *part_m;          // [split][Tq*H_q] running max (log2 domain)
  float *part_l;          // [split][Tq*H_q] running sum
  const int32_t *doc_lim; // per query token: linked rows it sees (NULL: all of them)
  int32_t batch;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t group;          // n_q_heads / n_kv_heads
  int32_t d_k;
  int32_t d_v;
  int32_t total_q;        // Tq
  int32_t num_splits;     // 1: write out/lse directly; >1: write partials
  int32_t nrb;            // row blocks per (request, kv head)
  int32_t max_rows;       // most rows of one (request, kv head)
  int32_t n_groups;       // batch * n_kv_heads, padded as the kernel requires
  int32_t n_xcd;          // accelerator dies (XCDs) of the device, each with its own L2
  float scale_log2;       // softmax_scale * log2(e)
};

// Shape of the current device: compute units and XCDs. Workgroups with
// consecutive ids are dispatched round-robin to the XCDs, so a kernel that
// wants some of them to share an L2 maps ids with the XCD count.
struct DevShape {
  int32_t cus;
  int32_t xcds;
};
DevShape device_shape();

// Launchers (each returns the launch status).
hipError_t launch_put_rows(const void *src, void *dst, int64_t n_tokens, int32_t lp,
                           int32_t heads, int32_t width, int32_t esz, hipStream_t st);
hipError_t launch_put_transposed(const void *src, void *dst, int64_t n_tokens, int32_t lp,
                                 int32_t heads, int32_t width, int32_t esz, hipStream_t st);
hipError_t launch_gather(const LinkEntry *links, int32_t n_links, int64_t total_tokens,
                         int32_t heads, int32_t d_k, int32_t d_v, int32_t mla, int32_t esz,
                         void *k_out, void *v_out, hipStream_t st);

// Destination of one row written into a chunk slot: its K row of head 0
// (head h at + h * lp * d_k elements) and its V^T entry of head 0, dim 0
// (head h, dim e at + h * d_v * lp + e * kPanel; unused for MLA).
struct RowDst {
  void *k;
  void *v;
  int64_t lp;
};
// Scatters token-major rows src_k [n][heads][d_k] (and src_v [n][heads][d_v]
// unless mla) to the slot rows dst[0 .. n).
hipError_t launch_write_rows(const RowDst *dst, int32_t n, const void *src_k, const void *src_v,
                             int32_t heads, int32_t d_k, int32_t d_v, int32_t mla, int32_t esz,
                             hipStream_t st);

// Copies bytes (a multiple of 16) from a host-mapped buffer to the device.
hipError_t launch_table_copy(const void *src, void *dst, int64_t bytes, hipStream_t st);

// The dense MLA projections around the latent link (see pic.h).
hipError_t launch_mla_absorb_q(const void *q, const void *w_uk_t, void *q_out, int32_t n_tokens,
                               int32_t n_heads, const DevShape &ds, hipStream_t st);
hipError_t launch_mla_up_v(const void *o_lat, const void *w_uv, void *out, int32_t n_tokens,
                           int32_t n_heads, const DevShape &ds, hipStream_t st);
// The call's prologue: lays out the own KV of every request (token-major
// k_self / v_self) like a chunk slot at its own link (the request's last
// link), zero-padded to lp, in `work` (when max_own_lp > 0) and copies copy_bytes of tables from
// copy_src to copy_dst (when copy_bytes > 0). The layout takes each
// request's own rows and slot from `own` (host, batch entries, batch <=
// kOwnArgs: passed as kernel arguments, so it does not wait for a read of
// the tables over PCIe from the staging buffer), or, when own is NULL,
// from the tables at links / reqs.
struct OwnArg {
  int32_t s0, ls;     // own rows s0 .. s0+ls of k_self / v_self
  int64_t off;        // slot offset in the workspace (K block, then V^T block)
};
constexpr int kOwnArgs = 128;
hipError_t launch_prologue(const LinkParams &p, const LinkEntry *links, const ReqEntry *reqs,
                           int32_t mla, int32_t esz, int32_t max_own_lp, const OwnArg *own,
                           const void *work, const void *copy_src, void *copy_dst,
                           int64_t copy_bytes, hipStream_t st);

// Generic vector-ALU link attention: any d_k <= 576, d_v <= 512, fp32 or bf16.
hipError_t launch_link_valu(const LinkParams &p, int dtype, int mla, hipStream_t st,
                            const char **name);
int valu_rows_per_block();

// bf16 GQA link attention on MFMA, d_k = d_v = 128 (prefill-shaped).
hipError_t launch_link_mfma_d128(const LinkParams &p, hipStream_t st, const char **name);
int mfma_d128_rows_per_block();
int mfma_d128_blocks_per_cu();   // resident workgroups per CU (2 waves per SIMD)

// bf16 GQA decode-shaped link attention, d_k = d_v = 128, at most
// decode_d128_max_rows() rows per (request, kv head); one wave per split.
hipError_t launch_link_decode_d128(const LinkParams &p, hipStream_t st, const char **name);
int decode_d128_max_rows();

// bf16 MLA (absorbed) link attention: one 576-wide latent kv head, values
// are the first 512 entries of each latent row.
hipError_t launch_link_mla(const LinkParams &p, hipStream_t st, const char **name);
int mla_rows_per_block();

// Achievable-peak microbenchmarks (out: peak_out_floats() floats of scratch).
int64_t peak_out_floats();
double peak_mfma_flops(int32_t iters);
hipError_t launch_peak_mfma(float *out, int32_t iters, hipStream_t st);
hipError_t launch_peak_read(const void *src, int64_t bytes, float *out, hipStream_t st);
hipError_t launch_peak_write(void *dst, int64_t bytes, hipStream_t st);

// The library's static device scratch (a file-scope array, no allocation):
// its size, and its address on the current device (resolved once per
// device). Used by the entry points that must not allocate.
constexpr size_t kStaticScratchBytes = size_t(64) << 20;
constexpr int kMaxDevices = 64;
hipError_t static_scratch(void **out);

// Log-sum-exp merge of split partials into out / lse.
hipError_t launch_combine(const LinkParams &p, int dtype, hipStream_t st);

// Tables of a small generic-kernel call, passed by value as a kernel
// argument: the call then needs neither the table copy nor the own-KV
// layout of the prologue (see link_small_kernel).
constexpr int kSmallLinks = 32, kSmallReqs = 8;
struct SmallTabs {
  LinkEntry links[kSmallLinks];
  ReqEntry reqs[kSmallReqs];
  int32_t order[kSmallReqs];
};
hipError_t launch_link_small(const LinkParams &p, const SmallTabs &t, int dtype, int mla,
                             hipStream_t st, const char **name);

// Tables of a lean small call (link_lean_kernel): requests in dispatch
// order, and for every tile of every request the link that holds it
// (relative to the request's first link), so a workgroup finds its tiles
// with one table read instead of a walk over the links.
constexpr int kLeanTiles = 256;
struct LeanTabs {
  LinkEntry links[kSmallLinks];
  ReqEntry reqs[kSmallReqs];          // reqs[i]: the i-th request in dispatch order
  int32_t tile_base[kSmallReqs];      // first tile_link entry of reqs[i]
  uint8_t tile_link[kLeanTiles];
};
// GQA shapes the lean kernel is built for: d_k = d_v = d in {32, 64, 128}
// for fp32, {32, 64} for bf16, and a power-of-two query group.
bool lean_supported(int dtype, int d_k, int d_v, int group);
hipError_t launch_link_lean(const LinkParams &p, const LeanTabs &t, int dtype, hipStream_t st,
                            const char **name);

}  // namespace pic
