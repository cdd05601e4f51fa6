/*
 * pic.h -- link-stage attention over position-independent chunk caches, on
 * one AMD Instinct MI355X (gfx950).
 *
 * The method (Comb, "You Need an Encoder for Native Position-Independent
 * Caching"): each static context chunk is compiled once into key/value
 * caches computed from position zero (Sec. 1, Fig. 1; Sec. 4.2 stores the
 * cross-attention K and V). A request is a question plus zero or more
 * contexts in any order (Sec. 3). In the link stage the request's chunk
 * caches are looked up by id (Sec. 3, step 1), concatenated in request order
 * along the document axis (Sec. 4.2), and the request's dynamic tokens
 * attend over them -- without a mask (cross-attention, Sec. 4.2 Eq. 7-8) --
 * and over their own KV under a causal mask (Sec. 4.1 Eq. 2-3), all under
 * one softmax here. The PIC allocator owns a pool of GPU memory reserved
 * when the system starts (Sec. 5.3).
 *
 * Math computed for request r, query row i (0 <= i < L_q), query head h:
 *   keys  = [ K_{c_1} ; ... ; K_{c_n} ; K_own[0 .. i + L_s - L_q] ]
 *   s_j   = softmax_scale * <q[i,h], keys_j[h / (H_q/H_kv)]>
 *   out[i,h] = sum_j softmax(s)_j * values_j[h / (H_q/H_kv)]
 *   lse[i,h] = log(sum_j exp(s_j))   (natural log; -inf and out = 0 if no key)
 * The query rows are the last L_q of the L_s own tokens (bottom-right causal
 * alignment): new tokens are appended to the query sequence (Sec. 4).
 * MLA (absorbed latent form, Sec. 5.1 DeepSeek-V2-Lite backbone): one KV
 * "head" whose rows are [latent | rope] (d_k wide); the value of a row is its
 * first d_v entries, and the output is the latent (d_v wide) per head.
 *
 * Conventions for every call:
 *   - Status codes are negative on error. All validation happens on the host
 *     before any device work: an error launches nothing and writes nothing.
 *     pic_last_error() gives a thread-local message about the last error.
 *   - Device pointers are HIP device allocations on the current device;
 *     "host" arrays are ordinary host memory, read before the call returns.
 *   - `stream` is a hipStream_t (NULL = the null stream). All device work is
 *     enqueued on it; calls return before it runs.
 *   - Tensors are dense, row-major, with no padding, in the store's dtype
 *     (fp32, or bf16 as raw 16-bit patterns) unless stated; lse is fp32.
 *   - One host thread uses a store at a time. Outputs of calls that are in
 *     flight on different streams must not alias.
 *   - Each pic_link_attn / pic_link_decode call gets a device workspace of
 *     its own (the request's own KV laid out for the kernels, and partial
 *     results of split key ranges): a store keeps eight, handed out in turn,
 *     and one is reused only once the call that last used it has completed,
 *     so calls may be in flight on different streams at once; a ninth call
 *     waits on the host for the oldest of the eight. Runs of one link plan
 *     share the plan's workspace instead (see pic_link_plan_run).
 */
#ifndef PIC_H
#define PIC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PIC_OK = 0,
  PIC_ERR_INVALID = -1,      /* bad argument, shape or layout */
  PIC_ERR_NOT_FOUND = -2,    /* a linked chunk id is not in the store */
  PIC_ERR_EXISTS = -3,       /* put of an id already stored (chunks are immutable) */
  PIC_ERR_OOM = -4,          /* the store's pool has no room */
  PIC_ERR_HIP = -5,          /* a HIP runtime call failed */
  PIC_ERR_UNSUPPORTED = -6   /* valid request this build has no kernel for */
} pic_status;

enum { PIC_F32 = 0, PIC_BF16 = 1 };     /* pic_store_desc.dtype */
enum { PIC_GQA = 0, PIC_MLA = 1 };      /* pic_store_desc.kind  */

/* Shape of a store's chunk caches. d_k and d_v must be multiples of 8.
 * GQA: n_kv_heads >= 1, separate K [.., d_k] and V [.., d_v] per head.
 * MLA: n_kv_heads == 1, d_v <= d_k, the value is the first d_v of each key row.
 * n_layers: cross-attention layers per chunk, 0 or 1 for one. Comb
 *   interleaves L_cross cross-attention layers with the decoder (Sec. 4.2
 *   and 4.3, Fig. 3: 8 among 32 decoder layers; Eq. 12), and each reads its
 *   own K and V of every document; a chunk's caches of all layers are put
 *   together and each link call names its layer.
 * capacity_tokens: pool size in tokens per layer, in pages of 64 tokens.
 * Each chunk occupies its length rounded up to whole pages in every layer,
 * in one run of consecutive pages when a free run is long enough, else in
 * several (removal leaves holes; no copy ever moves a chunk). */
typedef struct pic_store_desc {
  int32_t kind;
  int32_t dtype;
  int32_t n_kv_heads;
  int32_t d_k;
  int32_t d_v;
  int32_t n_layers;          /* 0..256; 0 and 1 both mean one layer */
  int64_t capacity_tokens;
} pic_store_desc;

typedef struct pic_store pic_store;

/* Creates a chunk store on the current HIP device and reserves its pool
 * (the PIC allocator's reservation, Sec. 5.3): capacity_tokens per layer.
 * *out receives the handle.
 * Errors: INVALID (desc), UNSUPPORTED (shape), HIP (allocation failed). */
pic_status pic_store_create(const pic_store_desc *desc, pic_store **out);

/* Waits for the device, then frees the store and everything it owns.
 * NULL is accepted and ignored. Errors: INVALID while link plans of the
 * store are alive (destroy them first). */
pic_status pic_store_destroy(pic_store *store);

/* Compile-stage entry (Sec. 3 steps 3-4): copies one chunk's caches into the
 * pool and records chunk_id -> slot in the store's hash table.
 *   k: device, [n_layers][n_tokens][n_kv_heads][d_k] (token-major per layer)
 *   v: device, [n_layers][n_tokens][n_kv_heads][d_v] for GQA; NULL for MLA
 * The copy (into the store's internal layout) is ordered on `stream`; the
 * caller may reuse k and v once the stream has passed it.
 * Errors: INVALID, EXISTS (id present), OOM (pool full), HIP. */
pic_status pic_store_put(pic_store *store, uint64_t chunk_id, int64_t n_tokens, const void *k,
                         const void *v, void *stream);

/* Removes a chunk from the store and frees its pages (the paper's allocator
 * hands out free memory, Sec. 5.3, and says nothing of eviction; removal is
 * the caller's policy). The pages are reused only after the work enqueued on
 * `stream` up to this call has completed: pass the stream of the link calls
 * that may still read the chunk. A removed id may be put again.
 * Errors: INVALID (NULL store, or a live link plan links the chunk),
 * NOT_FOUND, HIP. */
pic_status pic_store_remove(pic_store *store, uint64_t chunk_id, void *stream);

/* A chunk that differs from a stored one in a few rows, for the link stage
 * of post-training PIC, which recomputes selected tokens of each document
 * and attends over the cached KV with those rows replaced (Sec. 2: EPIC
 * recomputes the first tokens of every chunk, CacheBlend the tokens whose
 * cached KV deviates most; Sec. 6.1 runs CacheBlend at 20%).
 * pic_store_derive: new_id becomes a chunk with base_id's length and
 *   content. The 64-token pages that hold `rows` (host int32 [n_rows],
 *   strictly increasing, each below the base's length) are private copies
 *   made on `stream`; every other page is shared with the base (no copy).
 *   The base may be removed first: shared pages live while a chunk holds
 *   them (a run of pages allocated together is freed once no chunk holds
 *   any of its pages). Errors: INVALID, NOT_FOUND (base), EXISTS (new_id),
 *   OOM, HIP.
 * pic_store_write_rows: writes token-major K / V rows of one layer into a
 *   derived chunk: k device [n_rows][n_kv_heads][d_k], v device
 *   [n_rows][n_kv_heads][d_v] (GQA) or NULL (MLA); rows as above, each on a
 *   page the chunk holds alone (a page named at pic_store_derive and not
 *   shared since by a later derive). Ordered on `stream`; k and v are read
 *   before the stream passes the call. Link calls already enqueued on
 *   another stream may see either content.
 *   Errors: INVALID (not a derived chunk, a row on a shared page, bad
 *   arguments), NOT_FOUND, HIP. */
pic_status pic_store_derive(pic_store *store, uint64_t new_id, uint64_t base_id, int32_t n_rows,
                            const int32_t *rows, void *stream);
pic_status pic_store_write_rows(pic_store *store, uint64_t chunk_id, int32_t layer,
                                int32_t n_rows, const int32_t *rows, const void *k,
                                const void *v, void *stream);

/* Handing a store to another process on the same GPU, in place: the PIC
 * manager of the paper sends the handles of the PICaches it collected to the
 * inference engine over the GPU's inter-process memory API, so tensors pass
 * between processes without copies (Sec. 5.3, System Details).
 * pic_store_export: waits for the device (every put and copy enqueued so far
 *   has landed), then writes a self-contained description of the store --
 *   its shape, an inter-process handle of its pool and its chunk index as it
 *   stands -- into buf (host, buf_bytes). *bytes_out receives the size
 *   needed; buf = NULL only asks for it. Chunks put or removed later are not
 *   in the description: the exporting process keeps the store and the
 *   exported chunks alive (no pic_store_remove, no pic_store_destroy) while
 *   importers use them. Errors: INVALID (NULL store or bytes_out, buffer too
 *   small, an imported store), UNSUPPORTED (pool of 2 GiB or more: the
 *   pool's n_layers * capacity_tokens * H_kv * (d_k + d_v) * esize must stay
 *   below 2^31 bytes), HIP.
 * pic_store_import: in another process on the same GPU (with that device
 *   current), maps the exported pool and rebuilds the chunk index. The result
 *   is a read-only store: link calls, link plans, pic_store_lookup,
 *   pic_store_usage and pic_debug_gather work as on the original;
 *   pic_store_put, pic_store_remove, pic_store_derive and
 *   pic_store_write_rows return INVALID. pic_store_destroy unmaps the pool
 *   (the exporter still owns it). Mapping a pool in the process that
 *   exported it is not supported. Errors: INVALID (not a description made by
 *   pic_store_export, or a corrupt one), HIP (the mapping failed), OOM. */
pic_status pic_store_export(pic_store *store, void *buf, size_t buf_bytes, size_t *bytes_out);
pic_status pic_store_import(const void *buf, size_t buf_bytes, pic_store **out);

/* Hash-table lookup (Sec. 3 step 1): *n_tokens_out = the chunk's length.
 * Errors: INVALID, NOT_FOUND. */
pic_status pic_store_lookup(const pic_store *store, uint64_t chunk_id, int64_t *n_tokens_out);

/* Pool usage in tokens of allocated 64-token pages (pages of removed chunks
 * count until their readers have finished; pages shared by derived chunks
 * count once), the capacity, and the number of stored chunks (derived ones
 * included). Any output pointer may be NULL. */
pic_status pic_store_usage(const pic_store *store, int64_t *used_tokens,
                           int64_t *capacity_tokens, int64_t *n_chunks);

/* A batch of requests (Sec. 3: a question plus zero or more contexts).
 * All arrays are host memory with batch+1 non-decreasing entries from 0.
 *   chunk_offsets/chunk_ids: the links of request r, in request order, are
 *     chunk_ids[chunk_offsets[r] .. chunk_offsets[r+1]-1]; an id may repeat.
 *   q_offsets: the query tokens of request r are rows q_offsets[r].. of q.
 *   self_offsets: own-KV tokens of request r (L_s >= L_q), or NULL for
 *     cross-attention only (no own KV, every row sees only the documents).
 *   chunk_starts: NULL (every link reads its whole chunk), or per link (same
 *     indexing as chunk_ids) the first token of the chunk the link reads: a
 *     multiple of 64 below the chunk's length. Lets a request splice chunk
 *     caches, e.g. the link of post-training PIC that recomputes the first
 *     tokens of every document (Sec. 1 and 2.2; Sec. 6.1 runs EPIC with 64
 *     per document): link [the recomputed tokens, put as a chunk of their
 *     own ; the cached chunk from token 64] for every document.
 *   q_doc_limits: NULL (every query token sees all of its request's linked
 *     rows), or per query token t (indexing as q) the number of leading
 *     linked rows it sees, 0 .. the request's linked rows. Recomputed
 *     tokens attend as in a prefill of the concatenated prompt (Sec. 2,
 *     post-training PIC): a token at position P of the linked rows passes
 *     P + 1 (and the call passes self_offsets = NULL). The own KV, if any,
 *     is not affected. */
typedef struct pic_link_req {
  int32_t batch;
  int32_t layer;             /* the store layer whose chunk caches are read (0 for one layer) */
  const int32_t *chunk_offsets;
  const uint64_t *chunk_ids;
  const int32_t *q_offsets;
  const int32_t *self_offsets;
  const int32_t *chunk_starts;
  const int32_t *q_doc_limits;
} pic_link_req;

/* Link-stage attention for prefill-shaped requests (Sec. 4.1-4.2).
 *   q      device [Tq][n_q_heads][d_k], Tq = q_offsets[batch]
 *   k_self device [Ts][n_kv_heads][d_k], Ts = self_offsets[batch] (NULL if none)
 *   v_self device [Ts][n_kv_heads][d_v] (GQA), NULL for MLA
 *   out    device [Tq][n_q_heads][d_v], store dtype
 *   lse    device [Tq][n_q_heads] fp32 natural-log log-sum-exp, or NULL
 * n_q_heads must be a multiple of n_kv_heads. softmax_scale (positive,
 * finite) multiplies the dot products (Eq. 2 and 7 use 1/sqrt(d)). The chunk table of the call is
 * copied to the device on `stream`; all host arrays are consumed on return.
 * When the batch has too few query rows to fill the GPU (short questions
 * over long documents), the library splits each request's keys and merges
 * the partial softmax states exactly, as pic_link_decode does; the result
 * is the same up to floating-point rounding order.
 * Errors: INVALID, NOT_FOUND, UNSUPPORTED, HIP. */
pic_status pic_link_attn(pic_store *store, const pic_link_req *req, int32_t n_q_heads,
                         const void *q, const void *k_self, const void *v_self,
                         float softmax_scale, void *out, float *lse, void *stream);

/* Link-stage attention for decode-shaped requests (few query tokens each):
 * the same function as pic_link_attn (a generated token is treated like a
 * query token, Sec. 4), computed by splitting each request's keys into
 * num_splits ranges whose partial softmax states are merged exactly
 * (log-sum-exp). num_splits = 0 lets the library choose; otherwise 1..256.
 * Each request may have at most 16 query tokens.
 * Errors: as pic_link_attn. */
pic_status pic_link_decode(pic_store *store, const pic_link_req *req, int32_t n_q_heads,
                           const void *q, const void *k_self, const void *v_self,
                           float softmax_scale, int32_t num_splits, void *out, float *lse,
                           void *stream);

/* pic_link_decode for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc. Same arguments, kernels, split choice and result as
 * pic_link_decode, but the call's tables, own-KV layout and split partials
 * live in the library's static device scratch, a file-scope array of
 * 64 MiB that each GPU the library runs on holds until the process ends;
 * the call allocates nothing (no hipMalloc, hipFree, pinned staging or
 * event). The host tables are copied with hipMemcpyAsync from pageable
 * memory, which the runtime completes before returning (the host therefore
 * waits for the stream's earlier work). Small calls (at most 32 links and 8
 * requests, no per-query limits, a shape without a matrix-core kernel) run
 * the kernels pic_link_decode runs for them, which take the tables as a
 * kernel argument and read the own KV in place: they use the scratch for
 * split partials only and copy nothing. Every kernel writes what it later
 * reads, so nothing in the scratch has to start at zero.
 * All calls on one GPU share its scratch: calls must not overlap on a GPU
 * (enqueue them on one stream, or order them); calls that overlap race.
 * Errors: as pic_link_decode, and INVALID when the call needs more than the
 * 64 MiB (about 256 B of tables per link and request, plus
 * ceil(L_s / 64) * 64 own tokens * H_kv * (d_k + d_v) * esize per request,
 * plus Tq * H_q * splits * (d_v + 2) * 4 B when the keys are split); such a
 * call launches nothing. */
pic_status pic_link_decode_noalloc(pic_store *store, const pic_link_req *req, int32_t n_q_heads,
                                   const void *q, const void *k_self, const void *v_self,
                                   float softmax_scale, int32_t num_splits, void *out, float *lse,
                                   void *stream);

/* A request batch resolved once for repeated calls. Comb runs the same
 * links in each of its cross-attention layers and again at every decode
 * step (generated tokens attend to the same documents, Sec. 4 and Eq. 12);
 * a plan looks the chunk ids up, chooses kernel and splits, and puts the
 * link tables of every layer and the call's workspace on the device once,
 * so that a run enqueues kernels only: no host-side lookup, no copy, no
 * allocation.
 * pic_link_plan_create: req as for pic_link_attn (req->layer must be 0);
 *   mode PIC_PREFILL (num_splits must be 0) computes as pic_link_attn,
 *   PIC_DECODE as pic_link_decode with the given num_splits (0 = auto),
 *   with the same kernels and split choice, so a run returns the bits the
 *   direct call returns (small calls, at most 32 links and 8 requests on
 *   the generic kernel, pass the tables as a kernel argument from the
 *   plan's host copy of each layer's table, as the direct calls do).
 *   Blocking: copies the tables to the device before returning. The plan
 *   keeps no pointer into req; the store must outlive it
 *   (pic_store_destroy refuses while plans are alive).
 * pic_link_plan_run: one call of the planned batch on cross-attention layer
 *   `layer`, with tensors as for pic_link_attn (sizes from the plan's
 *   offsets). Runs of one plan share its workspace: enqueue them on one
 *   stream, or order them.
 * pic_link_plan_destroy: waits for the device and frees the plan; NULL is
 *   ignored.
 * Errors: INVALID, NOT_FOUND, UNSUPPORTED, OOM, HIP. */
enum { PIC_PREFILL = 0, PIC_DECODE = 1 };   /* pic_link_plan_create mode */
typedef struct pic_link_plan pic_link_plan;
pic_status pic_link_plan_create(pic_store *store, const pic_link_req *req, int32_t n_q_heads,
                                int32_t mode, int32_t num_splits, pic_link_plan **out);
pic_status pic_link_plan_run(pic_link_plan *plan, int32_t layer, const void *q,
                             const void *k_self, const void *v_self, float softmax_scale,
                             void *out, float *lse, void *stream);
pic_status pic_link_plan_destroy(pic_link_plan *plan);

/* Test hook: materialises the concatenation (Sec. 4.2) of the listed chunks
 * of one layer, in the given order, reading the pool through the same
 * address resolution the attention kernels use. k_out: device token-major
 * [sum len][H_kv][d_k]; v_out: device [sum len][H_kv][d_v] (GQA) or NULL
 * (MLA). Bit-exact copies.
 * Errors: INVALID, NOT_FOUND, HIP. */
pic_status pic_debug_gather(pic_store *store, const uint64_t *ids, int32_t n, int32_t layer,
                            void *k_out, void *v_out, void *stream);

/* Test hook, host only (no device work, no store): the request order the
 * planner gives a bf16 d=128 prefill call, whose row blocks (256 rows of
 * one request and kv head) are dispatched in that order, each on the first
 * free CU of its XCD. Request r has q_len[r] query tokens, self_len[r] own
 * tokens (causal, Sec. 4.1) and doc_tiles[r] 64-key tiles of linked
 * documents (Sec. 4.2); the GQA group is n_q_heads / n_kv_heads; cus and
 * xcds describe the device (workgroup ids go round-robin to the XCDs).
 * order_out: host [batch], the request at each position: heaviest first
 * (tiles x query tokens), improved by pairwise swaps when the row blocks
 * of an XCD take several rounds of its CUs. finish_out: host [2] or NULL,
 * the simulated finish time in tiles of the busiest XCD (a workgroup takes
 * its visible tiles plus 1.5) for heaviest first and for the returned
 * order; both 0 when no search runs.
 * Errors: INVALID (NULL arrays, negative lengths, n_q_heads not a multiple
 * of n_kv_heads, cus not a multiple of xcds). */
pic_status pic_debug_request_order(const int32_t *q_len, const int32_t *self_len,
                                   const int32_t *doc_tiles, int32_t batch, int32_t n_q_heads,
                                   int32_t n_kv_heads, int32_t cus, int32_t xcds,
                                   int32_t *order_out, double *finish_out);

/* Dense per-head projections around absorbed MLA link attention, for the
 * DeepSeek-V2-Lite backbone (Sec. 5.1): per head h its latent rows c (512)
 * give non-absorbed keys [W_UK[h] c | k_rope] and values W_UV[h] c, with
 * W_UK[h] and W_UV[h] 128 x 512. Absorbing W_UK into the query turns the
 * attention into the latent form pic_link_attn computes on an MLA store
 * (d_k 576, d_v 512); W_UV then maps its latent output to the 128 value dims.
 * bf16 in and out (round to nearest even), fp32 accumulation.
 * pic_mla_absorb_q: q_out[t,h,0:512] = W_UK[h]^T q[t,h,0:128] and
 *   q_out[t,h,512:576] = q[t,h,128:192] (the rope part, copied).
 *   q device [n_tokens][n_heads][192] (q_nope 128 | q_rope 64)
 *   w_uk_t device [n_heads][512][128]: W_UK[h] transposed (row j holds the
 *     128 weights of latent dim j)
 *   q_out device [n_tokens][n_heads][576]
 * pic_mla_up_v: out[t,h,0:128] = W_UV[h] o_lat[t,h,0:512].
 *   o_lat device [n_tokens][n_heads][512] (pic_link_attn's output)
 *   w_uv device [n_heads][128][512]
 *   out device [n_tokens][n_heads][128]
 * All pointers 16-byte aligned; n_heads 1..1024; n_tokens 0 does nothing.
 * Errors: INVALID, HIP. */
pic_status pic_mla_absorb_q(int32_t n_tokens, int32_t n_heads, const void *q, const void *w_uk_t,
                            void *q_out, void *stream);
pic_status pic_mla_up_v(int32_t n_tokens, int32_t n_heads, const void *o_lat, const void *w_uv,
                        void *out, void *stream);

/* Kernel timing for measurement. pic_prof_begin() clears and enables
 * recording of HIP events around every launch of the main attention kernel;
 * pic_prof_begin_sampled(every) around one launch in `every` (1..1000000;
 * the event pair adds a few microseconds between kernels, so sampling keeps
 * the timed steps close to an uninstrumented run); pic_prof_end() waits for
 * them, disables recording and returns the summed kernel time in
 * milliseconds, the number of timed launches and the kernel's name
 * (name_buf may be NULL). Errors: INVALID (every out of range), HIP. */
pic_status pic_prof_begin(void);
pic_status pic_prof_begin_sampled(int32_t every);
pic_status pic_prof_end(double *kernel_ms, int64_t *launches, char *name_buf, int32_t name_len);

/* Achievable peaks of this GPU, a second roofline denominator next to the
 * spec peaks (measurement helpers, not part of the method; blocking, they
 * synchronise `stream`, allocate and free a 512 KB scratch buffer).
 * pic_peak_mfma_bf16: bf16 dense matrix-core rate in TFLOP/s of `iters`
 *   rounds of four independent 32x32x16 MFMAs per wave, two waves per SIMD
 *   on every CU (iters 1..2^22; ~4096 gives a ~10 ms run).
 * pic_peak_hbm_read: HBM read rate in GB/s of one streaming pass over buf
 *   (device memory, 16-byte aligned, bytes a positive multiple of 16; use a
 *   buffer far larger than the last-level cache).
 * pic_peak_hbm_write: the same for one streaming pass of stores over buf
 *   (overwrites it). One dispatch of either moves exactly `bytes`, which
 *   also calibrates the HBM traffic counters of a profiler.
 * Errors: INVALID, HIP. */
pic_status pic_peak_mfma_bf16(int32_t iters, double *tflops, void *stream);
pic_status pic_peak_hbm_read(const void *buf, int64_t bytes, double *gbs, void *stream);
pic_status pic_peak_hbm_write(void *buf, int64_t bytes, double *gbs, void *stream);

const char *pic_status_str(pic_status status);
const char *pic_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* PIC_H */
