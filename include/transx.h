/*
 * transx.h -- C ABI of the TransX amortized serving path on MI355X (gfx950).
 *
 * TransX (arXiv 2607.28940) encodes each user's behavior stream once with a
 * causal Transformer encoder, caches the keys/values that every decoder layer's
 * cross-attention needs, extends that cache incrementally as new behavior
 * events arrive, and at serving time lets the serving-event tokens and the
 * candidate tokens of a request cross-attend to it (Sec. 4.1-4.3, App. B, App. D).
 * This library implements that path with hand-written HIP kernels:
 *
 *   kv_cache_build    encode behavior sequences, fill the paged per-request cache
 *   kv_cache_append   encode only newly appended events against the cached prefix
 *   score_candidates  decoder over serving + candidate tokens, linear head
 *   score_events      the same per serving event of a user, each against its
 *                     own prefix of the cache (seq-to-seq training forward)
 *   score_candidates_static
 *                     score_candidates without a workspace argument and
 *                     without allocating, for callers that cannot allocate
 *
 * Conventions
 *   - All tensors the caller hands over are device pointers unless marked
 *     "host". Row-major, tokens packed request after request; host int64 offset
 *     arrays of length n_req+1 index the packed rows (offsets[0] >= 0,
 *     non-decreasing).
 *   - Element type of tokens, weights and cache is the model's dtype (TX_BF16:
 *     bfloat16 storage, fp32 accumulation, softmax and LayerNorm; TX_F32: fp32
 *     throughout). Scores are always fp32.
 *   - The library never allocates device memory: the caller provides the
 *     repacked-weight buffer, the page pool and a workspace for each call.
 *     (The one exception is the fixed array that score_candidates_static uses
 *     in place of a workspace, part of the library's code object.) Host-side
 *     bookkeeping (page tables, free list, pinned staging for small uploads)
 *     is owned by the library.
 *   - Calls are asynchronous on the given stream. Build, append and score of the
 *     same request must be ordered on one stream by the caller. A handle must
 *     not be used from two host threads at once.
 *   - Every argument check runs on the host before any launch: a call that
 *     returns TX_E_INVALID, TX_E_NOMEM, TX_E_NOCACHE or TX_E_UNSUPPORTED has
 *     changed nothing. When a HIP call fails inside kv_cache_build or
 *     kv_cache_append (TX_E_HIP), the call's requests are left without a cache
 *     (length -1) and keep their pages until tx_kv_cache_release returns them
 *     to the free list (work already enqueued on the stream may still write
 *     to them); the other requests are untouched. tx_last_error() describes
 *     the last error of the calling thread.
 */
#ifndef TRANSX_H
#define TRANSX_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TX_OK = 0,
  TX_E_INVALID = -1,     /* bad argument: offsets, ids, sizes, alignment, mismatched model */
  TX_E_NOMEM = -2,       /* page pool or workspace too small */
  TX_E_NOCACHE = -3,     /* request has no cache (cold start: App. D, the caller falls back) */
  TX_E_HIP = -4,         /* a HIP runtime call or launch failed */
  TX_E_UNSUPPORTED = -5  /* configuration outside what the kernels implement */
} tx_status;

typedef enum { TX_F32 = 0, TX_BF16 = 1 } tx_dtype;

/* Model shape (Sec. 4.1; encoder relative-position bias from the App. D
 * remark on incremental encoding). d_model = n_heads * d_head. */
typedef struct {
  int32_t d_model;
  int32_t n_heads;
  int32_t d_ffn;
  int32_t n_enc_layers;
  int32_t n_dec_layers;
  int32_t rel_pos_buckets; /* R: logit bias beta_h[min(i - j, R - 1)]; 0 = none */
  float ln_eps;
  int32_t dtype;           /* tx_dtype */
  /* Local-global sparse cross-attention (Sec. 4.1.2, Eq. sparse-cross-attn;
   * the experiments use L_local = 10 with an attention-pooled global token,
   * Sec. 5 setup). l_local = 0: every decoder query attends to every cached
   * token. 1 <= l_local <= 64: only to the request's last l_local cached
   * tokens, plus, when global_pool = 1, one global anchor token: the
   * attention pooling g = sum_j a_j h_j of the encoded rows with
   * a = softmax_j(h_j . w_pool / sqrt(d_model)), projected by each decoder
   * layer's cross-attention K/V weights. global_pool requires l_local > 0. */
  int32_t l_local;
  int32_t global_pool;
  /* Decoder head (Sec. 4.1.3, Eq. action-decoding). 0: one logit per
   * candidate, s = z . w_s + b_s (the two-action case). k = 2..16: the
   * query-key softmax over k learned action embeddings, p = softmax(z W_dec +
   * b_dec), W_dec [d_model][k] (column a = action a's embedding), where z is
   * the candidate's decoder output row. */
  int32_t n_actions;
} tx_config;

typedef struct tx_model tx_model;
typedef struct tx_kv_cache tx_kv_cache;

/* Message for the last non-OK status returned on this thread. */
const char* tx_last_error(void);

/* ------------------------------------------------------------------ model */

/* Number of parameter tensors in canonical order:
 *   per encoder layer (17): Wq bq Wk bk Wv bv Wo bo ln1_g ln1_b W1 b1 W2 b2 ln2_g ln2_b rel[H][R]
 *   per decoder layer (26): self Wq bq Wk bk Wv bv Wo bo ln1_g ln1_b,
 *                           cross Wq bq Wk bk Wv bv Wo bo ln2_g ln2_b,
 *                           FFN W1 b1 W2 b2 ln3_g ln3_b
 *   head (2): w_s[d] b_s[1], or with n_actions = k: W_dec[d][k] b_dec[k]
 *   global-token pooling (1, only when global_pool): w_pool[d]
 * Matrices are [d_in][d_out] row-major (a layer computes y = x W + b). */
int32_t tx_num_weights(const tx_config* cfg);

/* Bytes of the device buffer that receives the repacked (transposed, fused,
 * biases widened to fp32) weights. */
size_t tx_model_repack_bytes(const tx_config* cfg);

/* Validate cfg and lay the repacked parameters out in dev_repack (256-byte
 * aligned, at least tx_model_repack_bytes). Host only: nothing is launched and
 * dev_repack is not touched until tx_model_set_weights. model_id stamps every
 * cache made from this model (versioned cache entries, App. D).
 * Errors: TX_E_INVALID, TX_E_UNSUPPORTED (d_head not 32, 64 or 128),
 * TX_E_NOMEM (repack_bytes too small). */
int tx_model_create(const tx_config* cfg, void* dev_repack, size_t repack_bytes, uint64_t model_id,
                    tx_model** out);

/* Repack the parameters (device pointers, canonical order, model dtype) into
 * the model's buffer on `stream`: matrices transposed to [d_out][d_in], the
 * self-attention Q/K/V fused, the cross-attention K/V of all decoder layers
 * fused, biases and LayerNorm parameters widened to fp32. The source tensors
 * may be freed once the stream has passed this call. Must precede any build,
 * append or score. Errors: TX_E_INVALID (count, null or misaligned pointer),
 * TX_E_HIP. */
int tx_model_set_weights(tx_model* model, const void* const* dev_weights, int32_t n_weights, hipStream_t stream);

void tx_model_destroy(tx_model* model);

/* -------------------------------------------------------------- KV cache */

/* Tokens per cache page (fixed). */
#define TX_PAGE_TOKENS 64

/* Bytes of one page: for each encoder layer then each decoder layer, K as
 * [H][64][d_head] and V transposed as [H][d_head][64], each V^T row holding
 * the page's tokens in 16-token groups ordered 0-3, 8-11, 4-7, 12-15 (the k
 * order of the attention MFMAs; tx_kv_cache_export returns plain order). */
size_t tx_kv_page_bytes(const tx_config* cfg);

/* Bytes of the device pool for n_pages pages plus the device page table of
 * max_requests requests of up to max_tokens tokens each; with global_pool
 * also, per request, the pooling state (fp32 max, sum and weighted row sum)
 * and the global token's cross-attention K/V of every decoder layer. */
size_t tx_kv_pool_bytes(const tx_config* cfg, int64_t n_pages, int32_t max_requests, int64_t max_tokens);

/* Create a cache over a caller-owned device pool (256-byte aligned): the
 * per-user store of encoded behavior K/V that amortized serving reads
 * (Sec. 4.3; App. D, cache management, warm start: the caller builds entries
 * ahead of serving). Request ids are 0 .. max_requests-1. Also reserves the pinned host staging that
 * score_candidates_static uploads its metadata through (4 x 512 KiB; without a
 * usable device the cache is still created and that call later reports
 * TX_E_NOMEM). Errors: TX_E_INVALID, TX_E_NOMEM (pool too small). */
int tx_kv_cache_create(const tx_model* model, void* dev_pool, size_t pool_bytes, int64_t n_pages,
                       int32_t max_requests, int64_t max_tokens, tx_kv_cache** out);
/* Release the cache's host bookkeeping (the caller frees the device pool
 * afterwards, once the stream's work on it has completed). */
void tx_kv_cache_destroy(tx_kv_cache* cache);

/* Evict requests (their pages return to the free list): the eviction step of
 * the cache lifecycle (App. D, cache management: entries carry a time-to-live
 * and are evicted by recency of access; the policy stays with the caller,
 * this call frees the pages). Releasing a request without a cache is not an
 * error. Errors: TX_E_INVALID (id out of range). */
int tx_kv_cache_release(tx_kv_cache* cache, int32_t n_req, const int32_t* req_ids /* host */);

/* Cached length of a request (the encoded prefix that kv_cache_append
 * extends, App. D nearline updates); -1 if it has no cache (cold start). */
int tx_kv_cache_length(const tx_kv_cache* cache, int32_t req_id, int64_t* len_out /* host */);

/* Pages on the free list: the headroom the caller's eviction policy (App. D
 * cache lifecycle) works against. */
int64_t tx_kv_cache_free_pages(const tx_kv_cache* cache);

/* Model id the cache was created for (App. D, cache management, versioning
 * and consistency: entries are tied to the model identifier, so a caller that
 * upgrades the model creates a new cache instead of reusing stale entries). */
uint64_t tx_kv_cache_model_id(const tx_kv_cache* cache);

/* Copy one cached tensor of a request into a dense device buffer out
 * [len][d_model] (model dtype), head h in columns h*d_head .. h*d_head+d_head-1.
 * part: 0 encoder K, 1 encoder V (layer < n_enc), 2 cross-attention K,
 * 3 cross-attention V (layer < n_dec); with global_pool, 4 and 5 are the
 * global token's cross-attention K and V of decoder layer `layer` (one row).
 * For inspection and tests. */
int tx_kv_cache_export(const tx_kv_cache* cache, int32_t req_id, int32_t part, int32_t layer, void* out,
                       hipStream_t stream);

/* ------------------------------------------------------------ workspace */

enum { TX_OP_BUILD = 0, TX_OP_APPEND = 1, TX_OP_SCORE = 2 };

/* Workspace bytes for one call that processes all n_req requests in a single
 * pass. BUILD: offs_a = behavior offsets. APPEND: offs_a = event offsets.
 * SCORE: offs_a = serving offsets, offs_b = candidate offsets. A smaller
 * workspace (at least tx_workspace_min_bytes) makes the call run in several
 * passes over groups of requests. */
size_t tx_workspace_bytes(const tx_kv_cache* cache, int32_t op, int32_t n_req, const int64_t* offs_a,
                          const int64_t* offs_b);
size_t tx_workspace_min_bytes(const tx_kv_cache* cache, int32_t op, int32_t n_req, const int64_t* offs_a,
                              const int64_t* offs_b);

/* ------------------------------------------------------------ the path */

/* kv_cache_build -- nearline encoding of whole behavior sequences (Sec. 4.3,
 * amortized encoding and caching; Sec. 4.1.1 causal encoder).
 *   behavior          device [sum L][d_model]: behavior tokens H of each request
 *   behavior_offsets  host [n_req+1]; request i owns rows offsets[i]..offsets[i+1]-1,
 *                     L_i >= 1 and L_i <= max_tokens
 * Runs the encoder over each sequence, keeps every encoder layer's K/V (for
 * later appends) and every decoder layer's cross-attention K/V
 * (K = Phi_b W_K, V = Phi_b W_V, Sec. 4.1.2) in the request's pages. Replaces
 * any existing cache of those ids. Errors: TX_E_INVALID (duplicate / out-of-range
 * ids, bad offsets, L < 1, misaligned pointers), TX_E_NOMEM (pool or workspace),
 * TX_E_HIP. */
int kv_cache_build(tx_kv_cache* cache, int32_t n_req, const int32_t* req_ids /* host */, const void* behavior,
                   const int64_t* behavior_offsets /* host */, void* ws, size_t ws_bytes, hipStream_t stream);

/* kv_cache_append -- incremental encoding of new behavior events (App. D
 * remark: with a causal encoder and relative position bias the cached tokens'
 * states do not change; only the new tokens are encoded, against the stored
 * per-layer K/V of the prefix). The new rows take positions len .. len+n-1
 * and the cache grows in place.
 *   events         device [sum n][d_model]
 *   event_offsets  host [n_req+1], n_i >= 1
 * Errors: TX_E_NOCACHE (a request has no cache), TX_E_INVALID, TX_E_NOMEM,
 * TX_E_HIP. */
int kv_cache_append(tx_kv_cache* cache, int32_t n_req, const int32_t* req_ids /* host */, const void* events,
                    const int64_t* event_offsets /* host */, void* ws, size_t ws_bytes, hipStream_t stream);

/* score_candidates -- online serving of one serving event per request
 * (Sec. 4.1.2 cross-attention onto the cached K/V shared by all queries of the
 * request; App. B candidate-isolating mask; Sec. 4.1.3 with a linear head).
 *   serving            device [sum S][d_model]: serving-event tokens, causal among themselves
 *   serving_offsets    host [n_req+1], S_i >= 0
 *   candidates         device [sum C][d_model]: candidate tokens; each sees every serving
 *                      token of its request and itself, never another candidate
 *   candidate_offsets  host [n_req+1], C_i >= 0
 *   scores             device fp32 [sum C]: scores[candidate_offsets[i] + c] is the
 *                      logit of candidate c of request i (sigmoid = click probability);
 *                      with n_actions = k, [sum C][k]: row candidate_offsets[i] + c holds
 *                      that candidate's probabilities over the k actions (sum 1)
 * A request with C_i = 0 contributes nothing. Errors: TX_E_NOCACHE (a request
 * has no cache: cold start, App. D), TX_E_INVALID, TX_E_NOMEM, TX_E_HIP. */
int score_candidates(const tx_kv_cache* cache, int32_t n_req, const int32_t* req_ids /* host */,
                     const void* serving, const int64_t* serving_offsets /* host */, const void* candidates,
                     const int64_t* candidate_offsets /* host */, float* scores, void* ws, size_t ws_bytes,
                     hipStream_t stream);

/* score_events -- event-sliced decoding for seq-to-seq training (Sec. 4.2:
 * the behavior stream is encoded once and every serving event decodes against
 * its own prefix of it, sliced rather than re-encoded; exact because the
 * encoder is causal). Event e uses the cache of request req_ids[e] (ids may
 * repeat: several events of one user) but only its first prefix_len[e]
 * cached tokens as cross-attention keys (1 <= prefix_len[e] <= cached length).
 * With the local-global sparse form the window is the prefix's last l_local
 * tokens; a pooled global token exists only for the whole history, so with
 * global_pool every prefix_len[e] must equal the cached length
 * (TX_E_UNSUPPORTED otherwise). Other arguments, outputs and errors as in
 * score_candidates, with events in place of requests. */
int score_events(const tx_kv_cache* cache, int32_t n_events, const int32_t* req_ids /* host */,
                 const int64_t* prefix_len /* host */, const void* serving, const int64_t* serving_offsets /* host */,
                 const void* candidates, const int64_t* candidate_offsets /* host */, float* scores, void* ws,
                 size_t ws_bytes, hipStream_t stream);

/* score_candidates_static -- score_candidates for callers that cannot
 * allocate device memory or call allocating routines: code under HIP graph
 * capture, serving loops and harnesses that forbid allocation. Arguments,
 * outputs and errors as in score_candidates, without the workspace: the call
 * uses a fixed array of TX_STATIC_SCRATCH_BYTES (128 MiB) in the library's own
 * device memory, one per GPU the library runs on, held from the library's
 * first use on that GPU until the process ends, and the pinned staging for
 * its metadata that tx_kv_cache_create reserved. A batch larger than the
 * array runs in several passes over groups of requests; a request whose own
 * activations or metadata exceed it is rejected with TX_E_NOMEM before any
 * launch. It calls no hipMalloc, hipFree or other allocating routine. Every
 * call on one GPU shares that GPU's array, which keeps the last call's
 * contents (nothing in it needs to start at zero): calls that overlap on one
 * GPU, on different streams or from different threads, race. The stream must
 * belong to the current device (TX_E_INVALID otherwise). */
#define TX_STATIC_SCRATCH_BYTES ((size_t)128 << 20)
int score_candidates_static(const tx_kv_cache* cache, int32_t n_req, const int32_t* req_ids /* host */,
                            const void* serving, const int64_t* serving_offsets /* host */, const void* candidates,
                            const int64_t* candidate_offsets /* host */, float* scores, hipStream_t stream);

/* ------------------------------------------------------------ measurement */

/* Per-kernel timing for roofline reports. While enabled, every kernel launch
 * of the calls above is bracketed by a HIP event pair recorded on the caller's
 * stream, and tagged with its kernel class and the algorithmic flops and bytes
 * of that launch (the work the method defines for it, not what the kernel
 * happens to move). tx_profile_enable clears earlier records; enabling makes
 * 2048 events up front (call it while the GPU is idle: creating events while
 * kernels run stalled a running kernel by milliseconds when the runtime grew
 * its signal pool), enough for 1024 launches between reads. */
int tx_profile_enable(int32_t on);
/* Restricts recording to the classes whose bit (1 << class index) is set in
 * class_mask, so that a timed region carries event pairs only around the
 * launches it reports; tx_profile_enable resets it to every class. Always
 * TX_OK (bits past tx_profile_classes() are ignored). */
int tx_profile_select(uint64_t class_mask);
int32_t tx_profile_classes(void);
const char* tx_profile_class_name(int32_t i);
/* Per class (arrays of tx_profile_classes() entries, any may be NULL): summed
 * event time in ms, number of launches, algorithmic flops and bytes. Waits
 * for the recorded events. */
int tx_profile_read(double* total_ms, int64_t* launches, double* flops, double* bytes);

#ifdef __cplusplus
}
#endif

#endif /* TRANSX_H */
