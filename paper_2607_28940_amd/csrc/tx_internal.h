// Internal declarations of the TransX HIP library: element types, device
// helpers, the metadata records the host hands to kernels, and the launch
// functions each kernel file exports to the API layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tx {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
// Storage of a post-LN sublayer's pre-LayerNorm sum (bias + residual +
// sublayer output) in bf16 models: 11 mantissa bits at the width of bf16.
typedef _Float16 f16;
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kPage = 64;  // tokens per cache page

// ------------------------------------------------------------ metadata records

// One request as seen by an attention launch. Query i of the request lives in
// activation row (i < qa_n ? qa_row + i : qb_row + i - qa_n); when causal it sits
// at sequence position pos0 + i. Keys are cache positions 0 .. kv_len-1 of the
// request whose page-table row is `slot`.
struct AttnReq {
  int32_t qa_row, qa_n, qb_row, qb_n;
  int32_t kv_len, pos0, slot, pad;
};

// A unit of attention work: queries q_begin .. q_begin+q_count-1 of request
// `req` (index into the AttnReq array) for head `head`.
struct AttnTile {
  int32_t req, head, q_begin, q_count;
};

// One request of the decoder self-attention: serving rows s_row .. s_row+S-1
// (causal among themselves), candidate rows c_row .. c_row+C-1 (see every
// serving row and themselves).
struct SelfReq {
  int32_t s_row, S, c_row, C;
};

// A tile of the decoder cross-attention: queries q_begin ..
// q_begin + q_count - 1 (at most 128) of one request and head against the
// request's key pages page_begin .. page_end - 1. Query i of the request lives
// in activation row (i < qa_n ? qa_row + i : qb_row + i - qa_n); kv_len is the
// request's cached length (keys past it, on its last page, are masked), slot
// its page-table row. part < 0: the tile covers every page and writes the
// output rows; part >= 0: a kv-split tile that writes its unnormalised output,
// running max and sum to partial slot `part` (128 x (d_h + 2) floats).
struct XTile {
  int32_t head, q_begin, q_count, part;
  int32_t page_begin, page_end, kv_len, slot;
  int32_t qa_row, qa_n, qb_row, pad;
};
// Merge of the n_parts partial slots part0 .. part0 + n_parts - 1 of one
// (request, head, query block) into its output rows.
struct XMerge {
  int32_t head, q_begin, q_count, part0;
  int32_t n_parts, qa_row, qa_n, qb_row;
};

// Self-attention tile: queries q_begin.. (in the request's [serving; candidate]
// order) of request `req`, head `head`.
typedef AttnTile SelfTile;

// Rows to scatter into cache pages: rows row0 .. row0+n-1 of the source matrix
// take sequence positions pos0 .. pos0+n-1 of the request in page-table row slot.
struct ScatterReq {
  int32_t row0, n, pos0, slot;
};

// Part of one cache page written by a scatter: positions t0 .. t1-1 of page
// `page` of request slot `slot`, position t0 coming from source row `row`.
struct ScatterTile {
  int32_t slot, page, t0, t1, row;
};

// Attention pooling work: rows row0 .. row0+n-1 (n <= 64) of the encoded
// matrix, one chunk of the request at index `req` of the pass.
struct PoolChunk {
  int32_t req, row0, n, pad;
};
// Per request of a pass: its chunks chunk0 .. chunk0+n_chunks-1, its page-table
// row (which also indexes the per-request pooling state and global-token K/V),
// and whether the pooling starts afresh (build) or continues the stored state
// (append).
struct PoolReq {
  int32_t chunk0, n_chunks, slot, fresh;
};

// Geometry of a cache page: for each layer slot (encoder layers, then decoder
// layers), K as [H][64][dh] then V transposed as [H][dh][64].
// Column of token t (0..63 within its page) in a stored V^T row: every group
// of 16 tokens is kept in the order 0-3, 8-11, 4-7, 12-15, the k order the
// bf16 attention kernels feed to the PV MFMA (the map is its own inverse).
__host__ __device__ inline int vt_col(int t) { return (t & ~15) | (t & 3) | ((t & 4) << 1) | ((t & 8) >> 1); }

struct PageGeom {
  int32_t H, dh, n_slots;
  int64_t page_elems;  // elements per page
  __host__ __device__ int64_t k_off(int slot, int h) const {
    return ((int64_t)(slot * 2 + 0) * H + h) * kPage * dh;
  }
  __host__ __device__ int64_t v_off(int slot, int h) const {
    return ((int64_t)(slot * 2 + 1) * H + h) * kPage * dh;
  }
};

// ------------------------------------------------------------ launch functions
// Every launcher returns hipSuccess or the launch error. Element type of the
// activations is given by `bf16` (true) or fp32 (false).

// Epilogues of C = A * Bt^T + bias:
//   EPI_BIAS        C = acc + bias                          (C in the model type)
//   EPI_BIAS_GELU   C = GELU(acc + bias)                    (C in the model type)
//   EPI_BIAS_RESID  C = acc + bias + R, R in the model type (C in the sum type)
//   EPI_BIAS_RESLN  C = acc + bias + LN(R), R in the sum type, where
//                   LN(R)[m][n] = (R[m][n] * st[m].x + st[m].y) * g[n] + b[n]
//                   recomputes in fp32 the LayerNorm output whose rounded copy
//                   the sublayer read as its operand       (C in the sum type)
//   EPI_LN          C = LN(A) * W + b, computed as (acc * st[m].x + st[m].y *
//   EPI_LN_GELU     cs[n]) + b'[n] (then GELU): the consumer of a LayerNorm
//                   output multiplies the stored pre-LN sum itself (A in the
//                   sum type, fp16) by the gain-scaled weight W'[k][n] =
//                   g[k] W[k][n] (Bt in fp16), cs[n] = sum_k W'[k][n] and
//                   b'[n] = b[n] + sum_k LNb[k] W[k][n] (ln.g = cs, bias = b');
//                   bf16 models, MFMA-kernel shapes only (gemm_ln_ok)
//                                                           (C in the model type)
// The sum type holds a post-LN sublayer's pre-LayerNorm sum: fp16 for bf16
// models (same width, 8x finer rounding), fp32 for fp32 models.
enum Epilogue { EPI_BIAS = 0, EPI_BIAS_GELU = 1, EPI_BIAS_RESID = 2, EPI_BIAS_RESLN = 3, EPI_LN = 4, EPI_LN_GELU = 5 };
__host__ __device__ constexpr bool epi_resid(int e) { return e == EPI_BIAS_RESID || e == EPI_BIAS_RESLN; }
__host__ __device__ constexpr bool epi_gelu(int e) { return e == EPI_BIAS_GELU || e == EPI_LN_GELU; }
__host__ __device__ constexpr bool epi_lnfold(int e) { return e == EPI_LN || e == EPI_LN_GELU; }

// Row statistics of a LayerNorm in the form its consumers apply it:
// x = 1 / sqrt(var + eps), y = -mean * x (so LN(v) = (v * x + y) * g + b).
struct LnRow {
  float x, y;
};
struct LnResid {
  const LnRow* stats = nullptr;
  const float* g = nullptr;
  const float* b = nullptr;
};

// C[M][N] (ldc) = epi(A[M][K] (lda) * Bt[N][K]^T + bias[N] (+ residual)).
// C must not overlap A or R.
bool gemm_ln_ok(int N, int K, int lda, int ldc);  // EPI_LN* runs on this shape (any M)
hipError_t launch_gemm(bool bf, const void* A, int lda, const void* Bt, const float* bias, const void* R, int ldr,
                       void* C, int ldc, int M, int N, int K, Epilogue epi, hipStream_t s, LnResid ln = LnResid());

// y[i] = LN(x[i]) * g + b over d features for M rows; x in the sum type, y in
// the model type; the row statistics go to stats[i] when it is not null. With
// y null only the statistics are written (their consumers fold the LayerNorm).
hipError_t launch_layernorm(bool bf, const void* x, void* y, LnRow* stats, const float* g, const float* b, int M,
                            int d, float eps, hipStream_t s);
// Decoder head on LN(x[i]) = z_i, x in the sum type (fp32 out): n_act == 0: scores[i] = z_i . w + b0;
// n_act = k >= 2: scores[i][a] = softmax_a(z_i . w[a] + b0[a]), w fp32 [k][d].
hipError_t launch_layernorm_score(bool bf, const void* x, const float* g, const float* b, const float* w,
                                  const float* b0, float* scores, int M, int d, float eps, int n_act, hipStream_t s);

// Paged attention: out[row] = softmax(q k^T / sqrt(dh) (+ rel bias)) v over the
// request's cached keys (causal: keys at positions <= the query's position).
hipError_t launch_paged_attention(bool bf, const void* q, int ldq, void* out, int ldo, const void* pool,
                                  const int32_t* page_table, int max_pages, PageGeom g, int layer_slot,
                                  const AttnReq* reqs, const AttnTile* tiles, int n_tiles, bool causal,
                                  const float* rel, int R, int q_block, hipStream_t s);
// Query block (queries per tile) each attention kernel variant expects.
// Causal tiles of kDecodeQBlock queries (bf16, dh 64 or 128, at most
// kDecodeMaxRel relative-position buckets) select the kernel that streams
// pages into registers: for encoder passes with at most that many new tokens
// per request (appends), where no page is shared by several waves.
int paged_attention_q_block(bool bf, int dh);
constexpr int kDecodeQBlock = 32;
constexpr int kDecodeMaxRel = 256;  // relative-position buckets the register kernel holds
inline bool paged_attention_decode_ok(bool bf, int dh, int R) { return bf && (dh == 64 || dh == 128) && R <= kDecodeMaxRel; }

// Decoder self-attention over the packed QKV matrix (ld 3d).
hipError_t launch_self_attention(bool bf, const void* qkv, int d, int H, void* out, const SelfReq* reqs,
                                 const SelfTile* tiles, int n_tiles, bool candidates_only, hipStream_t s);
int self_attention_q_block(bool bf, int dh);

// Write K and V columns of src (per layer: K in cols [l*2d, l*2d+d), V in
// [l*2d+d, l*2d+2d); ld = lds) into the pages of layer slots
// slot0 .. slot0+n_layers-1, one page tile (page_tiles) at a time.
hipError_t launch_scatter_kv(bool bf, const void* src, int lds, int n_layers, int slot0, void* pool,
                             const int32_t* page_table, int max_pages, PageGeom g, const ScatterTile* tiles,
                             int n_tiles, hipStream_t s);
// Export one cached tensor (K or V of a layer slot) of a request into a dense
// [len][H*dh] matrix.
hipError_t launch_export_kv(bool bf, const void* pool, const int32_t* page_row, PageGeom g, int layer_slot, int is_v,
                            int64_t len, void* out, hipStream_t s);

// Attention pooling of encoded rows H [rows][d] with vector w (fp32 [d]):
// per chunk the running max, sum and weighted row sum of exp(h.w*zscale)
// (part: fp32 [n_chunks][d + 2] = max, sum, acc[d]), then per request the
// merge of its chunks with the stored state (ml: fp32 [max_req][2], acc:
// fp32 [max_req][d]), which is updated in place, and the pooled token
// acc / sum written to g_out [n_req][d] in the model's element type.
hipError_t launch_pool(bool bf, const void* H, int d, const float* w, float zscale, const PoolChunk* chunks,
                       int n_chunks, const PoolReq* reqs, int n_req, float* part, float* ml, float* acc, void* g_out,
                       hipStream_t s);
// dst[slot][0 .. W) = src[i][0 .. W) for every request i of the pass
hipError_t launch_store_rows(bool bf, const void* src, int W, const PoolReq* reqs, int n_req, void* dst,
                             hipStream_t s);
// Local-global sparse cross-attention: each query attends to the last
// min(l_local, kv_len) cached tokens of its request (layer slot layer_slot)
// and, when gkv is not null, to the request's global token, whose key and
// value are columns [2*dec_layer*d + h*dh ..) and [(2*dec_layer+1)*d + h*dh ..)
// of row `slot` of gkv (row stride gkv_ld). Tiles of q_block =
// lg_attention_q_block(bf, l_local, gkv != nullptr, H, dh) queries (checked),
// each serving heads [head * hb, head * hb + hb) of its queries with
// hb = lg_attention_heads_per_tile(...) (tiles planned with H / hb heads).
int lg_attention_q_block(bool bf, int l_local, bool gpool, int H, int dh);
int lg_attention_heads_per_tile(bool bf, int l_local, bool gpool, int H, int dh);
hipError_t launch_lg_attention(bool bf, const void* q, int ldq, void* out, int ldo, const void* pool,
                               const int32_t* page_table, int max_pages, PageGeom g, int layer_slot,
                               const AttnReq* reqs, const AttnTile* tiles, int n_tiles, int q_block, int l_local,
                               const void* gkv, int gkv_ld, int dec_layer, hipStream_t s);
// Decoder cross-attention over per-XCD tile lists (bf16, d_h = 128): XCD x
// owns tiles[xoff[x] .. xoff[x + 1]); block b (which the hardware runs on XCD
// b % 8) takes entry b / 8 of its XCD's list, on a grid of 8 x longest_list
// blocks. The whole-request tiles write their rows; the kv-split tiles, a
// tile set and a launch of their own, write partial slots (kXPartBytes
// each), which the merge items then combine into the output rows.
bool cross_attention_split_ok(bool bf, int dh);
constexpr int kXQueryBlock = 128;  // queries per tile
constexpr int kXBlocksPerCu = 3;   // resident blocks per CU
constexpr size_t kXPartBytes = (size_t)128 * (128 + 2) * 4;  // one partial slot
hipError_t launch_cross_attention(const void* q, int ldq, void* out, int ldo, const void* pool,
                                  const int32_t* page_table, int max_pages, PageGeom g, int layer_slot,
                                  const XTile* tiles, const int32_t* xoff, int longest_list,
                                  const XTile* split_tiles, const int32_t* split_xoff, int split_longest,
                                  float* partial, const XMerge* merges, int n_merges, hipStream_t s);
constexpr int kMaxActions = 16;  // largest supported action vocabulary of the decoder head
constexpr int kMaxLocal = 64;  // largest supported l_local

// Workspace of the no-allocation entry point: a fixed array in the library's
// device memory, one per GPU, of kStaticScratchBytes. static_scratch() gives
// the current device's address of it (looked up once per device).
constexpr size_t kStaticScratchBytes = (size_t)128 << 20;
hipError_t static_scratch(void** out);

// dst[n][k] = src[k][n] (src [K][N] row-major), same element type
hipError_t launch_transpose(bool bf, const void* src, void* dst, int K, int N, int dst_ld, hipStream_t s);
// The weight of a LayerNorm-folding GEMM (EPI_LN*) from the repacked bf16
// weight Bt [N][K], the LayerNorm's gain g and offset lnb [K] and the bias [N]:
// Wf [N][K] fp16 = g[k] Bt[n][k], cs[n] = sum_k Wf[n][k], bf[n] = bias[n] +
// sum_k lnb[k] Bt[n][k]; *overflow set to 1 when a scaled weight is not finite
// in fp16.
hipError_t launch_fold_ln_weight(const void* Bt, int N, int K, const float* g, const float* lnb, const float* bias,
                                 void* Wf, float* cs, float* bf, int* overflow, hipStream_t s);
// *p = 0 on the stream; *host = *dev after the stream's work so far.
hipError_t launch_zero_int(int* p, hipStream_t s);
hipError_t read_int(const int* dev, int* host, hipStream_t s);
// dst fp32 [N][K] = src [K][N]
hipError_t launch_transpose_to_f32(bool bf, const void* src, float* dst, int K, int N, hipStream_t s);
// dst fp32[n] = src[n]
hipError_t launch_to_f32(bool bf, const void* src, float* dst, int64_t n, hipStream_t s);

}  // namespace tx
