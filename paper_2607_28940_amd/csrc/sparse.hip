// Local-global sparse cross-attention of the TransX decoder (Sec. 4.1.2,
// paragraph on local-global sparse cross attention and Eq. sparse-cross-attn):
// every decoder query attends to the index set I_t = the L_local most recent
// cached behavior tokens plus one global anchor token. The anchor is the
// attention pooling of the encoded behavior rows (the experiments' choice,
// Sec. 5 setup): weights softmax_j(h_j . w / sqrt(d)) with a learned vector
// w, pooled token g = sum_j weight_j h_j, projected by the same cross-attention
// K/V weights as any cached row.
//
// The pooling keeps a running (max, sum, weighted sum) per request, the
// online-softmax state, so appending events folds only the new rows into it
// (the incremental form App. D asks of every cached quantity).
//
// Both parts are small next to the decoder GEMMs: the pooling reads the
// encoded rows once, and the attention touches at most 65 keys per query, so
// these kernels use plain fp32 arithmetic rather than MFMA tiles.
#include "tx_internal.h"
#include "wave_reduce.h"

namespace tx {

// ---------------------------------------------------------------- pooling

template <typename T>
__global__ __launch_bounds__(256) void pool_partial(const T* __restrict__ H, int d, const float* __restrict__ w,
                                                    float zscale, const PoolChunk* __restrict__ chunks,
                                                    float* __restrict__ part) {
  __shared__ float z[64], e[64];
  const PoolChunk ck = chunks[blockIdx.x];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // logits: wave w takes rows w, w+4, ...; lanes split the features
  for (int r = wave; r < ck.n; r += 4) {
    const T* h = H + (size_t)(ck.row0 + r) * d;
    float s = 0.f;
    for (int f = lane; f < d; f += 64) s = fmaf((float)h[f], w[f], s);
    s = wave_sum(s);
    if (lane == 0) z[r] = s * zscale;
  }
  __syncthreads();
  float m = -INFINITY;
  for (int r = 0; r < ck.n; ++r) m = fmaxf(m, z[r]);
  if (tid < ck.n) e[tid] = expf(z[tid] - m);
  __syncthreads();
  float* out = part + (size_t)blockIdx.x * (d + 2);
  for (int f = tid; f < d; f += 256) {
    float a = 0.f;
    for (int r = 0; r < ck.n; ++r) a = fmaf(e[r], (float)H[(size_t)(ck.row0 + r) * d + f], a);
    out[2 + f] = a;
  }
  if (tid == 0) {
    float l = 0.f;
    for (int r = 0; r < ck.n; ++r) l += e[r];
    out[0] = m;
    out[1] = l;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void pool_combine(const float* __restrict__ part, const PoolReq* __restrict__ reqs,
                                                    int d, float* __restrict__ ml, float* __restrict__ acc,
                                                    T* __restrict__ g_out) {
  const PoolReq rq = reqs[blockIdx.x];
  const int tid = threadIdx.x;
  const float m_old = rq.fresh ? -INFINITY : ml[2 * rq.slot];
  const float l_old = rq.fresh ? 0.f : ml[2 * rq.slot + 1];
  float m = m_old;
  for (int c = 0; c < rq.n_chunks; ++c) m = fmaxf(m, part[(size_t)(rq.chunk0 + c) * (d + 2)]);
  float l = rq.fresh ? 0.f : l_old * expf(m_old - m);
  for (int c = 0; c < rq.n_chunks; ++c) {
    const float* pc = part + (size_t)(rq.chunk0 + c) * (d + 2);
    l += pc[1] * expf(pc[0] - m);
  }
  __syncthreads();  // every thread has read the old state before it is replaced
  const float old_scale = rq.fresh ? 0.f : expf(m_old - m);
  const float inv = 1.f / l;
  for (int f = tid; f < d; f += 256) {
    float a = rq.fresh ? 0.f : acc[(size_t)rq.slot * d + f] * old_scale;
    for (int c = 0; c < rq.n_chunks; ++c) {
      const float* pc = part + (size_t)(rq.chunk0 + c) * (d + 2);
      a = fmaf(pc[2 + f], expf(pc[0] - m), a);
    }
    acc[(size_t)rq.slot * d + f] = a;
    g_out[(size_t)blockIdx.x * d + f] = (T)(a * inv);
  }
  if (tid == 0) {
    ml[2 * rq.slot] = m;
    ml[2 * rq.slot + 1] = l;
  }
}

hipError_t launch_pool(bool bf, const void* H, int d, const float* w, float zscale, const PoolChunk* chunks,
                       int n_chunks, const PoolReq* reqs, int n_req, float* part, float* ml, float* acc, void* g_out,
                       hipStream_t s) {
  if (n_chunks <= 0 || n_req <= 0) return hipSuccess;
  if (bf) {
    pool_partial<bf16><<<n_chunks, 256, 0, s>>>((const bf16*)H, d, w, zscale, chunks, part);
    pool_combine<bf16><<<n_req, 256, 0, s>>>(part, reqs, d, ml, acc, (bf16*)g_out);
  } else {
    pool_partial<float><<<n_chunks, 256, 0, s>>>((const float*)H, d, w, zscale, chunks, part);
    pool_combine<float><<<n_req, 256, 0, s>>>(part, reqs, d, ml, acc, (float*)g_out);
  }
  return hipGetLastError();
}

template <typename T>
__global__ __launch_bounds__(256) void store_rows(const T* __restrict__ src, int W, const PoolReq* __restrict__ reqs,
                                                  T* __restrict__ dst) {
  const int slot = reqs[blockIdx.x].slot;
  for (int i = threadIdx.x; i < W; i += 256) dst[(size_t)slot * W + i] = src[(size_t)blockIdx.x * W + i];
}

hipError_t launch_store_rows(bool bf, const void* src, int W, const PoolReq* reqs, int n_req, void* dst,
                             hipStream_t s) {
  if (n_req <= 0) return hipSuccess;
  if (bf) store_rows<bf16><<<n_req, 256, 0, s>>>((const bf16*)src, W, reqs, (bf16*)dst);
  else store_rows<float><<<n_req, 256, 0, s>>>((const float*)src, W, reqs, (float*)dst);
  return hipGetLastError();
}

// ---------------------------------------------------------------- attention

// One block per tile of 64 queries of one (request, head): the keys and
// values (at most l_local + 1) go to LDS as fp32, sized for the launch's
// window so that many blocks share a CU (K rows are read feature-fastest, V
// from the page's transposed, k-permuted layout key-fastest, both
// contiguous), then every query is served by 4 lanes, each owning DH/4
// features, with the online softmax in the exp2 domain. In LDS each key row
// keeps the four lanes' feature runs 16-byte aligned and DH/4 + 4 floats
// apart, so a lane reads its run with 16-byte loads and the four runs of a
// query fall in different banks (the 16 queries of a wave read the same row:
// broadcast).
template <typename T, int DH>
__global__ __launch_bounds__(256) void lg_cross_attn(const T* __restrict__ q, int ldq, T* __restrict__ out, int ldo,
                                                     const T* __restrict__ pool, const int32_t* __restrict__ page_table,
                                                     int max_pages, PageGeom g, int layer_slot,
                                                     const AttnReq* __restrict__ reqs,
                                                     const AttnTile* __restrict__ tiles, int l_local,
                                                     const T* __restrict__ gkv, int gkv_ld, int dec_layer,
                                                     float scale_log2) {
  constexpr int DP = DH / 4, PS = DP + 4, LD = 4 * PS;  // part stride, row stride (floats)
  extern __shared__ __attribute__((aligned(16))) float smem[];
  float* sK = smem;                               // [l_local + 1][LD]
  float* sV = smem + (size_t)(l_local + 1) * LD;  // [l_local + 1][LD]
  auto at = [](int j, int f) { return j * LD + (f / DP) * PS + (f % DP); };
  const AttnTile tile = tiles[blockIdx.x];
  if (tile.q_count <= 0) return;
  const AttnReq rq = reqs[tile.req];
  const int h = tile.head, tid = threadIdx.x, qi = tid >> 2, part = tid & 3;
  const int len = rq.kv_len;
  const int k0 = max(0, len - l_local), nl = len - k0;
  const int32_t* ptab = page_table + (size_t)rq.slot * max_pages;
  for (int e = tid; e < nl * DH; e += 256) {
    const int j = e / DH, f = e % DH;  // feature fastest: one K row is contiguous
    const int pos = k0 + j;
    const T* base = pool + (size_t)ptab[pos / kPage] * g.page_elems;
    sK[at(j, f)] = (float)base[g.k_off(layer_slot, h) + (size_t)(pos % kPage) * DH + f];
  }
  for (int e = tid; e < nl * DH; e += 256) {
    const int f = e / nl, j = e % nl;  // key fastest: one V^T row is contiguous
    const int pos = k0 + j;
    const T* base = pool + (size_t)ptab[pos / kPage] * g.page_elems;
    sV[at(j, f)] = (float)base[g.v_off(layer_slot, h) + (size_t)f * kPage + vt_col(pos % kPage)];
  }
  int nk = nl;
  if (gkv) {
    const int d = g.H * DH;
    const T* kr = gkv + (size_t)rq.slot * gkv_ld + (size_t)(2 * dec_layer) * d + h * DH;
    for (int f = tid; f < DH; f += 256) {
      sK[at(nl, f)] = (float)kr[f];
      sV[at(nl, f)] = (float)kr[d + f];
    }
    ++nk;
  }
  __syncthreads();
  if (qi >= tile.q_count) return;
  const int i = tile.q_begin + qi;
  const int row = i < rq.qa_n ? rq.qa_row + i : rq.qb_row + (i - rq.qa_n);
  float qv[DP], acc[DP];
#pragma unroll
  for (int e = 0; e < DP; ++e) {
    qv[e] = (float)q[(size_t)row * ldq + h * DH + part * DP + e];
    acc[e] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int j = 0; j < nk; ++j) {
    const floatx4* kr = reinterpret_cast<const floatx4*>(sK + j * LD + part * PS);
    const floatx4* vr = reinterpret_cast<const floatx4*>(sV + j * LD + part * PS);
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < DP / 4; ++e) {
      const floatx4 k4 = kr[e];
#pragma unroll
      for (int c = 0; c < 4; ++c) s = fmaf(qv[4 * e + c], k4[c], s);
    }
    s = quad_sum(s);  // the query's four lanes
    s *= scale_log2;
    const float m_new = fmaxf(m, s);
    const float alpha = __builtin_amdgcn_exp2f(m - m_new);  // 0 while m is -inf
    const float p = __builtin_amdgcn_exp2f(s - m_new);
    l = l * alpha + p;
#pragma unroll
    for (int e = 0; e < DP / 4; ++e) {
      const floatx4 v4 = vr[e];
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[4 * e + c] = fmaf(p, v4[c], acc[4 * e + c] * alpha);
    }
    m = m_new;
  }
  const float inv = 1.f / l;
#pragma unroll
  for (int e = 0; e < DP; ++e) out[(size_t)row * ldo + h * DH + part * DP + e] = (T)(acc[e] * inv);
}

hipError_t launch_lg_attention(bool bf, const void* q, int ldq, void* out, int ldo, const void* pool,
                               const int32_t* page_table, int max_pages, PageGeom g, int layer_slot,
                               const AttnReq* reqs, const AttnTile* tiles, int n_tiles, int l_local,
                               const void* gkv, int gkv_ld, int dec_layer, hipStream_t s) {
  if (n_tiles <= 0) return hipSuccess;
  if (l_local < 1 || l_local > kMaxLocal) return hipErrorInvalidValue;
  const float sl2 = 1.4426950408889634f / sqrtf((float)g.dh);
  const size_t lds = (size_t)(l_local + 1) * 4 * (g.dh / 4 + 4) * 2 * sizeof(float);
#define TX_LG(TT, DH)                                                                                            \
  lg_cross_attn<TT, DH><<<n_tiles, 256, lds, s>>>((const TT*)q, ldq, (TT*)out, ldo, (const TT*)pool, page_table, \
                                                max_pages, g, layer_slot, reqs, tiles, l_local, (const TT*)gkv,  \
                                                gkv_ld, dec_layer, sl2)
  switch (g.dh) {
    case 32: if (bf) TX_LG(bf16, 32); else TX_LG(float, 32); break;
    case 64: if (bf) TX_LG(bf16, 64); else TX_LG(float, 64); break;
    case 128: if (bf) TX_LG(bf16, 128); else TX_LG(float, 128); break;
    default: return hipErrorInvalidValue;
  }
#undef TX_LG
  return hipGetLastError();
}

}  // namespace tx
