// Row-wise and data-movement kernels of the TransX path:
//   LayerNorm of post-LN sublayers (Sec. 4.1.2 crossAttend block) over the
//   stored pre-LN sums, with its row statistics kept for later residuals, optionally
//   fused with the decoder head (Sec. 4.1.3, Eq. action-decoding: either the
//   softmax over k action embeddings, or with two actions one logit), the
//   scatter of projected K/V rows into
//   the paged cache layout, cache export, and weight repacking.
#include "tx_internal.h"
#include "wave_reduce.h"

#include <algorithm>

namespace tx {

// Decoder head on one wave's row, given this lane's share of the normalised
// row (z at features c0 + e * stride, e < cnt). n_act == 0:
// scores[row] = z . w + b0[0]. n_act = k >= 2: w is [k][d] (row a = action
// a's embedding, repacked that way so a lane reads its features of one
// action contiguously), lane a ends up with logit a, and the softmax over the
// k lanes gives scores[row * k + a].
template <int CNT>
__device__ __forceinline__ void head_out(const float (&z)[CNT], int c0, int stride, int cnt, int lane, int d,
                                         const float* __restrict__ w, const float* __restrict__ b0,
                                         float* __restrict__ scores, int row, int n_act) {
  if (n_act == 0) {
    float dot = 0.f;
#pragma unroll
    for (int e = 0; e < CNT; ++e)
      if (e < cnt) dot += z[e] * w[c0 + e * stride];
    dot = wave_sum(dot);
    if (lane == 0) scores[row] = dot + b0[0];
    return;
  }
  float mine = -INFINITY;
  for (int a = 0; a < n_act; ++a) {
    float dot = 0.f;
#pragma unroll
    for (int e = 0; e < CNT; ++e)
      if (e < cnt) dot += z[e] * w[(size_t)a * d + c0 + e * stride];
    dot = wave_sum(dot);
    if (lane == a) mine = dot + b0[a];
  }
  float mx = mine;
  mx = wave_max(mx);
  const float e = lane < n_act ? expf(mine - mx) : 0.f;
  float den = e;
  den = wave_sum(den);
  if (lane < n_act) scores[(size_t)row * n_act + lane] = e / den;
}

// One wave per row at a time; EPL features per lane held in registers
// (EPL = d / 64). Each wave walks rows wave_id, wave_id + n_waves, ... so the
// gain and bias it needs are loaded once, and the next row's features are
// requested before the current row is normalised. Two-pass mean / variance
// in fp32 from the register copy. The input is the sublayer's pre-LN sum (sum
// type TX); the output row goes out in the model type T, and the row's
// statistics to `stats` (when given) for the epilogue that adds this LayerNorm
// output as a residual later.
template <typename TX, typename T, int EPL, bool SCORE>
__global__ __launch_bounds__(256) void layernorm_rows(const TX* __restrict__ x, T* __restrict__ y,
                                                      LnRow* __restrict__ stats, const float* __restrict__ g,
                                                      const float* __restrict__ b, const float* __restrict__ w,
                                                      const float* __restrict__ b0, float* __restrict__ scores, int M,
                                                      int d, float eps, int n_act) {
  const int lane = threadIdx.x & 63;
  const int n_waves = gridDim.x * 4;
  int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const int c0 = lane * EPL;
  float gv[EPL], bv[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    gv[e] = g[c0 + e];
    bv[e] = b[c0 + e];
  }
  TX nx[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) nx[e] = x[(size_t)row * d + c0 + e];
  for (; row < M; row += n_waves) {
    float v[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) v[e] = (float)nx[e];
    const int next = row + n_waves;
    if (next < M) {
#pragma unroll
      for (int e = 0; e < EPL; ++e) nx[e] = x[(size_t)next * d + c0 + e];
    }
    float sum = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) sum += v[e];
    sum = wave_sum(sum);
    const float mean = sum / d;
    float sq = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      const float t = v[e] - mean;
      sq += t * t;
    }
    sq = wave_sum(sq);
    const float inv = rsqrtf(sq / d + eps);
    const float sh = -mean * inv;
    if (SCORE) {
      float z[EPL];
#pragma unroll
      for (int e = 0; e < EPL; ++e) z[e] = fmaf(fmaf(v[e], inv, sh), gv[e], bv[e]);
      head_out<EPL>(z, c0, 1, EPL, lane, d, w, b0, scores, row, n_act);
    } else {
      if (y) {
        T* yr = y + (size_t)row * d + c0;
#pragma unroll
        for (int e = 0; e < EPL; ++e) yr[e] = (T)fmaf(fmaf(v[e], inv, sh), gv[e], bv[e]);
      }
      if (stats && lane == 0) stats[row] = LnRow{inv, sh};
    }
  }
}

// Generic width: one wave per row, strided features, three passes over the row.
template <typename TX, typename T, bool SCORE>
__global__ __launch_bounds__(256) void layernorm_rows_any(const TX* __restrict__ x, T* __restrict__ y,
                                                          LnRow* __restrict__ stats, const float* __restrict__ g,
                                                          const float* __restrict__ b, const float* __restrict__ w,
                                                          const float* __restrict__ b0, float* __restrict__ scores,
                                                          int M, int d, float eps, int n_act) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= M) return;
  const TX* xr = x + (size_t)row * d;
  float sum = 0.f;
  for (int c = lane; c < d; c += 64) sum += (float)xr[c];
  sum = wave_sum(sum);
  const float mean = sum / d;
  float sq = 0.f;
  for (int c = lane; c < d; c += 64) {
    const float t = (float)xr[c] - mean;
    sq += t * t;
  }
  sq = wave_sum(sq);
  const float inv = rsqrtf(sq / d + eps);
  const float sh = -mean * inv;
  if (!SCORE) {
    if (y)
      for (int c = lane; c < d; c += 64) y[(size_t)row * d + c] = (T)fmaf(fmaf((float)xr[c], inv, sh), g[c], b[c]);
    if (stats && lane == 0) stats[row] = LnRow{inv, sh};
    return;
  }
  // widths without a register-resident variant are at most 64 * 64 here
  constexpr int MAXC = 64;
  float z[MAXC];
  const int cnt = (d - lane + 63) / 64;
#pragma unroll
  for (int e = 0; e < MAXC; ++e) {
    const int c = lane + 64 * e;
    z[e] = (e < cnt) ? fmaf(fmaf((float)xr[c], inv, sh), g[c], b[c]) : 0.f;
  }
  head_out<MAXC>(z, lane, 64, cnt, lane, d, w, b0, scores, row, n_act);
}

template <typename TX, typename T, bool SCORE>
static hipError_t ln_dispatch(const void* x, void* y, LnRow* stats, const float* g, const float* b, const float* w,
                              const float* b0, float* scores, int M, int d, float eps, int n_act, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  const int blocks = (M + 3) / 4;
  // register-resident widths: at most 8 rows per wave (2048 blocks of 4 waves)
  const int rblocks = std::min(blocks, std::max(2048, (blocks + 7) / 8));
  const TX* xx = (const TX*)x;
  T* yy = (T*)y;
#define TX_LN(E) \
  layernorm_rows<TX, T, E, SCORE><<<rblocks, 256, 0, s>>>(xx, yy, stats, g, b, w, b0, scores, M, d, eps, n_act)
  switch (d) {
    case 64: TX_LN(1); break;
    case 128: TX_LN(2); break;
    case 256: TX_LN(4); break;
    case 512: TX_LN(8); break;
    case 1024: TX_LN(16); break;
    case 2048: TX_LN(32); break;
    default:
      if (SCORE && d > 64 * 64) return hipErrorInvalidValue;
      layernorm_rows_any<TX, T, SCORE><<<blocks, 256, 0, s>>>(xx, yy, stats, g, b, w, b0, scores, M, d, eps, n_act);
  }
#undef TX_LN
  return hipGetLastError();
}

hipError_t launch_layernorm(bool bf, const void* x, void* y, LnRow* stats, const float* g, const float* b, int M,
                            int d, float eps, hipStream_t s) {
  return bf ? ln_dispatch<f16, bf16, false>(x, y, stats, g, b, nullptr, nullptr, nullptr, M, d, eps, 0, s)
            : ln_dispatch<float, float, false>(x, y, stats, g, b, nullptr, nullptr, nullptr, M, d, eps, 0, s);
}

hipError_t launch_layernorm_score(bool bf, const void* x, const float* g, const float* b, const float* w,
                                  const float* b0, float* scores, int M, int d, float eps, int n_act, hipStream_t s) {
  if (n_act < 0 || n_act == 1 || n_act > 64) return hipErrorInvalidValue;
  return bf ? ln_dispatch<f16, bf16, true>(x, nullptr, nullptr, g, b, w, b0, scores, M, d, eps, n_act, s)
            : ln_dispatch<float, float, true>(x, nullptr, nullptr, g, b, w, b0, scores, M, d, eps, n_act, s);
}

// ---------------------------------------------------------------- cache scatter
// One block per (page tile, layer, head): positions t0 .. t1-1 of one page of
// one request, source rows row .. row + t1 - t0 - 1. K rows are copied 16 bytes
// per lane. The page keeps V transposed ([dh][kPage], columns in vt_col order),
// so the V^T tile is assembled in LDS (starting from the page's current
// contents when the tile covers only part of the page) and written back as
// whole 16-byte pieces of its rows.
template <typename T>
__global__ __launch_bounds__(256) void scatter_pages(const T* __restrict__ src, int lds, int slot0,
                                                     T* __restrict__ pool, const int32_t* __restrict__ page_table,
                                                     int max_pages, PageGeom g, const ScatterTile* __restrict__ tiles) {
  constexpr int VEC = 16 / sizeof(T);  // elements per 16 bytes
  constexpr int LDP = kPage + 2;       // padded V^T row in LDS
  __shared__ T sv[128 * LDP];
  const ScatterTile tl = tiles[blockIdx.x];
  const int layer = blockIdx.y / g.H, h = blockIdx.y % g.H;
  const int d = g.H * g.dh, dh = g.dh, cpr = dh / VEC, n = tl.t1 - tl.t0;
  T* base = pool + (size_t)page_table[(size_t)tl.slot * max_pages + tl.page] * g.page_elems;
  T* kdst = base + g.k_off(slot0 + layer, h);
  T* vdst = base + g.v_off(slot0 + layer, h);
  const T* ksrc = src + (size_t)tl.row * lds + (size_t)layer * 2 * d + h * dh;
  const T* vsrc = ksrc + d;
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  for (int c = threadIdx.x; c < n * cpr; c += 256) {
    const int t = c / cpr, ch = c % cpr;
    *reinterpret_cast<u32x4*>(kdst + (size_t)(tl.t0 + t) * dh + ch * VEC) =
        *reinterpret_cast<const u32x4*>(ksrc + (size_t)t * lds + ch * VEC);
  }
  constexpr int RC = kPage / VEC;  // 16-byte pieces per V^T row
  // A page tile that ends before the page does is its request's last: the
  // columns of positions t1 .. 63 are set to zero, so that a kernel reading
  // the whole page multiplies the masked keys' zero probabilities by zeros
  // rather than by whatever the pool held there.
  if (n < kPage)
    for (int c = threadIdx.x; c < dh * RC; c += 256) {
      const int r = c / RC, q = c % RC;
      u32x4 raw = *reinterpret_cast<const u32x4*>(vdst + (size_t)r * kPage + q * VEC);
      T* v = reinterpret_cast<T*>(&raw);
#pragma unroll
      for (int e = 0; e < VEC; ++e)
        if (vt_col(q * VEC + e) >= tl.t1) v[e] = (T)0.f;
      *reinterpret_cast<u32x4*>(&sv[r * LDP + q * VEC]) = raw;
    }
  __syncthreads();
  for (int c = threadIdx.x; c < n * cpr; c += 256) {
    const int t = c / cpr, ch = c % cpr;
    const u32x4 raw = *reinterpret_cast<const u32x4*>(vsrc + (size_t)t * lds + ch * VEC);
    const T* v = reinterpret_cast<const T*>(&raw);
    const int col = vt_col(tl.t0 + t);
#pragma unroll
    for (int e = 0; e < VEC; ++e) sv[(ch * VEC + e) * LDP + col] = v[e];
  }
  __syncthreads();
  for (int c = threadIdx.x; c < dh * RC; c += 256) {
    const int r = c / RC, q = c % RC;
    *reinterpret_cast<u32x4*>(vdst + (size_t)r * kPage + q * VEC) = *reinterpret_cast<const u32x4*>(&sv[r * LDP + q * VEC]);
  }
}

hipError_t launch_scatter_kv(bool bf, const void* src, int lds, int n_layers, int slot0, void* pool,
                             const int32_t* page_table, int max_pages, PageGeom g, const ScatterTile* tiles,
                             int n_tiles, hipStream_t s) {
  if (n_tiles <= 0 || n_layers <= 0) return hipSuccess;
  if (g.dh > 128 || g.dh % 8 != 0 || lds % 8 != 0) return hipErrorInvalidValue;
  const dim3 grid((unsigned)n_tiles, (unsigned)(n_layers * g.H));
  if (bf)
    scatter_pages<bf16><<<grid, 256, 0, s>>>((const bf16*)src, lds, slot0, (bf16*)pool, page_table, max_pages, g,
                                             tiles);
  else
    scatter_pages<float><<<grid, 256, 0, s>>>((const float*)src, lds, slot0, (float*)pool, page_table, max_pages, g,
                                              tiles);
  return hipGetLastError();
}

// ---------------------------------------------------------------- cache export
template <typename T>
__global__ __launch_bounds__(256) void export_kv(const T* __restrict__ pool, const int32_t* __restrict__ page_row,
                                                 PageGeom g, int layer_slot, int is_v, int64_t len,
                                                 T* __restrict__ out) {
  const int d = g.H * g.dh;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= len * d) return;
  const int64_t pos = idx / d;
  const int c = (int)(idx % d), h = c / g.dh, f = c % g.dh;
  const T* base = pool + (size_t)page_row[pos / kPage] * g.page_elems;
  const int t = (int)(pos % kPage);
  out[idx] = is_v ? base[g.v_off(layer_slot, h) + (size_t)f * kPage + vt_col(t)] : base[g.k_off(layer_slot, h) + (size_t)t * g.dh + f];
}

hipError_t launch_export_kv(bool bf, const void* pool, const int32_t* page_row, PageGeom g, int layer_slot, int is_v,
                            int64_t len, void* out, hipStream_t s) {
  const int64_t n = len * g.H * g.dh;
  if (n <= 0) return hipSuccess;
  const unsigned blocks = (unsigned)((n + 255) / 256);
  if (bf) export_kv<bf16><<<blocks, 256, 0, s>>>((const bf16*)pool, page_row, g, layer_slot, is_v, len, (bf16*)out);
  else export_kv<float><<<blocks, 256, 0, s>>>((const float*)pool, page_row, g, layer_slot, is_v, len, (float*)out);
  return hipGetLastError();
}

// ---------------------------------------------------------------- weight repack
template <typename T>
__global__ __launch_bounds__(256) void transpose_tiles(const T* __restrict__ src, T* __restrict__ dst, int K, int N,
                                                       int dst_ld) {
  __shared__ T tile[32][33];
  const int n0 = blockIdx.x * 32, k0 = blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 32 x 8
  for (int r = ty; r < 32; r += 8) {
    const int k = k0 + r, n = n0 + tx;
    if (k < K && n < N) tile[r][tx] = src[(size_t)k * N + n];
  }
  __syncthreads();
  for (int r = ty; r < 32; r += 8) {
    const int n = n0 + r, k = k0 + tx;
    if (k < K && n < N) dst[(size_t)n * dst_ld + k] = tile[tx][r];
  }
}

hipError_t launch_transpose(bool bf, const void* src, void* dst, int K, int N, int dst_ld, hipStream_t s) {
  dim3 grid((N + 31) / 32, (K + 31) / 32);
  if (bf) transpose_tiles<bf16><<<grid, 256, 0, s>>>((const bf16*)src, (bf16*)dst, K, N, dst_ld);
  else transpose_tiles<float><<<grid, 256, 0, s>>>((const float*)src, (float*)dst, K, N, dst_ld);
  return hipGetLastError();
}

// dst fp32 [N][K] = src [K][N] (one-time repack of small matrices)
template <typename T>
__global__ __launch_bounds__(256) void transpose_to_f32_kernel(const T* __restrict__ src, float* __restrict__ dst,
                                                               int K, int N) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (int64_t)K * N) return;
  const int n = (int)(i / K), k = (int)(i % K);
  dst[i] = (float)src[(size_t)k * N + n];
}

hipError_t launch_transpose_to_f32(bool bf, const void* src, float* dst, int K, int N, hipStream_t s) {
  const int64_t n = (int64_t)K * N;
  if (n <= 0) return hipSuccess;
  const unsigned blocks = (unsigned)((n + 255) / 256);
  if (bf) transpose_to_f32_kernel<bf16><<<blocks, 256, 0, s>>>((const bf16*)src, dst, K, N);
  else transpose_to_f32_kernel<float><<<blocks, 256, 0, s>>>((const float*)src, dst, K, N);
  return hipGetLastError();
}

template <typename T>
__global__ __launch_bounds__(256) void to_f32_kernel(const T* __restrict__ src, float* __restrict__ dst, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) dst[i] = (float)src[i];
}

hipError_t launch_to_f32(bool bf, const void* src, float* dst, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const unsigned blocks = (unsigned)((n + 255) / 256);
  if (bf) to_f32_kernel<bf16><<<blocks, 256, 0, s>>>((const bf16*)src, dst, n);
  else to_f32_kernel<float><<<blocks, 256, 0, s>>>((const float*)src, dst, n);
  return hipGetLastError();
}

// The LayerNorm fold of a consumer GEMM (EPI_LN*): for output column n of the
// repacked weight Bt [N][K] (bf16), W'[n][k] = g[k] Bt[n][k] in fp16,
// cs[n] = sum_k W'[n][k] (of the rounded values, as the GEMM multiplies them)
// and b'[n] = bias[n] + sum_k lnb[k] Bt[n][k]. One block per column; the sums
// run in a fixed order. *overflow is set when a scaled weight leaves the fp16
// range (the caller then keeps the unfolded LayerNorm).
__global__ __launch_bounds__(256) void fold_ln_weight(const bf16* __restrict__ Bt, int K, const float* __restrict__ g,
                                                      const float* __restrict__ lnb, const float* __restrict__ bias,
                                                      f16* __restrict__ Wf, float* __restrict__ cs,
                                                      float* __restrict__ bf, int* __restrict__ overflow) {
  __shared__ float part[2][4];
  const int n = blockIdx.x, tid = threadIdx.x;
  float c = 0.f, bb = 0.f;
  bool bad = false;
  for (int k = tid; k < K; k += 256) {
    const float w = (float)Bt[(size_t)n * K + k];
    const float gw = g[k] * w;
    bad |= !(fabsf(gw) <= 65504.f);
    const f16 wf = (f16)gw;
    Wf[(size_t)n * K + k] = wf;
    c += (float)wf;
    bb = fmaf(lnb[k], w, bb);
  }
  if (bad) *overflow = 1;
  c = wave_sum(c);
  bb = wave_sum(bb);
  if ((tid & 63) == 0) {
    part[0][tid >> 6] = c;
    part[1][tid >> 6] = bb;
  }
  __syncthreads();
  if (tid == 0) {
    cs[n] = (part[0][0] + part[0][1]) + (part[0][2] + part[0][3]);
    bf[n] = bias[n] + ((part[1][0] + part[1][1]) + (part[1][2] + part[1][3]));
  }
}

__global__ void zero_int(int* p) { *p = 0; }
hipError_t launch_zero_int(int* p, hipStream_t s) {
  zero_int<<<1, 1, 0, s>>>(p);
  return hipGetLastError();
}
hipError_t read_int(const int* dev, int* host, hipStream_t s) {
  hipError_t e = hipMemcpyAsync(host, dev, sizeof(int), hipMemcpyDeviceToHost, s);
  return e == hipSuccess ? hipStreamSynchronize(s) : e;
}

hipError_t launch_fold_ln_weight(const void* Bt, int N, int K, const float* g, const float* lnb, const float* bias,
                                 void* Wf, float* cs, float* bf, int* overflow, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  fold_ln_weight<<<N, 256, 0, s>>>((const bf16*)Bt, K, g, lnb, bias, (f16*)Wf, cs, bf, overflow);
  return hipGetLastError();
}

}  // namespace tx
