// Projection and FFN GEMMs of the TransX path: C = epi(A * Bt^T + bias [+ R]).
//
// A is the packed activation matrix [M][K] (token rows), Bt the repacked weight
// [N][K] (the layer's W [K][N] transposed so that both operands are contiguous
// along K). Epilogues: +bias, +bias then exact-erf GELU (FFN), +bias + residual
// (post-LN sublayers add the block input before LayerNorm, Sec. 4.1.2).
//
// bf16 path: v_mfma_f32_32x32x16_bf16 with fp32 accumulation. The weight tile
// is the MFMA "A" operand and the activation tile the "B" operand, so each
// lane's accumulator holds 4 consecutive output columns of one row. Operand
// tiles are staged global -> registers -> LDS (rows padded by 16 bytes, no bank
// conflicts), double-buffered, prefetched one K step ahead. Blocks are
// renumbered so that each of the 8 XCDs (the hardware deals workgroup b to XCD
// b % 8) works through a contiguous range of tiles, walked in groups of row
// blocks so that operand blocks are reused from that XCD's L2.
#include "tx_internal.h"

namespace tx {

// GELU(x) = x * Phi(x) = 0.5 x erfc(-x / sqrt 2), with erfc from the Chebyshev
// fit of Press et al. (Numerical Recipes, erfcc; fractional error below 1.2e-7
// for every argument, so the negative tail keeps its relative accuracy):
//   erfc(z) = t exp(-z^2 + P(t)),  t = 1 / (1 + z/2),  z >= 0.
// One reciprocal, one exp2 and 9 FMAs instead of the library erff.
__device__ __forceinline__ float gelu_erf(float x) {
  const float z = fabsf(x) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(1.0f + 0.5f * z);
  float p = 0.17087277f;
  p = fmaf(p, t, -0.82215223f);
  p = fmaf(p, t, 1.48851587f);
  p = fmaf(p, t, -1.13520398f);
  p = fmaf(p, t, 0.27886807f);
  p = fmaf(p, t, -0.18628806f);
  p = fmaf(p, t, 0.09678418f);
  p = fmaf(p, t, 0.37409196f);
  p = fmaf(p, t, 1.00002368f);
  p = fmaf(p, t, -1.26551223f);
  const float e = t * __builtin_amdgcn_exp2f((p - z * z) * 1.4426950408889634f);  // erfc(|x| / sqrt 2)
  const float h = 0.5f * x * e;
  return x >= 0.f ? x - h : h;
}

template <int EPI>
__device__ __forceinline__ float epilogue(float acc, float bias, float resid) {
  float v = acc + bias;
  if (EPI == EPI_BIAS_GELU) v = gelu_erf(v);
  if (EPI == EPI_BIAS_RESID) v += resid;
  return v;
}

constexpr int GM = 128, GN = 128, GK = 64, GLD = GK + 8;

template <int EPI>
__global__ __launch_bounds__(256, 2) void gemm_bf16_mfma(const bf16* __restrict__ A, int lda,
                                                          const bf16* __restrict__ Bt, const float* __restrict__ bias,
                                                          const bf16* __restrict__ R, int ldr, bf16* __restrict__ C,
                                                          int ldc, int M, int N, int K, int tiles_n, int n_tiles) {
  __shared__ __attribute__((aligned(16))) bf16 sA[2][GM * GLD];
  __shared__ __attribute__((aligned(16))) bf16 sB[2][GN * GLD];

  const int per_xcd = (n_tiles + 7) >> 3;
  const int t = (int)(blockIdx.x & 7) * per_xcd + (int)(blockIdx.x >> 3);
  if (t >= n_tiles) return;
  const int m0 = (t / tiles_n) * GM, n0 = (t % tiles_n) * GN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int l32 = lane & 31, hi = lane >> 5;

  // global -> register staging: 128 rows x 8 chunks of 16 B per operand, 4 chunks per thread
  bf16x8 ra[4], rb[4];
  auto gload = [&](int k0) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = tid + 256 * u, r = c >> 3, col = (c & 7) * 8;
      const int gm = min(m0 + r, M - 1);
      ra[u] = *reinterpret_cast<const bf16x8*>(A + (size_t)gm * lda + k0 + col);
      rb[u] = *reinterpret_cast<const bf16x8*>(Bt + (size_t)(n0 + r) * K + k0 + col);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = tid + 256 * u, r = c >> 3, col = (c & 7) * 8;
      *reinterpret_cast<bf16x8*>(&sA[buf][r * GLD + col]) = ra[u];
      *reinterpret_cast<bf16x8*>(&sB[buf][r * GLD + col]) = rb[u];
    }
  };

  floatx16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const int nk = K / GK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * GK);
#pragma unroll
    for (int ks = 0; ks < GK / 16; ++ks) {
      bf16x8 fw[2], fx[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        fw[i] = *reinterpret_cast<const bf16x8*>(&sB[cur][(wn * 64 + i * 32 + l32) * GLD + ks * 16 + hi * 8]);
        fx[i] = *reinterpret_cast<const bf16x8*>(&sA[cur][(wm * 64 + i * 32 + l32) * GLD + ks * 16 + hi * 8]);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[i], fx[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) lstore(cur ^ 1);
    __syncthreads();
  }

  // accumulator (i, j), element v: column n = n0 + wn*64 + i*32 + 8*(v/4) + 4*hi + v%4,
  // row m = m0 + wm*64 + j*32 + l32
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int m = m0 + wm * 64 + j * 32 + l32;
    if (m >= M) continue;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = n0 + wn * 64 + i * 32 + 8 * g + 4 * hi;
        const floatx4 b4 = *reinterpret_cast<const floatx4*>(bias + n);
        float r4[4] = {0.f, 0.f, 0.f, 0.f};
        if (EPI == EPI_BIAS_RESID) {
          const bf16x4 rv = *reinterpret_cast<const bf16x4*>(R + (size_t)m * ldr + n);
#pragma unroll
          for (int q = 0; q < 4; ++q) r4[q] = (float)rv[q];
        }
        bf16x4 o;
#pragma unroll
        for (int q = 0; q < 4; ++q) o[q] = (bf16)epilogue<EPI>(acc[i][j][4 * g + q], b4[q], r4[q]);
        *reinterpret_cast<bf16x4*>(C + (size_t)m * ldc + n) = o;
      }
    }
  }
}


// Large-tile kernel: 256x256 block tile, K step 64, 8 waves (2 per SIMD) as
// 2x4, each wave 128 rows x 64 columns of C (2x4 MFMA tiles). Fragments of the
// next 16-wide k step are read from LDS while the MFMAs of the current one run
// (the scheduling barriers keep the compiler from sinking those reads next to
// their use). The epilogue goes through LDS: each wave parks 32 rows x 64
// columns of fp32 results in its own slice of the (then idle) tile buffers and
// reads them back row-contiguously, so every global store writes 16 bytes per
// lane and 8 lanes fill one 128-byte row segment; bias, GELU and residual are
// applied in that phase, with a single rounding to bf16.
constexpr int BM = 256, BN = 256, BK = 64, BLD = BK + 8, kGroupM = 8;

template <int EPI>
__global__ __launch_bounds__(512, 1) void gemm_bf16_mfma_256(const bf16* __restrict__ A, int lda,
                                                             const bf16* __restrict__ Bt,
                                                             const float* __restrict__ bias,
                                                             const bf16* __restrict__ R, int ldr,
                                                             bf16* __restrict__ C, int ldc, int M, int N, int K,
                                                             int tiles_m, int tiles_n, int n_tiles) {
  __shared__ __attribute__((aligned(16))) bf16 sA[2][BM * BLD];
  __shared__ __attribute__((aligned(16))) bf16 sB[2][BN * BLD];

  const int per_xcd = (n_tiles + 7) >> 3;
  const int t = (int)(blockIdx.x & 7) * per_xcd + (int)(blockIdx.x >> 3);
  if (t >= n_tiles) return;
  // grouped order: kGroupM row blocks share each column block in turn
  const int group = t / (kGroupM * tiles_n);
  const int first_m = group * kGroupM;
  const int gm_size = min(tiles_m - first_m, kGroupM);
  const int tm = first_m + (t % (kGroupM * tiles_n)) % gm_size;
  const int tn = (t % (kGroupM * tiles_n)) / gm_size;
  const int m0 = tm * BM, n0 = tn * BN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  const int l32 = lane & 31, hi = lane >> 5;

  bf16x8 ra[4], rb[4];
  auto gload = [&](int k0) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = tid + 512 * u, r = c >> 3, col = (c & 7) * 8;
      const int gm = min(m0 + r, M - 1);
      ra[u] = *reinterpret_cast<const bf16x8*>(A + (size_t)gm * lda + k0 + col);
      rb[u] = *reinterpret_cast<const bf16x8*>(Bt + (size_t)(n0 + r) * K + k0 + col);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = tid + 512 * u, r = c >> 3, col = (c & 7) * 8;
      *reinterpret_cast<bf16x8*>(&sA[buf][r * BLD + col]) = ra[u];
      *reinterpret_cast<bf16x8*>(&sB[buf][r * BLD + col]) = rb[u];
    }
  };

  floatx16 acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const int nk = K / BK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * BK);
    bf16x8 fw[2][2], fx[2][4];
#pragma unroll
    for (int i = 0; i < 2; ++i)
      fw[0][i] = *reinterpret_cast<const bf16x8*>(&sB[cur][(wn * 64 + i * 32 + l32) * BLD + hi * 8]);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      fx[0][j] = *reinterpret_cast<const bf16x8*>(&sA[cur][(wm * 128 + j * 32 + l32) * BLD + hi * 8]);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int f = ks & 1;
      if (ks + 1 < BK / 16) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
          fw[f ^ 1][i] =
              *reinterpret_cast<const bf16x8*>(&sB[cur][(wn * 64 + i * 32 + l32) * BLD + (ks + 1) * 16 + hi * 8]);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          fx[f ^ 1][j] =
              *reinterpret_cast<const bf16x8*>(&sA[cur][(wm * 128 + j * 32 + l32) * BLD + (ks + 1) * 16 + hi * 8]);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[f][i], fx[f][j], acc[i][j], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (kt + 1 < nk) lstore(cur ^ 1);
    __syncthreads();
  }

  // accumulator (i, j), element v: column wn*64 + i*32 + 8*(v/4) + 4*hi + v%4,
  // row wm*128 + j*32 + l32 (within the block tile)
  constexpr int ELD = 64 + 4;  // fp32 row stride of a wave's staging slice
  float* stage = reinterpret_cast<float*>(&sA[0][0]) + wave * 32 * ELD;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const floatx4 v4 = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]};
        *reinterpret_cast<floatx4*>(stage + l32 * ELD + i * 32 + 8 * g + 4 * hi) = v4;
      }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int q = lane + 64 * u, r = q >> 3, cc = (q & 7) * 8;
      const int m = m0 + wm * 128 + j * 32 + r, n = n0 + wn * 64 + cc;
      const floatx4 x0 = *reinterpret_cast<const floatx4*>(stage + r * ELD + cc);
      const floatx4 x1 = *reinterpret_cast<const floatx4*>(stage + r * ELD + cc + 4);
      if (m < M) {
        const floatx4 b0 = *reinterpret_cast<const floatx4*>(bias + n);
        const floatx4 b1 = *reinterpret_cast<const floatx4*>(bias + n + 4);
        float rr[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        if (EPI == EPI_BIAS_RESID) {
          const bf16x8 rv = *reinterpret_cast<const bf16x8*>(R + (size_t)m * ldr + n);
#pragma unroll
          for (int e = 0; e < 8; ++e) rr[e] = (float)rv[e];
        }
        bf16x8 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          o[e] = (bf16)epilogue<EPI>(x0[e], b0[e], rr[e]);
          o[e + 4] = (bf16)epilogue<EPI>(x1[e], b1[e], rr[e + 4]);
        }
        *reinterpret_cast<bf16x8*>(C + (size_t)m * ldc + n) = o;
      }
    }
  }
}

// Plain tiled GEMM for fp32 models and shapes the MFMA tiling does not cover:
// 64x64 block tile, K step 16, each thread computes 4x4 outputs in fp32.
template <typename T, int EPI>
__global__ __launch_bounds__(256) void gemm_plain(const T* __restrict__ A, int lda, const T* __restrict__ Bt,
                                                  const float* __restrict__ bias, const T* __restrict__ R, int ldr,
                                                  T* __restrict__ C, int ldc, int M, int N, int K) {
  __shared__ float sA[16][64 + 4];
  __shared__ float sB[16][64 + 4];
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = tid + 256 * u, r = e >> 4, c = e & 15;
      const int gm = m0 + r, gn = n0 + r, gk = k0 + c;
      sA[c][r] = (gm < M && gk < K) ? (float)A[(size_t)gm * lda + gk] : 0.f;
      sB[c][r] = (gn < N && gk < K) ? (float)Bt[(size_t)gn * K + gk] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = sA[kk][ty * 4 + i];
        b[i] = sB[kk][tx * 4 + i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (n >= N) continue;
      const float r = (EPI == EPI_BIAS_RESID) ? (float)R[(size_t)m * ldr + n] : 0.f;
      C[(size_t)m * ldc + n] = (T)epilogue<EPI>(acc[i][j], bias[n], r);
    }
  }
}

template <typename T>
static hipError_t plain(const void* A, int lda, const void* Bt, const float* bias, const void* R, int ldr, void* C,
                        int ldc, int M, int N, int K, Epilogue epi, hipStream_t s) {
  dim3 grid((N + 63) / 64, (M + 63) / 64);
  const T* a = (const T*)A;
  const T* b = (const T*)Bt;
  const T* r = (const T*)R;
  T* c = (T*)C;
  switch (epi) {
    case EPI_BIAS: gemm_plain<T, EPI_BIAS><<<grid, 256, 0, s>>>(a, lda, b, bias, r, ldr, c, ldc, M, N, K); break;
    case EPI_BIAS_GELU:
      gemm_plain<T, EPI_BIAS_GELU><<<grid, 256, 0, s>>>(a, lda, b, bias, r, ldr, c, ldc, M, N, K);
      break;
    case EPI_BIAS_RESID:
      gemm_plain<T, EPI_BIAS_RESID><<<grid, 256, 0, s>>>(a, lda, b, bias, r, ldr, c, ldc, M, N, K);
      break;
  }
  return hipGetLastError();
}

hipError_t launch_gemm(bool bf, const void* A, int lda, const void* Bt, const float* bias, const void* R, int ldr,
                       void* C, int ldc, int M, int N, int K, Epilogue epi, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (!bf) return plain<float>(A, lda, Bt, bias, R, ldr, C, ldc, M, N, K, epi, s);
  const bool aligned = (lda % 8 == 0) && (ldc % 8 == 0) && (ldr % 8 == 0) && (((uintptr_t)A & 15) == 0) &&
                       (((uintptr_t)Bt & 15) == 0) && (((uintptr_t)C & 15) == 0) && (((uintptr_t)R & 15) == 0) &&
                       (((uintptr_t)bias & 15) == 0);
  if (N % GN != 0 || K % GK != 0 || !aligned)
    return plain<bf16>(A, lda, Bt, bias, R, ldr, C, ldc, M, N, K, epi, s);
  if (N % BN == 0 && M >= 2048) {
    const int tiles_n = N / BN, tiles_m = (M + BM - 1) / BM, n_tiles = tiles_n * tiles_m;
    const int grid = ((n_tiles + 7) / 8) * 8;
    const bf16* a = (const bf16*)A;
    const bf16* b = (const bf16*)Bt;
    const bf16* r = (const bf16*)R;
    bf16* c = (bf16*)C;
#define TX_G256(E) \
  gemm_bf16_mfma_256<E><<<grid, 512, 0, s>>>(a, lda, b, bias, r, ldr, c, ldc, M, N, K, tiles_m, tiles_n, n_tiles)
    switch (epi) {
      case EPI_BIAS: TX_G256(EPI_BIAS); break;
      case EPI_BIAS_GELU: TX_G256(EPI_BIAS_GELU); break;
      case EPI_BIAS_RESID: TX_G256(EPI_BIAS_RESID); break;
    }
#undef TX_G256
    return hipGetLastError();
  }
  const int tiles_n = N / GN, tiles_m = (M + GM - 1) / GM, n_tiles = tiles_n * tiles_m;
  const int grid = ((n_tiles + 7) / 8) * 8;
  const bf16* a = (const bf16*)A;
  const bf16* b = (const bf16*)Bt;
  const bf16* r = (const bf16*)R;
  bf16* c = (bf16*)C;
  switch (epi) {
    case EPI_BIAS:
      gemm_bf16_mfma<EPI_BIAS><<<grid, 256, 0, s>>>(a, lda, b, bias, r, ldr, c, ldc, M, N, K, tiles_n, n_tiles);
      break;
    case EPI_BIAS_GELU:
      gemm_bf16_mfma<EPI_BIAS_GELU><<<grid, 256, 0, s>>>(a, lda, b, bias, r, ldr, c, ldc, M, N, K, tiles_n, n_tiles);
      break;
    case EPI_BIAS_RESID:
      gemm_bf16_mfma<EPI_BIAS_RESID><<<grid, 256, 0, s>>>(a, lda, b, bias, r, ldr, c, ldc, M, N, K, tiles_n,
                                                          n_tiles);
      break;
  }
  return hipGetLastError();
}

}  // namespace tx
