// Projection and FFN GEMMs of the TransX path: C = epi(A * Bt^T + bias [+ R]).
//
// A is the packed activation matrix [M][K] (token rows), Bt the repacked weight
// [N][K] (the layer's W [K][N] transposed so that both operands are contiguous
// along K). Epilogues: +bias, +bias then exact-erf GELU (FFN), +bias + residual
// (post-LN sublayers add the block input before LayerNorm, Sec. 4.1.2).
//
// bf16 path: 128x128 block tile, K step 64, 4 waves as 2x2, each wave 64x64 of
// C built from 2x2 v_mfma_f32_32x32x16_bf16 tiles with fp32 accumulation. The
// weight tile is the MFMA "A" operand and the activation tile the "B" operand,
// so each lane's accumulator holds 4 consecutive output columns of one row and
// the epilogue stores 8 bytes per lane. Tiles are double-buffered in LDS (rows
// padded by 16 bytes against bank conflicts) and prefetched into registers one
// K step ahead. Blocks are renumbered so that each of the 8 XCDs works through a
// contiguous range of row blocks (the hardware deals workgroup b to XCD b % 8),
// keeping an activation row block in one XCD's L2 for all its column tiles.
#include "tx_internal.h"

namespace tx {

__device__ __forceinline__ float gelu_erf(float x) { return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f)); }

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
  const bool aligned = (lda % 8 == 0) && (ldc % 4 == 0) && (ldr % 4 == 0) && (((uintptr_t)A & 15) == 0) &&
                       (((uintptr_t)Bt & 15) == 0) && (((uintptr_t)C & 7) == 0) && (((uintptr_t)R & 7) == 0) &&
                       (((uintptr_t)bias & 15) == 0);
  if (N % GN != 0 || K % GK != 0 || !aligned)
    return plain<bf16>(A, lda, Bt, bias, R, ldr, C, ldc, M, N, K, epi, s);
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
