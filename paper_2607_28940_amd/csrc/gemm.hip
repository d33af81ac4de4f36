// Projection and FFN GEMMs of the TransX path: C = epi(A * Bt^T + bias [+ R]).
//
// A is the packed activation matrix [M][K] (token rows), Bt the repacked weight
// [N][K] (the layer's W [K][N] transposed so that both operands are contiguous
// along K). Epilogues: +bias, +bias then exact-erf GELU (FFN), +bias + residual
// (post-LN sublayers add the block input before LayerNorm, Sec. 4.1.2).
//
// bf16 path: v_mfma_f32_32x32x16_bf16 with fp32 accumulation. The weight tile
// is the MFMA "A" operand and the activation tile the "B" operand, so each
// lane's accumulator holds 4 consecutive output columns of one row. Large
// products run on a persistent kernel (one block per CU walking 256x256 tiles,
// see gemm_bf16_p4); the others on one block per tile with operands staged
// global -> registers -> LDS (rows padded by 16 bytes, no bank conflicts),
// double-buffered, prefetched one K step ahead. Tiles are numbered so that each
// of the 8 XCDs (the hardware deals workgroup b to XCD b % 8) works through a
// contiguous range of them, walked in groups of row blocks so that operand
// blocks are reused from that XCD's L2.
#include <atomic>

#include "tx_internal.h"

#include <algorithm>
#include <type_traits>

namespace tx {

// GELU(x) = x Phi(x) = max(x, 0) - u Phi(-u) with u = |x|, for either sign
// of x. Phi(-u) = erfc(u / sqrt 2) / 2, with erfc(z) = t exp(-z^2 + P(t)),
// t = 1 / (1 + z / 2) (the form of Press et al., Numerical Recipes erfcc) and
// P a degree-7 least-squares fit on Chebyshev nodes (gelu_fit.py; fractional
// error below 7.4e-7 for every argument, so the negative tail keeps its
// relative accuracy). Evaluated as Phi(-u) = t 2^(P'(t) - (c u)^2) with
// P' = log2(e) P - 1 and c^2 = log2(e) / 2: one reciprocal, one exp2 and 10
// FMA-type operations.
__device__ __forceinline__ float gelu_erf(float x) {
  const float u = fabsf(x);
  const float t = __builtin_amdgcn_rcpf(fmaf(u, 0.35355339059327373f, 1.0f));
  float p = -0.2718776930163839f;
  p = fmaf(p, t, 1.0879713150078754f);
  p = fmaf(p, t, -1.449840280957486f);
  p = fmaf(p, t, 0.5090884597583125f);
  p = fmaf(p, t, -0.05895698505211376f);
  p = fmaf(p, t, 0.5686708691445311f);
  p = fmaf(p, t, 1.4406420004433174f);
  p = fmaf(p, t, -2.825698746517148f);
  const float w = u * 0.8493218002880191f;
  const float q = t * __builtin_amdgcn_exp2f(fmaf(-w, w, p));  // Phi(-u)
  return fmaf(-u, q, fmaxf(x, 0.f));
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

// Persistent four-wave kernel: one block per CU walks a run of 256x256 output
// tiles. Four waves (one per SIMD) as 2x2, each wave 128x128 of C from 4x4
// v_mfma_f32_32x32x16_bf16 tiles with the fp32 accumulators in AGPRs, so every
// 1 KB fragment read from LDS feeds four MFMAs. K advances 64 at a time through
// two LDS stages (A and B tiles of 128-byte rows; 16-byte slot s of row r is
// held at slot s ^ ((r / 2) % 8), so row-wise stores and column-wise fragment
// reads are both free of bank conflicts without padding).
//
// Operands travel global -> registers -> LDS in four groups of 64 bytes per
// thread. Group q >= 1 of k step t + 1 is parked during sub-step q - 1 of step t
// and group 0 of step t + 2 during its sub-step 3 (right after the barrier that
// frees the stage), each group being refetched as soon as it is parked: every
// load has one whole k step of MFMA work to land, and the loads are spread
// evenly over the step instead of arriving in one burst. The load stream runs
// across tile boundaries and the epilogue parks results in an LDS area of its
// own, so the pipeline never drains between tiles.
constexpr int PT = 256, PK = 64, kPStage = 2 * PT * PK;

#define TX_LGKM_BARRIER() asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory")

template <int EPI>
__global__ __launch_bounds__(256, 1) void gemm_bf16_p4(const bf16* __restrict__ A, int lda,
                                                       const bf16* __restrict__ Bt,
                                                       const float* __restrict__ bias,
                                                       const bf16* __restrict__ R, int ldr, bf16* __restrict__ C,
                                                       int ldc, int M, int N, int K, int tiles_m, int tiles_n,
                                                       int n_tiles, int per_xcd) {
  __shared__ __attribute__((aligned(16))) bf16 lds[2 * kPStage];
  __shared__ __attribute__((aligned(16))) float park_all[4 * 32 * 64];

  const int nloc = gridDim.x >> 3, local = blockIdx.x >> 3;
  const int t_begin = (blockIdx.x & 7) * per_xcd, t_end = min(n_tiles, t_begin + per_xcd);
  const int my_tiles = t_begin + local < t_end ? (t_end - t_begin - local + nloc - 1) / nloc : 0;
  if (my_tiles == 0) return;
  const int nk = K / PK;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int l32 = lane & 31, hi = lane >> 5;

  auto tile_origin = [&](int i, int& m0, int& n0) {
    const int t = t_begin + local + min(i, my_tiles - 1) * nloc;
    const int group = t / (kGroupM * tiles_n);
    const int first_m = group * kGroupM;
    const int gm_size = min(tiles_m - first_m, kGroupM);
    m0 = (first_m + (t % (kGroupM * tiles_n)) % gm_size) * PT;
    n0 = ((t % (kGroupM * tiles_n)) / gm_size) * PT;
  };

  // staging: chunk u of this thread is row (tid / 8) + 32 u, 16-byte slot
  // tid % 8 of both operand tiles; group q holds chunks 2q and 2q + 1
  const int srow = tid >> 3, sslot = tid & 7;
  const int wofs = srow * PK + ((sslot ^ ((srow >> 1) & 7)) << 3);
  bf16x8 ga[8], gb[8];
  // Operands through raw buffer loads: the lane's byte offset within a tile is
  // fixed (row srow + 32 u, slot sslot), the tile's row base is added as one
  // 32-bit value and k0 travels in the scalar offset. Rows past M fall beyond
  // the A resource's extent and read as zeros; their results are not stored.
  // (extents in bytes: the launcher keeps M lda and N K below 2^31 elements;
  // word 3 of the resource as CDNA wants it for raw loads)
  const __amdgpu_buffer_rsrc_t ra =
      __builtin_amdgcn_make_buffer_rsrc((void*)A, 0, (int)(2u * (uint32_t)M * (uint32_t)lda), 0x00020000);
  const __amdgpu_buffer_rsrc_t rb =
      __builtin_amdgcn_make_buffer_rsrc((void*)Bt, 0, (int)(2u * (uint32_t)N * (uint32_t)K), 0x00020000);
  const uint32_t la = 2u * (uint32_t)(srow * lda + sslot * 8), lb = 2u * (uint32_t)(srow * K + sslot * 8);
  auto gload = [&](auto Q_, int m0, int n0, int k0) {
    constexpr int Q = decltype(Q_)::value;
#pragma unroll
    for (int v = 0; v < 2; ++v) {
      const int u = 2 * Q + v;
      const uint32_t oa = 2u * ((uint32_t)(m0 + 32 * u) * (uint32_t)lda) + la;
      const uint32_t ob = 2u * ((uint32_t)(n0 + 32 * u) * (uint32_t)K) + lb;
      ga[u] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(ra, (int)oa, 2 * k0, 0));
      gb[u] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rb, (int)ob, 2 * k0, 0));
    }
  };
  auto lstore = [&](auto Q_, int stage) {
    constexpr int Q = decltype(Q_)::value;
    bf16* sa = lds + stage * kPStage;
#pragma unroll
    for (int v = 0; v < 2; ++v) {
      const int u = 2 * Q + v;
      *reinterpret_cast<bf16x8*>(sa + wofs + u * 32 * PK) = ga[u];
      *reinterpret_cast<bf16x8*>(sa + PT * PK + wofs + u * 32 * PK) = gb[u];
    }
  };

  // fragment reads: A rows wm*128 + 32 j + l32, B rows wn*128 + 32 i + l32;
  // k sub-step ks covers slots 2 ks + hi
  int rofs[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) rofs[ks] = l32 * PK + (((2 * ks + hi) ^ ((l32 >> 1) & 7)) << 3);
  const int a_base = wm * 128 * PK, b_base = PT * PK + wn * 128 * PK;
  auto fread = [&](bf16x8(&fa)[4], bf16x8(&fb)[4], int stage, int ks) {
    const bf16* s = lds + stage * kPStage;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      fa[q] = *reinterpret_cast<const bf16x8*>(s + a_base + q * 32 * PK + rofs[ks]);
      fb[q] = *reinterpret_cast<const bf16x8*>(s + b_base + q * 32 * PK + rofs[ks]);
    }
  };

  floatx16 acc[4][4];
  bf16x8 fa0[4], fb0[4], fa1[4], fb1[4];
  auto mfma16 = [&](auto Z_, const bf16x8(&fa)[4], const bf16x8(&fb)[4]) {
    constexpr bool Z = decltype(Z_)::value;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[i], fa[j], Z ? floatx16{} : acc[i][j], 0, 0, 0);
  };
  using F0 = std::false_type;
  using T1 = std::true_type;
  // 16 MFMAs with 8 fragment reads, 4 LDS stores and 4 global loads between them
  auto interleave = [&]() {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;

  // tile-local k step -> (tile origin, column): steps past the tile belong to
  // the next one (the last tile stands in for a next tile that does not exist)
  int m0, n0, nm0, nn0;
  auto target = [&](int kt, int& tm0, int& tn0, int& k0) {
    const bool nxt = kt >= nk;
    tm0 = nxt ? nm0 : m0;
    tn0 = nxt ? nn0 : n0;
    k0 = (nxt ? kt - nk : kt) * PK;
  };

  // One k step on stage S (= kt % 2); see the kernel comment for the order
  auto step = [&](auto S_, auto Z_, int kt) {
    constexpr int S = decltype(S_)::value;
    int am0, an0, ak0, bm0, bn0, bk0;
    target(kt + 2, am0, an0, ak0);
    target(kt + 3, bm0, bn0, bk0);
    fread(fa1, fb1, S, 1);
    lstore(I1{}, S ^ 1);
    gload(I1{}, am0, an0, ak0);
    mfma16(Z_, fa0, fb0);
    interleave();
    fread(fa0, fb0, S, 2);
    lstore(I2{}, S ^ 1);
    gload(I2{}, am0, an0, ak0);
    mfma16(F0{}, fa1, fb1);
    interleave();
    fread(fa1, fb1, S, 3);
    lstore(I3{}, S ^ 1);
    gload(I3{}, am0, an0, ak0);
    mfma16(F0{}, fa0, fb0);
    interleave();
    TX_LGKM_BARRIER();
    fread(fa0, fb0, S ^ 1, 0);
    lstore(I0{}, S);
    gload(I0{}, bm0, bn0, bk0);
    mfma16(F0{}, fa1, fb1);
    interleave();
  };

  // prologue: stage 0 = step 0, group 0 of step 1 in stage 1; registers hold
  // group 0 of step 2 and groups 1..3 of step 1
  tile_origin(0, m0, n0);
  tile_origin(1, nm0, nn0);
  {
    int tm0, tn0, k0;
    gload(I0{}, m0, n0, 0);
    gload(I1{}, m0, n0, 0);
    gload(I2{}, m0, n0, 0);
    gload(I3{}, m0, n0, 0);
    lstore(I0{}, 0);
    lstore(I1{}, 0);
    lstore(I2{}, 0);
    lstore(I3{}, 0);
    target(1, tm0, tn0, k0);
    gload(I0{}, tm0, tn0, k0);
    lstore(I0{}, 1);
    gload(I1{}, tm0, tn0, k0);
    gload(I2{}, tm0, tn0, k0);
    gload(I3{}, tm0, tn0, k0);
    target(2, tm0, tn0, k0);
    gload(I0{}, tm0, tn0, k0);
  }
  TX_LGKM_BARRIER();
  fread(fa0, fb0, 0, 0);

  float* park = park_all + wave * 32 * 64;
  const int er = lane >> 3, ec = lane & 7;  // row (plus 8 u) and 8-float chunk of the read-back

  for (int i = 0; i < my_tiles; ++i) {
    // the tile's first MFMAs take a zero accumulator input
    step(I0{}, T1{}, 0);
    step(I1{}, F0{}, 1);
    for (int kt = 2; kt < nk; kt += 2) {
      step(I0{}, F0{}, kt);
      step(I1{}, F0{}, kt + 1);
    }
    const int cm0 = m0, cn0 = n0;
    m0 = nm0;
    n0 = nn0;
    tile_origin(i + 2, nm0, nn0);

    // epilogue: per round each wave parks 32 rows x 64 columns of fp32 results
    // (16-byte unit q of row r at unit q ^ (r % 16): conflict-free both ways)
    // and reads them back row-contiguously, 8 lanes per 128-byte row segment;
    // bias, GELU or residual applied with one rounding to bf16. Rows past M
    // (computed from zero rows) are not stored.
    floatx4 bv[2][2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      bv[h][0] = *reinterpret_cast<const floatx4*>(bias + cn0 + wn * 128 + 64 * h + ec * 8);
      bv[h][1] = *reinterpret_cast<const floatx4*>(bias + cn0 + wn * 128 + 64 * h + ec * 8 + 4);
    }
    bf16x8 rres[4];
    auto rload = [&](int j, int h) {
      if (EPI == EPI_BIAS_RESID) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int m = min(cm0 + wm * 128 + j * 32 + er + 8 * u, M - 1);
          rres[u] = *reinterpret_cast<const bf16x8*>(R + (size_t)m * ldr + cn0 + wn * 128 + 64 * h + ec * 8);
        }
      }
    };
    rload(0, 0);
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
#pragma unroll
        for (int ii = 0; ii < 2; ++ii)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const floatx4 v4 = {acc[2 * h + ii][j][4 * g], acc[2 * h + ii][j][4 * g + 1], acc[2 * h + ii][j][4 * g + 2],
                                acc[2 * h + ii][j][4 * g + 3]};
            const int q = ii * 8 + 2 * g + hi;
            *reinterpret_cast<floatx4*>(park + l32 * 64 + ((q ^ (l32 & 15)) << 2)) = v4;
          }
        bf16x8 rcur[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) rcur[u] = rres[u];
        if (j * 2 + h + 1 < 8) rload((j * 2 + h + 1) >> 1, (j * 2 + h + 1) & 1);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int r = er + 8 * u;
          const floatx4 x0 = *reinterpret_cast<const floatx4*>(park + r * 64 + (((2 * ec) ^ (r & 15)) << 2));
          const floatx4 x1 = *reinterpret_cast<const floatx4*>(park + r * 64 + (((2 * ec + 1) ^ (r & 15)) << 2));
          const int m = cm0 + wm * 128 + j * 32 + r;
          bf16x8 o;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float r0 = EPI == EPI_BIAS_RESID ? (float)rcur[u][e] : 0.f;
            const float r1 = EPI == EPI_BIAS_RESID ? (float)rcur[u][e + 4] : 0.f;
            o[e] = (bf16)epilogue<EPI>(x0[e], bv[h][0][e], r0);
            o[e + 4] = (bf16)epilogue<EPI>(x1[e], bv[h][1][e], r1);
          }
          if (m < M) *reinterpret_cast<bf16x8*>(C + (size_t)m * ldc + cn0 + wn * 128 + 64 * h + ec * 8) = o;
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
  // Persistent kernel: K a multiple of 128 and at least 256 (its load stream
  // runs three k steps ahead), element offsets within int32.
  if (N % PT == 0 && K % (2 * PK) == 0 && K >= 4 * PK && M >= 2048 && (long long)M * lda < (1ll << 31) &&
      (long long)N * K < (1ll << 31)) {
    // the current device's CU count, looked up once per device
    static std::atomic<int> cu_of_device[64];
    int dev = 0, n_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = -1;
    if (dev >= 0) n_cu = cu_of_device[dev].load(std::memory_order_relaxed);
    if (n_cu <= 0) {
      if (dev < 0 || hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
          n_cu < 8)
        n_cu = 256;
      if (dev >= 0) cu_of_device[dev].store(n_cu, std::memory_order_relaxed);
    }
    const int tiles_n = N / PT, tiles_m = (M + PT - 1) / PT, n_tiles = tiles_n * tiles_m;
    const int per_xcd = (n_tiles + 7) / 8;
    const int grid = 8 * std::max(1, std::min(n_cu / 8, per_xcd));
    const bf16* a = (const bf16*)A;
    const bf16* b = (const bf16*)Bt;
    const bf16* r = (const bf16*)R;
    bf16* c = (bf16*)C;
#define TX_GP4(E)                                                                                             \
  gemm_bf16_p4<E><<<grid, 256, 0, s>>>(a, lda, b, bias, r, ldr, c, ldc, M, N, K, tiles_m, tiles_n, n_tiles, \
                                       per_xcd)
    switch (epi) {
      case EPI_BIAS: TX_GP4(EPI_BIAS); break;
      case EPI_BIAS_GELU: TX_GP4(EPI_BIAS_GELU); break;
      case EPI_BIAS_RESID: TX_GP4(EPI_BIAS_RESID); break;
    }
#undef TX_GP4
    return hipGetLastError();
  }
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
