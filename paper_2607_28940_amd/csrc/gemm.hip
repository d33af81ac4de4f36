// Projection and FFN GEMMs of the TransX path: C = epi(A * Bt^T + bias [+ R]).
//
// A is the packed activation matrix [M][K] (token rows), Bt the repacked weight
// [N][K] (the layer's W [K][N] transposed so that both operands are contiguous
// along K). Epilogues: +bias, +bias then exact-erf GELU (FFN), +bias + residual
// (post-LN sublayers add the block input before LayerNorm, Sec. 4.1.2). A
// residual that is itself a LayerNorm output is recomputed in fp32 from the
// stored pre-LN sum and its row statistics, so the residual stream never
// passes through the rounded bf16 copy the sublayer used as its operand, and
// the new pre-LN sum is stored in fp16 (see EPI_BIAS_RESLN).
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
// of x. Phi(-u) = 2^Q(min(u, 6)) with Q a degree-7 least-squares fit to
// log2 Phi(-u) on Chebyshev nodes of [0, 6] (gelu_fit.py): fractional error
// below 5.5e-6 for |x| <= 6 (evaluated in fp32), 360 times below the bf16
// output's half unit; beyond, where |GELU(x)| < 1e-9 |x|, the clamp keeps the
// error below that. Seven FMAs, one exp2 and no reciprocal.
__device__ __forceinline__ float gelu_erf(float x) {
  const float u = fminf(fabsf(x), 6.0f);
  float q = -1.889626233332388e-06f;
  q = fmaf(q, u, 6.268140100811885e-05f);
  q = fmaf(q, u, -0.0009388679332881356f);
  q = fmaf(q, u, 0.008539461331933599f);
  q = fmaf(q, u, -0.05402068711617134f);
  q = fmaf(q, u, -0.45840977680772027f);
  q = fmaf(q, u, -1.1512691471649812f);
  q = fmaf(q, u, -0.9999943403320692f);
  return fmaf(-fabsf(x), __builtin_amdgcn_exp2f(q), fmaxf(x, 0.f));
}

template <int EPI>
__device__ __forceinline__ float epilogue(float acc, float bias, float resid) {
#pragma clang fp contract(off)
  float v = acc + bias;
  if (epi_gelu(EPI)) v = gelu_erf(v);
  if (epi_resid(EPI)) v += resid;
  return v;
}

// Residual element e of a 16-byte piece of R: the model-type value itself
// (EPI_BIAS_RESID) or the LayerNorm of the fp16 pre-LN sum with row
// statistics st and the column's gain g (EPI_BIAS_RESLN), whose offset every
// kernel adds to the bias instead: (acc + (bias + b)) + (y * x + y') * g, the
// same operations in the same order in each kernel, so that they agree
// bitwise.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ float ln_resid(float y, LnRow st, float g) {
#pragma clang fp contract(off)
  return fmaf(y, st.x, st.y) * g;
}
template <int EPI>
__device__ __forceinline__ float resid8(const u32x4& raw, int e, LnRow st, float g) {
  if (EPI == EPI_BIAS_RESID) return (float)__builtin_bit_cast(bf16x8, raw)[e];
  if (EPI == EPI_BIAS_RESLN) return ln_resid((float)__builtin_bit_cast(f16x8, raw)[e], st, g);
  return 0.f;
}
template <int EPI>
__device__ __forceinline__ float resid4(const u32x2& raw, int e, LnRow st, float g) {
  if (EPI == EPI_BIAS_RESID) return (float)__builtin_bit_cast(bf16x4, raw)[e];
  if (EPI == EPI_BIAS_RESLN) return ln_resid((float)__builtin_bit_cast(f16x4, raw)[e], st, g);
  return 0.f;
}

constexpr int GM = 128, GN = 128, GK = 64, GLD = GK + 8;

template <int EPI>
__global__ __launch_bounds__(256, 2) void gemm_bf16_mfma(const bf16* __restrict__ A, int lda,
                                                          const bf16* __restrict__ Bt, const float* __restrict__ bias,
                                                          const void* __restrict__ R, int ldr, void* __restrict__ C,
                                                          int ldc, int M, int N, int K, int tiles_n, int n_tiles,
                                                          LnResid ln) {
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
        for (int j = 0; j < 2; ++j) {
          if (epi_lnfold(EPI))  // fp16 operands (see gemm_bf16_p4)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, fw[i]),
                                                               __builtin_bit_cast(f16x8, fx[j]), acc[i][j], 0, 0, 0);
          else
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[i], fx[j], acc[i][j], 0, 0, 0);
        }
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
    LnRow st{0.f, 0.f};
    if (EPI == EPI_BIAS_RESLN || epi_lnfold(EPI)) st = ln.stats[m];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = n0 + wn * 64 + i * 32 + 8 * g + 4 * hi;
        floatx4 b4 = *reinterpret_cast<const floatx4*>(bias + n);
        if (epi_lnfold(EPI)) {
          // the same operations as the persistent kernel's epilogue
          const floatx4 cs4 = *reinterpret_cast<const floatx4*>(ln.g + n);
          bf16x4 o;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            float v = fmaf(acc[i][j][4 * g + q], st.x, fmaf(st.y, cs4[q], b4[q]));
            if (epi_gelu(EPI)) v = gelu_erf(v);
            o[q] = (bf16)v;
          }
          *reinterpret_cast<bf16x4*>((bf16*)C + (size_t)m * ldc + n) = o;
        } else if (epi_resid(EPI)) {
          const u32x2 raw = *reinterpret_cast<const u32x2*>((const bf16*)R + (size_t)m * ldr + n);
          floatx4 g4 = {0.f, 0.f, 0.f, 0.f};
          if (EPI == EPI_BIAS_RESLN) {
            g4 = *reinterpret_cast<const floatx4*>(ln.g + n);
            b4 += *reinterpret_cast<const floatx4*>(ln.b + n);
          }
          f16x4 o;
#pragma unroll
          for (int q = 0; q < 4; ++q)
            o[q] = (f16)epilogue<EPI>(acc[i][j][4 * g + q], b4[q], resid4<EPI>(raw, q, st, g4[q]));
          *reinterpret_cast<f16x4*>((f16*)C + (size_t)m * ldc + n) = o;
        } else {
          bf16x4 o;
#pragma unroll
          for (int q = 0; q < 4; ++q) o[q] = (bf16)epilogue<EPI>(acc[i][j][4 * g + q], b4[q], 0.f);
          *reinterpret_cast<bf16x4*>((bf16*)C + (size_t)m * ldc + n) = o;
        }
      }
    }
  }
}


constexpr int kGroupM = 8;  // row blocks that share each column block in turn (L2 reuse)

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
                                                       const void* __restrict__ R, int ldr, void* __restrict__ C,
                                                       int ldc, int M, int N, int K, int tiles_m, int tiles_n,
                                                       int n_tiles, int per_xcd, LnResid ln) {
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
  // the LayerNorm-folding epilogues take fp16 operands (the stored pre-LN sum
  // and the gain-scaled weight); the fragments are the same 16-byte units
  auto mfma16 = [&](auto Z_, const bf16x8(&fa)[4], const bf16x8(&fb)[4]) {
    constexpr bool Z = decltype(Z_)::value;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (epi_lnfold(EPI))
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, fb[i]),
                                                             __builtin_bit_cast(f16x8, fa[j]),
                                                             Z ? floatx16{} : acc[i][j], 0, 0, 0);
        else
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[i], fa[j], Z ? floatx16{} : acc[i][j], 0, 0, 0);
      }
  };
  using F0 = std::false_type;
  using T1 = std::true_type;
  // 16 MFMAs with 8 fragment reads, 4 LDS stores and 4 global loads between
  // them: the reads (the next sub-step's fragments) between the first eight
  // MFMAs, so that they have the second half to land, then the stores and
  // loads (~1% faster than spreading the reads over all sixteen)
  auto interleave = [&]() {
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
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
  // epilogue resources (extents in bytes, below 2^32: checked by the launcher)
  // and the lane's fixed offsets: row wm * 128 + er (+ 32 j + 8 u), column
  // wn * 128 + 8 ec (+ 64 h) of the tile, and the LayerNorm statistics of the
  // same rows
  constexpr bool kStats = EPI == EPI_BIAS_RESLN || epi_lnfold(EPI);  // row statistics used
  const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
      (void*)R, 0, epi_resid(EPI) ? (int)(2u * (uint32_t)M * (uint32_t)ldr) : 0, 0x00020000);
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)ln.stats, 0, kStats ? (int)(8u * (uint32_t)M) : 0, 0x00020000);
  const __amdgpu_buffer_rsrc_t rc =
      __builtin_amdgcn_make_buffer_rsrc(C, 0, (int)(2u * (uint32_t)M * (uint32_t)ldc), 0x00020000);
  const uint32_t lr = 2u * (uint32_t)((wm * 128 + er) * ldr + wn * 128 + ec * 8);
  const uint32_t lc = 2u * (uint32_t)((wm * 128 + er) * ldc + wn * 128 + ec * 8);
  const uint32_t ls = 8u * (uint32_t)(wm * 128 + er);

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
    // bias, GELU or residual applied with one rounding (bf16, or fp16 for a
    // pre-LN sum). Rows past M (computed from zero rows) are not stored.
    // Rounds (j, h): 32 rows (32 j ..) x 64 columns (64 h ..) of the wave's
    // 128 x 128. The residual pieces of a round are fetched one round ahead,
    // and the LayerNorm statistics of the lane's four rows (shared by both
    // rounds of j) a j ahead, each lane loading its own rows' (a broadcast
    // within the load: no lane permutes). The column vectors (bias, and for a
    // LayerNorm residual its gain and offset, the offset folded into the bias;
    // for a folded LayerNorm the weight's column sums) are read again each
    // round (L1 hits) rather than held through the epilogue. Residual, statistics
    // and outputs go through raw buffer operations with 32-bit offsets: rows
    // past M lie beyond the resources, read as zeros and are not written.
    u32x4 rres[4];
    LnRow stn[4], stc[4];  // statistics of the lane's rows er + 8 u (next j, current j)
    auto rload = [&](int j, int h) {
      if (epi_resid(EPI)) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const uint32_t o = 2u * ((uint32_t)(cm0 + j * 32 + 8 * u) * (uint32_t)ldr + (uint32_t)(cn0 + 64 * h)) + lr;
          rres[u] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rr, (int)o, 0, 0));
        }
      }
      if (kStats && h == 0) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const uint32_t o = 8u * (uint32_t)(cm0 + j * 32 + 8 * u) + ls;
          const u32x2 v = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(rs, (int)o, 0, 0));
          stn[u] = LnRow{__uint_as_float(v[0]), __uint_as_float(v[1])};
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
        u32x4 rcur[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) rcur[u] = rres[u];
        if (h == 0)
#pragma unroll
          for (int u = 0; u < 4; ++u) stc[u] = stn[u];
        if (j * 2 + h + 1 < 8) rload((j * 2 + h + 1) >> 1, (j * 2 + h + 1) & 1);
        asm volatile("" ::: "memory");  // keeps the column vectors from being held across rounds
        const int ncol = cn0 + wn * 128 + 64 * h + ec * 8;
        floatx4 cb[2], lg[2];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          cb[q] = *reinterpret_cast<const floatx4*>(bias + ncol + 4 * q);
          if (EPI == EPI_BIAS_RESLN) cb[q] += *reinterpret_cast<const floatx4*>(ln.b + ncol + 4 * q);
          if (kStats) lg[q] = *reinterpret_cast<const floatx4*>(ln.g + ncol + 4 * q);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int r = er + 8 * u;
          const floatx4 x0 = *reinterpret_cast<const floatx4*>(park + r * 64 + (((2 * ec) ^ (r & 15)) << 2));
          const floatx4 x1 = *reinterpret_cast<const floatx4*>(park + r * 64 + (((2 * ec + 1) ^ (r & 15)) << 2));
          const uint32_t o_off = 2u * ((uint32_t)(cm0 + j * 32 + 8 * u) * (uint32_t)ldc + (uint32_t)(cn0 + 64 * h)) + lc;
          u32x4 ov;
          if (epi_lnfold(EPI)) {
            // LN(A) W + b = (acc * x + y * cs) + b' for the row's statistics (x, y)
            const LnRow st = stc[u];
            bf16x8 o;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              float v0 = fmaf(x0[e], st.x, fmaf(st.y, lg[0][e], cb[0][e]));
              float v1 = fmaf(x1[e], st.x, fmaf(st.y, lg[1][e], cb[1][e]));
              if (epi_gelu(EPI)) {
                v0 = gelu_erf(v0);
                v1 = gelu_erf(v1);
              }
              o[e] = (bf16)v0;
              o[e + 4] = (bf16)v1;
            }
            ov = __builtin_bit_cast(u32x4, o);
          } else if (epi_resid(EPI)) {
            LnRow st{0.f, 0.f};
            if (EPI == EPI_BIAS_RESLN) st = stc[u];
            f16x8 o;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float r0 = resid8<EPI>(rcur[u], e, st, EPI == EPI_BIAS_RESLN ? lg[0][e] : 0.f);
              const float r1 = resid8<EPI>(rcur[u], e + 4, st, EPI == EPI_BIAS_RESLN ? lg[1][e] : 0.f);
              o[e] = (f16)epilogue<EPI>(x0[e], cb[0][e], r0);
              o[e + 4] = (f16)epilogue<EPI>(x1[e], cb[1][e], r1);
            }
            ov = __builtin_bit_cast(u32x4, o);
          } else {
            bf16x8 o;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              o[e] = (bf16)epilogue<EPI>(x0[e], cb[0][e], 0.f);
              o[e + 4] = (bf16)epilogue<EPI>(x1[e], cb[1][e], 0.f);
            }
            ov = __builtin_bit_cast(u32x4, o);
          }
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(__attribute__((ext_vector_type(4))) unsigned, ov),
                                                 rc, (int)o_off, 0, 0);
        }
      }
  }
}

// Plain tiled GEMM for fp32 models and shapes the MFMA tiling does not cover:
// 64x64 block tile, K step 16, each thread computes 4x4 outputs in fp32.
// Sum type (pre-LN sums of the residual epilogues): fp16 beside bf16, fp32
// beside fp32.
template <typename T>
using SumT = typename std::conditional<std::is_same<T, float>::value, float, f16>::type;

template <typename T, int EPI>
__global__ __launch_bounds__(256) void gemm_plain(const T* __restrict__ A, int lda, const T* __restrict__ Bt,
                                                  const float* __restrict__ bias, const void* __restrict__ R, int ldr,
                                                  void* __restrict__ C, int ldc, int M, int N, int K, LnResid ln) {
  typedef SumT<T> S;
  typedef typename std::conditional<EPI == EPI_BIAS_RESLN, S, T>::type RT;  // residual element type
  typedef typename std::conditional<epi_resid(EPI), S, T>::type CT;  // output element type
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
  const RT* Rt = (const RT*)R;
  CT* Ct = (CT*)C;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= M) continue;
    LnRow st{0.f, 0.f};
    if (EPI == EPI_BIAS_RESLN) st = ln.stats[m];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (n >= N) continue;
      float r = 0.f, bn = bias[n];
      if (EPI == EPI_BIAS_RESID) r = (float)Rt[(size_t)m * ldr + n];
      if (EPI == EPI_BIAS_RESLN) {
        r = ln_resid((float)Rt[(size_t)m * ldr + n], st, ln.g[n]);
        bn += ln.b[n];
      }
      Ct[(size_t)m * ldc + n] = (CT)epilogue<EPI>(acc[i][j], bn, r);
    }
  }
}

template <typename T>
static hipError_t plain(const void* A, int lda, const void* Bt, const float* bias, const void* R, int ldr, void* C,
                        int ldc, int M, int N, int K, Epilogue epi, LnResid ln, hipStream_t s) {
  dim3 grid((N + 63) / 64, (M + 63) / 64);
  const T* a = (const T*)A;
  const T* b = (const T*)Bt;
#define TX_PL(E) gemm_plain<T, E><<<grid, 256, 0, s>>>(a, lda, b, bias, R, ldr, C, ldc, M, N, K, ln)
  switch (epi) {
    case EPI_BIAS: TX_PL(EPI_BIAS); break;
    case EPI_BIAS_GELU: TX_PL(EPI_BIAS_GELU); break;
    case EPI_BIAS_RESID: TX_PL(EPI_BIAS_RESID); break;
    case EPI_BIAS_RESLN: TX_PL(EPI_BIAS_RESLN); break;
    default: return hipErrorInvalidValue;  // the LayerNorm-folding epilogues run on the persistent kernel only
  }
#undef TX_PL
  return hipGetLastError();
}

// Shapes the persistent kernel takes without splitting rows: N a multiple of
// the tile, K of two k steps and at least four, M at least 2048 rows (below,
// the launch covers too few of the CUs), element offsets within int32.
static bool persistent_shape(int M, int N, int K, long long ld_max) {
  return N % PT == 0 && K % (2 * PK) == 0 && K >= 4 * PK && M >= 2048 && (long long)M * ld_max < (1ll << 31) &&
         (long long)N * K < (1ll << 31);
}
bool gemm_ln_ok(int N, int K, int lda, int ldc) { return N % GN == 0 && K % GK == 0 && lda % 8 == 0 && ldc % 8 == 0; }

hipError_t launch_gemm(bool bf, const void* A, int lda, const void* Bt, const float* bias, const void* R, int ldr,
                       void* C, int ldc, int M, int N, int K, Epilogue epi, hipStream_t s, LnResid ln) {
  if (M <= 0) return hipSuccess;
  if (epi == EPI_BIAS_RESLN && (!ln.stats || !ln.g || !ln.b)) return hipErrorInvalidValue;
  if (epi_resid(epi) && !R) return hipErrorInvalidValue;
  if (epi_lnfold(epi) && (!bf || !ln.stats || !ln.g || !gemm_ln_ok(N, K, lda, ldc))) return hipErrorInvalidValue;
  if (!bf) return plain<float>(A, lda, Bt, bias, R, ldr, C, ldc, M, N, K, epi, ln, s);
  // The MFMA kernels address A, R and C with 32-bit byte offsets: a product
  // whose operands span 2^31 elements or more runs as several row chunks.
  {
    const long long ld_max = std::max({(long long)lda, (long long)ldc, epi_resid(epi) ? (long long)ldr : 1ll});
    const long long rows_max = std::max(256ll, ((1ll << 31) - 1) / ld_max / 256 * 256);
    if (M > rows_max) {
      for (long long m0 = 0; m0 < M; m0 += rows_max) {
        const int mc = (int)std::min(rows_max, (long long)M - m0);
        LnResid lc = ln;
        if (lc.stats) lc.stats += m0;
        const hipError_t e = launch_gemm(bf, (const bf16*)A + m0 * lda, lda, Bt, bias,
                                         R ? (const void*)((const bf16*)R + m0 * ldr) : nullptr, ldr,
                                         (bf16*)C + m0 * ldc, ldc, mc, N, K, epi, s, lc);
        if (e != hipSuccess) return e;
      }
      return hipSuccess;
    }
  }
  const bool aligned = (lda % 8 == 0) && (ldc % 8 == 0) && (ldr % 8 == 0) && (((uintptr_t)A & 15) == 0) &&
                       (((uintptr_t)Bt & 15) == 0) && (((uintptr_t)C & 15) == 0) && (((uintptr_t)R & 15) == 0) &&
                       (((uintptr_t)bias & 15) == 0) && (((uintptr_t)ln.g & 15) == 0) &&
                       (((uintptr_t)ln.b & 15) == 0);
  if (N % GN != 0 || K % GK != 0 || !aligned)
    return plain<bf16>(A, lda, Bt, bias, R, ldr, C, ldc, M, N, K, epi, ln, s);
  const bf16* a = (const bf16*)A;
  const bf16* b = (const bf16*)Bt;
  // Persistent kernel: K a multiple of 128 and at least 256 (its load stream
  // runs three k steps ahead), element offsets within int32.
  if (persistent_shape(M, N, K, std::max({(long long)lda, (long long)ldc, (long long)ldr}))) {
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
#define TX_GP4(E)                                                                                               \
  gemm_bf16_p4<E><<<grid, 256, 0, s>>>(a, lda, b, bias, R, ldr, C, ldc, M, N, K, tiles_m, tiles_n, n_tiles, \
                                       per_xcd, ln)
    switch (epi) {
      case EPI_BIAS: TX_GP4(EPI_BIAS); break;
      case EPI_BIAS_GELU: TX_GP4(EPI_BIAS_GELU); break;
      case EPI_BIAS_RESID: TX_GP4(EPI_BIAS_RESID); break;
      case EPI_BIAS_RESLN: TX_GP4(EPI_BIAS_RESLN); break;
      case EPI_LN: TX_GP4(EPI_LN); break;
      case EPI_LN_GELU: TX_GP4(EPI_LN_GELU); break;
    }
#undef TX_GP4
    return hipGetLastError();
  }
  const int tiles_n = N / GN, tiles_m = (M + GM - 1) / GM, n_tiles = tiles_n * tiles_m;
  const int grid = ((n_tiles + 7) / 8) * 8;
#define TX_G128(E) \
  gemm_bf16_mfma<E><<<grid, 256, 0, s>>>(a, lda, b, bias, R, ldr, C, ldc, M, N, K, tiles_n, n_tiles, ln)
  switch (epi) {
    case EPI_BIAS: TX_G128(EPI_BIAS); break;
    case EPI_BIAS_GELU: TX_G128(EPI_BIAS_GELU); break;
    case EPI_BIAS_RESID: TX_G128(EPI_BIAS_RESID); break;
    case EPI_BIAS_RESLN: TX_G128(EPI_BIAS_RESLN); break;
    case EPI_LN: TX_G128(EPI_LN); break;
    case EPI_LN_GELU: TX_G128(EPI_LN_GELU); break;
  }
#undef TX_G128
  return hipGetLastError();
}

}  // namespace tx
