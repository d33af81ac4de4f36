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
// encoded rows once, and the attention touches at most 65 keys per query.
// The attention is bound by its Q and O rows in HBM: bf16 models run its two
// small products on matrix cores (lg_cross_attn_mfma), fp32 models in plain
// fp32 arithmetic (lg_cross_attn).
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

// fp32 models. One block per tile of 64 queries of one (request, head): the keys and
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

constexpr int kLgQueries = 64;  // queries per block of the general kernel

// The same windows on matrix cores, for every bf16 model: NS key slots
// (16, 32, ..., 80) hold the window after its start is rounded down to a
// multiple of 4, plus the pooled token (NS = 16 for the paper's 10 + 1).
// Every query of a (request, head) sees the same keys, so per group of 16
// queries and 16 slots the scores are one small product S^T = K Q^T
// (v_mfma_f32_16x16x32_bf16, keys as rows: lane (q, g) ends with slots
// 4 g .. 4 g + 3 of the chunk for query q) and the output is a sum of more,
// O^T = V^T P^T over the chunks (v_mfma_f32_16x16x16_bf16), whose P^T
// operand wants exactly that layout: four slots of one query per lane. The
// softmax runs in the accumulator registers (row maximum and sum over the
// query's four lanes by row swaps), and no value changes lanes between the
// two products.
// Slot j is cache position p0 + j with p0 = k0 rounded down to a multiple of
// 4, and the pooled token takes the slot of position len; four slots are
// four consecutive positions, which a page's V^T slab keeps side by side (its
// column permutation moves bits 2 and 3 of the position only), so V^T is
// staged in 8-byte quads and K in 16-byte row pieces. Slots outside the
// window are masked and staged as zeros (nothing past the request's cached
// positions is read), so stale or poisoned page contents cannot reach the
// result. The slots that hold cached positions (at most 64 + 3 from a
// multiple of 4) span at most two pages.
// A block serves a tile of queries of one request for hb heads (all of them
// at the paper's window: 8 heads of 16 slots fit 74 KB of LDS; fewer for
// longer windows, hb a divisor of H): it stages those heads' windows once,
// and its 8 waves take (group of 16 queries, head) pairs eight consecutive
// ones at a time (with 8 heads, the 8 head pieces of the same 16 rows), the
// next pair's Q fragments requested before the current one is worked on. So
// each query's Q row is read, and its O row written, as whole rows or
// pieces of hb heads within a short span (head by head in blocks of their
// own, the 256-byte pieces of a row went to memory far apart in time, and
// the launch ran at the ~4 TB/s such a sweep gets). The output accumulator
// holds 4 features of one query per lane and 16-feature chunk; two row swaps
// per pair of chunks leave each lane 8 consecutive features (64 contiguous
// bytes of a row per query over the four key groups, as the Q loads read:
// the B operand takes 8 consecutive features per lane), and a rotation by 8
// lanes pairs two such halves, so that each store writes whole 128-byte
// lines of 8 queries.
constexpr int kLgMfmaMaxSlots = 80;
constexpr int kLgMfmaPairs = 144;  // (16-query group, head) pairs per tile
constexpr int kLgMfmaLds = 77824;  // LDS budget of a block's windows (76 KB: two blocks per CU)

// LDS bytes of one head's window: K rows of DH + 8 elements, V^T rows of NS + 4
constexpr int lg_head_bytes(int ns, int dh) { return 2 * (ns * (dh + 8) + dh * (ns + 4)); }
// heads a block's LDS holds: the largest power of two up to 8 within the budget
constexpr int lg_max_heads(int ns, int dh) {
  return 8 * lg_head_bytes(ns, dh) <= kLgMfmaLds   ? 8
         : 4 * lg_head_bytes(ns, dh) <= kLgMfmaLds ? 4
         : 2 * lg_head_bytes(ns, dh) <= kLgMfmaLds ? 2
                                                   : 1;
}

template <int DH, int NS>
__global__ __launch_bounds__(512) void lg_cross_attn_mfma(const bf16* __restrict__ q, int ldq, bf16* __restrict__ out,
                                                          int ldo, const bf16* __restrict__ pool,
                                                          const int32_t* __restrict__ page_table, int max_pages,
                                                          PageGeom g, int layer_slot, const AttnReq* __restrict__ reqs,
                                                          const AttnTile* __restrict__ tiles, int l_local, int hb,
                                                          const bf16* __restrict__ gkv, int gkv_ld, int dec_layer,
                                                          float scale_log2) {
  constexpr int NC = DH / 32;       // k chunks of the score product
  constexpr int NO = DH / 16;       // feature chunks of the output product
  constexpr int NCH = NS / 16;      // slot chunks
  constexpr int KS = DH + 8;        // K row stride (elements): rows 16 bytes apart in the banks
  constexpr int VS = NS + 4;        // V^T row stride (elements)
  constexpr int KH = NS * KS, VH = DH * VS;  // elements per head
  constexpr int HB = lg_max_heads(NS, DH);
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  __shared__ __attribute__((aligned(16))) bf16 sK[HB * KH];
  __shared__ __attribute__((aligned(16))) bf16 sV[HB * VH];
  const AttnTile tile = tiles[blockIdx.x];
  if (tile.q_count <= 0) return;
  const AttnReq rq = reqs[tile.req];
  const int h0 = tile.head * hb;  // the tile's first head
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int qn = lane & 15, kg = lane >> 4;
  const int n_groups = (tile.q_count + 15) / 16;
  // token row of query j of 16-query group gi
  auto row_of = [&](int gi, int j) {
    const int i = tile.q_begin + 16 * gi + j;
    return i < rq.qa_n ? rq.qa_row + i : rq.qb_row + (i - rq.qa_n);
  };
  // Q fragments of (group gi, head h): features 32 c + 8 kg .. of query qn,
  // zeros past the tile
  auto load_q = [&](int gi, int h, bf16x8(&qf)[NC]) {
    const bool ok = gi < n_groups && 16 * gi + qn < tile.q_count;
    const int row = ok ? row_of(gi, qn) : 0;
#pragma unroll
    for (int c = 0; c < NC; ++c)
      qf[c] = ok ? *reinterpret_cast<const bf16x8*>(q + (size_t)row * ldq + h * DH + 32 * c + 8 * kg) : bf16x8{};
  };
  bf16x8 qa[NC], qb[NC];
  load_q(wave / hb, h0 + wave % hb, qa);
  const int len = rq.kv_len;
  const int k0 = max(0, len - l_local), p0 = k0 & ~3;
  const bool gpool = gkv != nullptr;
  auto is_key = [&](int p) { return (p >= k0 && p < len) || (gpool && p == len); };
  // the window's (at most two) pages: the slots' cached positions end at len - 1
  const int32_t* ptab = page_table + (size_t)rq.slot * max_pages;
  const int pg0 = p0 / kPage, pg1 = max(pg0, (len - 1) / kPage);
  const bf16* page0 = pool + (size_t)ptab[pg0] * g.page_elems;
  const bf16* page1 = pool + (size_t)ptab[pg1] * g.page_elems;
  auto page_of = [&](int p) { return p / kPage == pg0 ? page0 : page1; };
  const int d = g.H * DH;
  const bf16* grow = gpool ? gkv + (size_t)rq.slot * gkv_ld + (size_t)(2 * dec_layer) * d : nullptr;
  // the heads' K pieces (slot j, features 8 c ..) and V^T quads (feature f,
  // slots 4 u ..), zeros outside the window
  for (int e = tid; e < hb * NS * DH / 8; e += 512) {
    const int hl = e / (NS * DH / 8), r = e % (NS * DH / 8), h = h0 + hl;
    const int j = r / (DH / 8), c = r % (DH / 8), p = p0 + j;
    bf16x8 v = {};
    if (p >= k0 && p < len)
      v = *reinterpret_cast<const bf16x8*>(page_of(p) + g.k_off(layer_slot, h) + (size_t)(p % kPage) * DH + 8 * c);
    else if (gpool && p == len)
      v = *reinterpret_cast<const bf16x8*>(grow + h * DH + 8 * c);
    *reinterpret_cast<bf16x8*>(sK + hl * KH + j * KS + 8 * c) = v;
  }
  for (int e = tid; e < hb * DH * NS / 4; e += 512) {
    const int hl = e / (DH * NS / 4), r = e % (DH * NS / 4), h = h0 + hl;
    const int f = r / (NS / 4), u = r % (NS / 4), pq = p0 + 4 * u;
    bf16x4 v = {};
    if (pq < len)
      v = *reinterpret_cast<const bf16x4*>(page_of(pq) + g.v_off(layer_slot, h) + (size_t)f * kPage + vt_col(pq % kPage));
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      if (pq + t >= len) v[t] = (bf16)0.f;
      if (gpool && pq + t == len) v[t] = grow[d + h * DH + f];
    }
    *reinterpret_cast<bf16x4*>(sV + hl * VH + f * VS + 4 * u) = v;
  }
  __syncthreads();
  bool key[NCH][4];
#pragma unroll
  for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
    for (int r = 0; r < 4; ++r) key[ch][r] = is_key(p0 + 16 * ch + 4 * kg + r);
  // A operands, read from LDS per (group, head): K (slot 16 ch + qn,
  // features 32 c + 8 kg ..) and V^T (feature 16 c + qn, slots
  // 16 ch + 4 kg ..); the lane offsets pass through an empty asm so the
  // reads are not hoisted
  const int kofs = qn * KS + 8 * kg, vofs = qn * VS + 4 * kg;
  auto work = [&](int gi, int hl, const bf16x8(&qf)[NC]) {
    int ko = kofs + hl * KH, vo = vofs + hl * VH;
    asm volatile("" : "+v"(ko), "+v"(vo));
    floatx4 sc[NCH];
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      sc[ch] = floatx4{};
#pragma unroll
      for (int c = 0; c < NC; ++c)
        sc[ch] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            *reinterpret_cast<const bf16x8*>(sK + ko + 16 * KS * ch + 32 * c), qf[c], sc[ch], 0, 0, 0);
    }
    // sc[ch][r]: slot 16 ch + 4 kg + r of query qn
    float m = -INFINITY;
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        sc[ch][r] = key[ch][r] ? sc[ch][r] * scale_log2 : -INFINITY;
        m = fmaxf(m, sc[ch][r]);
      }
    m = xor32_max(row16_max(m));
    s16x4 pp[NCH];
    float l = 0.f;
#pragma unroll
    for (int ch = 0; ch < NCH; ++ch) {
      bf16x4 pb;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        pb[r] = (bf16)__builtin_amdgcn_exp2f(sc[ch][r] - m);  // 0 where masked
        l += (float)pb[r];
      }
      pp[ch] = __builtin_bit_cast(s16x4, pb);
    }
    l = xor32_sum(row16_sum(l));
    const float inv = 1.f / l;
    // features 16 c .. 16 c + 31 of query qn: 8 consecutive ones per key group
    auto out_chunks = [&](int c) {
      // o0[r], o1[r]: features 16 c + 4 kg + r and 16 (c + 1) + 4 kg + r
      floatx4 o0 = {}, o1 = {};
#pragma unroll
      for (int ch = 0; ch < NCH; ++ch) {
        o0 = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(
            *reinterpret_cast<const s16x4*>(sV + vo + 16 * VS * c + 16 * ch), pp[ch], o0, 0, 0, 0);
        o1 = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(
            *reinterpret_cast<const s16x4*>(sV + vo + 16 * VS * (c + 1) + 16 * ch), pp[ch], o1, 0, 0, 0);
      }
      bf16x4 b0, b1;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        b0[r] = (bf16)(o0[r] * inv);
        b1[r] = (bf16)(o1[r] * inv);
      }
      u32x2_t x = __builtin_bit_cast(u32x2_t, b0), y = __builtin_bit_cast(u32x2_t, b1);
      // lanes of key groups 2, 3 trade x for the y of groups 0, 1, then odd
      // groups trade x for the y of even ones: group kg ends with features
      // 16 c + 8 kg .. + 7 as (x, y)
#pragma unroll
      for (int w = 0; w < 2; ++w) {
        const auto a = __builtin_amdgcn_permlane32_swap(x[w], y[w], false, false);
        const auto b = __builtin_amdgcn_permlane16_swap(a[0], a[1], false, false);
        x[w] = b[0];
        y[w] = b[1];
      }
      return u32x4_t{x[0], x[1], y[0], y[1]};
    };
    const int h = h0 + hl;
    if constexpr (DH % 64 == 0) {
      // Whole 128-byte lines per store: features 16 c .. 16 c + 63 of a
      // query are e0 (first half) and e1 (second half) of its four lanes.
      // Rotating e1 by 8 lanes within each row of 16 puts the second half of
      // query j next to the first half of query j + 8 or j - 8, so a store
      // serves queries 0..7 (a) or 8..15 (b) with whole lines: query
      // (qn & 7) (+ 8 for b), features 16 c + 8 kg, + 32 where the lane took
      // the rotated half. A store of half lines from 16 queries costs ~15% of
      // the kernel's time.
      const int j = qn & 7;
      const bool lo = qn < 8;
      const bool ok_a = 16 * gi + j < tile.q_count, ok_b = 16 * gi + j + 8 < tile.q_count;
      const int row_a = ok_a ? row_of(gi, j) : 0, row_b = ok_b ? row_of(gi, j + 8) : 0;
#pragma unroll
      for (int c = 0; c < NO; c += 4) {
        const u32x4_t e0 = out_chunks(c), e1 = out_chunks(c + 2);
        u32x4_t a, b;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const uint32_t r = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)e1[w], 0x128 /* row_ror:8 */, 0xf, 0xf, false);
          a[w] = lo ? e0[w] : r;
          b[w] = lo ? r : e0[w];
        }
        const int col = h * DH + 16 * c + 8 * kg;
        if (ok_a) *reinterpret_cast<u32x4_t*>(out + (size_t)row_a * ldo + col + (lo ? 0 : 32)) = a;
        if (ok_b) *reinterpret_cast<u32x4_t*>(out + (size_t)row_b * ldo + col + (lo ? 32 : 0)) = b;
      }
    } else {
      // a head piece of 32 features is half a line, whichever lanes hold it
      const bool ok = 16 * gi + qn < tile.q_count;
      const int row = ok ? row_of(gi, qn) : 0;
#pragma unroll
      for (int c = 0; c < NO; c += 2) {
        const u32x4_t e = out_chunks(c);
        if (ok) *reinterpret_cast<u32x4_t*>(out + (size_t)row * ldo + h * DH + 16 * c + 8 * kg) = e;
      }
    }
  };
  // (group, head) pair k = 16-query group k / hb, head h0 + k % hb: wave w
  // takes pairs w, w + 8, ..., so the 8 waves work on 8 consecutive pairs at
  // a time (with 8 heads, the 8 pieces of the same rows); Q of the wave's
  // next pair requested first
  const int n_pairs = n_groups * hb;
  for (int k = wave; k < n_pairs; k += 16) {
    load_q((k + 8) / hb, h0 + (k + 8) % hb, qb);
    work(k / hb, k % hb, qa);
    if (k + 8 >= n_pairs) break;
    load_q((k + 16) / hb, h0 + (k + 16) % hb, qa);
    work((k + 8) / hb, (k + 8) % hb, qb);
  }
}

// slots of the MFMA kernel: the window from its start rounded down to a
// multiple of 4, and the pooled token (0: the window does not fit)
static int lg_mfma_slots(bool bf, int l_local, bool gpool) {
  const int need = l_local + (gpool ? 1 : 0) + 3;
  return bf && need <= kLgMfmaMaxSlots ? (need + 15) / 16 * 16 : 0;
}
static int lg_mfma_max_heads(int ns, int dh) {
  switch (ns) {
#define TX_LGH(NS) \
  case NS: return dh == 32 ? lg_max_heads(NS, 32) : dh == 64 ? lg_max_heads(NS, 64) : lg_max_heads(NS, 128);
    TX_LGH(16) TX_LGH(32) TX_LGH(48) TX_LGH(64) TX_LGH(80)
#undef TX_LGH
    default: return 0;
  }
}
int lg_attention_heads_per_tile(bool bf, int l_local, bool gpool, int H, int dh) {
  const int ns = lg_mfma_slots(bf, l_local, gpool);
  if (ns == 0) return 1;
  int hb = std::min(H, lg_mfma_max_heads(ns, dh));
  while (H % hb) --hb;
  return hb;
}
int lg_attention_q_block(bool bf, int l_local, bool gpool, int H, int dh) {
  if (lg_mfma_slots(bf, l_local, gpool) == 0) return kLgQueries;
  const int hb = lg_attention_heads_per_tile(bf, l_local, gpool, H, dh);
  return 16 * ((kLgMfmaPairs + hb - 1) / hb);
}

hipError_t launch_lg_attention(bool bf, const void* q, int ldq, void* out, int ldo, const void* pool,
                               const int32_t* page_table, int max_pages, PageGeom g, int layer_slot,
                               const AttnReq* reqs, const AttnTile* tiles, int n_tiles, int q_block, int l_local,
                               const void* gkv, int gkv_ld, int dec_layer, hipStream_t s) {
  if (n_tiles <= 0) return hipSuccess;
  if (l_local < 1 || l_local > kMaxLocal) return hipErrorInvalidValue;
  if (g.dh != 32 && g.dh != 64 && g.dh != 128) return hipErrorInvalidValue;
  const bool gp = gkv != nullptr;
  if (q_block != lg_attention_q_block(bf, l_local, gp, g.H, g.dh)) return hipErrorInvalidValue;
  const float sl2 = 1.4426950408889634f / sqrtf((float)g.dh);
  if (const int ns = lg_mfma_slots(bf, l_local, gp)) {
    const int hb = lg_attention_heads_per_tile(bf, l_local, gp, g.H, g.dh);
#define TX_LGM(DH, NS)                                                                                            \
  lg_cross_attn_mfma<DH, NS><<<n_tiles, 512, 0, s>>>((const bf16*)q, ldq, (bf16*)out, ldo, (const bf16*)pool,        \
                                                     page_table, max_pages, g, layer_slot, reqs, tiles, l_local, hb, \
                                                     (const bf16*)gkv, gkv_ld, dec_layer, sl2)
#define TX_LGM_NS(DH)                 \
  switch (ns) {                       \
    case 16: TX_LGM(DH, 16); break;   \
    case 32: TX_LGM(DH, 32); break;   \
    case 48: TX_LGM(DH, 48); break;   \
    case 64: TX_LGM(DH, 64); break;   \
    default: TX_LGM(DH, 80); break;   \
  }
    switch (g.dh) {
      case 32: TX_LGM_NS(32); break;
      case 64: TX_LGM_NS(64); break;
      default: TX_LGM_NS(128); break;
    }
#undef TX_LGM_NS
#undef TX_LGM
    return hipGetLastError();
  }
  // fp32 models (every bf16 window has its MFMA slot count)
  if (bf) return hipErrorInvalidValue;
  const size_t lds = (size_t)(l_local + 1) * 4 * (g.dh / 4 + 4) * 2 * sizeof(float);
#define TX_LG(DH)                                                                                                   \
  lg_cross_attn<float, DH><<<n_tiles, 256, lds, s>>>((const float*)q, ldq, (float*)out, ldo, (const float*)pool,   \
                                                   page_table, max_pages, g, layer_slot, reqs, tiles, l_local,       \
                                                   (const float*)gkv, gkv_ld, dec_layer, sl2)
  switch (g.dh) {
    case 32: TX_LG(32); break;
    case 64: TX_LG(64); break;
    default: TX_LG(128); break;
  }
#undef TX_LG
  return hipGetLastError();
}

}  // namespace tx
