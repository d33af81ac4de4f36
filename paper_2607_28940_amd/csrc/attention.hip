// Attention kernels of the TransX path.
//
// paged attention  softmax(q k^T / sqrt(d_h) [+ rel bias]) v with keys/values
//                  read from the request's cache pages. Serves the decoder
//                  cross-attention (every query of a request sees every cached
//                  token: Sec. 4.1.2, Eq. sparse-cross-attn with the index set
//                  = all tokens, K/V shared by all the request's queries) and the
//                  causal encoder (queries at positions pos0+i see positions
//                  <= their own, logit + beta_h[min(i - j, R - 1)]: Sec. 4.1.1,
//                  App. D remark on incremental encoding).
// self-attention   decoder self-attention with the candidate-isolating mask
//                  (App. B): serving tokens causal among themselves, candidate
//                  c sees every serving token and itself.
//
// Softmax is the online (running max / running sum) form in fp32 in the base-2
// domain: logits are scaled by log2(e) and exponentiated with exp2.
#include "tx_internal.h"
#include "wave_reduce.h"

namespace tx {

constexpr float kLog2e = 1.4426950408889634f;


// Running state of one wave's 32 queries: O^T accumulators (rows = features,
// columns = queries), running max and sum (base-2 domain).
template <int DH>
struct MfmaAcc {
  floatx16 o[DH / 32];
  float m, l;
  __device__ __forceinline__ void init() {
#pragma unroll
    for (int db = 0; db < DH / 32; ++db)
#pragma unroll
      for (int v = 0; v < 16; ++v) o[db][v] = 0.f;
    m = -INFINITY;
    l = 0.f;
  }
};

// One 64-key tile for one wave: S^T = K Q^T on MFMA (keys as rows, so lane
// l32 + 32*hi holds 32 keys of query l32), online softmax update, then
// O^T += V^T P^T with P^T taken from the S^T accumulators: the MFMA k index
// 8*hi + t stands for key base + 8*(t/4) + 4*hi + t%4 on both operands, so no
// register shuffle is needed, and a V^T tile held in the stored column order
// (vt_col: 16-key groups as 0-3, 8-11, 4-7, 12-15) supplies exactly those keys
// with one 16-byte LDS read.
// The running max is kept in raw logit units, so scaling and max subtraction
// fuse into one FMA before exp2. When `masked` (uniform across the wave) every
// raw logit goes through `mask(key, s)`, which returns it (plus any bias, in
// raw units) or -inf; other tiles skip that work. The O^T rescale is skipped when no lane's
// max moved.
// LDS addresses of the MFMA fragments. Padded tiles: K rows of KLD elements,
// V^T rows of VLD. Swizzled tiles (SWZ, filled by direct-to-LDS loads): K
// rows of DH elements with 16-byte slot s of row r holding chunk s ^ (r mod
// DH/8), V^T rows of 64 with slot s holding chunk s ^ ((r / 2) mod 8); both
// keep the fragment reads of 8 consecutive rows on distinct banks.
template <int DH, int KLD, bool SWZ>
__device__ __forceinline__ int k_frag(int row, int slot) {
  return SWZ ? row * DH + ((slot ^ (row & (DH / 8 - 1))) << 3) : row * KLD + (slot << 3);
}
template <int VLD, bool SWZ>
__device__ __forceinline__ int v_frag(int row, int slot) {
  return SWZ ? row * 64 + ((slot ^ ((row >> 1) & 7)) << 3) : row * VLD + (slot << 3);
}

// The tile arithmetic takes its operands from fragment sources:
// kfrag(kb, kk) is K row kb * 32 + l32, features 16 kk + 8 hi .. + 7;
// vfrag(ks, db) is V^T row 32 db + l32, stored columns
// 32 (ks / 2) + 16 (ks % 2) + 8 hi .. + 7. FROM_LDS adds scheduling hints
// for fragments read from LDS (each read four ahead of the MFMA that uses it).
template <int N>  // N fragment reads for N MFMAs
__device__ __forceinline__ void pace_lds_reads() {
  __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
  for (int g = 0; g < N - 4; ++g) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
}

// First half: S^T = K Q^T, the online softmax update and P^T in bf16.
template <int DH, bool FROM_LDS, class KFrag, class Mask>
__device__ __forceinline__ void mfma_qk_softmax(KFrag kfrag, const bf16x8 (&qf)[DH / 16], MfmaAcc<DH>& acc,
                                                float scale_log2, int hi, bool masked, Mask mask, bf16x8 (&pf)[4],
                                                float thr = -1.f) {
  floatx16 s[2];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
    for (int v = 0; v < 16; ++v) s[kb][v] = 0.f;
#pragma unroll
    for (int kk = 0; kk < DH / 16; ++kk) s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kfrag(kb, kk), qf[kk], s[kb], 0, 0, 0);
  }
  if (FROM_LDS) pace_lds_reads<DH / 8>();
  if (masked) {  // wave-uniform
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) s[kb][v] = mask(kb * 32 + 8 * (v >> 2) + 4 * hi + (v & 3), s[kb][v]);
  }
  float mx = -INFINITY;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int v = 0; v < 16; ++v) mx = fmaxf(mx, s[kb][v]);
  mx = xor32_max(mx);
  // Lazy reference max: probabilities are exp2((s - m) * scale) against a
  // reference m that only moves when this tile would push one above 2^8
  // (fine for fp32 sums and bf16 P); O and l are rescaled only then. The
  // final O / l does not depend on which reference was used.
  // (thr, when given, is 8 / scale_log2 computed once by the caller)
  const bool bump = mx > acc.m + (thr >= 0.f ? thr : 8.f / scale_log2);
  if (__any(bump)) {
    const float m_new = bump ? mx : acc.m;
    // 1 where the reference stays (also at -inf), 0 where it leaves -inf
    const float alpha = bump ? __builtin_amdgcn_exp2f((acc.m - m_new) * scale_log2) : 1.f;
    acc.l *= alpha;
#pragma unroll
    for (int db = 0; db < DH / 32; ++db)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc.o[db][v] *= alpha;
    acc.m = m_new;
  }
  const float off = (acc.m == -INFINITY) ? 0.f : -acc.m * scale_log2;
  float rs = 0.f;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const float e = __builtin_amdgcn_exp2f(fmaf(s[kb][v], scale_log2, off));
      s[kb][v] = e;
      rs += e;
    }
  rs = xor32_sum(rs);
  acc.l += rs;
#pragma unroll
  for (int ks = 0; ks < 4; ++ks)
#pragma unroll
    for (int t = 0; t < 8; ++t) pf[ks][t] = (bf16)s[ks >> 1][8 * (ks & 1) + t];
}

// Second half: O^T += V^T P^T. From LDS the V^T fragment reads run four ahead
// of their MFMAs, as the K reads do, instead of all sixteen being hoisted
// above the softmax (which would hold 64 more registers through it).
template <int DH, bool FROM_LDS, class VFrag>
__device__ __forceinline__ void mfma_pv(VFrag vfrag, const bf16x8 (&pf)[4], MfmaAcc<DH>& acc) {
#pragma unroll
  for (int ks = 0; ks < 4; ++ks)
#pragma unroll
    for (int db = 0; db < DH / 32; ++db) acc.o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vfrag(ks, db), pf[ks], acc.o[db], 0, 0, 0);
  if (FROM_LDS) pace_lds_reads<DH / 8>();
}

template <int DH, bool FROM_LDS, class KFrag, class VFrag, class Mask>
__device__ __forceinline__ void mfma_attend_frags(KFrag kfrag, VFrag vfrag, const bf16x8 (&qf)[DH / 16],
                                                  MfmaAcc<DH>& acc, float scale_log2, int hi, bool masked, Mask mask) {
  bf16x8 pf[4];
  mfma_qk_softmax<DH, FROM_LDS>(kfrag, qf, acc, scale_log2, hi, masked, mask, pf);
  mfma_pv<DH, FROM_LDS>(vfrag, pf, acc);
}

// The same tile with K and V^T staged in LDS.
template <int DH, int KLD, int VLD, class Mask, bool SWZ = false>
__device__ __forceinline__ void mfma_attend_tile(const bf16* __restrict__ sK, const bf16* __restrict__ sV,
                                                 const bf16x8 (&qf)[DH / 16], MfmaAcc<DH>& acc, float scale_log2,
                                                 int l32, int hi, bool masked, Mask mask) {
  auto kfrag = [&](int kb, int kk) {
    return *reinterpret_cast<const bf16x8*>(&sK[k_frag<DH, KLD, SWZ>(kb * 32 + l32, 2 * kk + hi)]);
  };
  auto vfrag = [&](int ks, int db) {
    const int kbase = (ks >> 1) * 32 + 16 * (ks & 1) + 8 * hi;  // in the V^T tile's permuted key order
    return *reinterpret_cast<const bf16x8*>(&sV[v_frag<VLD, SWZ>(32 * db + l32, kbase >> 3)]);
  };
  mfma_attend_frags<DH, true>(kfrag, vfrag, qf, acc, scale_log2, hi, masked, mask);
}

// Normalises the wave's 32 output rows, parks them in LDS (stage: 32 x DH
// elements of free LDS for this wave) and stores them row-contiguously, DH / 8
// lanes per row, instead of 8-byte pieces of 32 rows per store. 16-byte unit u
// of row r sits at u ^ swz(r): conflict-free for the 8-byte writes and the
// 16-byte reads. The wave's query r (r < nq) is query q0 + r of its request,
// whose output row is row_a + q for q < split and row_b + (q - split) after.
template <int DH>
__device__ __forceinline__ void mfma_store_out_staged(const MfmaAcc<DH>& acc, bf16* __restrict__ stage,
                                                      bf16* __restrict__ out, int ldo, int col0, int lane, int q0,
                                                      int nq, int split, int row_a, int row_b) {
  constexpr int UPR = DH / 8;    // 16-byte units per row
  constexpr int RPI = 64 / UPR;  // rows per read
  auto swz = [](int r) { return UPR == 16 ? (r & 15) : ((r >> 1) & 7); };
  const int l32 = lane & 31, hi = lane >> 5;
  const float inv = acc.l > 0.f ? 1.f / acc.l : 0.f;
#pragma unroll
  for (int db = 0; db < DH / 32; ++db)
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      bf16x4 w;
#pragma unroll
      for (int t = 0; t < 4; ++t) w[t] = (bf16)(acc.o[db][4 * gq + t] * inv);
      *reinterpret_cast<bf16x4*>(stage + l32 * DH + (((4 * db + gq) ^ swz(l32)) << 3) + 4 * hi) = w;
    }
#pragma unroll
  for (int k = 0; k < 32 / RPI; ++k) {
    const int r = k * RPI + lane / UPR, q = lane % UPR;
    const bf16x8 v = *reinterpret_cast<const bf16x8*>(stage + r * DH + ((q ^ swz(r)) << 3));
    if (r < nq) {
      const int qq = q0 + r;
      const int o = qq < split ? row_a + qq : row_b + (qq - split);
      *reinterpret_cast<bf16x8*>(out + (size_t)o * ldo + col0 + q * 8) = v;
    }
  }
}

// Direct HBM/L2 -> LDS copy of one page's 64 x DH K slab or DH x 64 V^T slab
// by the four waves of a block: wave w moves the 1 KB pieces w, w + 4, ...;
// lane l of a piece fills 16-byte LDS slot l with the chunk the XOR swizzle
// puts there (K: row r, slot s holds chunk s ^ (r mod DH/8); V^T: slot s
// holds chunk s ^ ((r / 2) mod 8)). Piece w + 4u lies 4u KB after piece w in
// the slab and in LDS with the same swizzle, so one 32-bit lane offset per
// slab and a scalar step serve every piece, and per page only the slab base
// (scalar registers, in a raw buffer resource) changes.
template <int DH>
struct PageDma {
  typedef __attribute__((address_space(3))) void* lds_ptr_t;
  uint32_t koff, voff;  // bytes from the slab start to the lane's chunk of piece w
  int piece0;           // element offset of piece w in LDS
  __device__ __forceinline__ PageDma(int wave, int lane) {
    const int e = wave * 512 + lane * 8;  // the lane's first element in piece w
    const int kr = e / DH, ks = (e % DH) >> 3;
    const int vr = e >> 6, vs = (e & 63) >> 3;
    koff = 2u * (uint32_t)(kr * DH + ((ks ^ (kr & (DH / 8 - 1))) << 3));
    voff = 2u * (uint32_t)(vr * 64 + ((vs ^ ((vr >> 1) & 7)) << 3));
    piece0 = wave * 512;
  }
  __device__ __forceinline__ void load(const bf16* slab, uint32_t off, bf16* dst) const {
    // word 3 of the resource as CDNA wants it for raw loads; extent = the slab
    const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc((void*)slab, 0, 128 * DH, 0x00020000);
#pragma unroll
    for (int u = 0; u < DH / 32; ++u)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_ptr_t)(dst + piece0 + 2048 * u), 16, (int)off, 4096 * u, 0, 0);
  }
};

// ============================================================================
// bf16 paged attention on MFMA.
//
// A block of 4 waves serves up to 128 queries of one (request, head); each
// wave owns 32 queries. For every 64-token page the block stages K [64][dh]
// and V^T [dh][64] in LDS (double-buffered: the next page travels from HBM/L2
// straight into LDS with buffer loads to LDS while the current one is used, no
// register staging), so every K/V byte fetched from HBM/L2 feeds all queries
// of the block. The page keeps V^T in the column order the PV MFMA wants; the
// tiles are XOR-swizzled in LDS (the swizzle applied on the global side, since
// each lane's 16 bytes land at a fixed slot) so fragment reads are
// bank-conflict free without padding.
//
// Per wave and page:  S^T = K Q^T  (v_mfma_f32_32x32x16_bf16, keys as rows so
// that a lane holds 32 keys of one query: the softmax row reduction is within
// the lane plus one exchange with lane l^32), online softmax update, then
// O^T += V^T P^T with P^T taken straight from the S^T accumulators (the MFMA
// k index is permuted consistently on both operands, so no register shuffle
// is needed; V^T supplies the matching keys with one 16-byte LDS read).
// Keys past the request's length are masked by selection and their V columns
// are zeroed in LDS so that unused page slots (of any content) never reach
// the output.
// ============================================================================
template <int DH, bool CAUSAL>
__global__ __launch_bounds__(256, 2) void paged_attn_mfma(const bf16* __restrict__ q, int ldq, bf16* __restrict__ out,
                                                           int ldo, const bf16* __restrict__ pool,
                                                           const int32_t* __restrict__ page_table, int max_pages,
                                                           PageGeom g, int layer_slot, const AttnReq* __restrict__ reqs,
                                                           const AttnTile* __restrict__ tiles,
                                                           const float* __restrict__ rel, int R, float scale_log2) {
  constexpr int KLD = DH, VLD = 64;  // swizzled, unpadded tiles
  // K page buffers 0, 1, then V^T page buffers 0, 1
  __shared__ __attribute__((aligned(16))) bf16 sKV[4 * 64 * DH];
  bf16* const sK0 = sKV;
  bf16* const sK1 = sKV + 64 * DH;
  bf16* const sV0 = sKV + 2 * 64 * DH;

  const AttnTile tile = tiles[blockIdx.x];
  if (tile.q_count <= 0) return;
  const AttnReq rq = reqs[tile.req];
  const int h = tile.head;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, hi = lane >> 5;

  const int qi = wave * 32 + l32;
  const bool wave_active = wave * 32 < tile.q_count;
  const int i = tile.q_begin + min(qi, tile.q_count - 1);
  const int row = i < rq.qa_n ? rq.qa_row + i : rq.qb_row + (i - rq.qa_n);
  const int qpos = rq.pos0 + i;
  const float bias_scale = kLog2e / scale_log2;  // logit bias expressed in raw q.k units

  // Q as the MFMA B operand: lane holds Q[query l32][16*kk + 8*hi .. +8]
  bf16x8 qf[DH / 16];
  {
    const bf16* qr = q + (size_t)row * ldq + h * DH + 8 * hi;
#pragma unroll
    for (int kk = 0; kk < DH / 16; ++kk) qf[kk] = *reinterpret_cast<const bf16x8*>(qr + 16 * kk);
  }

  MfmaAcc<DH> acc;
  acc.init();

  const int kv_len = rq.kv_len;
  int n_pages = (kv_len + kPage - 1) / kPage;
  if (CAUSAL) {
    const int last_pos = rq.pos0 + tile.q_begin + tile.q_count - 1;
    n_pages = min(n_pages, last_pos / kPage + 1);
  }
  const int32_t* ptab = page_table + (size_t)rq.slot * max_pages;

  // Pages travel HBM/L2 -> LDS with buffer_load_dwordx4 ... lds: each wave
  // moves DH/32 KB of the K slab and as much of the V^T slab per page; lane l
  // of a 1 KB load fills 16-byte slot l of it with the chunk the swizzle puts
  // there. Page p+1 is requested while page p is used; every wave waits for
  // its own loads before the page's closing barrier.
  const PageDma<DH> pd(wave, lane);
  auto dma = [&](int p, bf16* dK, bf16* dV) {
    const bf16* base = pool + (size_t)ptab[p] * g.page_elems;
    pd.load(base + g.k_off(layer_slot, h), pd.koff, dK);
    pd.load(base + g.v_off(layer_slot, h), pd.voff, dV);
  };
  // keys past the request's length on its last page: V^T columns zeroed in LDS
  // (the page may hold anything there; their K logits are masked anyway)
  auto zero_tail = [&](int p, bf16* dV) {
    const int valid = kv_len - p * kPage;
    for (int e = tid; e < DH * 64; e += 256) {
      const int r = e >> 6, col = e & 63;
      const int chunk = (col >> 3) ^ ((r >> 1) & 7);  // stored chunk held at this slot
      if (vt_col(chunk * 8 + (col & 7)) >= valid) dV[e] = (bf16)0.f;
    }
  };
  const bool partial = kv_len % kPage != 0;
  dma(0, sK0, sV0);
  __syncthreads();
  if (n_pages == 1 && partial) {
    zero_tail(0, sV0);
    __syncthreads();
  }
  auto step = [&](int p, const bf16* cK, const bf16* cV, bf16* nK, bf16* nV) {
    if (p + 1 < n_pages) dma(p + 1, nK, nV);
    if (wave_active) {
      const int key0 = p * kPage;
      // masking is needed on the request's last (partial) page and, when
      // causal, on pages that reach past this wave's first query position;
      // the relative-position bias applies to every causal tile
      const bool needs_mask = CAUSAL || key0 + kPage > kv_len;
      auto mask = [&](int kl, float x) {
        const int key = key0 + kl;
        bool ok = key < kv_len;
        if (CAUSAL) {
          ok = ok && key <= qpos;
          if (R > 0) x += rel[h * R + min(max(qpos - key, 0), R - 1)] * bias_scale;
        }
        return ok ? x : -INFINITY;
      };
      mfma_attend_tile<DH, KLD, VLD, decltype(mask), true>(cK, cV, qf, acc, scale_log2, l32, hi, needs_mask, mask);
    }
    __syncthreads();  // page p+1 in LDS for every wave; page p no longer read
    if (p + 2 == n_pages && partial) {
      zero_tail(p + 1, nV);
      __syncthreads();
    }
  };
  // one loop body for both buffers (the buffer offset is uniform), so the
  // fragment addresses are not held twice
  for (int p = 0; p < n_pages; ++p) {
    const int b = (p & 1) * (64 * DH);
    step(p, sK0 + b, sV0 + b, sK0 + (64 * DH - b), sV0 + (64 * DH - b));
  }
  // every step ends on a barrier, so no page buffer is read any more: waves
  // 0-1 park their output rows in sK0, waves 2-3 in sK1
  mfma_store_out_staged<DH>(acc, (wave < 2 ? sK0 : sK1) + (wave & 1) * 32 * DH, out, ldo, h * DH, lane,
                            tile.q_begin + wave * 32, tile.q_count - wave * 32, rq.qa_n, rq.qa_row, rq.qb_row);
}

// ============================================================================
// The decoder cross-attention (no causal mask, d_h = 128) with three blocks per
// CU, i.e. three waves per SIMD to overlap each wave's dependent page chain
// (QK on MFMA, softmax on the VALU, PV on MFMA) with two others instead of
// one: 48 KB of LDS (K double-buffered, V^T single-buffered) and at most 168
// registers. Page p + 1's K is requested at the top of page p's body, page
// p + 1's V^T once page p's PV has left the buffer; before the PV each wave
// waits for its own V^T loads only (the K loads issued after them may stay in
// flight) and the block meets at a barrier. Same arithmetic in the same order
// as paged_attn_mfma.
// The tiles come as one list per XCD (XCD x: tiles[xoff[x] .. xoff[x + 1])).
// A tile (XTile) covers up to 128 queries of one request and head against the
// key pages page_begin .. page_end - 1: all of the request's pages (its rows
// are written normalised), or one part of them (a kv-split tile: the
// unnormalised output, reference max and running sum go to a partial slot,
// combined later by xattn_merge). Keys past the request's length on its last
// page are masked; the cache keeps zeros in their V^T columns (the page
// scatter writes them), so their zero probabilities never meet other values.
// ============================================================================
template <int DH, bool SPLIT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3, 3))) void paged_attn_mfma3(
    const bf16* __restrict__ q, int ldq, bf16* __restrict__ out, int ldo, const bf16* __restrict__ pool,
    const int32_t* __restrict__ page_table, int max_pages, PageGeom g, int layer_slot,
    const XTile* __restrict__ tiles, const int32_t* __restrict__ xoff, float* __restrict__ partial,
    float scale_log2, float bump_thr) {
  // K page buffers 0, 1, then the V^T page buffer
  __shared__ __attribute__((aligned(16))) bf16 sKV[3 * 64 * DH];
  bf16* const sK0 = sKV;
  bf16* const sK1 = sKV + 64 * DH;
  bf16* const sV = sKV + 2 * 64 * DH;

  // block b runs on XCD b % 8 and takes entry b / 8 of that XCD's tile list
  const int t_idx = xoff[blockIdx.x & 7] + (int)(blockIdx.x >> 3);
  if (t_idx >= xoff[(blockIdx.x & 7) + 1]) return;
  const XTile tile = tiles[t_idx];
  const int h = tile.head;
  // the wave index is uniform in its wave: a scalar, as is all derived from it
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, hi = lane >> 5;
  const bool wave_active = wave * 32 < tile.q_count;
  const int i = tile.q_begin + min(wave * 32 + l32, tile.q_count - 1);
  const int row = i < tile.qa_n ? tile.qa_row + i : tile.qb_row + (i - tile.qa_n);

  bf16x8 qf[DH / 16];
  {
    const bf16* qr = q + (size_t)row * ldq + h * DH + 8 * hi;
#pragma unroll
    for (int kk = 0; kk < DH / 16; ++kk) qf[kk] = *reinterpret_cast<const bf16x8*>(qr + 16 * kk);
  }
  MfmaAcc<DH> acc;
  acc.init();

  const int kv_len = tile.kv_len;
  const int p0 = tile.page_begin, n_pages = tile.page_end - tile.page_begin;
  const int32_t* ptab = page_table + (size_t)tile.slot * max_pages + p0;
  const PageDma<DH> pd(wave, lane);
  // page-table window: lane l holds the pool index of page wbase + l of the
  // range; a page's index is read from its lane into a scalar, so the page
  // loads take a uniform address and no memory read of their own
  int wbase = 0;
  int pwin = ptab[min(lane, n_pages - 1)];
  auto page = [&](int p) { return pool + (size_t)__builtin_amdgcn_readlane(pwin, p - wbase) * g.page_elems; };
  pd.load(page(0) + g.k_off(layer_slot, h), pd.koff, sK0);
  pd.load(page(0) + g.v_off(layer_slot, h), pd.voff, sV);
  // LDS byte offsets of the lane's MFMA fragments, the swizzles of k_frag
  // and v_frag in closed form: K row kb * 32 + l32, slot 2 kk + hi at
  // kb * 64 DH * 2 + (kxor ^ 32 kk); V^T row 32 db + l32, slot 2 ks + hi at
  // db * 4096 + (vxor ^ 32 ks). One register each; every read costs one XOR.
  const int kxor = (l32 * DH * 2) | ((hi ^ (l32 & (DH / 8 - 1))) << 4);
  const int vxor = (l32 * 128) | ((hi ^ ((l32 >> 1) & 7)) << 4);
  const char* const lds = reinterpret_cast<const char*>(sKV);
  __syncthreads();
  for (int p = 0; p < n_pages; ++p) {
    const int b = (p & 1) * (64 * DH);
    if (p + 1 < n_pages) pd.load(page(p + 1) + g.k_off(layer_slot, h), pd.koff, sK0 + (64 * DH - b));
    const int key0 = (p0 + p) * kPage;
    bf16x8 pf[4];
    // the K buffer's offset joins the base before the XORs (it lies above
    // their bits); the opaque copies keep the per-read addresses from being
    // hoisted out of the loop into registers held across it
    int kx = kxor + 2 * b, vx = vxor + 2 * 2 * 64 * DH;
    asm volatile("" : "+v"(kx), "+v"(vx));
    if (wave_active) {
      auto kfrag = [&](int kb, int kk) {
        return *reinterpret_cast<const bf16x8*>(lds + (kx ^ (32 * kk)) + kb * 64 * DH);
      };
      mfma_qk_softmax<DH, true>(kfrag, qf, acc, scale_log2, hi, key0 + kPage > kv_len, [&](int kl, float x) {
        return key0 + kl < kv_len ? x : -INFINITY;
      }, pf, bump_thr);
    }
    if (p > 0) {
      // V^T of page p (requested after page p - 1's PV) in LDS for every wave;
      // the DH / 32 K loads of page p + 1 issued since may stay in flight
      if (p + 1 < n_pages) asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(DH / 32) : "memory");
      else asm volatile("s_waitcnt vmcnt(0)\n\ts_barrier" ::: "memory");
    }
    if (wave_active) {
      auto vfrag = [&](int ks, int db) {
        return *reinterpret_cast<const bf16x8*>(lds + (vx ^ (32 * ks)) + db * 4096);
      };
      mfma_pv<DH, true>(vfrag, pf, acc);
    }
    __syncthreads();  // K and V^T of page p no longer read; K of page p + 1 landed
    // no load is in flight here: the window moves when the next body's K
    // load (page p + 2) would leave it
    if (p + 2 - wbase >= 64 && p + 2 < n_pages) {
      wbase = p + 1;
      pwin = ptab[min(p + 1 + lane, n_pages - 1)];
      // consumed here, where it is the only load in flight (so that no later
      // read of the window waits on the page loads issued after it)
      asm volatile("" : "+v"(pwin));
    }
    if (p + 1 < n_pages) pd.load(page(p + 1) + g.v_off(layer_slot, h), pd.voff, sV);
  }
  if (SPLIT) {
    // kv-split tile: fp32 O (unnormalised, features 32 db + 8 gq + 4 hi ..),
    // reference max and running sum of each of the wave's queries
    const int lq = wave * 32 + l32;
    if (lq < tile.q_count) {
      float* ps = partial + (size_t)tile.part * (128 * (DH + 2));
#pragma unroll
      for (int db = 0; db < DH / 32; ++db)
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
          const floatx4 w = {acc.o[db][4 * gq], acc.o[db][4 * gq + 1], acc.o[db][4 * gq + 2], acc.o[db][4 * gq + 3]};
          *reinterpret_cast<floatx4*>(ps + (size_t)lq * DH + 32 * db + 8 * gq + 4 * hi) = w;
        }
      if (hi == 0) {
        ps[128 * DH + lq] = acc.m;
        ps[128 * DH + 128 + lq] = acc.l;
      }
    }
    return;
  }
  // every body ends on a barrier and the last requests nothing: waves 0-1
  // park their output rows in K buffer 0, waves 2-3 in K buffer 1
  mfma_store_out_staged<DH>(acc, (wave < 2 ? sK0 : sK1) + (wave & 1) * 32 * DH, out, ldo, h * DH, lane,
                            tile.q_begin + wave * 32, tile.q_count - wave * 32, tile.qa_n, tile.qa_row, tile.qb_row);
}

// ============================================================================
// Log-sum-exp merge of kv-split partial results: for every query of a
// (request, head, query block) split over n_parts page ranges,
//   O = sum_s 2^((m_s - M) c) O_s / sum_s 2^((m_s - M) c) l_s,  M = max_s m_s
// (m_s in raw logit units, c = log2(e) / sqrt(d_h)), rounded once to bf16.
// One block per item; thread t takes query t / 2, features 64 (t % 2) .. + 63.
// ============================================================================
__global__ __launch_bounds__(256) void xattn_merge(const float* __restrict__ partial, const XMerge* __restrict__ items,
                                                   bf16* __restrict__ out, int ldo, float scale_log2) {
  constexpr int DH = 128;
  const XMerge it = items[blockIdx.x];
  const int lq = threadIdx.x >> 1, half = threadIdx.x & 1;
  if (lq >= it.q_count) return;
  constexpr size_t kSlot = 128 * (DH + 2);
  float M = -INFINITY;
  for (int s = 0; s < it.n_parts; ++s) M = fmaxf(M, partial[(it.part0 + s) * kSlot + 128 * DH + lq]);
  float acc[64];
#pragma unroll
  for (int e = 0; e < 64; ++e) acc[e] = 0.f;
  float l = 0.f;
  for (int s = 0; s < it.n_parts; ++s) {
    const float* ps = partial + (it.part0 + s) * kSlot;
    const float ms = ps[128 * DH + lq];
    const float w = ms == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((ms - M) * scale_log2);
    l = fmaf(w, ps[128 * DH + 128 + lq], l);
    const floatx4* o = reinterpret_cast<const floatx4*>(ps + (size_t)lq * DH + 64 * half);
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const floatx4 v = o[e];
#pragma unroll
      for (int k = 0; k < 4; ++k) acc[4 * e + k] = fmaf(w, v[k], acc[4 * e + k]);
    }
  }
  const float inv = l > 0.f ? 1.f / l : 0.f;
  const int i = it.q_begin + lq;
  const int row = i < it.qa_n ? it.qa_row + i : it.qb_row + (i - it.qa_n);
  bf16* orow = out + (size_t)row * ldo + it.head * DH + 64 * half;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    bf16x8 v;
#pragma unroll
    for (int k = 0; k < 8; ++k) v[k] = (bf16)(acc[8 * e + k] * inv);
    *reinterpret_cast<bf16x8*>(orow + 8 * e) = v;
  }
}

bool cross_attention_split_ok(bool bf, int dh) { return bf && dh == 128; }

hipError_t launch_cross_attention(const void* q, int ldq, void* out, int ldo, const void* pool,
                                  const int32_t* page_table, int max_pages, PageGeom g, int layer_slot,
                                  const XTile* tiles, const int32_t* xoff, int longest_list,
                                  const XTile* split_tiles, const int32_t* split_xoff, int split_longest,
                                  float* partial, const XMerge* merges, int n_merges, hipStream_t s) {
  if (g.dh != 128) return hipErrorInvalidValue;
  const float sl2 = kLog2e / sqrtf(128.f);
  if (longest_list > 0)
    paged_attn_mfma3<128, false><<<8 * longest_list, 256, 0, s>>>((const bf16*)q, ldq, (bf16*)out, ldo,
                                                                   (const bf16*)pool, page_table, max_pages, g,
                                                                   layer_slot, tiles, xoff, partial, sl2, 8.f / sl2);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || split_longest <= 0) return e;
  paged_attn_mfma3<128, true><<<8 * split_longest, 256, 0, s>>>((const bf16*)q, ldq, (bf16*)out, ldo,
                                                                 (const bf16*)pool, page_table, max_pages, g,
                                                                 layer_slot, split_tiles, split_xoff, partial, sl2,
                                                                 8.f / sl2);
  e = hipGetLastError();
  if (e != hipSuccess || n_merges <= 0) return e;
  xattn_merge<<<n_merges, 256, 0, s>>>(partial, merges, (bf16*)out, ldo, sl2);
  return hipGetLastError();
}

// ============================================================================
// bf16 paged attention for few queries per (request, head): one wave per tile
// of at most 32 queries, four independent tiles per block, pages not staged
// in LDS. With no other wave to share a page there is nothing to stage it
// for: each lane loads its K and V^T MFMA fragments straight from the page
// into registers, the next page's while the current one is used (at d_h = 128
// one wave per SIMD, 128 KB of pages in flight per CU against 64 KB for the
// staged kernel), which is what a tile of the incremental append (16 new
// tokens against thousands of cached ones) is bound by.
// ============================================================================
template <int DH>
struct PageFrags {
  bf16x8 k[2][DH / 16];  // K rows kb * 32 + l32, features 16 kk + 8 hi
  bf16x8 v[4][DH / 32];  // V^T rows 32 db + l32, stored columns 32 (ks / 2) + 16 (ks % 2) + 8 hi
};

template <int DH, bool CAUSAL>
__global__ __launch_bounds__(256, 1) void paged_attn_decode(const bf16* __restrict__ q, int ldq, bf16* __restrict__ out,
                                                            int ldo, const bf16* __restrict__ pool,
                                                            const int32_t* __restrict__ page_table, int max_pages,
                                                            PageGeom g, int layer_slot,
                                                            const AttnReq* __restrict__ reqs,
                                                            const AttnTile* __restrict__ tiles, int n_tiles,
                                                            const float* __restrict__ rel, int R, float scale_log2) {
  const int t_idx = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t_idx >= n_tiles) return;  // whole waves; the kernel has no block-wide barrier
  const AttnTile tile = tiles[t_idx];
  if (tile.q_count <= 0) return;
  const AttnReq rq = reqs[tile.req];
  const int h = tile.head, lane = threadIdx.x & 63, l32 = lane & 31, hi = lane >> 5;
  const int i = tile.q_begin + min(l32, tile.q_count - 1);
  const int row = i < rq.qa_n ? rq.qa_row + i : rq.qb_row + (i - rq.qa_n);
  const int qpos = rq.pos0 + i;
  const float bias_scale = kLog2e / scale_log2;

  bf16x8 qf[DH / 16];
  {
    const bf16* qr = q + (size_t)row * ldq + h * DH + 8 * hi;
#pragma unroll
    for (int kk = 0; kk < DH / 16; ++kk) qf[kk] = *reinterpret_cast<const bf16x8*>(qr + 16 * kk);
  }
  MfmaAcc<DH> acc;
  acc.init();

  const int kv_len = rq.kv_len;
  int n_pages = (kv_len + kPage - 1) / kPage;
  if (CAUSAL) n_pages = min(n_pages, (rq.pos0 + tile.q_begin + tile.q_count - 1) / kPage + 1);
  const int32_t* ptab = page_table + (size_t)rq.slot * max_pages;
  // the head's relative-position table, per wave in LDS: the mask reads it
  // without a vector-memory wait, which would also wait for the page in flight
  __shared__ float s_rel[4][kDecodeMaxRel];
  float* wrel = s_rel[threadIdx.x >> 6];
  if (CAUSAL)
    for (int j = lane; j < R; j += 64) wrel[j] = rel[h * R + j];

  auto fetch = [&](int p, PageFrags<DH>& f) {
    const bf16* base = pool + (size_t)ptab[p] * g.page_elems;
    const bf16* kp = base + g.k_off(layer_slot, h) + (size_t)l32 * DH + 8 * hi;
    const bf16* vp = base + g.v_off(layer_slot, h) + (size_t)l32 * kPage + 8 * hi;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int kk = 0; kk < DH / 16; ++kk)
        f.k[kb][kk] = *reinterpret_cast<const bf16x8*>(kp + (size_t)kb * 32 * DH + 16 * kk);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int db = 0; db < DH / 32; ++db)
        f.v[ks][db] = *reinterpret_cast<const bf16x8*>(vp + (size_t)db * 32 * kPage + 32 * (ks >> 1) + 16 * (ks & 1));
  };
  // Causal pages whose every key lies at least R - 1 positions before the
  // tile's first query are visible to all its queries with the bias at the
  // last bucket: one added constant instead of the per-logit mask.
  const int q_first = rq.pos0 + tile.q_begin;
  const float far_bias = (CAUSAL && R > 0) ? wrel[R - 1] * bias_scale : 0.f;
  auto attend = [&](int p, PageFrags<DH>& f, bool tail) {
    const int key0 = p * kPage;
    const bool far = CAUSAL && !tail && key0 + kPage - 1 + max(R - 1, 0) <= q_first;
    auto mask = [&](int kl, float x) {
      if (far) return x + far_bias;
      const int key = key0 + kl;
      bool ok = key < kv_len;
      if (CAUSAL) {
        ok = ok && key <= qpos;
        if (R > 0) x += wrel[min(max(qpos - key, 0), R - 1)] * bias_scale;
      }
      return ok ? x : -INFINITY;
    };
    mfma_attend_frags<DH, false>([&](int kb, int kk) { return f.k[kb][kk]; },
                                 [&](int ks, int db) { return f.v[ks][db]; }, qf, acc, scale_log2, hi,
                                 tail || (CAUSAL && (!far || R > 0)), mask);
  };
  // keys past the request's length on the last page: V^T columns zeroed (the
  // page may hold anything there; their logits are masked)
  auto zero_tail = [&](int p, PageFrags<DH>& f) {
    const int valid = kv_len - p * kPage;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int db = 0; db < DH / 32; ++db)
#pragma unroll
        for (int t = 0; t < 8; ++t)
          if (vt_col(32 * (ks >> 1) + 16 * (ks & 1) + 8 * hi + t) >= valid) f.v[ks][db][t] = (bf16)0.f;
  };
  // full pages in pairs (page p + 1 travels while page p is used), then the
  // remaining full page and the partial last page, if any
  const int n_full = n_pages * kPage > kv_len ? n_pages - 1 : n_pages;
  PageFrags<DH> fa, fb;
  fetch(0, fa);
  int p = 0;
  for (; p + 1 < n_full; p += 2) {
    fetch(p + 1, fb);
    attend(p, fa, false);
    if (p + 2 < n_pages) fetch(p + 2, fa);
    attend(p + 1, fb, false);
  }
  if (p < n_full) {
    if (p + 1 < n_pages) fetch(p + 1, fb);
    attend(p, fa, false);
    if (++p < n_pages) {
      zero_tail(p, fb);
      attend(p, fb, true);
    }
  } else if (p < n_pages) {
    zero_tail(p, fa);
    attend(p, fa, true);
  }
  if (l32 < tile.q_count) {
    const float inv = acc.l > 0.f ? 1.f / acc.l : 0.f;
    bf16* orow = out + (size_t)row * ldo + h * DH + 4 * hi;
#pragma unroll
    for (int db = 0; db < DH / 32; ++db)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        bf16x4 w;
#pragma unroll
        for (int t = 0; t < 4; ++t) w[t] = (bf16)(acc.o[db][4 * gq + t] * inv);
        *reinterpret_cast<bf16x4*>(orow + 32 * db + 8 * gq) = w;
      }
  }
}

// ============================================================================
// bf16 decoder self-attention on MFMA (App. B mask). Same tile arithmetic as
// the paged kernel: the request's serving tokens are the keys, staged 64 at a
// time in LDS (K as rows, V transposed while it is written to LDS); serving
// query i sees serving keys j <= i, every candidate sees all serving keys and
// then its own key/value, folded in as one more online-softmax step.
// ============================================================================
template <int DH>
__global__ __launch_bounds__(256, 2) void self_attn_mfma(const bf16* __restrict__ qkv, int d, bf16* __restrict__ out,
                                                          const SelfReq* __restrict__ reqs,
                                                          const SelfTile* __restrict__ tiles, bool cand_only,
                                                          float scale_log2) {
  constexpr int KLD = DH + 8, VLD = 64 + 8;
  __shared__ __attribute__((aligned(16))) bf16 sK[64 * KLD];
  __shared__ __attribute__((aligned(16))) bf16 sV[DH * VLD];
  const SelfTile tile = tiles[blockIdx.x];
  if (tile.q_count <= 0) return;
  const SelfReq rq = reqs[tile.req];
  const int h = tile.head, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, hi = lane >> 5;
  const int ld = 3 * d;
  const int qi = wave * 32 + l32;
  const bool wave_active = wave * 32 < tile.q_count;
  const int i = tile.q_begin + min(qi, tile.q_count - 1);
  bool is_cand;
  int row;
  if (cand_only) {
    is_cand = true;
    row = rq.c_row + i;
  } else {
    is_cand = i >= rq.S;
    row = is_cand ? rq.c_row + (i - rq.S) : rq.s_row + i;
  }
  const int visible = is_cand ? rq.S : i + 1;

  bf16x8 qf[DH / 16];
  {
    const bf16* qr = qkv + (size_t)row * ld + h * DH + 8 * hi;
#pragma unroll
    for (int kk = 0; kk < DH / 16; ++kk) qf[kk] = *reinterpret_cast<const bf16x8*>(qr + 16 * kk);
  }
  // a candidate's own key and value, fetched now so that their latency
  // overlaps the serving keys
  // (V in 16-byte pieces: lane hi takes the 8-feature group 2 p + hi of each
  // 16 features, and the halves the other lane of the query needs are
  // exchanged just before use, so each load covers 32 contiguous bytes of the
  // row instead of 16)
  bf16x8 kown[DH / 16];
  u32x4_t vraw[DH / 32][2] = {};
  if (is_cand) {
    const bf16* kr = qkv + (size_t)row * ld + d + h * DH + 8 * hi;
#pragma unroll
    for (int kk = 0; kk < DH / 16; ++kk) kown[kk] = *reinterpret_cast<const bf16x8*>(kr + 16 * kk);
    const bf16* vr = qkv + (size_t)row * ld + 2 * d + h * DH + 8 * hi;
#pragma unroll
    for (int db = 0; db < DH / 32; ++db)
#pragma unroll
      for (int p = 0; p < 2; ++p) vraw[db][p] = *reinterpret_cast<const u32x4_t*>(vr + 32 * db + 16 * p);
  }
  MfmaAcc<DH> acc;
  acc.init();

  for (int c0 = 0; c0 < rq.S; c0 += 64) {
    const int valid = rq.S - c0;
    // each thread moves a pair of adjacent keys x 8 features: K rows go to LDS
    // as they are; V is transposed with 4-byte writes (the two keys of a pair
    // stay adjacent in the permuted V^T order), 32 lanes filling one 128-byte
    // V^T row segment, so neither store has bank conflicts
#pragma unroll
    for (int u = 0; u < DH / 64; ++u) {
      const int c = tid + 256 * u;
      const int pair = c & 31, col = (c >> 5) * 8;
      const int k0 = 2 * pair;
      bf16x8 kv[2], vv[2];
#pragma unroll
      for (int w = 0; w < 2; ++w) {
        const size_t r = (size_t)(rq.s_row + c0 + min(k0 + w, valid - 1)) * ld + h * DH + col;
        kv[w] = *reinterpret_cast<const bf16x8*>(qkv + r + d);
        vv[w] = *reinterpret_cast<const bf16x8*>(qkv + r + 2 * d);
        if (k0 + w >= valid) {
#pragma unroll
          for (int t = 0; t < 8; ++t) vv[w][t] = (bf16)0.f;
        }
        *reinterpret_cast<bf16x8*>(&sK[(k0 + w) * KLD + col]) = kv[w];
      }
      const int vp = vt_col(k0);
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
        *reinterpret_cast<bf16x2*>(&sV[(col + t) * VLD + vp]) = bf16x2{vv[0][t], vv[1][t]};
      }
    }
    __syncthreads();
    if (wave_active)
      mfma_attend_tile<DH, KLD, VLD>(sK, sV, qf, acc, scale_log2, l32, hi, true,
                                     [&](int kl, float x) { return (c0 + kl < visible) ? x : -INFINITY; });
    __syncthreads();
  }

  if (is_cand) {
    // the candidate's own key: dot over this lane's half of the features, then
    // the other half from lane l ^ 32 (same query)
    float dot = 0.f;
#pragma unroll
    for (int kk = 0; kk < DH / 16; ++kk) {
      const bf16x8 kv = kown[kk];
#pragma unroll
      for (int t = 0; t < 8; ++t) dot = fmaf((float)qf[kk][t], (float)kv[t], dot);
    }
    dot = xor32_sum(dot);
    const float m_new = fmaxf(acc.m, dot);
    const float alpha = exp2f((acc.m - m_new) * scale_log2);
    const float pself = exp2f((dot - m_new) * scale_log2);
    acc.l = acc.l * alpha + pself;
    acc.m = m_new;
    // features 32 db + 8 gq + 4 hi .. + 3 of the own value: after swapping the
    // upper half of lane hi = 0's group with the lower half of lane hi = 1's,
    // dwords 0-1 of piece p hold group 2 p and dwords 2-3 group 2 p + 1
    bf16x4 vown[DH / 32][4];
#pragma unroll
    for (int db = 0; db < DH / 32; ++db)
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        u32x4_t w = vraw[db][p];
        const auto s0 = __builtin_amdgcn_permlane32_swap(w[0], w[2], false, false);
        const auto s1 = __builtin_amdgcn_permlane32_swap(w[1], w[3], false, false);
        const u32x2_t lo = {s0[0], s1[0]}, up = {s0[1], s1[1]};
        vown[db][2 * p] = __builtin_bit_cast(bf16x4, lo);
        vown[db][2 * p + 1] = __builtin_bit_cast(bf16x4, up);
      }
#pragma unroll
    for (int db = 0; db < DH / 32; ++db)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const bf16x4 v4 = vown[db][gq];
#pragma unroll
        for (int t = 0; t < 4; ++t) acc.o[db][4 * gq + t] = fmaf(pself, (float)v4[t], acc.o[db][4 * gq + t] * alpha);
      }
  }
  // The K/V tiles are free now (the loop ended on a barrier): waves 0-1 park
  // their output rows in sK, waves 2-3 in sV, and store them as
  // mfma_store_out_staged does (written out here: the helper's form of the
  // row mapping costs this kernel four spilled registers).
  constexpr int UPR = DH / 8;
  auto swz = [](int r) { return UPR == 16 ? (r & 15) : ((r >> 1) & 7); };
  bf16* stage = (wave < 2 ? sK : sV) + (wave & 1) * 32 * DH;
  {
    const float inv = acc.l > 0.f ? 1.f / acc.l : 0.f;
#pragma unroll
    for (int db = 0; db < DH / 32; ++db)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        bf16x4 w;
#pragma unroll
        for (int t = 0; t < 4; ++t) w[t] = (bf16)(acc.o[db][4 * gq + t] * inv);
        *reinterpret_cast<bf16x4*>(stage + l32 * DH + (((4 * db + gq) ^ swz(l32)) << 3) + 4 * hi) = w;
      }
  }
  constexpr int RPI = 64 / UPR;  // rows per read instruction
#pragma unroll
  for (int k = 0; k < 32 / RPI; ++k) {
    const int r = k * RPI + lane / UPR, q = lane % UPR;
    const bf16x8 v = *reinterpret_cast<const bf16x8*>(stage + r * DH + ((q ^ swz(r)) << 3));
    const int qr = wave * 32 + r;
    if (qr < tile.q_count) {
      const int ir = tile.q_begin + qr;
      const int orow = cand_only ? rq.c_row + ir : (ir >= rq.S ? rq.c_row + (ir - rq.S) : rq.s_row + ir);
      *reinterpret_cast<bf16x8*>(out + (size_t)orow * d + h * DH + q * 8) = v;
    }
  }
}

// ============================================================================
// Plain paged attention (fp32 models, head widths without an MFMA variant).
// 64 queries per block, 4 lanes per query, each lane owning dh/4 features;
// pages staged in LDS; keys processed one at a time with the online softmax.
// ============================================================================
template <typename T, int DH>
__global__ __launch_bounds__(256) void paged_attn_plain(const T* __restrict__ q, int ldq, T* __restrict__ out, int ldo,
                                                        const T* __restrict__ pool, const int32_t* __restrict__ page_table,
                                                        int max_pages, PageGeom g, int layer_slot,
                                                        const AttnReq* __restrict__ reqs,
                                                        const AttnTile* __restrict__ tiles, bool causal,
                                                        const float* __restrict__ rel, int R, float scale_log2) {
  constexpr int DP = DH / 4;
  __shared__ float sK[kPage][DH + 1];
  __shared__ float sV[DH][kPage + 1];
  const AttnTile tile = tiles[blockIdx.x];
  if (tile.q_count <= 0) return;
  const AttnReq rq = reqs[tile.req];
  const int h = tile.head, tid = threadIdx.x, qi = tid >> 2, part = tid & 3;
  const bool active = qi < tile.q_count;
  const int i = tile.q_begin + min(qi, tile.q_count - 1);
  const int row = i < rq.qa_n ? rq.qa_row + i : rq.qb_row + (i - rq.qa_n);
  const int qpos = rq.pos0 + i;

  float qv[DP], acc[DP];
#pragma unroll
  for (int e = 0; e < DP; ++e) {
    qv[e] = (float)q[(size_t)row * ldq + h * DH + part * DP + e];
    acc[e] = 0.f;
  }
  float m_run = -INFINITY, l_run = 0.f;
  const int kv_len = rq.kv_len;
  int n_pages = (kv_len + kPage - 1) / kPage;
  if (causal) n_pages = min(n_pages, (rq.pos0 + tile.q_begin + tile.q_count - 1) / kPage + 1);
  const int32_t* ptab = page_table + (size_t)rq.slot * max_pages;

  for (int p = 0; p < n_pages; ++p) {
    const size_t base = (size_t)ptab[p] * g.page_elems;
    const T* kp = pool + base + g.k_off(layer_slot, h);
    const T* vp = pool + base + g.v_off(layer_slot, h);
    const int valid = min(kPage, kv_len - p * kPage);
    for (int e = tid; e < kPage * DH; e += 256) {
      sK[e / DH][e % DH] = (float)kp[e];
      const int vr = e / kPage, key = vt_col(e % kPage);
      sV[vr][key] = key < valid ? (float)vp[e] : 0.f;
    }
    __syncthreads();
    if (active) {
      for (int j = 0; j < valid; ++j) {
        const int key = p * kPage + j;
        if (causal && key > qpos) break;
        float s = 0.f;
#pragma unroll
        for (int e = 0; e < DP; ++e) s = fmaf(qv[e], sK[j][part * DP + e], s);
        s = quad_sum(s);  // the query's four lanes
        s *= scale_log2;
        if (causal && R > 0) s += rel[h * R + min(qpos - key, R - 1)] * kLog2e;
        const float m_new = fmaxf(m_run, s);
        const float alpha = exp2f(m_run - m_new);
        const float pj = exp2f(s - m_new);
        l_run = l_run * alpha + pj;
#pragma unroll
        for (int e = 0; e < DP; ++e) acc[e] = fmaf(pj, sV[part * DP + e][j], acc[e] * alpha);
        m_run = m_new;
      }
    }
    __syncthreads();
  }
  if (active) {
    const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
#pragma unroll
    for (int e = 0; e < DP; ++e) out[(size_t)row * ldo + h * DH + part * DP + e] = (T)(acc[e] * inv);
  }
}

int paged_attention_q_block(bool bf, int dh) { return (bf && (dh == 64 || dh == 128)) ? 128 : 64; }

hipError_t launch_paged_attention(bool bf, const void* q, int ldq, void* out, int ldo, const void* pool,
                                  const int32_t* page_table, int max_pages, PageGeom g, int layer_slot,
                                  const AttnReq* reqs, const AttnTile* tiles, int n_tiles, bool causal,
                                  const float* rel, int R, int q_block, hipStream_t s) {
  if (n_tiles <= 0) return hipSuccess;
  const float sl2 = kLog2e / sqrtf((float)g.dh);
  if (q_block == kDecodeQBlock && causal && paged_attention_decode_ok(bf, g.dh, R)) {
    const bf16* qq = (const bf16*)q;
    bf16* oo = (bf16*)out;
    const bf16* pp = (const bf16*)pool;
    const unsigned blocks = (unsigned)((n_tiles + 3) / 4);
#define TX_PD(DH, CZ)                                                                                              \
  paged_attn_decode<DH, CZ><<<blocks, 256, 0, s>>>(qq, ldq, oo, ldo, pp, page_table, max_pages, g, layer_slot, reqs, \
                                                    tiles, n_tiles, rel, R, sl2)
    if (g.dh == 64) TX_PD(64, true); else TX_PD(128, true);
#undef TX_PD
    return hipGetLastError();
  }
  if (q_block != paged_attention_q_block(bf, g.dh)) return hipErrorInvalidValue;
  if (bf && (g.dh == 64 || g.dh == 128)) {
    const bf16* qq = (const bf16*)q;
    bf16* oo = (bf16*)out;
    const bf16* pp = (const bf16*)pool;
#define TX_PA(DH, CZ)                                                                                              \
  paged_attn_mfma<DH, CZ><<<n_tiles, 256, 0, s>>>(qq, ldq, oo, ldo, pp, page_table, max_pages, g, layer_slot, reqs, \
                                                   tiles, rel, R, sl2)
    if (g.dh == 64) {
      if (causal) TX_PA(64, true); else TX_PA(64, false);
    } else {
      if (causal) TX_PA(128, true);
      else TX_PA(128, false);
    }
#undef TX_PA
    return hipGetLastError();
  }
#define TX_PP(T, DH)                                                                                              \
  paged_attn_plain<T, DH><<<n_tiles, 256, 0, s>>>((const T*)q, ldq, (T*)out, ldo, (const T*)pool, page_table,     \
                                                  max_pages, g, layer_slot, reqs, tiles, causal, rel, R, sl2)
  if (bf) {
    if (g.dh == 32) TX_PP(bf16, 32); else if (g.dh == 64) TX_PP(bf16, 64); else if (g.dh == 128) TX_PP(bf16, 128);
    else return hipErrorInvalidValue;
  } else {
    if (g.dh == 32) TX_PP(float, 32); else if (g.dh == 64) TX_PP(float, 64); else if (g.dh == 128) TX_PP(float, 128);
    else return hipErrorInvalidValue;
  }
#undef TX_PP
  return hipGetLastError();
}

// ============================================================================
// Decoder self-attention (App. B mask). 64 queries per block, 4 lanes per
// query. Serving keys/values are staged 64 at a time in LDS; a candidate then
// adds its own key/value, read from its row.
// ============================================================================
template <typename T, int DH>
__global__ __launch_bounds__(256) void self_attn_plain(const T* __restrict__ qkv, int d, T* __restrict__ out,
                                                       const SelfReq* __restrict__ reqs,
                                                       const SelfTile* __restrict__ tiles, bool cand_only,
                                                       float scale_log2) {
  constexpr int DP = DH / 4;
  __shared__ float sK[64][DH + 1];
  __shared__ float sV[64][DH + 1];
  const SelfTile tile = tiles[blockIdx.x];
  if (tile.q_count <= 0) return;
  const SelfReq rq = reqs[tile.req];
  const int h = tile.head, tid = threadIdx.x, qi = tid >> 2, part = tid & 3;
  const int ld = 3 * d;
  const bool active = qi < tile.q_count;
  const int i = tile.q_begin + min(qi, tile.q_count - 1);
  bool is_cand;
  int row;
  if (cand_only) {
    is_cand = true;
    row = rq.c_row + i;
  } else {
    is_cand = i >= rq.S;
    row = is_cand ? rq.c_row + (i - rq.S) : rq.s_row + i;
  }
  const int visible = is_cand ? rq.S : i + 1;  // serving keys this query sees

  float qv[DP], acc[DP];
#pragma unroll
  for (int e = 0; e < DP; ++e) {
    qv[e] = (float)qkv[(size_t)row * ld + h * DH + part * DP + e];
    acc[e] = 0.f;
  }
  float m_run = -INFINITY, l_run = 0.f;
  auto consume = [&](float s, const float* vrow_part, int vstride) {
    s = quad_sum(s);  // the query's four lanes
    s *= scale_log2;
    const float m_new = fmaxf(m_run, s);
    const float alpha = exp2f(m_run - m_new);
    const float pj = exp2f(s - m_new);
    l_run = l_run * alpha + pj;
#pragma unroll
    for (int e = 0; e < DP; ++e) acc[e] = fmaf(pj, vrow_part[e * vstride], acc[e] * alpha);
    m_run = m_new;
  };

  for (int c0 = 0; c0 < rq.S; c0 += 64) {
    const int nk = min(64, rq.S - c0);
    for (int e = tid; e < nk * DH; e += 256) {
      const int j = e / DH, f = e % DH;
      const size_t r = (size_t)(rq.s_row + c0 + j) * ld;
      sK[j][f] = (float)qkv[r + d + h * DH + f];
      sV[j][f] = (float)qkv[r + 2 * d + h * DH + f];
    }
    __syncthreads();
    if (active) {
      const int jmax = min(nk, visible - c0);
      for (int j = 0; j < jmax; ++j) {
        float s = 0.f;
#pragma unroll
        for (int e = 0; e < DP; ++e) s = fmaf(qv[e], sK[j][part * DP + e], s);
        consume(s, &sV[j][part * DP], 1);
      }
    }
    __syncthreads();
  }
  if (active && is_cand) {
    float kv[DP], vv[DP];
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < DP; ++e) {
      kv[e] = (float)qkv[(size_t)row * ld + d + h * DH + part * DP + e];
      vv[e] = (float)qkv[(size_t)row * ld + 2 * d + h * DH + part * DP + e];
      s = fmaf(qv[e], kv[e], s);
    }
    consume(s, vv, 1);
  }
  if (active) {
    const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
#pragma unroll
    for (int e = 0; e < DP; ++e) out[(size_t)row * d + h * DH + part * DP + e] = (T)(acc[e] * inv);
  }
}

int self_attention_q_block(bool bf, int dh) { return (bf && (dh == 64 || dh == 128)) ? 128 : 64; }

hipError_t launch_self_attention(bool bf, const void* qkv, int d, int H, void* out, const SelfReq* reqs,
                                 const SelfTile* tiles, int n_tiles, bool candidates_only, hipStream_t s) {
  if (n_tiles <= 0) return hipSuccess;
  const int dh = d / H;
  const float sl2 = kLog2e / sqrtf((float)dh);
  if (bf && (dh == 64 || dh == 128)) {
    if (dh == 64)
      self_attn_mfma<64><<<n_tiles, 256, 0, s>>>((const bf16*)qkv, d, (bf16*)out, reqs, tiles, candidates_only, sl2);
    else
      self_attn_mfma<128><<<n_tiles, 256, 0, s>>>((const bf16*)qkv, d, (bf16*)out, reqs, tiles, candidates_only, sl2);
    return hipGetLastError();
  }
#define TX_SA(T, DH)                                                                                             \
  self_attn_plain<T, DH><<<n_tiles, 256, 0, s>>>((const T*)qkv, d, (T*)out, reqs, tiles, candidates_only, sl2)
  if (bf) {
    if (dh == 32) TX_SA(bf16, 32); else if (dh == 64) TX_SA(bf16, 64); else if (dh == 128) TX_SA(bf16, 128);
    else return hipErrorInvalidValue;
  } else {
    if (dh == 32) TX_SA(float, 32); else if (dh == 64) TX_SA(float, 64); else if (dh == 128) TX_SA(float, 128);
    else return hipErrorInvalidValue;
  }
#undef TX_SA
  return hipGetLastError();
}

}  // namespace tx
