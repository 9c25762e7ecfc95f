// Forward pass on gfx950 matrix cores (bf16 data, head_dim 64 or 128, w2 <= 64).
//
// Formulation. The trilinear logit of Section 4, Eq. (3d-attention), factors as
//     A[i,j,k] = < scale * q_i o k'_k , k_j >,
// so every pair r = (i, k) with k in (i-w2, i] is a "row" with the modulated
// query q~_r = scale * q_i o k'_k, and its key window j in (i-w1, i] depends on
// i only. The joint softmax of Eq. (softmax) over (j, k) is a per-row online
// softmax over j followed by a log-sum-exp merge of the w2 rows of a query:
//     U_r = sum_j 2^(s_rj - m_r) v_j,  l_r = sum_j 2^(s_rj - m_r)      (s in log2 units)
//     LSE_i = log sum_k l_r 2^(m_r),  O_i = sum_k 2^(m_r - LSE_i) v'_k o U_r
// which is Eq. (attenval) regrouped. Both contractions are matrix products:
// S^T = K_blk q~^T (over d) and U^T += V_blk^T P^T (over j), bf16 MFMA with fp32
// accumulation. Elementwise work is only w2*D per query (forming q~), versus
// w1*D for the pairwise q o k_j product of the paper's Figure 2 tiling.
//
// Tiling. A workgroup of 4 wavefronts owns QW consecutive queries of one
// (batch, head); each wavefront owns 32 rows (one query's 32 k-rows; w2 = 64
// uses two wavefronts per query). All accumulators live in VGPRs so that two
// workgroups share a CU (two wavefronts per SIMD). The j-window union of the
// workgroup is walked in 32-key blocks through a 4-stage ring of swizzled
// row-major K/V tiles in LDS; K fragments are read row-wise, V fragments with
// the gfx950 transposing LDS read (no transposed copy of V).
//
// Pipeline. K and V blocks go from HBM/L2 straight into LDS (buffer loads
// with an LDS destination, 16 bytes per lane), each into its own 4-stage
// ring, so no VGPRs are spent on staging and the loads run 2-3 iterations
// ahead. Iteration n of the loop
//   - issues the loads of K(n+4) and V(n+3),
//   - masks and takes the running maximum of S(n), exponentiates and packs
//     P(n), while the matrix cores compute S(n+1) from K fragments that were
//     read one iteration earlier,
//   - accumulates P(n) V(n) while the K fragments of block n+2 are read.
// The last block's iteration is a separate copy without the products of a
// block after it (which would be discarded).
// With w2 <= 32 the prologue brings the workgroup's k' and q rows into a
// staging tile with the same LDS-DMA loads and forms q~ from LDS (one 16-byte
// load per row instead of per-wavefront register loads of overlapping rows),
// waits only for K(0) and K(1) before the first products and issues V(1),
// K(3), V(2) behind them; the staging tile then receives the v' rows. Tiles
// whose key window lies inside the sequence skip the per-block bounds test:
// the loop is bound by instruction issue, scalar instructions included.
// The iteration is unrolled over the 4 ring stages so every LDS address is a
// per-lane base plus an immediate; each stage is a separate LDS array so the
// compiler's wait for a stage's loads does not also wait for the others. Within a wavefront all rows share one
// query, so a block is fully valid or masked by column only; masked columns
// are set to -inf before the maximum.
// The running maximum m is raised lazily: P(n) is formed with the current m
// and only if some row's block sum of p leaves (0, 2^16] (p far from fp32
// overflow) is m raised to the block maximum and P(n) formed again; after the
// first block with a valid column this is rare, and the per-block maximum is
// not computed otherwise. The row sum l adds the bf16-rounded p that the P V
// product consumes, so O is a convex combination of V rows.
// Rows with k < 0 or k <= i - w2 get q~ = 0 and weight 0 in the merge.
#include "fwd_schedule.h"
#include "mfma_common.h"

namespace sa {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kStages = fwd_schedule::kStages;
constexpr float kPmax = 65536.0f;  // largest block row sum of p before the running max is raised

template <int X>
using IC = std::integral_constant<int, X>;

// s_waitcnt vmcnt(N) with the other counters left alone (gfx9 encoding:
// vmcnt low bits 3:0, high bits 15:14; expcnt 6:4 = 7, lgkmcnt 11:8 = 15).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}


// FORM 0: trilinear logits (Section 4); FORM 1: determinant logits (Section 5,
// w2 <= 32 only), which differ only in the modulated query formed below.
// BIAS: K' and V' values get the constants s.kp_bias / s.vp_bias added on load.
// HF (grouped-query attention with a multiple of 4 query heads per K-side
// head, w2 <= 32): the 4 wavefronts take 4 query heads of one K-side head at
// the same position i instead of 4 consecutive positions of one head, so they
// share one key window: ceil(w1 / 32) blocks with no masked columns away from
// the start of the sequence (the query-head tiling of Section 6).
template <int D, int G, int FORM, bool BIAS, bool HF>
__global__ __launch_bounds__(kThreads, 2) void fwd_mfma_kernel(Shape s, const uint16_t* __restrict__ q,
                                                               const uint16_t* __restrict__ k,
                                                               const uint16_t* __restrict__ kp,
                                                               const uint16_t* __restrict__ v,
                                                               const uint16_t* __restrict__ vp,
                                                               uint16_t* __restrict__ out,
                                                               float* __restrict__ lse) {
  constexpr int NT = D / 16;     // K-steps of the logit product
  constexpr int NDT = D / 32;    // 32-wide d tiles of the output product
  constexpr int QW = kWaves / G; // queries per workgroup
  constexpr int W2P = 32 * G;    // rows per query (w2 padded up to a multiple of 32)
  using T = SwzTile<D>;
  __shared__ __attribute__((aligned(16))) char kst0[T::bytes], kst1[T::bytes], kst2[T::bytes], kst3[T::bytes];
  __shared__ __attribute__((aligned(16))) char vst0[T::bytes], vst1[T::bytes], vst2[T::bytes], vst3[T::bytes];
  // Staging tile (w2 <= 32): rows 0 .. KR-1 hold k'_k for k = i0-31 ... (35
  // needed) and rows KR .. KR+3 the workgroup's q rows until q~ is formed;
  // from the first iteration on rows 0 .. 34 hold v'_k of the same k for the
  // epilogue. Rows of 2D bytes, 16-byte chunk ch of row r at slot ch ^ (r % CH).
  constexpr int KI = (35 * T::CH + 63) / 64;  // 64-lane loads of 35 rows
  constexpr int KR = KI * 64 / T::CH;         // rows they cover
  constexpr int SR = KR + 64 / T::CH;         // + one 64-lane load of q rows
  __shared__ __attribute__((aligned(16))) char stg[G == 1 ? SR * 2 * D : 16];
  __shared__ float stat[G == 1 ? 1 : kWaves * 32];
  __shared__ float xchg[G == 1 ? 1 : kWaves * 64 * (D / 64)];
  auto kst = [&](auto SC) __attribute__((always_inline)) {
    constexpr int X = decltype(SC)::value;
    return to_lds(X == 0 ? kst0 : X == 1 ? kst1 : X == 2 ? kst2 : kst3);
  };
  auto vst = [&](auto SC) __attribute__((always_inline)) {
    constexpr int X = decltype(SC)::value;
    return to_lds(X == 0 ? vst0 : X == 1 ? vst1 : X == 2 ? vst2 : vst3);
  };

  // XCD-aware tile order: hardware deals workgroups round-robin over the 8
  // XCDs; remap so each XCD walks a contiguous run of tiles of one head and
  // the overlapping K/V windows of neighbouring tiles hit the same L2.
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63, c = lane & 31, h = lane >> 5;
  const int qs = wave / G, g = wave % G;
  static_assert(!HF || G == 1, "head-folded tiles take one wavefront per query");
  // Q-side tensors (q, out) have H heads; K-side ones (k, k', v, v') Hkv,
  // query head hh reading K-side head hk = hh / (H / Hkv) (grouped-query
  // attention; Hkv == H otherwise). A tile is QW consecutive queries of one
  // head, or (HF) QW query heads hq0 .. hq0 + QW - 1 of one K-side head at one
  // position; tiles sharing K / V rows are adjacent in the XCD order below.
  int b, hk, hh, i0, hq0 = 0;
  {
    const int per_bh = HF ? s.N * (s.H / s.Hkv / QW) : (s.N + QW - 1) / QW;
    const int total = per_bh * s.B * (HF ? s.Hkv : s.H);
    const int per_xcd = (total + 7) / 8;
    const int logical = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
    if (logical >= total) return;
    const int bhx = logical / per_bh;
    const int tile = logical - bhx * per_bh;
    if constexpr (HF) {
      const int quads = s.H / s.Hkv / QW;
      b = bhx / s.Hkv;
      hk = bhx - b * s.Hkv;
      i0 = tile / quads;
      hq0 = hk * (s.H / s.Hkv) + (tile - i0 * quads) * QW;
      hh = hq0 + qs;
    } else {
      b = bhx / s.H;
      hh = bhx - b * s.H;
      hk = hh / (s.H / s.Hkv);
      i0 = tile * QW;
    }
  }
  const int bh = b * s.H + hh;  // query head row of lse
  const int qoff = HF ? 0 : qs;  // position of this wavefront's query after i0
  const size_t rs = static_cast<size_t>(s.H) * D;
  const size_t base = (static_cast<size_t>(b) * s.N * s.H + hh) * D;
  const size_t rskv = static_cast<size_t>(s.Hkv) * D;
  const size_t kvbase = (static_cast<size_t>(b) * s.N * s.Hkv + hk) * D;
  const int N = s.N, w1 = s.w1, w2 = s.w2;
  const int i = i0 + qoff;
  const bool qvalid = i < N;

  const int kk = i - W2P + 1 + 32 * g + c;
  const bool rowvalid = qvalid && kk >= 0 && kk > i - w2;
  const float qscale = s.scale * kLog2e;

  const int jlo = i0 - w1 + 1;
  const int nb = (w1 + (HF ? 0 : QW - 1) + 31) / 32;
  const int rsbq = static_cast<int>(rs) * 2;     // bytes between rows of q, out
  const int rsb = static_cast<int>(rskv) * 2;    // bytes between rows of k, k', v, v'
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(k + kvbase, head_bytes(N, rsb, D));
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(v + kvbase, head_bytes(N, rsb, D));

  // Per-lane LDS byte offsets inside a tile. K row fragment t: row c,
  // columns 16t + 8h .. + 7. Transposed V fragment (dt, u): two
  // ds_read_b64_tr_b16 at vo[dt][0] and vo[dt][1] plus 32 D u (16 rows on).
  int ko[NT], vo[NDT][2];
#pragma unroll
  for (int t = 0; t < NT; ++t) ko[t] = T::off(c, 2 * t + h);
  {
    const int grp = lane >> 4, sl = lane & 15;
    const int r0 = 4 * (grp >> 1) + (sl >> 2);
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      const int col = 32 * dt + 16 * (grp & 1) + 4 * (sl & 3);
      const int ch = col >> 3, within = (col & 7) * 2;
      vo[dt][0] = T::off(r0, ch) + within;
      vo[dt][1] = T::off(r0 + 8, ch) + within;
    }
  }
  auto kfrag = [&](auto SC, int t) __attribute__((always_inline)) {
    return lds_ld<u32x4_t>(kst(SC) + ko[t]);
  };
  auto vfrag = [&](auto SC, int dt, int u) __attribute__((always_inline)) {
    const lds_char* p = vst(SC) + 32 * D * u;
    const u32x2_t a = lds_tr16(p + vo[dt][0]);
    const u32x2_t bb = lds_tr16(p + vo[dt][1]);
    return u32x4_t{a[0], a[1], bb[0], bb[1]};
  };

  // Block loads: wavefront x-th share of a 32 x D tile is the 1 KB at
  // 1024 (x kWaves + wave) of the tile, lane l supplying the 16-byte chunk at
  // offset 16 l of it (row p / CH, swizzled chunk of p = 64 (x kWaves + wave)
  // + l). The hardware writes lane l's chunk to the LDS address given plus
  // 16 l. Rows outside [0, N) are loaded from the clamped row: they are
  // masked (p = 0), and finite data keeps 0 * v finite.
  constexpr int SPW = (T::instrs + kWaves - 1) / kWaves;  // loads per tile per wavefront
  // Every wavefront issues exactly SPW loads per tile (head_dim 64: 4 loads,
  // 128: 8, over 4 wavefronts), so each vmcnt wait below, which counts the
  // issuing wavefront's own loads, holds for every wavefront.
  static_assert(T::instrs % kWaves == 0, "tile loads must divide evenly over the wavefronts");
  auto wait_tiles = [&](auto NC) __attribute__((always_inline)) {
    wait_vmcnt<decltype(NC)::value * SPW>();  // that many tiles' loads may stay in flight
  };
  int lrow[SPW], lcol[SPW];
#pragma unroll
  for (int x = 0; x < SPW; ++x) {
    const int kx = x * kWaves + wave;
    const int p = 64 * kx + lane;
    lrow[x] = p / T::CH;
    lcol[x] = 16 * ((p % T::CH) ^ T::swz(lrow[x]));
  }
  // Tiles whose whole key window lies inside the sequence (all but the first
  // and last few of each head) skip the per-block bounds test.
  const bool interior = jlo >= 0 && jlo + 32 * nb <= N;
  auto load_tile = [&](__amdgpu_buffer_rsrc_t r, lds_char* dst, int blk) __attribute__((always_inline)) {
    const int jb = jlo + 32 * blk;
    if (interior || (jb >= 0 && jb + 31 < N)) {
      // Block inside the sequence: the block's row offset goes in the
      // scalar offset, the lane's offset within the block is fixed.
#pragma unroll
      for (int x = 0; x < SPW; ++x) {
        const int kx = x * kWaves + wave;
        if (T::instrs % kWaves == 0 || kx < T::instrs)
          load_lds16(r, dst + 1024 * kx, lrow[x] * rsb + lcol[x], jb * rsb);
      }
    } else {
#pragma unroll
      for (int x = 0; x < SPW; ++x) {
        const int kx = x * kWaves + wave;
        const int row = min(max(jb + lrow[x], 0), N - 1);
        if (T::instrs % kWaves == 0 || kx < T::instrs) load_lds16(r, dst + 1024 * kx, row * rsb + lcol[x]);
      }
    }
  };
  const __amdgpu_buffer_rsrc_t rq = make_rsrc(q + base, head_bytes(N, rsbq, D));
  const __amdgpu_buffer_rsrc_t rkp = make_rsrc(kp + kvbase, head_bytes(N, rsb, D));
  const __amdgpu_buffer_rsrc_t rvp = make_rsrc(vp + kvbase, head_bytes(N, rsb, D));
  const int kk0 = i0 - 31;  // first k of the staged k' / v' rows (w2 <= 32)
  // 64-lane loads x of staging rows: row r of the 64 x 16 bytes is p / CH
  // for p = 64 x + lane, its chunk goes to slot (p % CH) ^ (r % CH).
  auto stage = [&](__amdgpu_buffer_rsrc_t r, int rstride, int x, int row0) __attribute__((always_inline)) {
    const int p = 64 * x + lane, rr = p / T::CH;
    const int ch = (p % T::CH) ^ (rr % T::CH);
    const int row = min(max(row0 + rr, 0), N - 1);
    load_lds16(r, to_lds(stg) + 1024 * x, row * rstride + 16 * ch);
  };
  u32x4_t qt[NT];
  if constexpr (G == 1) {
    // The workgroup's k' rows and q rows go to the staging tile, then the
    // blocks the first products and iteration 0 need: K(0), K(1), V(0), K(2).
    // V(1), K(3), V(2) follow once S(0) is under way, so that the wait of
    // every iteration below (K(blk + 2) and V(blk) loaded) holds from the
    // first one on. Blocks past the window only cost the loads.
#pragma unroll
    for (int x = wave; x < KI + 1; x += kWaves) {
      if (x < KI) {
        stage(rkp, rsb, x, kk0);
      } else if constexpr (HF) {
        // q rows of the QW heads at position i0: contiguous, QW * 2D bytes
        // (a resource of exactly that size zero-fills the rest of the load).
        const __amdgpu_buffer_rsrc_t rqh = make_rsrc(q + (static_cast<size_t>(b) * N + i0) * rs +
                                                     static_cast<size_t>(hq0) * D, QW * 2 * D);
        const int rr = lane / T::CH;
        const int ch = (lane % T::CH) ^ ((KR + rr) % T::CH);
        load_lds16(rqh, to_lds(stg) + 1024 * x, rr * 2 * D + 16 * ch);
      } else {
        stage(rq, rsbq, x, i0 - KR);
      }
    }
    load_tile(rk, kst(IC<0>{}), 0);
    load_tile(rk, kst(IC<1>{}), 1);
    load_tile(rv, vst(IC<0>{}), 0);
    load_tile(rk, kst(IC<2>{}), 2);
  } else {
    // Blocks 0-3 of K and 0-2 of V go out before the q~ loads, so their
    // latencies overlap (blocks past the window only cost the loads).
    load_tile(rk, kst(IC<0>{}), 0);
    load_tile(rk, kst(IC<1>{}), 1);
    load_tile(rk, kst(IC<2>{}), 2);
    load_tile(rk, kst(IC<3>{}), 3);
    load_tile(rv, vst(IC<0>{}), 0);
    load_tile(rv, vst(IC<1>{}), 1);
    load_tile(rv, vst(IC<2>{}), 2);
    // modulated queries q~ = (scale*log2 e) * q_i o k'_k as B operands
    // (rows outside the window or the sequence load as zeros: offset -1)
    u32x4_t qa[NT], ka[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      qa[t] = ldbuf128(rq, rowvalid ? i * rsbq + 32 * t + 16 * h : -1);
      ka[t] = ldbuf128(rkp, rowvalid ? kk * rsb + 32 * t + 16 * h : -1);
    }
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        qt[t][e] = pack_bf16x2(bf16_lo(qa[t][e]) * plus_bias<BIAS>(bf16_lo(ka[t][e]), s.kp_bias) * qscale,
                               bf16_hi(qa[t][e]) * plus_bias<BIAS>(bf16_hi(ka[t][e]), s.kp_bias) * qscale);
  }

  f32x16_t acc[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) acc[dt] = f32x16_t{};
  // Running row maximum m and sum l (log2 units; logits come out of the
  // products unshifted and p = 2^(s - m)). m starts finite so that a block
  // masked entirely (s = -inf) before any valid one gives p = 0, not NaN;
  // the first block with a valid column always raises it.
  float m = -1e30f, l = 0.f;
  f32x16_t sc[2];
  u32x4_t kf[NT];
  auto logits = [&](f32x16_t& dst) __attribute__((always_inline)) {
    dst = mfma32(kf[0], qt[0], f32x16_t{});
#pragma unroll
    for (int t = 1; t < NT; ++t) dst = mfma32(kf[t], qt[t], dst);
  };

  if constexpr (G == 1) {
    // Staging rows, K(0) and K(1) in LDS for every wavefront; V(0) and K(2)
    // may still be in flight.
    wait_tiles(IC<2>{});
    lds_barrier_tracked();
    // modulated queries q~ = (scale*log2 e) * q_i o k'_k as B operands, from
    // the staged rows (local k' row qs + c, q row KR + qs); rows outside the
    // window or the sequence are zero.
    const int rr = qoff + c, rq_ = KR + qs;
    const lds_char* krow = to_lds(stg) + rr * 2 * D;
    const lds_char* qrow = to_lds(stg) + rq_ * 2 * D;
    const unsigned keep = rowvalid ? 0xFFFFFFFFu : 0u;
    if constexpr (FORM == 0) {
      u32x4_t qa[NT], ka[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const int ch = 2 * t + h;
        ka[t] = lds_ld<u32x4_t>(krow + 16 * (ch ^ (rr % T::CH)));
        qa[t] = lds_ld<u32x4_t>(qrow + 16 * (ch ^ (rq_ % T::CH)));
      }
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          qt[t][e] = keep & pack_bf16x2(bf16_lo(qa[t][e]) * plus_bias<BIAS>(bf16_lo(ka[t][e]), s.kp_bias) * qscale,
                                        bf16_hi(qa[t][e]) * plus_bias<BIAS>(bf16_hi(ka[t][e]), s.kp_bias) * qscale);
    } else {
      // Determinant logits: per 3-component chunk, det([q; k; k']) =
      // k . (k' x q), so q~ = (scale log2 e) * (k'_k x q_i) chunk by chunk and
      // <q~, k_j> is the logit. The lane's fragment t holds components
      // 8 ch .. 8 ch + 7 (ch = 2t + h); a chunk reaches at most 2 components
      // into the neighbouring 16-byte slots, read as 4-byte words (clamped at
      // the row ends, where they are not used). Components past the last whole
      // chunk (D mod 3 of them) are 0.
      constexpr int DC = 3 * (D / 3);
      const int swk = rr % T::CH, swq = rq_ % T::CH;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const int ch = 2 * t + h;
        const int chp = ch > 0 ? ch - 1 : 0, chn = ch < T::CH - 1 ? ch + 1 : ch;
        const u32x4_t kc = lds_ld<u32x4_t>(krow + 16 * (ch ^ swk));
        const u32x4_t qc = lds_ld<u32x4_t>(qrow + 16 * (ch ^ swq));
        const unsigned kw[2] = {lds_ld<unsigned>(krow + 16 * (chp ^ swk) + 12),
                                lds_ld<unsigned>(krow + 16 * (chn ^ swk))};
        const unsigned qw[2] = {lds_ld<unsigned>(qrow + 16 * (chp ^ swq) + 12),
                                lds_ld<unsigned>(qrow + 16 * (chn ^ swq))};
        // window x = 0 .. 11 holds components 8 ch - 2 .. 8 ch + 9
        float fk[12], fq[12];
        const float kb = s.kp_bias;
        fk[0] = plus_bias<BIAS>(bf16_lo(kw[0]), kb), fk[1] = plus_bias<BIAS>(bf16_hi(kw[0]), kb);
        fk[10] = plus_bias<BIAS>(bf16_lo(kw[1]), kb), fk[11] = plus_bias<BIAS>(bf16_hi(kw[1]), kb);
        fq[0] = bf16_lo(qw[0]), fq[1] = bf16_hi(qw[0]), fq[10] = bf16_lo(qw[1]), fq[11] = bf16_hi(qw[1]);
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          fk[2 + 2 * w] = plus_bias<BIAS>(bf16_lo(kc[w]), kb);
          fk[3 + 2 * w] = plus_bias<BIAS>(bf16_hi(kc[w]), kb);
          fq[2 + 2 * w] = bf16_lo(qc[w]), fq[3 + 2 * w] = bf16_hi(qc[w]);
        }
        // component e of the fragment sits at position m of its chunk, which
        // starts at window index e + 2 - m; m = (8 ch + e) mod 3 = (t + 2h + e) mod 3.
        auto cross = [&](int e, int m) __attribute__((always_inline)) {
          const int b = e + 2 - m;
          return m == 0 ? fk[b + 1] * fq[b + 2] - fk[b + 2] * fq[b + 1]
               : m == 1 ? fk[b + 2] * fq[b] - fk[b] * fq[b + 2]
                        : fk[b] * fq[b + 1] - fk[b + 1] * fq[b];
        };
        float cr[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float x = h == 0 ? cross(e, (t + e) % 3) : cross(e, (t + 2 + e) % 3);
          cr[e] = 8 * ch + e < DC ? x * qscale : 0.f;
        }
#pragma unroll
        for (int w = 0; w < 4; ++w) qt[t][w] = keep & pack_bf16x2(cr[2 * w], cr[2 * w + 1]);
      }
    }
  } else {
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wavefront's block loads are in LDS
    lds_barrier();
  }
#pragma unroll
  for (int t = 0; t < NT; ++t) kf[t] = kfrag(IC<0>{}, t);
  __builtin_amdgcn_sched_barrier(0);  // all fragment reads ahead of the products
  logits(sc[0]);
  if constexpr (G == 1) {
    load_tile(rv, vst(IC<1>{}), 1);
    load_tile(rk, kst(IC<3>{}), 3);
    load_tile(rv, vst(IC<2>{}), 2);
  }
#pragma unroll
  for (int t = 0; t < NT; ++t) kf[t] = kfrag(IC<1>{}, t);

  const bf16x2_t ones = {static_cast<__bf16>(1.0f), static_cast<__bf16>(1.0f)};
  auto iteration = [&](auto SC, int blk, auto LASTC) __attribute__((always_inline)) {
    constexpr int S = decltype(SC)::value;  // ring stage of block blk
    constexpr bool LAST = decltype(LASTC)::value;  // blk == nb - 1: no S(blk + 1)
    constexpr int cur = S & 1, nxt = cur ^ 1;
    // K(blk + 2) (loaded in iteration blk - 2) and V(blk) (iteration
    // blk - 3) must be in LDS for every wavefront: wait until at most the
    // loads this wavefront issued after them are in flight (3 tiles in
    // steady state, fewer in the last three iterations, where the ring
    // issues no more loads), then synchronise.
    switch (fwd_schedule::inflight_tiles(blk, nb)) {
      case 3: wait_tiles(IC<3>{}); break;
      case 2: wait_tiles(IC<2>{}); break;
      case 1: wait_tiles(IC<1>{}); break;
      default: wait_tiles(IC<0>{}); break;
    }
    lds_barrier_tracked();
    // K(blk + 4) replaces K(blk), read in iteration blk - 2; V(blk + 3)
    // replaces V(blk - 1), read in iteration blk - 1.
    if (fwd_schedule::loads_k(blk, nb)) load_tile(rk, kst(IC<S>{}), blk + 4);
    if (fwd_schedule::loads_v(blk, nb)) load_tile(rv, vst(IC<(S + 3) % kStages>{}), blk + 3);
    if constexpr (G == 1 && S == 0) {
      // v' rows into the staging tile, whose q and k' rows every wavefront
      // has read before the barrier above.
      if (blk == 0) {
#pragma unroll
        for (int x = wave; x < KI; x += kWaves) stage(rvp, rsb, x, kk0);
      }
    }
    // V(blk) fragments, in flight while S(blk + 1) and P(blk) are formed.
    u32x4_t vf[2][NDT];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) vf[u][dt] = vfrag(SC, dt, u);

    // Valid block-local columns of this wavefront's query.
    const int lo = max(qoff, -jlo) - 32 * blk;
    const int hi = min(qoff + w1 - 1, N - 1 - jlo) - 32 * blk;
    if (lo > 0 || hi < 31) {
#pragma unroll
      for (int vv = 0; vv < 16; ++vv) {
        const int jl = acc_row(vv, h);
        if (jl < lo || jl > hi) sc[cur][vv] = -INFINITY;
      }
    }
    // P(blk) on the vector units while the matrix cores form S(blk + 1).
    // From here to the end of the block this wavefront issues ahead of the
    // other one on its SIMD while that one is at the barrier or issuing its
    // loads (wavefront priority 1; back to 0 at the end of the block).
    __builtin_amdgcn_s_setprio(1);
    if constexpr (!LAST) logits(sc[nxt]);
    u32x4_t pf[2];
    float lb = 0.f;
    auto form_p = [&]() __attribute__((always_inline)) {
      lb = 0.f;
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const unsigned pp =
              pack_bf16x2(fast_exp2(sc[cur][8 * u + 2 * e] - m), fast_exp2(sc[cur][8 * u + 2 * e + 1] - m));
          pf[u][e] = pp;
          lb = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, pp), ones, lb, false);
        }
    };
    form_p();
    // The running maximum is raised only when some row's block sum leaves
    // (0, kPmax] (always on the first block with a valid column, where
    // m = -1e30 makes p = inf): then m becomes the block maximum, the state
    // is rescaled and P(blk) is formed again.
    if (__builtin_amdgcn_ballot_w64(!(lb <= kPmax)) != 0) {
      float mx = fmaxf(sc[cur][0], sc[cur][1]);
#pragma unroll
      for (int vv = 2; vv < 16; vv += 2) mx = fmaxf(fmaxf(mx, sc[cur][vv]), sc[cur][vv + 1]);
      mx = fmaxf(mx, swap_halves(mx));
      const float mnew = fmaxf(m, mx);
      const float alpha = fast_exp2(m - mnew);
      l *= alpha;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) acc[dt] *= alpha;
      m = mnew;
      form_p();
    }
    l += lb;
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) acc[dt] = mfma32(vf[u][dt], pf[u], acc[dt]);
    // K fragments of block blk + 2 (stage written in iteration blk - 1).
#pragma unroll
    for (int t = 0; t < NT; ++t)
      if constexpr (!LAST) kf[t] = kfrag(IC<(S + 2) % kStages>{}, t);
    __builtin_amdgcn_s_setprio(0);
  };
  // Blocks 0 .. nb-2, then the last block without the products of a next one.
  const int nmain = nb - 1;
  for (int b0 = 0; b0 < nmain; b0 += kStages) {
    iteration(IC<0>{}, b0, std::false_type{});
    if (b0 + 1 < nmain) iteration(IC<1>{}, b0 + 1, std::false_type{});
    if (b0 + 2 < nmain) iteration(IC<2>{}, b0 + 2, std::false_type{});
    if (b0 + 3 < nmain) iteration(IC<3>{}, b0 + 3, std::false_type{});
  }
  switch (nmain & 3) {
    case 0: iteration(IC<0>{}, nmain, std::true_type{}); break;
    case 1: iteration(IC<1>{}, nmain, std::true_type{}); break;
    case 2: iteration(IC<2>{}, nmain, std::true_type{}); break;
    default: iteration(IC<3>{}, nmain, std::true_type{}); break;
  }
  // ---- epilogue: merge the k-rows of each query (log-sum-exp), apply v'_k ----
  // v'_k of this lane's row in the accumulator layout (d = 32 dt + 8 (v/4) +
  // 4 h + v%4): from the LDS tile when w2 <= 32, else loaded here, before the
  // merge below covers their latency.
  u32x2_t vpr[4 * NDT];
  if constexpr (G == 1) {
    // The v' rows (issued in iteration 0) are in LDS for every wavefront
    // once the last iteration (n = nb - 1 >= 1) has waited for every load
    // and passed its barrier; a one-block window waits here.
    if (fwd_schedule::epilogue_waits(nb)) {
      wait_vmcnt<0>();
      lds_barrier_tracked();
    }
    const int r = qoff + c;
    const lds_char* vrow = to_lds(stg) + r * 2 * D + 8 * h;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) vpr[4 * dt + qd] = lds_ld<u32x2_t>(vrow + 16 * ((4 * dt + qd) ^ (r % T::CH)));
  } else {
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int qd = 0; qd < 4; ++qd)
        vpr[4 * dt + qd] = ldbuf64(rvp, rowvalid ? kk * rsb + 2 * (32 * dt + 8 * qd + 4 * h) : -1);
  }
  const float lsum = l + swap_halves(l);
  const float lse2_row = rowvalid ? m + fast_log2(lsum) : -INFINITY;
  float mq, z;
  if constexpr (G == 1) {
    // All 32 rows of the query are in this wavefront.
    mq = reduce32(lse2_row, [](float a, float bb) { return fmaxf(a, bb); });
    z = reduce32(lse2_row == -INFINITY ? 0.f : fast_exp2(lse2_row - mq), [](float a, float bb) { return a + bb; });
  } else {
    if (h == 0) stat[wave * 32 + c] = lse2_row;
    lds_barrier();
    mq = -INFINITY;
#pragma unroll
    for (int gg = 0; gg < G; ++gg) mq = fmaxf(mq, stat[(qs * G + gg) * 32 + c]);
    mq = reduce32(mq, [](float a, float bb) { return fmaxf(a, bb); });
    z = 0.f;
#pragma unroll
    for (int gg = 0; gg < G; ++gg) {
      const float x = stat[(qs * G + gg) * 32 + c];
      z += x == -INFINITY ? 0.f : fast_exp2(x - mq);
    }
    z = reduce32(z, [](float a, float bb) { return a + bb; });
  }
  const float lse2 = mq + fast_log2(z);
  const float wgt = rowvalid ? fast_exp2(m - lse2) : 0.f;

  // O_i = sum over the query's rows of w_r v'_k o U_r: the sums over the 32
  // rows of a wavefront run across lanes in registers; with w2 > 32 the two
  // wavefronts of a query add their halves through LDS.
  constexpr int NV = 16 * NDT;
  constexpr int NO = NV / 32;  // sums per lane
  float xv[NV];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int qd = 0; qd < 4; ++qd) {
      const u32x2_t x = vpr[4 * dt + qd];
      xv[16 * dt + 4 * qd + 0] = wgt * plus_bias<BIAS>(bf16_lo(x[0]), s.vp_bias) * acc[dt][4 * qd + 0];
      xv[16 * dt + 4 * qd + 1] = wgt * plus_bias<BIAS>(bf16_hi(x[0]), s.vp_bias) * acc[dt][4 * qd + 1];
      xv[16 * dt + 4 * qd + 2] = wgt * plus_bias<BIAS>(bf16_lo(x[1]), s.vp_bias) * acc[dt][4 * qd + 2];
      xv[16 * dt + 4 * qd + 3] = wgt * plus_bias<BIAS>(bf16_hi(x[1]), s.vp_bias) * acc[dt][4 * qd + 3];
    }
  reduce_lanes32<NV>(xv, lane);
  const int j0 = NV / 2 * ((c >> 4) & 1) + NV / 4 * ((c >> 3) & 1) + NV / 8 * ((c >> 2) & 1) +
                 NV / 16 * ((c >> 1) & 1) + NV / 32 * (c & 1);
  // j = 16 dt + 4 qd + e  <->  d = 32 dt + 8 qd + 4 h + e
  const int d0 = 32 * (j0 >> 4) + 8 * ((j0 >> 2) & 3) + 4 * h + (j0 & 3);
  if constexpr (G > 1) {
    float* part = xchg + wave * 64 * NO;
#pragma unroll
    for (int t = 0; t < NO; ++t) part[lane * NO + t] = xv[t];
    lds_barrier();
    if (g == 0) {
#pragma unroll
      for (int gg = 1; gg < G; ++gg)
#pragma unroll
        for (int t = 0; t < NO; ++t) xv[t] += part[gg * 64 * NO + lane * NO + t];
    }
  }
  if (qvalid && g == 0) {
    uint16_t* dst = out + base + static_cast<size_t>(i) * rs + d0;
    if constexpr (NO == 2) {
      *reinterpret_cast<unsigned*>(dst) = pack_bf16x2(xv[0], xv[1]);
    } else {
#pragma unroll
      for (int t = 0; t < NO; ++t) dst[t] = f32_to_bf16(xv[t]);
    }
    if (lane == 0) lse[static_cast<size_t>(bh) * N + i] = lse2 * kLn2;
  }
}

template <int D, int G, int FORM = 0, bool BIAS = false, bool HF = false>
hipError_t launch(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                  const void* vp, void* out, float* lse, hipStream_t st) {
  constexpr int QW = kWaves / G;
  const long total = HF ? static_cast<long>(s.N) * (s.H / QW) * s.B
                        : static_cast<long>((s.N + QW - 1) / QW) * s.B * s.H;
  const long grid = ((total + 7) / 8) * 8;
  hipLaunchKernelGGL((fwd_mfma_kernel<D, G, FORM, BIAS, HF>), dim3(static_cast<unsigned>(grid)), dim3(kThreads), 0,
                     st, s, static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                     static_cast<const uint16_t*>(kp), static_cast<const uint16_t*>(v),
                     static_cast<const uint16_t*>(vp), static_cast<uint16_t*>(out), lse);
  return hipGetLastError();
}

// Grouped-query attention with a multiple of 4 query heads per K-side head
// takes the head-folded tiles (trilinear logits).
bool head_folded(const Shape& s) { return s.form == 0 && s.Hkv < s.H && (s.H / s.Hkv) % kWaves == 0; }

}  // namespace

bool mfma_fwd_supported(const Shape& s) {
  // Per-head byte offsets are 32-bit in the buffer loads.
  const bool fits = static_cast<long long>(s.N) * s.H * s.D * 2 < (1ll << 31);
  return s.dtype == 1 && (s.D == 64 || s.D == 128) && s.w2 <= (s.form == 1 ? 32 : 64) && fits;
}

template <bool BIAS>
hipError_t mfma_fwd_b(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                      const void* vp, void* out, float* lse, hipStream_t st) {
  const int G = s.w2 <= 32 ? 1 : 2;
  if (s.form == 1) {  // determinant logits: w2 <= 32 only (mfma_fwd_supported)
    if (G != 1) return hipErrorInvalidValue;
    return s.D == 128 ? launch<128, 1, 1, BIAS>(s, q, k, kp, v, vp, out, lse, st)
                      : launch<64, 1, 1, BIAS>(s, q, k, kp, v, vp, out, lse, st);
  }
  if constexpr (!BIAS) {
    if (G == 1 && head_folded(s))
      return s.D == 128 ? launch<128, 1, 0, false, true>(s, q, k, kp, v, vp, out, lse, st)
                        : launch<64, 1, 0, false, true>(s, q, k, kp, v, vp, out, lse, st);
  }
  if (s.D == 128) return G == 1 ? launch<128, 1, 0, BIAS>(s, q, k, kp, v, vp, out, lse, st)
                                : launch<128, 2, 0, BIAS>(s, q, k, kp, v, vp, out, lse, st);
  if (s.D == 64) return G == 1 ? launch<64, 1, 0, BIAS>(s, q, k, kp, v, vp, out, lse, st)
                               : launch<64, 2, 0, BIAS>(s, q, k, kp, v, vp, out, lse, st);
  return hipErrorInvalidValue;
}

hipError_t mfma_fwd(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                    const void* vp, void* out, float* lse, hipStream_t st) {
  return s.kp_bias != 0.f || s.vp_bias != 0.f ? mfma_fwd_b<true>(s, q, k, kp, v, vp, out, lse, st)
                                              : mfma_fwd_b<false>(s, q, k, kp, v, vp, out, lse, st);
}

}  // namespace sa
