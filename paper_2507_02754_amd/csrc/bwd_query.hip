// Query-side backward (dQ, dK', dV') on gfx950 matrix cores, bf16, head_dim
// 64/128, w2 <= 32.
//
// With the rows r = (i, k) of the forward (q~_r = scale q_i o k'_k,
// do~_r = dO_i o v'_k, P_rj = exp(A_ijk - LSE_i)), Section 7's query-side
// gradients are
//     dQ~_r = sum_j dS_rj k_j,   U~_r = sum_j P_rj v_j,   dS_rj = P_rj (dP_rj - Delta_i),
//     dq_i  = scale sum_k k'_k o dQ~_r,  dk'_k = scale sum_i q_i o dQ~_r,
//     dv'_k = sum_i dO_i o U~_r.
//
// Work split. A workgroup walks a chunk of consecutive queries of one
// (batch, head) in tiles of four. Each query's 32 k-rows get two wavefronts:
//   role A (q~ in registers): S^T = K q~^T, P = exp2(S - LSE2), handed to the
//          partner through LDS, then U~^T += V^T P^T;
//   role B (do~ in registers): dP^T = V do~^T, then with the partner's P
//          dS = P (dP - Delta) and dQ~^T += K^T dS^T.
// Each role runs 16 of a key block's 32 matrix products and fits in 256
// registers, so two wavefronts share a SIMD. The roles run separate loops
// with the same barriers. Within a tile the loop is software-pipelined: in
// iteration n role A computes S and P of key block n + 1 and U~ of block n
// (with P(n) kept from the previous iteration), role B dP of block n + 1 and
// dS, dQ~ of block n (with P(n) written by A before the last barrier). K and V
// blocks are staged by all eight wavefronts through a four-stage LDS ring
// (block n + 2 written in iteration n) in one pipeline over (tile, block).
//
// Tile epilogue: B reduces dQ~ into dq_i and adds scale q_i o dQ~_r into an
// fp32 LDS ring of k-rows (dk'); A adds dO_i o U~_r into a second ring (dv').
// Each ring slice receives the four queries' contributions in a fixed order
// (four phases), so the result is deterministic. k-rows that no later query
// of the chunk touches are complete and written out; the w2 - 1 rows before
// each chunk boundary are split between two chunks, whose partial sums go to
// the workspace for the fix-up kernel (as in the other query-side path).
#include "mfma_common.h"

#include <type_traits>

namespace sa {
namespace {

constexpr int kQWaves = 8;
constexpr int kQThreads = 64 * kQWaves;

template <int D>
struct QueryLds {
  using T = SwzTile<D>;
  static constexpr int QW = 4;   // queries per tile
  static constexpr int W2P = 32;  // k-rows per query
  static constexpr int NS = 4;   // K/V block stages
  static constexpr int RL = 64 / T::CH;  // rows moved by one 64-lane row load
  static constexpr int stageBytes = 2 * FragTile<D>::bytes;  // K tile, then V tile
  static constexpr int xOff = NS * stageBytes;     // P exchange [2][QW][2 KB]
  static constexpr int xBytes = 2 * QW * 2048;
  static constexpr int rStride = D + 4;            // fp32 ring rows
  static constexpr int RB = W2P + QW;
  static constexpr int accOff = xOff + xBytes;
  static constexpr int RK = ((W2P + QW - 1 + RL + 15) / 16) * 16;
  static constexpr int RQ = 16;
  static constexpr int kringOff = accOff + 2 * RB * rStride * 4;
  static constexpr int qringOff = kringOff + 2 * RK * 2 * D;
  static constexpr int bytes = qringOff + 2 * RQ * 2 * D;
};

// FORM 1: determinant logits (Section 5): role A forms q~ = (scale log2 e)
// k'_k x q_i per 3-component chunk; role B stores its dQ~ rows (fp32, [B*H,
// N, 32, D]) in dqt instead of reducing them, because dq_i = scale sum_k
// dQ~_r x k'_k and dk'_k = scale sum_i q_i x dQ~_r mix components of a chunk
// that lie in different lane halves; a separate kernel forms them.
template <int D, bool BIAS, int FORM>
__global__ __launch_bounds__(kQThreads, 1) void bwd_query_kernel(
    Shape s, BwdPlan plan, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ kp, const uint16_t* __restrict__ v, const uint16_t* __restrict__ vp,
    const uint16_t* __restrict__ dout, const float* __restrict__ lse, const float* __restrict__ delta,
    uint16_t* __restrict__ dq, uint16_t* __restrict__ dkp, uint16_t* __restrict__ dvp,
    float* __restrict__ ws, float* __restrict__ dqt) {
  constexpr int NT = D / 16, NDT = D / 32;
  using L = QueryLds<D>;
  using T = typename L::T;  // layout of the k'/v' row ring
  constexpr int QW = L::QW, W2P = L::W2P, RB = L::RB, RK = L::RK, RQ = L::RQ, RL = L::RL, NS = L::NS;
  constexpr int SW = D / QW;  // columns of one ring phase slice
  static_assert(RQ >= QW + RL && SW % 8 == 0, "layout");
  __shared__ __attribute__((aligned(16))) char smem[L::bytes];
  lds_char* const lds = to_lds(smem);
  float* ring_kp = reinterpret_cast<float*>(smem + L::accOff);
  float* ring_vp = ring_kp + RB * L::rStride;
  char* kring = smem + L::kringOff;  // k' rows, then v' rows
  char* qring = smem + L::qringOff;  // q rows, then dO rows

  const int total = plan.nchunks * s.B * s.H;
  const int per_xcd = (total + 7) / 8;
  const int logical = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (logical >= total) return;
  const int bh = logical / plan.nchunks;
  const int chunk = logical - bh * plan.nchunks;
  const int b = bh / s.H, hh = bh - b * s.H;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // Roles alternate by wavefront. Wavefronts w and w + 4 of a 512-thread
  // workgroup share a SIMD, so each SIMD holds two wavefronts of one role;
  // pairing the two roles of a query on a SIMD instead measured slower here.
  const bool roleA = (wave & 1) == 0;
  const int qs = wave >> 1;  // query slot of this wavefront in a tile
  const int lane = tid & 63, c = lane & 31, h = lane >> 5;
  const size_t rs = static_cast<size_t>(s.H) * D;
  const int rsb = static_cast<int>(rs) * 2;
  const size_t base = (static_cast<size_t>(b) * s.N * s.H + hh) * D;
  // K, K', V, V' of the K-side head of query head hh (grouped-query attention)
  const int rsbk = s.Hkv * D * 2;
  const size_t basek = (static_cast<size_t>(b) * s.N * s.Hkv + hh / (s.H / s.Hkv)) * D;
  const int N = s.N, w1 = s.w1, w2 = s.w2;
  const int cs = chunk * plan.CQ, ce = min(N, cs + plan.CQ);
  const int kbase = cs - W2P + 1;  // k-row k: acc ring row (k - kbase) % RB, k' ring row (k - kbase) % RK
  const float qscale = s.scale * kLog2e;
  const size_t stat = static_cast<size_t>(bh) * N;
  const size_t halo = static_cast<size_t>(W2P - 1) * D;
  float* ws_head_kp = ws + (static_cast<size_t>(bh) * plan.nchunks + chunk) * halo;
  float* ws_head_vp = ws_head_kp + plan.halo_floats;
  float* ws_tail_kp = ws_head_vp + plan.halo_floats;
  float* ws_tail_vp = ws_tail_kp + plan.halo_floats;
  const unsigned hb = head_bytes(N, rsb, D), hbk = head_bytes(N, rsbk, D);

  for (int x = tid; x < 2 * RB * L::rStride; x += kQThreads) ring_kp[x] = 0.f;

  // Writes acc ring row k (complete or partial) to its destination and clears it.
  auto flush_row = [&](int kr, bool tail) {
    const int slot = (kr - kbase) % RB;
    for (int d = lane; d < D; d += 64) {
      float* a = ring_kp + slot * L::rStride + d;
      float* bv = ring_vp + slot * L::rStride + d;
      if (kr >= 0) {
        if (kr < cs) {
          const size_t o = static_cast<size_t>(kr - kbase) * D + d;
          ws_head_kp[o] = *a;
          ws_head_vp[o] = *bv;
        } else if (tail) {
          const size_t o = static_cast<size_t>(kr - (ce - W2P + 1)) * D + d;
          ws_tail_kp[o] = *a;
          ws_tail_vp[o] = *bv;
        } else {
          dkp[base + static_cast<size_t>(kr) * rs + d] = f32_to_bf16(*a);
          dvp[base + static_cast<size_t>(kr) * rs + d] = f32_to_bf16(*bv);
        }
      }
      *a = 0.f;
      *bv = 0.f;
    }
  };

  // ---- row rings: wavefronts 0..3 move RL consecutive rows of one tensor per
  // load (0: k', 1: v', 2: q, 3: dO); rows outside [0, N) load as zeros ----
  const int rw = wave & 3;
  const bool rowloader = wave < 4;
  const __amdgpu_buffer_rsrc_t rrow = rw < 2 ? make_rsrc((rw == 0 ? kp : vp) + basek, hbk)
                                              : make_rsrc((rw == 2 ? q : dout) + base, hb);
  const int rrsb = rw < 2 ? rsbk : rsb;
  const int rl_row = lane / T::CH, rl_ch = lane % T::CH;
  auto row_load = [&](int r0) { return ldbuf128(rrow, (r0 + rl_row) * rrsb + 16 * rl_ch); };
  auto row_put = [&](int r0, u32x4_t x) {
    const int r = r0 + rl_row;
    if (rw < 2) {
      const int slot = (r - kbase) % RK;
      *reinterpret_cast<u32x4_t*>(kring + rw * RK * 2 * D + slot * 2 * D + 16 * (rl_ch ^ T::swz(slot))) = x;
    } else {
      const int slot = (r - cs) % RQ;
      *reinterpret_cast<u32x4_t*>(qring + (rw - 2) * RQ * 2 * D + slot * 2 * D + 16 * rl_ch) = x;
    }
  };
  if (rowloader) {
    // Rows of the first tile: k-rows kbase .. cs + QW - 1, queries cs .. cs + QW - 1.
    constexpr int NG = (W2P + QW - 1 + RL - 1) / RL;
    const int r00 = rw < 2 ? kbase : cs;
    const int ng = rw < 2 ? NG : 1;
    u32x4_t x[NG];
#pragma unroll
    for (int gi = 0; gi < NG; ++gi) x[gi] = row_load(gi < ng ? r00 + gi * RL : -RL - 1);
#pragma unroll
    for (int gi = 0; gi < NG; ++gi)
      if (gi < ng) row_put(r00 + gi * RL, x[gi]);
  }

  // ---- K/V blocks: one staging pipeline over (query tile, 32-key block) ----
  // Wavefronts w < F::instrs move the K and V tiles of a block, 16 bytes per
  // lane, into the fragment-major layout; block `it` goes into stage it % NS.
  using F = FragTile<D>;
  const int nb = (w1 + QW - 1 + 31) / 32;
  const int ntiles = (ce - cs + QW - 1) / QW;
  const int total_it = ntiles * nb;
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(k + basek, hbk), rv = make_rsrc(v + basek, hbk);
  const bool stager = wave < F::instrs;
  const int st_row = (64 * wave + lane) / F::CH, st_ch = (64 * wave + lane) % F::CH;
  const int st_slot = F::slot(st_row, st_ch);
  u32x4_t skr = {0u, 0u, 0u, 0u}, svr = {0u, 0u, 0u, 0u};
  auto stage_fetch = [&](int it) {
    const int tile = it / nb, blk = it - tile * nb;
    const int jb = cs + tile * QW - w1 + 1 + 32 * blk;
    const int off = stager && it < total_it ? (jb + st_row) * rsbk + 16 * st_ch : -1;
    skr = ldbuf128(rk, off);
    svr = ldbuf128(rv, off);
  };
  auto stage_put = [&](int it) {
    if (stager) {
      const int o = (it % NS) * L::stageBytes + st_slot;
      lds_st(lds + o, skr);
      lds_st(lds + o + F::bytes, svr);
    }
  };
  // Blocks 0 and 1 into their stages, block 2 into the registers.
  stage_fetch(0);
  stage_put(0);
  stage_fetch(1);
  stage_put(1);
  stage_fetch(2);

  // ---- per-lane LDS bases of the operand fragments (fragment-major tiles) ----
  const int rbase0 = F::row_base(lane, 0), rbase1 = F::row_base(lane, 1);
  const int tbase0 = F::tr_base(lane, 0), tbase1 = F::tr_base(lane, 1);
  // Row fragment t of the tile at byte offset `off`.
  auto frag_row = [&](int off, int t) {
    return lds_ld<u32x4_t>(lds + ((t & 1) ? rbase1 : rbase0) + off + 1024 * t);
  };
  // Transposed fragment (dt, uu) of the tile at byte offset `off`.
  auto frag_tr = [&](int off, int dt, int uu) {
    const u32x2_t a = lds_tr16(lds + tbase0 + off + (2048 * dt + 256 * uu));
    const u32x2_t bb = lds_tr16(lds + tbase1 + off + (2048 * dt + 256 * uu));
    return u32x4_t{a[0], a[1], bb[0], bb[1]};
  };
  // P exchange of this query slot: [buffer][u] blocks of 1 KB, 16 bytes per lane.
  const int xlane = L::xOff + qs * 2048 + 16 * lane;

  lds_barrier();  // rings cleared, first rows and blocks 0, 1 in LDS

  // ---- pieces shared by both roles' tile loops (same barriers in both) ----
  // Staging step of iteration `it`: block it + 2 into its stage, block it + 3
  // into the registers.
  auto stage_step = [&](int it) {
    stage_put(it + 2);
    stage_fetch(it + 3);
  };
  // Rows that no later query of the chunk touches are complete.
  auto flush_tile = [&](int i0) {
    const int fl_lo = i0 - W2P + 1;
    const int fl_hi = min(i0 + QW, ce) - W2P;  // inclusive
    for (int kr = fl_lo + wave; kr <= fl_hi; kr += kQWaves) flush_row(kr, false);
  };
  // Adds this wavefront's per-row contributions (x, already scaled) into
  // ring `ring` in QW phases: in phase p the wavefront of query slot qs adds
  // column slice (qs + p) % QW, so every slice of a ring row receives the
  // contributions in a fixed order.
  // hook(IC<p>) runs in phase p before its barrier (register-only work that
  // fills the wait).
  auto ring_add = [&](float* ring, f32x16_t* x, bool rowvalid, int kk, auto hook) __attribute__((always_inline)) {
    const int aslot = (kk - kbase) % RB;
    float* rp = ring + aslot * L::rStride + 4 * h;
    auto phase = [&](auto PC) __attribute__((always_inline)) {
      constexpr int p = decltype(PC)::value;
      const int sl = (qs + p) % QW;
#pragma unroll
      for (int slc = 0; slc < QW; ++slc) {
        if (slc != sl || !rowvalid) continue;
        float4 xa[4 * NDT];
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
          for (int qd = 0; qd < 4; ++qd) {
            const int d0 = 32 * dt + 8 * qd;
            if (d0 / SW != slc) continue;
            xa[4 * dt + qd] = *reinterpret_cast<const float4*>(rp + d0);
          }
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
          for (int qd = 0; qd < 4; ++qd) {
            const int d0 = 32 * dt + 8 * qd;
            if (d0 / SW != slc) continue;
            float4& y = xa[4 * dt + qd];
            y.x += x[dt][4 * qd + 0];
            y.y += x[dt][4 * qd + 1];
            y.z += x[dt][4 * qd + 2];
            y.w += x[dt][4 * qd + 3];
            *reinterpret_cast<float4*>(rp + d0) = y;
          }
      }
      hook(PC);
      lds_barrier();
    };
    static_assert(QW == 4, "four ring phases");
    phase(std::integral_constant<int, 0>{});
    phase(std::integral_constant<int, 1>{});
    phase(std::integral_constant<int, 2>{});
    phase(std::integral_constant<int, 3>{});
  };

  // Per-query statistic of this wavefront's query (A: LSE, B: Delta), loaded
  // one tile ahead.
  float st_cur = (roleA ? lse : delta)[stat + min(cs + qs, N - 1)];
  if (roleA) {
    u32x4_t qt[NT];
    f32x16_t au[NDT];
    int it = 0;
    for (int tile = 0; tile < ntiles; ++tile) {
      const int i0 = cs + tile * QW;
      const int i = i0 + qs;
      const int kk = i - W2P + 1 + c;
      const bool qvalid = i < ce;
      const bool rowvalid = qvalid && kk >= 0 && kk > i - w2;
      const int jlo = i0 - w1 + 1;
      // Rows outside the window get an infinite normaliser: P = 0.
      const float lse2 = rowvalid ? st_cur * kLog2e : __builtin_inff();
      if (tile + 1 < ntiles) st_cur = lse[stat + min(i + QW, N - 1)];  // next tile's, ahead of use
      const u32x4_t nrow = row_load(rowloader && tile + 1 < ntiles ? i0 + QW : -RL - 1);
      {
        const int kslot = (kk - kbase) % RK;
        const char* krow = kring + kslot * 2 * D;
        const char* qrow = qring + ((i - cs) % RQ) * 2 * D;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const int ch = 2 * t + h;
          const u32x4_t qa = *reinterpret_cast<const u32x4_t*>(qrow + 16 * ch);
          const u32x4_t ka = *reinterpret_cast<const u32x4_t*>(krow + 16 * (ch ^ T::swz(kslot)));
          u32x4_t a4 = {0u, 0u, 0u, 0u};
          if constexpr (FORM == 1) {
            // windows of components 8 ch - 2 .. 8 ch + 9 of k' and q: the
            // slot and the 4-byte words on either side (clamped at the row
            // ends, where they are not used)
            const int chp = ch > 0 ? ch - 1 : 0, chn = ch < T::CH - 1 ? ch + 1 : ch;
            const int sw = T::swz(kslot);
            const unsigned kw0 = *reinterpret_cast<const unsigned*>(krow + 16 * (chp ^ sw) + 12);
            const unsigned kw1 = *reinterpret_cast<const unsigned*>(krow + 16 * (chn ^ sw));
            const unsigned qw0 = *reinterpret_cast<const unsigned*>(qrow + 16 * chp + 12);
            const unsigned qw1 = *reinterpret_cast<const unsigned*>(qrow + 16 * chn);
            float fk[12], fq[12], cr[8];
            fk[0] = bf16_lo(kw0), fk[1] = bf16_hi(kw0), fk[10] = bf16_lo(kw1), fk[11] = bf16_hi(kw1);
            fq[0] = bf16_lo(qw0), fq[1] = bf16_hi(qw0), fq[10] = bf16_lo(qw1), fq[11] = bf16_hi(qw1);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              fk[2 + 2 * e] = bf16_lo(ka[e]), fk[3 + 2 * e] = bf16_hi(ka[e]);
              fq[2 + 2 * e] = bf16_lo(qa[e]), fq[3 + 2 * e] = bf16_hi(qa[e]);
            }
            cross8_rt<3 * (D / 3)>(fk, fq, ch, cr);
            if (rowvalid) {
#pragma unroll
              for (int e = 0; e < 4; ++e) a4[e] = pack_bf16x2(cr[2 * e] * qscale, cr[2 * e + 1] * qscale);
            }
          } else if (rowvalid) {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              a4[e] = pack_bf16x2(bf16_lo(qa[e]) * plus_bias<BIAS>(bf16_lo(ka[e]), s.kp_bias) * qscale,
                                  bf16_hi(qa[e]) * plus_bias<BIAS>(bf16_hi(ka[e]), s.kp_bias) * qscale);
          }
          qt[t] = a4;
        }
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) au[dt] = f32x16_t{};
      }
      // S^T - LSE2 of the block in stage st, masked to this query's keys, as
      // probabilities packed for the U~ products and for the partner.
      auto probs = [&](int blk, int st, u32x4_t* pf) __attribute__((always_inline)) {
        u32x4_t ka[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) ka[t] = frag_row(st * L::stageBytes, t);  // K rows
        f32x16_t sacc = mfma32(ka[0], qt[0], f32x16_t{});
#pragma unroll
        for (int t = 1; t < NT; ++t) sacc = mfma32(ka[t], qt[t], sacc);
        const int lo = max(qs, -jlo) - 32 * blk;
        const int hi = min(qs + w1 - 1, N - 1 - jlo) - 32 * blk;
        float pr[16];
#pragma unroll
        for (int vv = 0; vv < 16; ++vv) pr[vv] = fast_exp2(sacc[vv] - lse2);
        if (lo > 0 || hi < 31) {
#pragma unroll
          for (int vv = 0; vv < 16; ++vv) {
            const int jl = acc_row(vv, h);
            pr[vv] = jl >= lo && jl <= hi ? pr[vv] : 0.f;
          }
        }
#pragma unroll
        for (int uu = 0; uu < 2; ++uu) {
          pf[uu] = pack_frag(pr, uu);
          lds_st(lds + xlane + ((blk & 1) * QW * 2048 + 1024 * uu), pf[uu]);
        }
      };
      // Iteration n of the tile (global block it): P and S of block n + 1
      // (when `next`), U~ of block n with pin = P(n); P(n + 1) into pout.
      auto step = [&](int n, int it_, const u32x4_t* pin, u32x4_t* pout, auto next) __attribute__((always_inline)) {
        const int so = (it_ % NS) * L::stageBytes;
        u32x4_t vtr[2][NDT];
#pragma unroll
        for (int uu = 0; uu < 2; ++uu)
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt) vtr[uu][dt] = frag_tr(so + F::bytes, dt, uu);
        if constexpr (decltype(next)::value) probs(n + 1, (it_ + 1) % NS, pout);
#pragma unroll
        for (int uu = 0; uu < 2; ++uu)
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt) au[dt] = mfma32(vtr[uu][dt], pin[uu], au[dt]);
        stage_step(it_);
        lds_barrier();
      };
      u32x4_t pa[2], pb[2];
      probs(0, it % NS, pa);
      lds_barrier();
      int n = 0;
      for (; n + 2 < nb; n += 2, it += 2) {
        step(n, it, pa, pb, std::true_type{});
        step(n + 1, it + 1, pb, pa, std::true_type{});
      }
      if (n + 1 < nb) {
        step(n, it, pa, pb, std::true_type{});
        step(n + 1, it + 1, pb, pa, std::false_type{});
        n += 2;
        it += 2;
      } else {
        step(n, it, pa, pb, std::false_type{});
        ++n;
        ++it;
      }
      // ---- tile epilogue (A): dO_i o U~_r into the dv' ring ----
      if (rowloader && tile + 1 < ntiles) row_put(i0 + QW, nrow);
      {
        const char* qrow = qring + RQ * 2 * D + ((i - cs) % RQ) * 2 * D;  // dO_i
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
          for (int qd = 0; qd < 4; ++qd) {
            const int d = 32 * dt + 8 * qd + 4 * h;
            const u32x2_t ov = *reinterpret_cast<const u32x2_t*>(qrow + 2 * d);
            au[dt][4 * qd + 0] *= bf16_lo(ov[0]);
            au[dt][4 * qd + 1] *= bf16_hi(ov[0]);
            au[dt][4 * qd + 2] *= bf16_lo(ov[1]);
            au[dt][4 * qd + 3] *= bf16_hi(ov[1]);
          }
      }
      lds_barrier();  // matches B's barrier after its dq reduction
      ring_add(ring_vp, au, rowvalid, kk, [](auto) {});
      // No barrier after the flush: the rows it reads and clears are next
      // written by the ring phases of the next tile, past its barriers.
      flush_tile(i0);
    }
  } else {
    u32x4_t ot[NT];
    f32x16_t adq[NDT];
    int it = 0;
    for (int tile = 0; tile < ntiles; ++tile) {
      const int i0 = cs + tile * QW;
      const int i = i0 + qs;
      const int kk = i - W2P + 1 + c;
      const bool qvalid = i < ce;
      const bool rowvalid = qvalid && kk >= 0 && kk > i - w2;
      const float dlt = qvalid ? st_cur : 0.f;
      if (tile + 1 < ntiles) st_cur = delta[stat + min(i + QW, N - 1)];  // next tile's, ahead of use
      const u32x4_t nrow = row_load(rowloader && tile + 1 < ntiles ? i0 + QW : -RL - 1);
      const int kslot = (kk - kbase) % RK;
      const char* krow = kring + kslot * 2 * D;
      {
        const char* orow = qring + RQ * 2 * D + ((i - cs) % RQ) * 2 * D;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const int ch = 2 * t + h;
          const u32x4_t oa = *reinterpret_cast<const u32x4_t*>(orow + 16 * ch);
          const u32x4_t va = *reinterpret_cast<const u32x4_t*>(krow + RK * 2 * D + 16 * (ch ^ T::swz(kslot)));
          u32x4_t b4 = {0u, 0u, 0u, 0u};
          if (rowvalid) {
#pragma unroll
            for (int e = 0; e < 4; ++e)
              b4[e] = pack_bf16x2(bf16_lo(oa[e]) * plus_bias<BIAS>(bf16_lo(va[e]), s.vp_bias),
                                  bf16_hi(oa[e]) * plus_bias<BIAS>(bf16_hi(va[e]), s.vp_bias));
          }
          ot[t] = b4;
        }
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) adq[dt] = f32x16_t{};
      }
      // dP^T = V do~^T of the block in stage st.
      auto dprod = [&](int st) __attribute__((always_inline)) {
        u32x4_t va[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) va[t] = frag_row(st * L::stageBytes + F::bytes, t);  // V rows
        f32x16_t pacc = mfma32(va[0], ot[0], f32x16_t{});
#pragma unroll
        for (int t = 1; t < NT; ++t) pacc = mfma32(va[t], ot[t], pacc);
        return pacc;
      };
      // Iteration n of the tile (global block it): dP of block n + 1 (when
      // `next`) into dout_, dS and dQ~ of block n from dpin = dP(n) and the
      // partner's P(n).
      auto step = [&](int n, int it_, const f32x16_t& dpin, f32x16_t& dout_, auto next) __attribute__((always_inline)) {
        const int so = (it_ % NS) * L::stageBytes;
        u32x4_t pf[2], ktr[2][NDT];
#pragma unroll
        for (int uu = 0; uu < 2; ++uu) pf[uu] = lds_ld<u32x4_t>(lds + xlane + ((n & 1) * QW * 2048 + 1024 * uu));
#pragma unroll
        for (int uu = 0; uu < 2; ++uu)
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt) ktr[uu][dt] = frag_tr(so, dt, uu);
        if constexpr (decltype(next)::value) dout_ = dprod((it_ + 1) % NS);
#pragma unroll
        for (int uu = 0; uu < 2; ++uu) {
          u32x4_t df;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float d0 = bf16_lo(pf[uu][e]) * (dpin[8 * uu + 2 * e] - dlt);
            const float d1 = bf16_hi(pf[uu][e]) * (dpin[8 * uu + 2 * e + 1] - dlt);
            df[e] = pack_bf16x2(d0, d1);
          }
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt) adq[dt] = mfma32(ktr[uu][dt], df, adq[dt]);
        }
        stage_step(it_);
        lds_barrier();
      };
      f32x16_t da = dprod(it % NS), db;
      lds_barrier();
      int n = 0;
      for (; n + 2 < nb; n += 2, it += 2) {
        step(n, it, da, db, std::true_type{});
        step(n + 1, it + 1, db, da, std::true_type{});
      }
      if (n + 1 < nb) {
        step(n, it, da, db, std::true_type{});
        step(n + 1, it + 1, db, da, std::false_type{});
        n += 2;
        it += 2;
      } else {
        step(n, it, da, db, std::false_type{});
        ++n;
        ++it;
      }
      // ---- tile epilogue (B): dq_i, then scale q_i o dQ~_r into the dk' ring ----
      if (rowloader && tile + 1 < ntiles) row_put(i0 + QW, nrow);
      if constexpr (FORM == 1) {
        // dQ~ rows to dqt (row c of query i, d = 32 dt + 8 qd + 4 h + e);
        // the ring phases keep their barriers (matching role A) without adds.
        if (qvalid) {
          float* dst = dqt + ((static_cast<size_t>(bh) * N + i) * 32 + c) * D;
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
            for (int qd = 0; qd < 4; ++qd)
              *reinterpret_cast<float4*>(dst + 32 * dt + 8 * qd + 4 * h) =
                  float4{adq[dt][4 * qd], adq[dt][4 * qd + 1], adq[dt][4 * qd + 2], adq[dt][4 * qd + 3]};
        }
        lds_barrier();  // matches the barrier before role A's ring phases
        ring_add(ring_kp, adq, false, kk, [](auto) {});
        flush_tile(i0);
        continue;
      }
      // dq_i = scale * sum_k k'_k o dQ~_(i,k): every lane multiplies its
      // accumulators (row c, d = 32 dt + 8 (v/4) + 4 h + v%4) by k'_k, then
      // the sums over the 32 rows run across lanes in registers: the first
      // level here, the other four in the ring phases below (their waits).
      constexpr int NV = 16 * NDT;
      float xv[NV];
      {
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
          for (int qd = 0; qd < 4; ++qd) {
            const int d = 32 * dt + 8 * qd + 4 * h;
            const u32x2_t m = *reinterpret_cast<const u32x2_t*>(krow + 16 * ((d >> 3) ^ T::swz(kslot)) + 8 * h);
            xv[16 * dt + 4 * qd + 0] = plus_bias<BIAS>(bf16_lo(m[0]), s.kp_bias) * adq[dt][4 * qd + 0];
            xv[16 * dt + 4 * qd + 1] = plus_bias<BIAS>(bf16_hi(m[0]), s.kp_bias) * adq[dt][4 * qd + 1];
            xv[16 * dt + 4 * qd + 2] = plus_bias<BIAS>(bf16_lo(m[1]), s.kp_bias) * adq[dt][4 * qd + 2];
            xv[16 * dt + 4 * qd + 3] = plus_bias<BIAS>(bf16_hi(m[1]), s.kp_bias) * adq[dt][4 * qd + 3];
          }
        reduce_lanes32_level<NV, 0>(xv, lane);
        const char* qrow = qring + ((i - cs) % RQ) * 2 * D;  // q_i
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
          for (int qd = 0; qd < 4; ++qd) {
            const int d = 32 * dt + 8 * qd + 4 * h;
            const u32x2_t qv = *reinterpret_cast<const u32x2_t*>(qrow + 2 * d);
            adq[dt][4 * qd + 0] *= s.scale * bf16_lo(qv[0]);
            adq[dt][4 * qd + 1] *= s.scale * bf16_hi(qv[0]);
            adq[dt][4 * qd + 2] *= s.scale * bf16_lo(qv[1]);
            adq[dt][4 * qd + 3] *= s.scale * bf16_hi(qv[1]);
          }
      }
      lds_barrier();  // every wavefront is past its reads of this tile's rows
      ring_add(ring_kp, adq, rowvalid, kk, [&](auto PC) __attribute__((always_inline)) {
        reduce_lanes32_level<NV, decltype(PC)::value + 1>(xv, lane);
      });
      {
        constexpr int NO = NV / 32;  // sums per lane: columns j0 .. j0 + NO - 1
        const int j0 = NV / 2 * ((c >> 4) & 1) + NV / 4 * ((c >> 3) & 1) + NV / 8 * ((c >> 2) & 1) +
                       NV / 16 * ((c >> 1) & 1) + NV / 32 * (c & 1);
        // j = 16 dt + 4 qd + e  <->  d = 32 dt + 8 qd + 4 h + e
        const int d0 = 32 * (j0 >> 4) + 8 * ((j0 >> 2) & 3) + 4 * h + (j0 & 3);
        if (qvalid) {
          uint16_t* dst = dq + base + static_cast<size_t>(i) * rs + d0;
          if constexpr (NO == 2) {
            *reinterpret_cast<unsigned*>(dst) = pack_bf16x2(xv[0] * s.scale, xv[1] * s.scale);
          } else {
#pragma unroll
            for (int t = 0; t < NO; ++t) dst[t] = f32_to_bf16(xv[t] * s.scale);
          }
        }
      }
      flush_tile(i0);
    }
  }
  // Rows still open at the end of the chunk.
  for (int kr = ce - W2P + 1 + wave; kr <= ce - 1; kr += kQWaves) flush_row(kr, ce < N);
}

}  // namespace

bool mfma_bwd_query_supported(const Shape& s) { return s.w2 <= 32 && (s.D == 64 || s.D == 128); }

hipError_t mfma_bwd_query(const Shape& s, const BwdPlan& plan, const void* q, const void* k,
                          const void* kp, const void* v, const void* vp, const void* dout,
                          const float* lse, const float* delta, void* dq, void* dkp, void* dvp,
                          float* halo, float* dqt, hipStream_t st) {
  const long tot = static_cast<long>(plan.nchunks) * s.B * s.H;
  const dim3 grid(static_cast<unsigned>(((tot + 7) / 8) * 8));
  const auto* Q = static_cast<const uint16_t*>(q);
  const auto* K = static_cast<const uint16_t*>(k);
  const auto* KP = static_cast<const uint16_t*>(kp);
  const auto* V = static_cast<const uint16_t*>(v);
  const auto* VP = static_cast<const uint16_t*>(vp);
  const auto* DO = static_cast<const uint16_t*>(dout);
  const bool bias = s.kp_bias != 0.f || s.vp_bias != 0.f;
  auto go = [&](auto kern) {
    hipLaunchKernelGGL(kern, grid, dim3(kQThreads), 0, st, s, plan, Q, K, KP, V, VP, DO, lse, delta,
                       static_cast<uint16_t*>(dq), static_cast<uint16_t*>(dkp), static_cast<uint16_t*>(dvp),
                       halo, dqt);
  };
  if (s.form == 1) {
    if (s.D == 128)
      go(bwd_query_kernel<128, false, 1>);
    else if (s.D == 64)
      go(bwd_query_kernel<64, false, 1>);
    else
      return hipErrorInvalidValue;
  } else if (s.D == 128) {
    bias ? go(bwd_query_kernel<128, true, 0>) : go(bwd_query_kernel<128, false, 0>);
  } else if (s.D == 64) {
    bias ? go(bwd_query_kernel<64, true, 0>) : go(bwd_query_kernel<64, false, 0>);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace sa
