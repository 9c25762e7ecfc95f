// Key-side backward (dK, dV) on gfx950 matrix cores, bf16, head_dim 64/128,
// w2 <= 64.
//
// With the rows r = (i, k) of the forward (q~_r = q_i o k'_k, do~_r = dO_i o v'_k,
// P_rj = exp(A_ijk - LSE_i)), the key gradients of Section 7 are
//     dV_j = sum_r P_rj do~_r,     dK_j = scale * sum_r dS_rj q~_r,
//     dS_rj = P_rj (dP_rj - Delta_i),  dP_rj = < do~_r, v_j >.
//
// Work split. A workgroup owns 128 consecutive keys of one (batch, head) and
// walks the row blocks (query i, 32 k-rows) whose windows reach them. Its eight
// wavefronts come in two roles per group of 32 keys, so that one SIMD holds two
// wavefronts whose instruction streams complement each other:
//   role A (K rows in registers): S = q~ K^T, P = exp2(S*scale*log2e - LSE2),
//          hands P to its partner through LDS, then dV += P^T do~;
//   role B (V rows in registers): dP = do~ V^T, then, with the partner's P,
//          dS = P (dP - Delta) and dK += dS^T q~.
// Each role runs 16 of the 32 matrix products of a row block and needs under
// 256 registers, so two wavefronts share a SIMD: the exponentials of one
// overlap the products of the other. The roles run separate loops (same
// number of barriers), so each keeps its accumulators in fixed registers.
//
// Row-block tiles q~ and do~ are formed cooperatively in swizzled row-major
// LDS tiles: role A forms the q~ half of tile t during phase 2 of row block
// t-2, role B the do~ half during phase 1 of row block t-1. Tiles rotate
// through four LDS slots and the loops are unrolled by four, so every LDS
// address is a per-lane base plus an immediate. One workgroup barrier per row
// block separates phase 1 (S/P and dP) from phase 2 (dV and dK); P goes
// through a double-buffered exchange area.
// Rows whose k lies outside the window are formed as zeros and contribute
// nothing; keys outside query i's window get an infinite normaliser (P = 0),
// and a group of 32 keys entirely outside it skips the row block's products.
#include "mfma_common.h"

#include <type_traits>

namespace sa {
namespace {

constexpr int kKeyWaves = 8;
constexpr int kKeyThreads = 64 * kKeyWaves;
constexpr int kSlots = 4;  // tile slots in LDS (the loop unroll factor)

template <int D>
struct KeyLds {
  using T = SwzTile<D>;
  static constexpr int tileBytes = 2 * T::bytes;         // q~ tile, then do~ tile
  static constexpr int xOff = kSlots * tileBytes;        // P exchange: [2][4 groups][2 KB]
  static constexpr int xBytes = 2 * 4 * 2048;
  static constexpr int mainBytes = xOff + xBytes;
  static constexpr int oStride = D + 4;                  // fp32 staging rows of the store
  static constexpr int outBytes = 4 * 32 * oStride * 4;  // one role at a time
  static constexpr int bytes = mainBytes > outBytes ? mainBytes : outBytes;
};

template <int X>
using ic = std::integral_constant<int, X>;

// FORM 1: determinant logits (Section 5): role A forms q~ = k'_k x q_i per
// 3-component chunk (unscaled), so S = q~ K^T is the determinant logit and
// dK = scale sum_r dS_rj q~_r as for the trilinear form.
template <int D, int G, bool BIAS, int FORM>
__global__ __launch_bounds__(kKeyThreads, 1) void bwd_key_kernel(
    Shape s, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ kp, const uint16_t* __restrict__ v, const uint16_t* __restrict__ vp,
    const uint16_t* __restrict__ dout, const float* __restrict__ lse, const float* __restrict__ delta,
    uint16_t* __restrict__ dk, uint16_t* __restrict__ dv) {
  constexpr int NT = D / 16, NDT = D / 32;
  constexpr int W2P = 32 * G;
  using L = KeyLds<D>;
  using T = typename L::T;
  constexpr int IPT = T::CH / 8;  // tile items (row, 16-byte chunk) per thread and role
  constexpr int RPI = 32 / IPT;   // rows covered by one pass of a role's 256 threads
  __shared__ __attribute__((aligned(16))) char smem[L::bytes];

  const int jblocks = (s.N + 127) / 128;
  const int total = jblocks * s.B * s.H;
  const int per_xcd = (total + 7) / 8;
  const int logical = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (logical >= total) return;
  const int bh = logical / jblocks;
  const int jblk = logical - bh * jblocks;
  const int b = bh / s.H, hh = bh - b * s.H;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // Roles by halves: wavefronts w and w + 4 of a 512-thread workgroup run on
  // the same SIMD, so each SIMD holds one role-A and one role-B wavefront
  // (measured faster than alternating roles, which pairs two wavefronts of the
  // same role on a SIMD). Role B's key groups are rotated by two, so the two
  // wavefronts sharing a SIMD belong to different key groups and do not reach
  // their exchange points in lockstep (measured 2.5% faster than pairing the
  // two roles of one key group).
  const bool roleA = wave < 4;
  const int kg = roleA ? wave : (wave + 2) & 3;  // key group of this wavefront
  const int lane = tid & 63, c = lane & 31, h = lane >> 5;
  const int rsb = s.H * D * 2;  // bytes between rows
  const size_t base = (static_cast<size_t>(b) * s.N * s.H + hh) * D;
  const int N = s.N, w1 = s.w1, w2 = s.w2;
  const float qscale = s.scale * kLog2e;
  const size_t stat = static_cast<size_t>(bh) * N;
  const int j0 = jblk * 128;
  const int jw = j0 + 32 * kg;  // keys jw .. jw + 31 of this wavefront
  const int jme = jw + c;       // key of this lane's accumulator column
  const unsigned hb = head_bytes(N, rsb, D);

  // K (role A) or V (role B) rows of the group as B operands: lane (h, c) holds
  // key jw + c, d = 16 t + 8 h .. + 7. Keys past the end load as zeros.
  u32x4_t kv[NT];
  {
    const __amdgpu_buffer_rsrc_t r = make_rsrc((roleA ? k : v) + base, hb);
#pragma unroll
    for (int t = 0; t < NT; ++t) kv[t] = ldbuf128(r, jme * rsb + 32 * t + 16 * h);
  }
  f32x16_t acc[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) acc[dt] = f32x16_t{};

  // Row blocks: (query i, k-chunk g) for i in [j0, min(N, j0 + 127 + w1)),
  // padded to a multiple of the unroll factor (the padding is inactive).
  const int i_end = min(N, j0 + 127 + w1);
  const int nrb = (i_end - j0) * G;
  const int nrb4 = (nrb + kSlots - 1) / kSlots * kSlots;

  // ---- loop-invariant LDS offsets of this lane ----
  // Row fragments (lane (h, c): row c, columns 16 t + 8 h .. + 7).
  int rowoff[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) rowoff[t] = T::off(c, 2 * t + h);
  // Transposed fragments (see frag_tr_swz): rows r0 and r0 + 8 of the first
  // 16-row half; the second half is 16 rows (a constant offset) further.
  int troff[NDT][2];
  {
    const int grp = lane >> 4, sl = lane & 15, hg = grp >> 1;
    const int r0 = 4 * hg + (sl >> 2);
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) {
      const int col = 32 * dt + 16 * (grp & 1) + 4 * (sl & 3);
      troff[dt][0] = T::off(r0, col >> 3) + (col & 7) * 2;
      troff[dt][1] = T::off(r0 + 8, col >> 3) + (col & 7) * 2;
    }
  }
  constexpr int kHalf16 = 16 * T::CH * 16;  // bytes of 16 tile rows
  lds_char* const lds = to_lds(smem);
  auto frag_row = [&](int tile_off, int t) { return lds_ld<u32x4_t>(lds + rowoff[t] + tile_off); };
  auto frag_tr = [&](int tile_off, int dt, int uu) {
    const u32x2_t a = lds_tr16(lds + troff[dt][0] + (tile_off + uu * kHalf16));
    const u32x2_t bb = lds_tr16(lds + troff[dt][1] + (tile_off + uu * kHalf16));
    return u32x4_t{a[0], a[1], bb[0], bb[1]};
  };
  // P exchange of this group: [buffer][u] blocks of 1 KB, 16 bytes per lane.
  const int xlane = L::xOff + kg * 2048 + 16 * lane;

  // ---- tile formation (role A: q~ = q_i o k'_k, role B: do~ = dO_i o v'_k) ----
  // Thread u of a role forms rows rho + RPI y (y < IPT), 16-byte chunk dc, so
  // the 16 lanes of a store group write 16 consecutive swizzled rows.
  const int u = kg * 64 + lane;  // index of this thread within its role
  const int rho = u % RPI, dc = u / RPI;
  const __amdgpu_buffer_rsrc_t rrow = make_rsrc((roleA ? q : dout) + base, hb);
  const __amdgpu_buffer_rsrc_t rmod = make_rsrc((roleA ? kp : vp) + base, hb);
  int formoff[IPT];
#pragma unroll
  for (int y = 0; y < IPT; ++y) formoff[y] = T::off(rho + RPI * y, dc) + (roleA ? 0 : T::bytes);
  // Two register sets for the formation loads (role A keeps loads in flight
  // for two iterations, role B for one). With bias constants, fb holds the
  // constant for rows inside the window and 0 for the others, which must stay
  // zero rows (their k' / v' load as zeros).
  u32x4_t fr[2], fm[2][IPT];
  float fb[2][IPT];
  // FORM 1, role A: the 4-byte words on either side of each 16-byte slot of
  // q and k' (a 3-chunk reaches 2 components into the neighbouring slots;
  // out-of-range offsets load zeros and are not used).
  unsigned frw[2][2], fmw[2][IPT][2];
  const float mbias = roleA ? s.kp_bias : s.vp_bias;
  auto fetch = [&](int rb, auto set) __attribute__((always_inline)) {
    constexpr int X = decltype(set)::value;
    const int i = j0 + rb / G, g = rb % G;
    fr[X] = ldbuf128(rrow, i * rsb + 16 * dc);
    if constexpr (FORM == 1) {
      if (roleA) {
        frw[X][0] = ldbuf32(rrow, i * rsb + 16 * dc - 4);
        frw[X][1] = ldbuf32(rrow, i * rsb + 16 * dc + 16);
      }
    }
#pragma unroll
    for (int y = 0; y < IPT; ++y) {
      const int kk = i - W2P + 1 + 32 * g + rho + RPI * y;
      const bool inwin = kk > i - w2 && (!BIAS || kk >= 0);  // kk < 0 also loads zeros
      fm[X][y] = ldbuf128(rmod, inwin ? kk * rsb + 16 * dc : -1);
      if constexpr (FORM == 1) {
        if (roleA) {
          fmw[X][y][0] = ldbuf32(rmod, inwin ? kk * rsb + 16 * dc - 4 : -1);
          fmw[X][y][1] = ldbuf32(rmod, inwin ? kk * rsb + 16 * dc + 16 : -1);
        }
      }
      if constexpr (BIAS) fb[X][y] = inwin ? mbias : 0.f;
    }
  };
  auto form_put = [&](int tile_off, auto set) __attribute__((always_inline)) {
    constexpr int X = decltype(set)::value;
    if constexpr (FORM == 1) {
      if (roleA) {
        // q~ = k'_k x q_i per chunk from the windows of components
        // 8 dc - 2 .. 8 dc + 9 (rows outside the window load as zeros).
        float fq[12];
        fq[0] = bf16_lo(frw[X][0]), fq[1] = bf16_hi(frw[X][0]);
        fq[10] = bf16_lo(frw[X][1]), fq[11] = bf16_hi(frw[X][1]);
#pragma unroll
        for (int e = 0; e < 4; ++e) fq[2 + 2 * e] = bf16_lo(fr[X][e]), fq[3 + 2 * e] = bf16_hi(fr[X][e]);
#pragma unroll
        for (int y = 0; y < IPT; ++y) {
          float fk[12], cr[8];
          fk[0] = bf16_lo(fmw[X][y][0]), fk[1] = bf16_hi(fmw[X][y][0]);
          fk[10] = bf16_lo(fmw[X][y][1]), fk[11] = bf16_hi(fmw[X][y][1]);
#pragma unroll
          for (int e = 0; e < 4; ++e) fk[2 + 2 * e] = bf16_lo(fm[X][y][e]), fk[3 + 2 * e] = bf16_hi(fm[X][y][e]);
          cross8_rt<3 * (D / 3)>(fk, fq, dc, cr);
          u32x4_t a4;
#pragma unroll
          for (int e = 0; e < 4; ++e) a4[e] = pack_bf16x2(cr[2 * e], cr[2 * e + 1]);
          lds_st(lds + formoff[y] + tile_off, a4);
        }
        return;
      }
    }
    float lo[4], hi[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      lo[e] = bf16_lo(fr[X][e]);
      hi[e] = bf16_hi(fr[X][e]);
    }
#pragma unroll
    for (int y = 0; y < IPT; ++y) {
      u32x4_t a4;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        a4[e] = pack_bf16x2(lo[e] * plus_bias<BIAS>(bf16_lo(fm[X][y][e]), fb[X][y]),
                            hi[e] * plus_bias<BIAS>(bf16_hi(fm[X][y][e]), fb[X][y]));
      lds_st(lds + formoff[y] + tile_off, a4);
    }
  };

  // Per-row-block statistic, 64 row blocks at a time: lane l holds the value
  // of row block (rb & ~63) + l (A: -LSE * log2 e, B: Delta), taken with a
  // lane read. The next 64 values are loaded half a window ahead. stat_at
  // must be called for every row block in order.
  const float* statp = roleA ? lse : delta;
  auto stat_load = [&](int rb0) {
    const int ii = min(j0 + (rb0 + lane) / G, N - 1);
    const float x = statp[stat + ii];
    return roleA ? -x * kLog2e : x;
  };
  float st_l = stat_load(0), st_nx = 0.f;
  auto stat_at = [&](int rb) {
    if ((rb & 63) == 32) st_nx = stat_load((rb & ~63) + 64);
    if ((rb & 63) == 0 && rb > 0) st_l = st_nx;
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, st_l), rb & 63));
  };
  // Keys of this group inside query i's window and the sequence, for a real row block.
  auto is_active = [&](int rb, int i) { return rb < nrb && jw <= i && jw + 31 > i - w1 && jw < N; };

  // Software pipeline: iteration n (one barrier at its end) computes the
  // logit-side product of row block n + 1 (A: S and P, B: dP) and the
  // gradient products of row block n (A: dV with P(n) kept from the previous
  // iteration; B: dS(n) with the partner's P(n), written before the last
  // barrier, then dK), and forms both halves of tile n + 2. Three tiles are
  // live at a time (n: transposed reads, n + 1: row reads, n + 2: written).
  // Prologue: tiles 0 and 1, then row block 0's logit side.
  fetch(0, ic<0>{});
  form_put(0, ic<0>{});
  fetch(1, ic<0>{});
  form_put(L::tileBytes, ic<0>{});
  fetch(2, ic<0>{});
  if (roleA) fetch(3, ic<1>{});
  // The loops start with every load complete (the wait-count pass would
  // otherwise keep the K/V operand loads pending into every iteration).
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  lds_barrier();

  // Row blocks [rb_lo, rb_hi) have every key group active for rb and rb + 1:
  // there the steps run without the activity tests, as straight-line code
  // the scheduler can interleave. Bounds are multiples of the unroll factor.
  int rb_lo = (96 * G + kSlots - 1) / kSlots * kSlots;
  int rb_hi = min((w1 + 30) * G - 1, min(nrb - 1, (N - j0) * G - 1));
  rb_hi = rb_hi / kSlots * kSlots;
  if (j0 + 96 >= N || rb_hi < rb_lo) rb_lo = rb_hi = nrb4;
  auto run_loops = [&](auto& step) __attribute__((always_inline)) {
    auto quad = [&](int rb, auto guard) __attribute__((always_inline)) {
      step(rb, ic<0>{}, guard);
      step(rb + 1, ic<1>{}, guard);
      step(rb + 2, ic<2>{}, guard);
      step(rb + 3, ic<3>{}, guard);
    };
    int rb = 0;
    for (; rb < rb_lo; rb += kSlots) quad(rb, ic<1>{});
    for (; rb < rb_hi; rb += kSlots) quad(rb, ic<0>{});
    for (; rb < nrb4; rb += kSlots) quad(rb, ic<1>{});
  };

  if (roleA) {
    // S = q~ K^T of the row block in the tile at tq.
    auto logits = [&](int tq) __attribute__((always_inline)) {
      u32x4_t qa[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) qa[t] = frag_row(tq, t);
      f32x16_t sacc = mfma32(qa[0], kv[0], f32x16_t{});
#pragma unroll
      for (int t = 1; t < NT; ++t) sacc = mfma32(qa[t], kv[t], sacc);
      return sacc;
    };
    // P of row block rb from its logits, packed, and written to the exchange
    // buffer at xb for the partner.
    auto probs = [&](int rb, float nlse2, const f32x16_t& sacc, int xb, u32x4_t* pf) __attribute__((always_inline)) {
      const int i = j0 + rb / G;
      const bool colok = jme <= i && jme > i - w1 && jme < N;
      const float nl = nlse2 - (colok ? 0.f : __builtin_inff());
      // p = 2^min(x, 0): at most 1, so rows formed as zeros (whose statistic
      // may belong to another query) stay finite. Written as a [0, 1] clamp of
      // 2^x, which the compiler folds into the exponential's clamp bit.
      float pr[16];
#pragma unroll
      for (int vv = 0; vv < 16; ++vv)
        pr[vv] = __builtin_amdgcn_fmed3f(fast_exp2(__builtin_fmaf(sacc[vv], qscale, nl)), 0.f, 1.f);
#pragma unroll
      for (int uu = 0; uu < 2; ++uu) {
        pf[uu] = pack_frag(pr, uu);
        lds_st(lds + xlane + (xb + 1024 * uu), pf[uu]);
      }
    };
    u32x4_t pcur[2];  // P of the row block whose dV is next (set only when active)
    {
      const float nl0 = stat_at(0);
      if (is_active(0, j0)) probs(0, nl0, logits(0), 0, pcur);
    }
    lds_barrier();
    // Iteration rb, tile slot S = rb % 4. The q~ half of tile rb + 2 is formed
    // from loads issued two iterations earlier (register set rb & 1).
    auto step = [&](int rb, auto slot, auto guard) __attribute__((always_inline)) {
      // Wavefront priority 1 while computing, 0 at the barrier (measured
      // faster: a wavefront that is computing issues ahead of one that is
      // about to wait).
      __builtin_amdgcn_s_setprio(1);
      constexpr int S = decltype(slot)::value;
      constexpr int S1 = (S + 1) % kSlots, S2 = (S + 2) % kSlots;
      constexpr bool kGuard = decltype(guard)::value != 0;
      const bool act0 = !kGuard || is_active(rb, j0 + rb / G);
      const bool act1 = !kGuard || is_active(rb + 1, j0 + (rb + 1) / G);
      const float nl1 = stat_at(rb + 1);
      f32x16_t snext;
      u32x4_t pnext[2];
      if constexpr (!kGuard) {
        // Straight-line: all fragment reads first, then the logit products
        // interleaved with the tile formation and the dV products with the
        // probabilities (about seven vector instructions per product).
        u32x4_t qa[NT], otr[2][NDT];
#pragma unroll
        for (int t = 0; t < NT; ++t) qa[t] = frag_row(S1 * L::tileBytes, t);
#pragma unroll
        for (int uu = 0; uu < 2; ++uu)
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt) otr[uu][dt] = frag_tr(S * L::tileBytes + T::bytes, dt, uu);
        snext = mfma32(qa[0], kv[0], f32x16_t{});
#pragma unroll
        for (int t = 1; t < NT; ++t) snext = mfma32(qa[t], kv[t], snext);
        form_put(S2 * L::tileBytes, ic<S & 1>{});
#pragma unroll
        for (int uu = 0; uu < 2; ++uu)
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt) acc[dt] = mfma32(pcur[uu], otr[uu][dt], acc[dt]);
        probs(rb + 1, nl1, snext, (S1 & 1) * 8192, pnext);
        __builtin_amdgcn_sched_group_barrier(0x100, NT, 0);  // q~ row fragments
#pragma unroll
        for (int x = 0; x < NT; ++x) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // S product
          __builtin_amdgcn_sched_group_barrier(0x100, 4 * NDT / NT, 0);  // do~ transposed fragments
          __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);  // formation
        }
#pragma unroll
        for (int x = 0; x < 2 * NDT; ++x) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // dV product
          __builtin_amdgcn_sched_group_barrier(0x002, 7, 0);  // probabilities
        }
      } else {
        if (act1) snext = logits(S1 * L::tileBytes);
        if (act0) {
          u32x4_t otr[2][NDT];
#pragma unroll
          for (int uu = 0; uu < 2; ++uu)
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) otr[uu][dt] = frag_tr(S * L::tileBytes + T::bytes, dt, uu);
#pragma unroll
          for (int uu = 0; uu < 2; ++uu)
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) acc[dt] = mfma32(pcur[uu], otr[uu][dt], acc[dt]);
        }
        if (act1) probs(rb + 1, nl1, snext, (S1 & 1) * 8192, pnext);
        form_put(S2 * L::tileBytes, ic<S & 1>{});
      }
      fetch(rb + 4, ic<S & 1>{});
      pcur[0] = pnext[0];
      pcur[1] = pnext[1];
      __builtin_amdgcn_s_setprio(0);
      lds_barrier();
    };
    run_loops(step);
  } else {
    // dP = do~ V^T of the row block in the tile whose do~ half is at to.
    auto logits_dp = [&](int to) __attribute__((always_inline)) {
      u32x4_t oa[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) oa[t] = frag_row(to, t);
      f32x16_t pacc = mfma32(oa[0], kv[0], f32x16_t{});
#pragma unroll
      for (int t = 1; t < NT; ++t) pacc = mfma32(oa[t], kv[t], pacc);
      return pacc;
    };
    f32x16_t dpcur;  // dP of the row block whose dK is next (set only when active)
    if (is_active(0, j0)) dpcur = logits_dp(T::bytes);
    lds_barrier();
    // dS = P (dP - Delta) of the current row block, packed (operand of dK).
    auto dsoft = [&](const u32x4_t* pf, float dlt, int uu) __attribute__((always_inline)) {
      u32x4_t df;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float d0 = bf16_lo(pf[uu][e]) * (dpcur[8 * uu + 2 * e] - dlt);
        const float d1 = bf16_hi(pf[uu][e]) * (dpcur[8 * uu + 2 * e + 1] - dlt);
        df[e] = pack_bf16x2(d0, d1);
      }
      return df;
    };
    auto step = [&](int rb, auto slot, auto guard) __attribute__((always_inline)) {
      __builtin_amdgcn_s_setprio(1);
      constexpr int S = decltype(slot)::value;
      constexpr int S1 = (S + 1) % kSlots, S2 = (S + 2) % kSlots;
      constexpr bool kGuard = decltype(guard)::value != 0;
      const bool act0 = !kGuard || is_active(rb, j0 + rb / G);
      const bool act1 = !kGuard || is_active(rb + 1, j0 + (rb + 1) / G);
      const float dlt = stat_at(rb);
      f32x16_t dpnext;
      if constexpr (!kGuard) {
        // Straight-line: reads first, then the dP products of row block rb + 1
        // interleaved with dS of row block rb, then the dK products with the
        // formation of tile rb + 2.
        u32x4_t pf[2], oa[NT], qtr[2][NDT];
#pragma unroll
        for (int uu = 0; uu < 2; ++uu) pf[uu] = lds_ld<u32x4_t>(lds + xlane + ((S & 1) * 8192 + 1024 * uu));
#pragma unroll
        for (int t = 0; t < NT; ++t) oa[t] = frag_row(S1 * L::tileBytes + T::bytes, t);
#pragma unroll
        for (int uu = 0; uu < 2; ++uu)
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt) qtr[uu][dt] = frag_tr(S * L::tileBytes, dt, uu);
        dpnext = mfma32(oa[0], kv[0], f32x16_t{});
#pragma unroll
        for (int t = 1; t < NT; ++t) dpnext = mfma32(oa[t], kv[t], dpnext);
        u32x4_t df[2];
#pragma unroll
        for (int uu = 0; uu < 2; ++uu) df[uu] = dsoft(pf, dlt, uu);
#pragma unroll
        for (int uu = 0; uu < 2; ++uu)
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt) acc[dt] = mfma32(df[uu], qtr[uu][dt], acc[dt]);
        form_put(S2 * L::tileBytes, ic<0>{});
        __builtin_amdgcn_sched_group_barrier(0x100, 2 + NT, 0);  // P, do~ row fragments
#pragma unroll
        for (int x = 0; x < NT; ++x) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // dP product
          __builtin_amdgcn_sched_group_barrier(0x100, 4 * NDT / NT, 0);  // q~ transposed fragments
          __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);  // dS
        }
#pragma unroll
        for (int x = 0; x < 2 * NDT; ++x) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // dK product
          __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);  // formation
        }
      } else {
        u32x4_t pf[2];
        if (act0) {
#pragma unroll
          for (int uu = 0; uu < 2; ++uu) pf[uu] = lds_ld<u32x4_t>(lds + xlane + ((S & 1) * 8192 + 1024 * uu));
        }
        if (act1) dpnext = logits_dp(S1 * L::tileBytes + T::bytes);
        if (act0) {
          u32x4_t qtr[2][NDT];
#pragma unroll
          for (int uu = 0; uu < 2; ++uu)
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) qtr[uu][dt] = frag_tr(S * L::tileBytes, dt, uu);
#pragma unroll
          for (int uu = 0; uu < 2; ++uu) {
            const u32x4_t df = dsoft(pf, dlt, uu);
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) acc[dt] = mfma32(df, qtr[uu][dt], acc[dt]);
          }
        }
        form_put(S2 * L::tileBytes, ic<0>{});
      }
      fetch(rb + 3, ic<0>{});
      dpcur = dpnext;
      __builtin_amdgcn_s_setprio(0);
      lds_barrier();
    };
    run_loops(step);
  }

  // ---- store: accumulator rows are keys, lanes are columns d; one role at a
  // time through fp32 staging rows ----
  const float oscale = roleA ? 1.f : s.scale;  // q~ is formed unscaled
  uint16_t* dst = roleA ? dv : dk;
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    lds_barrier();
    float* ob = reinterpret_cast<float*>(smem) + kg * 32 * L::oStride;
    const bool mine = (pass == 0) == roleA;
    if (mine) {
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int vv = 0; vv < 16; ++vv) ob[acc_row(vv, h) * L::oStride + 32 * dt + c] = acc[dt][vv] * oscale;
    }
    lds_barrier();
    if (mine) {
      constexpr int CH = D / 8;
      for (int x = lane; x < 32 * CH; x += 64) {
        const int row = x / CH, col = x % CH;
        const int j = jw + row;
        if (j < N) {
          const float* src = ob + row * L::oStride + 8 * col;
          u32x4_t w;
#pragma unroll
          for (int e = 0; e < 4; ++e) w[e] = pack_bf16x2(src[2 * e], src[2 * e + 1]);
          *reinterpret_cast<u32x4_t*>(dst + base + static_cast<size_t>(j) * s.H * D + 8 * col) = w;
        }
      }
    }
  }
}

template <int D, int G, bool BIAS, int FORM = 0>
hipError_t launch_key(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                      const void* vp, const void* dout, const float* lse, const float* delta, void* dk,
                      void* dv, hipStream_t st) {
  const long tot = static_cast<long>((s.N + 127) / 128) * s.B * s.H;
  hipLaunchKernelGGL((bwd_key_kernel<D, G, BIAS, FORM>), dim3(static_cast<unsigned>(((tot + 7) / 8) * 8)),
                     dim3(kKeyThreads), 0, st, s, static_cast<const uint16_t*>(q),
                     static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(kp),
                     static_cast<const uint16_t*>(v), static_cast<const uint16_t*>(vp),
                     static_cast<const uint16_t*>(dout), lse, delta, static_cast<uint16_t*>(dk),
                     static_cast<uint16_t*>(dv));
  return hipGetLastError();
}

}  // namespace

template <bool BIAS>
hipError_t mfma_bwd_key_b(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                          const void* vp, const void* dout, const float* lse, const float* delta,
                          void* dk, void* dv, hipStream_t st) {
  const int G = s.w2 <= 32 ? 1 : 2;
  if (s.D == 128)
    return G == 1 ? launch_key<128, 1, BIAS>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st)
                  : launch_key<128, 2, BIAS>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st);
  if (s.D == 64)
    return G == 1 ? launch_key<64, 1, BIAS>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st)
                  : launch_key<64, 2, BIAS>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st);
  return hipErrorInvalidValue;
}

hipError_t mfma_bwd_key(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                        const void* vp, const void* dout, const float* lse, const float* delta,
                        void* dk, void* dv, hipStream_t st) {
  if (s.form == 1) {  // determinant logits: w2 <= 32, no bias constants
    if (s.w2 > 32) return hipErrorInvalidValue;
    return s.D == 128 ? launch_key<128, 1, false, 1>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st)
                      : launch_key<64, 1, false, 1>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st);
  }
  return s.kp_bias != 0.f || s.vp_bias != 0.f
             ? mfma_bwd_key_b<true>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st)
             : mfma_bwd_key_b<false>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st);
}

}  // namespace sa
