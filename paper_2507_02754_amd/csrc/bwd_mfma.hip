// Backward pass on gfx950 matrix cores (bf16 data, head_dim 64 or 128, w2 <= 64).
//
// Gradients of Section 7, written over the rows r = (i, k) of the forward
// (q~_r = scale * q_i o k'_k, do~_r = dO_i o v'_k, P_rj = exp(A_ijk - LSE_i)):
//     dP_rj = < do~_r, v_j >            dS_rj = P_rj (dP_rj - Delta_i)
//     dK_j  = sum_r dS_rj q~_r           dV_j  = sum_r P_rj do~_r
//     dQ~_r = sum_j dS_rj k_j            U~_r  = sum_j P_rj v_j
//     dq_i  = scale sum_k k'_k o dQ~_r   dk'_k = scale sum_i q_i o dQ~_r
//     dv'_k = sum_i dO_i o U~_r
// (dsoftmax read as dS = P (dP - Delta) with Delta_i = <dO_i, O_i>.)
//
// Following Section 7's split into two kernels that avoid atomics:
//   * bwd_q  (query-stationary): recomputes S and dP per j-block of the window
//     and accumulates dQ~ and U~ on the matrix cores; its epilogue reduces the
//     k-rows into dq_i and adds the dk'/dv' contributions into an LDS ring of
//     k-rows. A workgroup walks a chunk of consecutive query tiles, so each
//     k-row is completed inside the chunk except the w2-1 rows at each chunk
//     boundary; those partial sums go to the workspace and a fix-up kernel adds
//     the two halves in a fixed order (deterministic, no atomics). This plays
//     the role of the paper's even/odd two-stage scheme (Algorithm 2).
//   * key side (bwd_key.hip, key-stationary): K and V rows stay in registers
//     and the kernel walks the query rows (i, k) that see them.
// Delta is computed by a small row-dot kernel first.
#include "mfma_common.h"


namespace sa {

// ---- workspace layout (shared with the host's size query) --------------------
BwdPlan mfma_bwd_plan(const Shape& s) {
  BwdPlan p{};
  p.G = s.w2 <= 32 ? 1 : 2;
  p.W2P = 32 * p.G;
  const long bh = static_cast<long>(s.B) * s.H;
  // Chunk length: enough workgroups to fill the chip several times, at least
  // one halo long, a multiple of every tile height.
  long cq = 128;
  while (cq < 1024 && bh * ((s.N + cq - 1) / cq) > 4096) cq *= 2;
  if (cq < p.W2P) cq = p.W2P;
  const size_t halo_rows = static_cast<size_t>(p.W2P - 1);
  const size_t delta_bytes = ((bh * static_cast<size_t>(s.N) * 4) + 255) & ~size_t(255);
  auto set_chunk = [&](long c) {
    p.CQ = static_cast<int>(c);
    p.nchunks = static_cast<int>((s.N + c - 1) / c);
    p.halo_floats = bh * static_cast<size_t>(p.nchunks) * halo_rows * s.D;
    p.bytes = delta_bytes + 4 * p.halo_floats * 4;
  };
  set_chunk(cq);
  // A capped workspace takes longer chunks (one chunk per head at most).
  while (s.ws_cap > 0 && p.bytes > s.ws_cap && cq < s.N) {
    cq *= 2;
    set_chunk(cq);
  }
  p.delta_off = 0;
  p.halo_off = delta_bytes;  // 4 arrays: head/tail x dk'/dv'
  p.dqt_off = 0;
  if (s.form == 1) {  // determinant logits: the dQ~ rows of every query
    p.dqt_off = (p.bytes + 255) & ~size_t(255);
    p.bytes = p.dqt_off + bh * static_cast<size_t>(s.N) * 32 * s.D * 4;
  }
  return p;
}

namespace {

// ------------------------------------------------------------------ delta ---
// Delta_i = <dO_i, O_i>; 16 lanes per query row (8 bf16 each for D = 128).
template <int D>
__global__ __launch_bounds__(256) void delta_kernel(Shape s, const uint16_t* __restrict__ out,
                                                     const uint16_t* __restrict__ dout,
                                                     float* __restrict__ delta) {
  constexpr int LPR = D / 8;  // lanes per row
  const long row = (static_cast<long>(blockIdx.x) * 256 + threadIdx.x) / LPR;
  const int part = threadIdx.x % LPR;
  const long total = static_cast<long>(s.B) * s.H * s.N;
  float acc = 0.f;
  long bh = 0, i = 0;
  if (row < total) {
    bh = row / s.N;
    i = row - bh * s.N;
    const long b = bh / s.H, h = bh - b * s.H;
    const size_t off = ((static_cast<size_t>(b) * s.N + i) * s.H + h) * D + 8 * part;
    const u32x4_t o = ldg128(out + off);
    const u32x4_t g = ldg128(dout + off);
#pragma unroll
    for (int e = 0; e < 4; ++e) acc += bf16_lo(o[e]) * bf16_lo(g[e]) + bf16_hi(o[e]) * bf16_hi(g[e]);
  }
#pragma unroll
  for (int off = LPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (row < total && part == 0) delta[row] = acc;
}

// ------------------------------------------------------------------ bwd_q ---

// LDS of the query-side kernel (D = 128: 101 KB for w2 <= 32, 148 KB for w2 = 64):
//   stage[2]  K and V tiles of one 32-key block (swizzled row-major), double
//             buffered; during a tile epilogue (w2 > 32) the stage just
//             consumed passes the two halves of each dq between wavefronts
//   acc       fp32 dk'/dv' ring of k-rows (RB rows)
//   kring     bf16 k' and v' rows (RK rows each, swizzled like the tiles)
//   qring     bf16 q and dO rows (RQ rows each)
template <int D, int G, int WAVES>
struct BwdQLds {
  using T = SwzTile<D>;
  static constexpr int QW = WAVES / G;
  static constexpr int W2P = 32 * G;
  static constexpr int RL = 64 / T::CH;  // rows moved by one 64-lane row load
  static constexpr int stageBytes = 2 * T::bytes;
  static constexpr int rStride = D + 4;  // fp32 acc ring rows
  static constexpr int RB = W2P + QW;
  // k' rows in use by a tile plus the RL rows loaded for the next one
  static constexpr int RK = ((W2P + QW - 1 + RL + 15) / 16) * 16;
  static constexpr int RQ = 16;
  static constexpr int accOff = 2 * stageBytes;
  static constexpr int kringOff = accOff + 2 * RB * rStride * 4;
  static constexpr int qringOff = kringOff + 2 * RK * 2 * D;
  static constexpr int bytes = qringOff + 2 * RQ * 2 * D;
};

template <int D, int G, int WAVES, bool BIAS>
__global__ __launch_bounds__(64 * WAVES) void bwd_q_kernel(
    Shape s, BwdPlan plan, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ kp, const uint16_t* __restrict__ v, const uint16_t* __restrict__ vp,
    const uint16_t* __restrict__ dout, const float* __restrict__ lse, const float* __restrict__ delta,
    uint16_t* __restrict__ dq, uint16_t* __restrict__ dkp, uint16_t* __restrict__ dvp,
    float* __restrict__ ws) {
  constexpr int NT = D / 16, NDT = D / 32;
  constexpr int NTH = 64 * WAVES;
  using L = BwdQLds<D, G, WAVES>;
  using T = typename L::T;
  constexpr int QW = L::QW, W2P = L::W2P, RB = L::RB, RK = L::RK, RQ = L::RQ, RL = L::RL;
  constexpr int SW = D / WAVES;  // columns of one ring phase slice
  static_assert(WAVES == 4, "one row tensor per wavefront in the row loads");
  static_assert(RQ >= QW + RL && SW % 8 == 0 && WAVES * 64 * D / 32 * 4 <= L::stageBytes, "layout");
  __shared__ __attribute__((aligned(16))) char smem[L::bytes];
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
  const int lane = tid & 63, c = lane & 31, h = lane >> 5;
  const int qs = wave / G, g = wave % G;
  const size_t rs = static_cast<size_t>(s.H) * D;
  const size_t base = (static_cast<size_t>(b) * s.N * s.H + hh) * D;
  const int N = s.N, w1 = s.w1, w2 = s.w2;
  const int cs = chunk * plan.CQ, ce = min(N, cs + plan.CQ);
  const int kbase = cs - W2P + 1;  // k-row k lives in acc ring row (k - kbase) % RB, k' ring row (k - kbase) % RK
  const float qscale = s.scale * kLog2e;
  const size_t stat = static_cast<size_t>(bh) * N;
  const size_t halo = static_cast<size_t>(W2P - 1) * D;
  float* ws_head_kp = ws + (static_cast<size_t>(bh) * plan.nchunks + chunk) * halo;
  float* ws_head_vp = ws_head_kp + plan.halo_floats;
  float* ws_tail_kp = ws_head_vp + plan.halo_floats;
  float* ws_tail_vp = ws_tail_kp + plan.halo_floats;
  const int rsb = static_cast<int>(rs) * 2;
  // K, K', V, V' of the K-side head of query head hh (grouped-query attention)
  const int rsbk = s.Hkv * D * 2;
  const size_t basek = (static_cast<size_t>(b) * s.N * s.Hkv + hh / (s.H / s.Hkv)) * D;
  const unsigned hb = head_bytes(N, rsb, D), hbk = head_bytes(N, rsbk, D);
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(k + basek, hbk), rv = make_rsrc(v + basek, hbk);

  for (int x = tid; x < 2 * RB * L::rStride; x += NTH) ring_kp[x] = 0.f;

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

  // ---- row rings ----
  // Wavefront w moves RL consecutive rows of one tensor per load (w = 0: k',
  // 1: v', 2: q, 3: dO), 16 bytes per lane; rows outside [0, N) come back as
  // zeros from the buffer range check. A tile's k' and v' rows (and q, dO of
  // its queries) are in the rings before its prologue; the RL rows after them
  // are loaded during the tile and written in its epilogue.
  const __amdgpu_buffer_rsrc_t rrow = wave < 2 ? make_rsrc((wave == 0 ? kp : vp) + basek, hbk)
                                                : make_rsrc((wave == 2 ? q : dout) + base, hb);
  const int rrsb = wave < 2 ? rsbk : rsb;
  const int rl_row = lane / T::CH, rl_ch = lane % T::CH;
  auto row_load = [&](int r0) { return ldbuf128(rrow, (r0 + rl_row) * rrsb + 16 * rl_ch); };
  auto row_put = [&](int r0, u32x4_t x) {
    const int r = r0 + rl_row;
    if (wave < 2) {
      const int slot = (r - kbase) % RK;
      *reinterpret_cast<u32x4_t*>(kring + wave * RK * 2 * D + slot * 2 * D + 16 * (rl_ch ^ T::swz(slot))) = x;
    } else {
      const int slot = (r - cs) % RQ;
      *reinterpret_cast<u32x4_t*>(qring + (wave - 2) * RQ * 2 * D + slot * 2 * D + 16 * rl_ch) = x;
    }
  };
  {
    // Rows of the first tile: k-rows kbase .. cs + QW - 1, queries cs .. cs + QW - 1.
    constexpr int NG = (W2P + QW - 1 + RL - 1) / RL;
    const int r00 = wave < 2 ? kbase : cs;
    const int ng = wave < 2 ? NG : 1;
    u32x4_t x[NG];
#pragma unroll
    for (int gi = 0; gi < NG; ++gi) x[gi] = row_load(gi < ng ? r00 + gi * RL : -RL - 1);
#pragma unroll
    for (int gi = 0; gi < NG; ++gi)
      if (gi < ng) row_put(r00 + gi * RL, x[gi]);
  }

  // ---- K/V blocks: one pipeline over (query tile, 32-key block) ----
  // stage_fetch loads this wavefront's share of block `it` into registers
  // (16 bytes per lane per load, the chunk that belongs at LDS offset
  // 1024 k + 16 lane of the swizzled tile); stage_put writes it into a stage
  // one block later.
  const int nb = (w1 + QW - 1 + 31) / 32;
  const int ntiles = (ce - cs + QW - 1) / QW;
  const int total_it = ntiles * nb;
  constexpr int SPW = (T::instrs + WAVES - 1) / WAVES;
  u32x4_t skr[SPW], svr[SPW];
  auto stage_fetch = [&](int it) {
    const int tile = it / nb, blk = it - tile * nb;
    const int jb = cs + tile * QW - w1 + 1 + 32 * blk;
#pragma unroll
    for (int x = 0; x < SPW; ++x) {
      const int kx = x * WAVES + wave;
      const int p = 64 * kx + lane;
      const int row = p / T::CH, ch = (p % T::CH) ^ T::swz(row);
      const int off = kx < T::instrs ? (jb + row) * rsbk + 16 * ch : -1;
      skr[x] = ldbuf128(rk, off);
      svr[x] = ldbuf128(rv, off);
    }
  };
  auto stage_put = [&](char* st) {
#pragma unroll
    for (int x = 0; x < SPW; ++x) {
      const int kx = x * WAVES + wave;
      if (kx < T::instrs) {
        *reinterpret_cast<u32x4_t*>(st + 1024 * kx + 16 * lane) = skr[x];
        *reinterpret_cast<u32x4_t*>(st + T::bytes + 1024 * kx + 16 * lane) = svr[x];
      }
    }
  };
  // Blocks 0 and 1 go into the two stages, block 2 into the registers.
  if (total_it > 0) {
    stage_fetch(0);
    stage_put(smem);
  }
  if (total_it > 1) {
    stage_fetch(1);
    stage_put(smem + L::stageBytes);
  }
  if (total_it > 2) stage_fetch(2);
  float nlse = lse[stat + min(cs + qs, N - 1)], ndlt = delta[stat + min(cs + qs, N - 1)];
  lds_barrier();  // acc ring cleared, first rows and blocks 0, 1 in LDS

  u32x4_t qt[NT], ot[NT];
  f32x16_t adq[NDT], au[NDT];
  int it = 0;
  for (int tile = 0; tile < ntiles; ++tile) {
    const int i0 = cs + tile * QW;
    const int i = i0 + qs;
    const int kk = i - W2P + 1 + 32 * g + c;
    const bool qvalid = i < ce;
    const bool rowvalid = qvalid && kk >= 0 && kk > i - w2;
    const int kslot = (kk - kbase) % RK;
    const char* krow = kring + kslot * 2 * D;
    const char* qrow = qring + ((i - cs) % RQ) * 2 * D;
    // Rows outside the window get an infinite normaliser: P = dS = 0.
    const float lse2 = rowvalid ? nlse * kLog2e : __builtin_inff();
    const float dlt = qvalid ? ndlt : 0.f;
    // ---- tile prologue: modulated operands of this wavefront's 32 rows ----
    {
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const int ch = 2 * t + h;
        const u32x4_t qa = *reinterpret_cast<const u32x4_t*>(qrow + 16 * ch);
        const u32x4_t oa = *reinterpret_cast<const u32x4_t*>(qrow + RQ * 2 * D + 16 * ch);
        const u32x4_t ka = *reinterpret_cast<const u32x4_t*>(krow + 16 * (ch ^ T::swz(kslot)));
        const u32x4_t va = *reinterpret_cast<const u32x4_t*>(krow + RK * 2 * D + 16 * (ch ^ T::swz(kslot)));
        u32x4_t a4 = {0u, 0u, 0u, 0u}, b4 = {0u, 0u, 0u, 0u};
        if (rowvalid) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            a4[e] = pack_bf16x2(bf16_lo(qa[e]) * plus_bias<BIAS>(bf16_lo(ka[e]), s.kp_bias) * qscale,
                                bf16_hi(qa[e]) * plus_bias<BIAS>(bf16_hi(ka[e]), s.kp_bias) * qscale);
            b4[e] = pack_bf16x2(bf16_lo(oa[e]) * plus_bias<BIAS>(bf16_lo(va[e]), s.vp_bias),
                                bf16_hi(oa[e]) * plus_bias<BIAS>(bf16_hi(va[e]), s.vp_bias));
          }
        }
        qt[t] = a4;
        ot[t] = b4;
      }
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        adq[dt] = f32x16_t{};
        au[dt] = f32x16_t{};
      }
    }
    // Rows of the next tile, written in this tile's epilogue.
    const bool more = tile + 1 < ntiles;
    const u32x4_t nrow = row_load(more ? i0 + QW : -RL - 1);
    if (more) {
      nlse = lse[stat + min(i + QW, N - 1)];
      ndlt = delta[stat + min(i + QW, N - 1)];
    }

    // ---- main loop, software-pipelined over the tile's 32-key blocks ----
    // Block it's logits S are computed at the end of block it - 1 (for a
    // tile's first block, here), so its exponentials overlap its dP products.
    // Stages: block it + 1 was written during block it - 1; after the barrier
    // in block it, block it's stage is free and takes block it + 2. At a
    // tile's last block that write waits for the next prologue, because the
    // epilogue uses the freed stage for the dq sums.
    // The products start from loop-invariant accumulator tiles: S from
    // -lse2 (the logits come out already normalised) and dP from -Delta.
    const int jlo = i0 - w1 + 1;
    if (tile > 0) {
      if (it + 1 < total_it) stage_put(smem + ((it + 1) & 1) * L::stageBytes);
      if (it + 2 < total_it) stage_fetch(it + 2);
    }
    lds_barrier();
    f32x16_t c_s, c_dp;
#pragma unroll
    for (int vv = 0; vv < 16; ++vv) {
      c_s[vv] = -lse2;
      c_dp[vv] = -dlt;
    }
    u32x4_t ka[NT], va[NT], ktr[2][NDT], vtr[2][NDT];
    f32x16_t sacc;
    // S^T - lse2 = K q~^T - lse2 of the block in stage `st`, with its V row
    // fragments read behind.
    auto logits = [&](const char* st) __attribute__((always_inline)) {
#pragma unroll
      for (int t = 0; t < NT; ++t) ka[t] = frag_row_swz<D>(st, c, h, t);
      sacc = mfma32(ka[0], qt[0], c_s);
#pragma unroll
      for (int t = 1; t < NT; ++t) sacc = mfma32(ka[t], qt[t], sacc);
#pragma unroll
      for (int t = 0; t < NT; ++t) va[t] = frag_row_swz<D>(st + T::bytes, c, h, t);
      __builtin_amdgcn_sched_group_barrier(0x100, NT, 0);
#pragma unroll
      for (int x = 0; x < NT; ++x) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
    };

    // One block, read from stage S.
    auto iter = [&](int S, int blk) __attribute__((always_inline)) {
      const char* kt = smem + S * L::stageBytes;
      const char* vt = kt + T::bytes;
      // Keys of this block inside query i's window and inside [0, N).
      const int lo = max(qs, -jlo) - 32 * blk;
      const int hi = min(qs + w1 - 1, N - 1 - jlo) - 32 * blk;
      const bool edge = lo > 0 || hi < 31;

      // (A) dP^T - Delta = V do~^T - Delta, overlapped with the
      // probabilities; the transposed V fragments are read behind it.
      f32x16_t pacc = mfma32(va[0], ot[0], c_dp);
#pragma unroll
      for (int t = 1; t < NT; ++t) pacc = mfma32(va[t], ot[t], pacc);
      float pr[16];
#pragma unroll
      for (int vv = 0; vv < 16; ++vv) pr[vv] = fast_exp2(sacc[vv]);
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) vtr[u][dt] = frag_tr_swz<D>(vt, lane, dt, u);
#pragma unroll
      for (int x = 0; x < NT; ++x) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 4 * NDT / NT, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
      // Blocks at the ends of the window (and of the sequence) mask their
      // keys; the empty asm keeps this a branch rather than selects on every block.
      if (edge) {
        asm volatile("" ::: "memory");
#pragma unroll
        for (int vv = 0; vv < 16; ++vv) {
          const int jl = acc_row(vv, h);
          pr[vv] = jl >= lo && jl <= hi ? pr[vv] : 0.f;
        }
      }
      u32x4_t pf[2], df[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) pf[u] = pack_frag(pr, u);
      __builtin_amdgcn_sched_barrier(0);

      // (B) U~^T += V^T P^T, overlapped with dS = P (dP - Delta); the
      // transposed K fragments are read behind it.
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) au[dt] = mfma32(vtr[u][dt], pf[u], au[dt]);
#pragma unroll
      for (int vv = 0; vv < 16; ++vv) pr[vv] *= pacc[vv];
#pragma unroll
      for (int u = 0; u < 2; ++u) df[u] = pack_frag(pr, u);
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) ktr[u][dt] = frag_tr_swz<D>(kt, lane, dt, u);
#pragma unroll
      for (int x = 0; x < 2 * NDT; ++x) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);
      }
      __builtin_amdgcn_sched_barrier(0);

      // (C) dQ~^T += K^T dS^T.
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) adq[dt] = mfma32(ktr[u][dt], df[u], adq[dt]);
      __builtin_amdgcn_sched_barrier(0);

      // (D) the next block's logits, after its stage is visible.
      if (blk + 1 < nb) {
        lds_barrier();
        if (it + 2 < total_it) stage_put(smem + S * L::stageBytes);
        if (it + 3 < total_it) stage_fetch(it + 3);
        __builtin_amdgcn_sched_barrier(0);
        logits(smem + (S ^ 1) * L::stageBytes);
        __builtin_amdgcn_sched_barrier(0);
      }
      ++it;
    };
    logits(smem + (it & 1) * L::stageBytes);
    __builtin_amdgcn_sched_barrier(0);
    for (int blk = 0; blk < nb; ++blk) iter(it & 1, blk);

    // ---- tile epilogue ----
    // The stage read by the last block is free once every wavefront is past
    // it. The next tile's rows go into the rings.
    lds_barrier();
    if (more) row_put(i0 + QW, nrow);
    // dq_i = scale * sum_k k'_k o dQ~_(i,k): every lane multiplies its
    // accumulators (row c, d = 32 dt + 8 (v/4) + 4 h + v%4) by k'_k, then the
    // sums over the 32 rows run across lanes in registers. With w2 > 32 the two
    // wavefronts of a query add their halves through LDS.
    {
      constexpr int NV = 16 * NDT;
      float xv[NV];
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
      reduce_lanes32<NV>(xv, lane);
      constexpr int NO = NV / 32;  // sums per lane: columns j0 .. j0 + NO - 1
      const int j0 = NV / 2 * ((c >> 4) & 1) + NV / 4 * ((c >> 3) & 1) + NV / 8 * ((c >> 2) & 1) +
                     NV / 16 * ((c >> 1) & 1) + NV / 32 * (c & 1);
      // j = 16 dt + 4 qd + e  <->  d = 32 dt + 8 qd + 4 h + e
      const int d0 = 32 * (j0 >> 4) + 8 * ((j0 >> 2) & 3) + 4 * h + (j0 & 3);
      if constexpr (G > 1) {
        float* part = reinterpret_cast<float*>(smem + ((it - 1) & 1) * L::stageBytes) + wave * 64 * NO;
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
        uint16_t* dst = dq + base + static_cast<size_t>(i) * rs + d0;
        if constexpr (NO == 2) {
          *reinterpret_cast<unsigned*>(dst) = pack_bf16x2(xv[0] * s.scale, xv[1] * s.scale);
        } else {
#pragma unroll
          for (int t = 0; t < NO; ++t) dst[t] = f32_to_bf16(xv[t] * s.scale);
        }
      }
    }

    // dk'/dv' contributions: every wavefront scales its accumulators in place
    // (scale q_i o dQ~ and dO_i o U~), then in phase p adds column slice
    // (wave + p) % WAVES of them into the acc ring. Each slice of a ring row
    // receives the wavefronts' contributions in a fixed order, so the sums
    // are deterministic, and no two wavefronts touch one slice in a phase.
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        const int d = 32 * dt + 8 * qd + 4 * h;
        const u32x2_t qv = *reinterpret_cast<const u32x2_t*>(qrow + 2 * d);
        const u32x2_t ov = *reinterpret_cast<const u32x2_t*>(qrow + RQ * 2 * D + 2 * d);
        adq[dt][4 * qd + 0] *= s.scale * bf16_lo(qv[0]);
        adq[dt][4 * qd + 1] *= s.scale * bf16_hi(qv[0]);
        adq[dt][4 * qd + 2] *= s.scale * bf16_lo(qv[1]);
        adq[dt][4 * qd + 3] *= s.scale * bf16_hi(qv[1]);
        au[dt][4 * qd + 0] *= bf16_lo(ov[0]);
        au[dt][4 * qd + 1] *= bf16_hi(ov[0]);
        au[dt][4 * qd + 2] *= bf16_lo(ov[1]);
        au[dt][4 * qd + 3] *= bf16_hi(ov[1]);
      }
    const int aslot = (kk - kbase) % RB;
    float* rk_ = ring_kp + aslot * L::rStride + 4 * h;
    float* rv_ = ring_vp + aslot * L::rStride + 4 * h;
    for (int p = 0; p < WAVES; ++p) {
      const int sl = (wave + p) % WAVES;
#pragma unroll
      for (int slc = 0; slc < WAVES; ++slc) {
        if (slc != sl || !rowvalid) continue;
        float4 xa[4 * NDT], ya[4 * NDT];
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
          for (int qd = 0; qd < 4; ++qd) {
            const int d0 = 32 * dt + 8 * qd;
            if (d0 / SW != slc) continue;
            xa[4 * dt + qd] = *reinterpret_cast<const float4*>(rk_ + d0);
            ya[4 * dt + qd] = *reinterpret_cast<const float4*>(rv_ + d0);
          }
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
          for (int qd = 0; qd < 4; ++qd) {
            const int d0 = 32 * dt + 8 * qd;
            if (d0 / SW != slc) continue;
            const int j = 4 * dt + qd;
            xa[j].x += adq[dt][4 * qd + 0];
            xa[j].y += adq[dt][4 * qd + 1];
            xa[j].z += adq[dt][4 * qd + 2];
            xa[j].w += adq[dt][4 * qd + 3];
            ya[j].x += au[dt][4 * qd + 0];
            ya[j].y += au[dt][4 * qd + 1];
            ya[j].z += au[dt][4 * qd + 2];
            ya[j].w += au[dt][4 * qd + 3];
            *reinterpret_cast<float4*>(rk_ + d0) = xa[j];
            *reinterpret_cast<float4*>(rv_ + d0) = ya[j];
          }
      }
      lds_barrier();
    }

    // Rows no later query of the chunk touches are complete. No barrier
    // after the flush: the rows it reads and clears are next written by the
    // ring phases of a later tile, past the next tile's barriers.
    const int fl_lo = i0 - W2P + 1;
    const int fl_hi = min(i0 + QW, ce) - W2P;  // inclusive
    for (int kr = fl_lo + wave; kr <= fl_hi; kr += WAVES) flush_row(kr, false);
  }
  // Rows still open at the end of the chunk.
  for (int kr = ce - W2P + 1 + wave; kr <= ce - 1; kr += WAVES) flush_row(kr, ce < N);
}

// Adds the tail partial of chunk c-1 and the head partial of chunk c for the
// W2P-1 k-rows before each chunk boundary and writes dk', dv'.
template <int D>
__global__ __launch_bounds__(256) void halo_fixup_kernel(Shape s, BwdPlan plan, const float* __restrict__ ws,
                                                         uint16_t* __restrict__ dkp, uint16_t* __restrict__ dvp) {
  const int W2P = plan.W2P;
  const long per_bound = static_cast<long>(W2P - 1) * D;
  const long nb = static_cast<long>(s.B) * s.H * (plan.nchunks - 1);
  const long idx = static_cast<long>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= nb * per_bound) return;
  const long bound = idx / per_bound;
  const long rem = idx - bound * per_bound;
  const int row = static_cast<int>(rem / D), d = static_cast<int>(rem % D);
  const int bh = static_cast<int>(bound / (plan.nchunks - 1));
  const int cb = static_cast<int>(bound % (plan.nchunks - 1)) + 1;  // chunk after the boundary
  const int kr = cb * plan.CQ - W2P + 1 + row;
  if (kr < 0 || kr >= s.N) return;
  const size_t halo = static_cast<size_t>(W2P - 1) * D;
  const float* head_kp = ws + (static_cast<size_t>(bh) * plan.nchunks + cb) * halo;
  const float* head_vp = head_kp + plan.halo_floats;
  const float* tail_kp = ws + 2 * plan.halo_floats + (static_cast<size_t>(bh) * plan.nchunks + cb - 1) * halo;
  const float* tail_vp = tail_kp + plan.halo_floats;
  const size_t o = static_cast<size_t>(row) * D + d;
  const int b = bh / s.H, hh = bh % s.H;
  const size_t dst = ((static_cast<size_t>(b) * s.N + kr) * s.H + hh) * D + d;
  dkp[dst] = f32_to_bf16(tail_kp[o] + head_kp[o]);
  dvp[dst] = f32_to_bf16(tail_vp[o] + head_vp[o]);
}

// Determinant logits (Section 5), from the dQ~ rows the query side stored:
//   dq_i  = scale sum_k  dQ~_(i,k) x k'_k   (k in the w2 window of i)
//   dk'_k = scale sum_i  q_i x dQ~_(i,k)    (i in [k, k + w2))
// per 3-component chunk (the gradients of <dQ~, k' x q> in q and in k'); the
// D mod 3 trailing components get 0. One thread per (query or key row,
// chunk), fixed summation order: deterministic.
template <int D, int WHICH>  // WHICH 0: dq, 1: dk'
__global__ __launch_bounds__(256) void det_grad_kernel(Shape s, const float* __restrict__ dqt,
                                                       const uint16_t* __restrict__ other,
                                                       uint16_t* __restrict__ out) {
  constexpr int NCH = (D + 2) / 3;  // chunks, the last one partial when D % 3 != 0
  const long idx = static_cast<long>(blockIdx.x) * 256 + threadIdx.x;
  const long total = static_cast<long>(s.B) * s.H * s.N * NCH;
  if (idx >= total) return;
  const int l = static_cast<int>(idx % NCH);
  const long row = idx / NCH;  // bh * N + n
  const int n = static_cast<int>(row % s.N);
  const int bh = static_cast<int>(row / s.N);
  const int b = bh / s.H, hh = bh - b * s.H;
  const size_t rs = static_cast<size_t>(s.H) * D;
  const size_t base = (static_cast<size_t>(b) * s.N * s.H + hh) * D;
  float acc[3] = {0.f, 0.f, 0.f};
  if (3 * l + 2 < D) {
    auto cross = [](const float* x, const float* y, float* a) {
      a[0] += x[1] * y[2] - x[2] * y[1];
      a[1] += x[2] * y[0] - x[0] * y[2];
      a[2] += x[0] * y[1] - x[1] * y[0];
    };
    if constexpr (WHICH == 0) {  // n = query i; rows r <-> k = i - 31 + r
      for (int r = 0; r < 32; ++r) {
        const int kk = n - 31 + r;
        if (kk < 0 || kk <= n - s.w2) continue;
        const float* a = dqt + ((static_cast<size_t>(row) * 32 + r) * D + 3 * l);
        const uint16_t* y = other + base + static_cast<size_t>(kk) * rs + 3 * l;  // k'
        const float xa[3] = {a[0], a[1], a[2]};
        const float ya[3] = {bf16_to_f32(y[0]), bf16_to_f32(y[1]), bf16_to_f32(y[2])};
        cross(xa, ya, acc);
      }
    } else {  // n = key row k; queries i = k .. k + w2 - 1, row r = k - i + 31
      const int iend = min(s.N, n + s.w2);
      for (int i = n; i < iend; ++i) {
        const float* a = dqt + (((static_cast<size_t>(bh) * s.N + i) * 32 + (n - i + 31)) * D + 3 * l);
        const uint16_t* x = other + base + static_cast<size_t>(i) * rs + 3 * l;  // q
        const float xq[3] = {bf16_to_f32(x[0]), bf16_to_f32(x[1]), bf16_to_f32(x[2])};
        const float ya[3] = {a[0], a[1], a[2]};
        cross(xq, ya, acc);
      }
    }
  }
  uint16_t* dst = out + base + static_cast<size_t>(n) * rs + 3 * l;
#pragma unroll
  for (int e = 0; e < 3; ++e)
    if (3 * l + e < D) dst[e] = f32_to_bf16(acc[e] * s.scale);
}

template <int D, int G>
hipError_t launch_stage(const Shape& s, BwdStage stage, const void* q, const void* k, const void* kp,
                        const void* v, const void* vp, const void* dout, const float* lse, void* g0,
                        void* g1, void* g2, void* workspace, hipStream_t st) {
  const BwdPlan plan = mfma_bwd_plan(s);
  char* wsb = static_cast<char*>(workspace);
  const float* delta = reinterpret_cast<const float*>(wsb + plan.delta_off);
  float* halo = reinterpret_cast<float*>(wsb + plan.halo_off);
  const auto* Q = static_cast<const uint16_t*>(q);
  const auto* K = static_cast<const uint16_t*>(k);
  const auto* KP = static_cast<const uint16_t*>(kp);
  const auto* V = static_cast<const uint16_t*>(v);
  const auto* VP = static_cast<const uint16_t*>(vp);
  const auto* DO = static_cast<const uint16_t*>(dout);
  if (stage == BwdStage::Query && mfma_bwd_query_supported(s)) {
    float* dqt = s.form == 1 ? reinterpret_cast<float*>(wsb + plan.dqt_off) : nullptr;
    const hipError_t e = mfma_bwd_query(s, plan, Q, K, KP, V, VP, DO, lse, delta, g0, g1, g2, halo, dqt, st);
    if (e != hipSuccess) return e;
    if (plan.nchunks > 1) {
      const long n = static_cast<long>(s.B) * s.H * (plan.nchunks - 1) * (plan.W2P - 1) * D;
      hipLaunchKernelGGL(halo_fixup_kernel<D>, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256),
                         0, st, s, plan, halo, static_cast<uint16_t*>(g1), static_cast<uint16_t*>(g2));
    }
    if (s.form == 1) {  // dq and dk' of the determinant logits (overwrite dk' entirely)
      const long n = static_cast<long>(s.B) * s.H * s.N * ((D + 2) / 3);
      const dim3 grid(static_cast<unsigned>((n + 255) / 256));
      hipLaunchKernelGGL((det_grad_kernel<D, 0>), grid, dim3(256), 0, st, s, dqt, KP, static_cast<uint16_t*>(g0));
      hipLaunchKernelGGL((det_grad_kernel<D, 1>), grid, dim3(256), 0, st, s, dqt, Q, static_cast<uint16_t*>(g1));
    }
  } else if (stage == BwdStage::Query) {
    if (s.form == 1) return hipErrorInvalidValue;  // determinant logits: w2 <= 32 only
    constexpr int WAVES = 4;
    const long totq = static_cast<long>(plan.nchunks) * s.B * s.H;
    auto go = [&](auto kern) {
      hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(((totq + 7) / 8) * 8)), dim3(64 * WAVES), 0, st,
                         s, plan, Q, K, KP, V, VP, DO, lse, delta, static_cast<uint16_t*>(g0),
                         static_cast<uint16_t*>(g1), static_cast<uint16_t*>(g2), halo);
    };
    if (s.kp_bias != 0.f || s.vp_bias != 0.f)
      go(bwd_q_kernel<D, G, WAVES, true>);
    else
      go(bwd_q_kernel<D, G, WAVES, false>);
    if (plan.nchunks > 1) {
      const long n = static_cast<long>(s.B) * s.H * (plan.nchunks - 1) * (plan.W2P - 1) * D;
      hipLaunchKernelGGL(halo_fixup_kernel<D>, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256),
                         0, st, s, plan, halo, static_cast<uint16_t*>(g1), static_cast<uint16_t*>(g2));
    }
  } else {
    return mfma_bwd_key(s, Q, K, KP, V, VP, DO, lse, delta, g0, g1, st);
  }
  return hipGetLastError();
}

}  // namespace

bool mfma_bwd_supported(const Shape& s) { return mfma_fwd_supported(s); }

hipError_t mfma_bwd_delta(const Shape& s, const void* out, const void* dout, void* workspace,
                          hipStream_t st) {
  const BwdPlan plan = mfma_bwd_plan(s);
  float* delta = reinterpret_cast<float*>(static_cast<char*>(workspace) + plan.delta_off);
  const long rows = static_cast<long>(s.B) * s.H * s.N;
  const auto* O = static_cast<const uint16_t*>(out);
  const auto* DO = static_cast<const uint16_t*>(dout);
  if (s.D == 128) {
    hipLaunchKernelGGL(delta_kernel<128>, dim3(static_cast<unsigned>((rows * 16 + 255) / 256)),
                       dim3(256), 0, st, s, O, DO, delta);
  } else if (s.D == 64) {
    hipLaunchKernelGGL(delta_kernel<64>, dim3(static_cast<unsigned>((rows * 8 + 255) / 256)),
                       dim3(256), 0, st, s, O, DO, delta);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t mfma_bwd_stage(const Shape& s, BwdStage stage, const void* q, const void* k,
                          const void* kp, const void* v, const void* vp, const void* dout,
                          const float* lse, void* g0, void* g1, void* g2, void* workspace,
                          hipStream_t st) {
  const int G = s.w2 <= 32 ? 1 : 2;
  if (s.D == 128)
    return G == 1 ? launch_stage<128, 1>(s, stage, q, k, kp, v, vp, dout, lse, g0, g1, g2, workspace, st)
                  : launch_stage<128, 2>(s, stage, q, k, kp, v, vp, dout, lse, g0, g1, g2, workspace, st);
  if (s.D == 64)
    return G == 1 ? launch_stage<64, 1>(s, stage, q, k, kp, v, vp, dout, lse, g0, g1, g2, workspace, st)
                  : launch_stage<64, 2>(s, stage, q, k, kp, v, vp, dout, lse, g0, g1, g2, workspace, st);
  return hipErrorInvalidValue;
}

}  // namespace sa
