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
// workgroups share a CU (two wavefronts per SIMD): one's exponentials overlap
// the other's matrix products. The j-window union of the workgroup is walked
// in 32-key blocks. K and V blocks are loaded into registers (16 bytes per
// lane, buffer loads whose range check zero-fills rows outside [0, N)) two
// blocks ahead and written one block ahead into a 2-stage ring of swizzled
// row-major LDS tiles. (Loads with an LDS destination measured slower here:
// their issue stalled the wavefront for hundreds of cycles per block.) K
// fragments are read row-wise; V fragments are read with the gfx950
// transposing LDS read, so V needs no transposed copy.
// Within a wavefront all rows share one query, so a block is skipped, fully
// valid, or masked by column only. The running maximum is rescaled lazily: only when some row's
// block maximum exceeds it by more than 2^8 (p stays <= 256, exact in fp32 and
// bf16 range), which after the first blocks is rare.
// Rows with k < 0 or k <= i - w2 get q~ = 0 and weight 0 in the merge.
#include "mfma_common.h"

namespace sa {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr float kLazyRescale = 8.0f;  // log2 headroom before the running max is raised

template <int D, int NS>
struct FwdLds {
  using T = SwzTile<D>;
  static constexpr int stageBytes = 2 * T::bytes;  // K tile + V tile of one 32-key block
  static constexpr int mainBytes = NS * stageBytes;  // also the epilogue's exchange area
  static constexpr int statOff = mainBytes;
  static constexpr int bytes = statOff + kWaves * 32 * 4;
};

// NS = stages of the ring of 32-key K/V blocks in LDS (2 suffices: a block is
// written one block before it is read, into the stage read two blocks ago).
template <int D, int G, int NS>
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
  using L = FwdLds<D, NS>;
  using T = typename L::T;
  __shared__ __attribute__((aligned(16))) char smem[L::bytes];
  float* stat = reinterpret_cast<float*>(smem + L::statOff);

  // XCD-aware tile order: hardware deals workgroups round-robin over the 8
  // XCDs; remap so each XCD walks a contiguous run of tiles of one head and
  // the overlapping K/V windows of neighbouring tiles hit the same L2.
  const int tiles = (s.N + QW - 1) / QW;
  const int total = tiles * s.B * s.H;
  const int per_xcd = (total + 7) / 8;
  const int logical = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (logical >= total) return;
  const int bh = logical / tiles;
  const int tile = logical - bh * tiles;
  const int b = bh / s.H, hh = bh - b * s.H;

  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63, c = lane & 31, h = lane >> 5;
  const int qs = wave / G, g = wave % G;
  const size_t rs = static_cast<size_t>(s.H) * D;
  const size_t base = (static_cast<size_t>(b) * s.N * s.H + hh) * D;
  const int N = s.N, w1 = s.w1, w2 = s.w2;
  const int i0 = tile * QW;
  const int i = i0 + qs;
  const bool qvalid = i < N;

  const int kk = i - W2P + 1 + 32 * g + c;
  const bool rowvalid = qvalid && kk >= 0 && kk > i - w2;
  const float qscale = s.scale * kLog2e;

  // ---- main loop over 32-key blocks of the workgroup's window union ----
  const int jlo = i0 - w1 + 1;
  const int nb = (w1 + QW - 1 + 31) / 32;
  const int rsb = static_cast<int>(rs) * 2;
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(k + base, head_bytes(N, rsb, D));
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(v + base, head_bytes(N, rsb, D));
  f32x16_t acc[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) acc[dt] = f32x16_t{};
  // Running row maximum m (log2 units). The logit products start from -m_used
  // in the accumulator, so they come out already shifted; m_used == m except
  // before the first block and inside a block where m was raised.
  float m = -INFINITY, l = 0.f, m_used = 0.f;
  f32x16_t negm = f32x16_t{};

  // K/V blocks are staged through registers: fetch loads this wavefront's
  // share of a block (16 bytes per lane per load, the chunk that belongs at
  // LDS offset 1024 k + 16 lane of the swizzled tile; rows outside [0, N)
  // come back as zeros from the buffer range check), put writes it into a
  // ring stage one block later.
  constexpr int SPW = (T::instrs + kWaves - 1) / kWaves;  // loads per tile per wavefront
  u32x4_t skr[SPW], svr[SPW];
  auto fetch = [&](int blk) {
    const int jb = jlo + 32 * blk;
#pragma unroll
    for (int x = 0; x < SPW; ++x) {
      const int kx = x * kWaves + wave;
      const int p = 64 * kx + lane;
      const int row = p / T::CH, ch = (p % T::CH) ^ T::swz(row);
      const int off = kx < T::instrs ? (jb + row) * rsb + 16 * ch : -1;
      skr[x] = ldbuf128(rk, off);
      svr[x] = ldbuf128(rv, off);
    }
  };
  auto put = [&](char* st) {
#pragma unroll
    for (int x = 0; x < SPW; ++x) {
      const int kx = x * kWaves + wave;
      if (kx < T::instrs) {
        *reinterpret_cast<u32x4_t*>(st + 1024 * kx + 16 * lane) = skr[x];
        *reinterpret_cast<u32x4_t*>(st + T::bytes + 1024 * kx + 16 * lane) = svr[x];
      }
    }
  };
  // The first block's K/V loads go out before the q~ loads, so their
  // latencies overlap.
  fetch(0);

  // ---- modulated queries q~ = (scale*log2 e) * q_i o k'_k as B operands ----
  // (rows outside the window or the sequence load as zeros: offset -1)
  u32x4_t qt[NT];
  {
    const __amdgpu_buffer_rsrc_t rq = make_rsrc(q + base, head_bytes(N, rsb, D));
    const __amdgpu_buffer_rsrc_t rkp = make_rsrc(kp + base, head_bytes(N, rsb, D));
    u32x4_t qa[NT], ka[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      qa[t] = ldbuf128(rq, rowvalid ? i * rsb + 32 * t + 16 * h : -1);
      ka[t] = ldbuf128(rkp, rowvalid ? kk * rsb + 32 * t + 16 * h : -1);
    }
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        qt[t][e] = pack_bf16x2(bf16_lo(qa[t][e]) * bf16_lo(ka[t][e]) * qscale,
                               bf16_hi(qa[t][e]) * bf16_hi(ka[t][e]) * qscale);
  }
  put(smem);
  if (nb > 1) fetch(1);

  for (int blk = 0; blk < nb; ++blk) {
    lds_barrier();
    // Block blk + 1 goes into its stage (last read in block blk - 1, which
    // every wavefront finished before the barrier), then block blk + 2 is
    // fetched into the registers.
    if (blk + 1 < nb) put(smem + ((blk + 1) % NS) * L::stageBytes);
    if (blk + 2 < nb) fetch(blk + 2);
    const char* kt = smem + (blk % NS) * L::stageBytes;
    const char* vt = kt + T::bytes;

    // Valid block-local columns of this wavefront's query.
    const int lo = max(qs, -jlo) - 32 * blk;
    const int hi = min(qs + w1 - 1, N - 1 - jlo) - 32 * blk;
    if (qvalid && hi >= 0 && lo <= 31 && lo <= hi) {
      u32x4_t kf[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) kf[t] = frag_row_swz<D>(kt, c, h, t);
      f32x16_t sacc = mfma32(kf[0], qt[0], negm);
#pragma unroll
      for (int t = 1; t < NT; ++t) sacc = mfma32(kf[t], qt[t], sacc);
      const float m_blk = m_used;
      float sv[16];
#pragma unroll
      for (int vv = 0; vv < 16; ++vv) sv[vv] = sacc[vv];
      if (lo > 0 || hi < 31) {
#pragma unroll
        for (int vv = 0; vv < 16; ++vv) {
          const int jl = acc_row(vv, h);
          if (jl < lo || jl > hi) sv[vv] = -INFINITY;
        }
      }
      float mx = fmaxf(sv[0], sv[1]);
#pragma unroll
      for (int vv = 2; vv < 16; vv += 2) mx = fmaxf(fmaxf(mx, sv[vv]), sv[vv + 1]);
      mx = fmaxf(mx, swap_halves(mx)) + m_blk;
      if (__builtin_amdgcn_ballot_w64(mx > m + kLazyRescale) != 0) {
        const float mnew = fmaxf(m, mx);
        const float alpha = fast_exp2(m - mnew);
        l *= alpha;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) acc[dt] *= alpha;
        m = mnew;
        m_used = mnew;
        const float off = m_blk - mnew;
#pragma unroll
        for (int vv = 0; vv < 16; ++vv) {
          sv[vv] += off;
          negm[vv] = -mnew;
        }
      }
#pragma unroll
      for (int vv = 0; vv < 16; ++vv) {
        sv[vv] = fast_exp2(sv[vv]);
        l += sv[vv];
      }
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const u32x4_t pf = pack_frag(sv, u);
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) acc[dt] = mfma32(frag_tr_swz<D>(vt, lane, dt, u), pf, acc[dt]);
      }
    }
  }
  // ---- epilogue: merge the k-rows of each query (log-sum-exp), apply v'_k ----
  // v'_k of this lane's row in the accumulator layout (d = 32 dt + 8 (v/4) +
  // 4 h + v%4), loaded first so the merge below covers their latency.
  const __amdgpu_buffer_rsrc_t rvp = make_rsrc(vp + base, head_bytes(N, rsb, D));
  u32x2_t vpr[4 * NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
    for (int qd = 0; qd < 4; ++qd)
      vpr[4 * dt + qd] = ldbuf64(rvp, rowvalid ? kk * rsb + 2 * (32 * dt + 8 * qd + 4 * h) : -1);
  const float lsum = l + swap_halves(l);
  const float lse2_row = rowvalid ? m + fast_log2(lsum) : -INFINITY;
  if (h == 0) stat[wave * 32 + c] = lse2_row;
  lds_barrier();  // also: every wavefront is past its last K/V stage reads
  float mq = -INFINITY;
#pragma unroll
  for (int gg = 0; gg < G; ++gg) mq = fmaxf(mq, stat[(qs * G + gg) * 32 + c]);
  mq = max32(mq);
  float z = 0.f;
#pragma unroll
  for (int gg = 0; gg < G; ++gg) {
    const float x = stat[(qs * G + gg) * 32 + c];
    z += x == -INFINITY ? 0.f : fast_exp2(x - mq);
  }
  z = sum32(z);
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
      xv[16 * dt + 4 * qd + 0] = wgt * bf16_lo(x[0]) * acc[dt][4 * qd + 0];
      xv[16 * dt + 4 * qd + 1] = wgt * bf16_hi(x[0]) * acc[dt][4 * qd + 1];
      xv[16 * dt + 4 * qd + 2] = wgt * bf16_lo(x[1]) * acc[dt][4 * qd + 2];
      xv[16 * dt + 4 * qd + 3] = wgt * bf16_hi(x[1]) * acc[dt][4 * qd + 3];
    }
  reduce_lanes32<NV>(xv, lane);
  const int j0 = NV / 2 * ((c >> 4) & 1) + NV / 4 * ((c >> 3) & 1) + NV / 8 * ((c >> 2) & 1) +
                 NV / 16 * ((c >> 1) & 1) + NV / 32 * (c & 1);
  // j = 16 dt + 4 qd + e  <->  d = 32 dt + 8 qd + 4 h + e
  const int d0 = 32 * (j0 >> 4) + 8 * ((j0 >> 2) & 3) + 4 * h + (j0 & 3);
  if constexpr (G > 1) {
    float* part = reinterpret_cast<float*>(smem) + wave * 64 * NO;
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

template <int D, int G>
hipError_t launch(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                  const void* vp, void* out, float* lse, hipStream_t st) {
  constexpr int QW = kWaves / G;
  constexpr int NS = 2;
  const long tiles = (s.N + QW - 1) / QW;
  const long total = tiles * s.B * s.H;
  const long grid = ((total + 7) / 8) * 8;
  hipLaunchKernelGGL((fwd_mfma_kernel<D, G, NS>), dim3(static_cast<unsigned>(grid)), dim3(kThreads), 0,
                     st, s, static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                     static_cast<const uint16_t*>(kp), static_cast<const uint16_t*>(v),
                     static_cast<const uint16_t*>(vp), static_cast<uint16_t*>(out), lse);
  return hipGetLastError();
}

}  // namespace

bool mfma_fwd_supported(const Shape& s) {
  // Per-head byte offsets are 32-bit in the buffer loads.
  const bool fits = static_cast<long long>(s.N) * s.H * s.D * 2 < (1ll << 31);
  return s.dtype == 1 && (s.D == 64 || s.D == 128) && s.w2 <= 64 && fits;
}

hipError_t mfma_fwd(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                    const void* vp, void* out, float* lse, hipStream_t st) {
  const int G = s.w2 <= 32 ? 1 : 2;
  if (s.D == 128) return G == 1 ? launch<128, 1>(s, q, k, kp, v, vp, out, lse, st)
                                : launch<128, 2>(s, q, k, kp, v, vp, out, lse, st);
  if (s.D == 64) return G == 1 ? launch<64, 1>(s, q, k, kp, v, vp, out, lse, st)
                               : launch<64, 2>(s, q, k, kp, v, vp, out, lse, st);
  return hipErrorInvalidValue;
}

}  // namespace sa
