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
// Tiling. A workgroup (4 wavefronts) owns QW consecutive queries of one
// (batch, head); each wavefront owns 64 rows = two 32-row groups (G = 1: two
// queries with 32 k-rows each; G = 2: one query with 64 k-rows). The j-window
// union of the workgroup is walked in 32-column blocks; K (row-major) and V
// (transposed) blocks are staged in double-buffered LDS with 16-byte coalesced
// global loads. Within a group all rows share one query, so a block is either
// skipped, fully valid, or masked by column only. Rows with k < 0 (queries
// i < w2 - 1) get q~ = 0 and weight 0 in the merge.
#include "mfma_common.h"

namespace sa {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;

template <int D>
struct FwdLds {
  static constexpr int kStride = D + 8;   // K rows (bf16): 16-byte pad keeps b128 reads conflict-free
  static constexpr int vStride = 32 + 4;  // V^T rows (bf16): 8-byte pad keeps b64 reads conflict-free
  static constexpr int rStride = D + 4;   // epilogue rows (fp32)
  static constexpr int kBytes = 32 * kStride * 2;
  static constexpr int vBytes = D * vStride * 2;
  static constexpr int bufBytes = kBytes + vBytes;
  static constexpr int mainBytes = 2 * bufBytes;
  static constexpr int redBytes = kWaves * 32 * rStride * 4;
  static constexpr int bytes = mainBytes > redBytes ? mainBytes : redBytes;
};

template <int D, int G>
__global__ __launch_bounds__(kThreads) void fwd_mfma_kernel(Shape s, const uint16_t* __restrict__ q,
                                                            const uint16_t* __restrict__ k,
                                                            const uint16_t* __restrict__ kp,
                                                            const uint16_t* __restrict__ v,
                                                            const uint16_t* __restrict__ vp,
                                                            uint16_t* __restrict__ out,
                                                            float* __restrict__ lse) {
  constexpr int NT = D / 16;   // K-steps of the logit product
  constexpr int NDT = D / 32;  // 32-wide d tiles of the output product
  constexpr int QW = 8 / G;    // queries per workgroup
  constexpr int W2P = 32 * G;  // rows per query (w2 padded up to a multiple of 32)
  using L = FwdLds<D>;
  __shared__ __attribute__((aligned(16))) char smem[L::bytes];

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
  const size_t rs = static_cast<size_t>(s.H) * D;
  const size_t base = (static_cast<size_t>(b) * s.N * s.H + hh) * D;
  const int N = s.N, w1 = s.w1, w2 = s.w2;
  const int i0 = tile * QW;

  // ---- modulated queries q~ = (scale*log2 e) * q_i o k'_k as B operands ----
  int qidx[2], kofs[2];
#pragma unroll
  for (int g = 0; g < 2; ++g) {
    qidx[g] = G == 1 ? 2 * wave + g : wave;
    kofs[g] = G == 1 ? 0 : 32 * g;
  }
  const float qscale = s.scale * kLog2e;
  u32x4_t qt[2][NT];
  bool rowvalid[2];
#pragma unroll
  for (int g = 0; g < 2; ++g) {
    const int i = i0 + qidx[g];
    const int kk = i - W2P + 1 + kofs[g] + c;
    rowvalid[g] = i < N && kk >= 0 && kk > i - w2;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      u32x4_t r4 = {0u, 0u, 0u, 0u};
      if (rowvalid[g]) {
        const u32x4_t a = ldg128(q + base + i * rs + 16 * t + 8 * h);
        const u32x4_t bb = ldg128(kp + base + kk * rs + 16 * t + 8 * h);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          r4[e] = pack_bf16x2(bf16_lo(a[e]) * bf16_lo(bb[e]) * qscale,
                              bf16_hi(a[e]) * bf16_hi(bb[e]) * qscale);
        }
      }
      qt[g][t] = r4;
    }
  }

  // ---- staging of K / V^T blocks --------------------------------------------
  const int jlo = i0 - w1 + 1;
  const int nb = (w1 + QW - 1 + 31) / 32;
  constexpr int KCH = 32 * D / 8;                 // 16-byte chunks of a K block
  constexpr int KPT = (KCH + kThreads - 1) / kThreads;
  constexpr int VCOLS = D / 8;                    // 8-wide column chunks of a V row
  const int vpair = tid & 15, vcol = tid >> 4;    // V: rows (2*vpair, 2*vpair+1), cols 8*vcol..
  const bool vactive = vcol < VCOLS;

  u32x4_t kreg[KPT];
  u32x4_t vreg[2];
  auto load_block = [&](int blk) {
    const int jb = jlo + 32 * blk;
#pragma unroll
    for (int x = 0; x < KPT; ++x) {
      const int ch = tid + x * kThreads;
      const int row = ch / (D / 8), col = ch % (D / 8);
      const int j = jb + row;
      u32x4_t z = {0u, 0u, 0u, 0u};
      if (ch < KCH && j >= 0 && j < N) z = ldg128(k + base + j * rs + 8 * col);
      kreg[x] = z;
    }
#pragma unroll
    for (int y = 0; y < 2; ++y) {
      const int j = jb + 2 * vpair + y;
      u32x4_t z = {0u, 0u, 0u, 0u};
      if (vactive && j >= 0 && j < N) z = ldg128(v + base + j * rs + 8 * vcol);
      vreg[y] = z;
    }
  };
  auto store_block = [&](int buf) {
    uint16_t* kb = reinterpret_cast<uint16_t*>(smem + buf * L::bufBytes);
    uint16_t* vb = reinterpret_cast<uint16_t*>(smem + buf * L::bufBytes + L::kBytes);
#pragma unroll
    for (int x = 0; x < KPT; ++x) {
      const int ch = tid + x * kThreads;
      if (ch < KCH) {
        const int row = ch / (D / 8), col = ch % (D / 8);
        *reinterpret_cast<u32x4_t*>(kb + row * L::kStride + 8 * col) = kreg[x];
      }
    }
    if (vactive) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        // columns 8*vcol + 2e (low halves) and 8*vcol + 2e + 1 (high halves)
        const unsigned a = vreg[0][e], bb = vreg[1][e];
        const unsigned lo = (a & 0xffffu) | (bb << 16);
        const unsigned hi = (a >> 16) | (bb & 0xffff0000u);
        *reinterpret_cast<unsigned*>(vb + (8 * vcol + 2 * e) * L::vStride + 2 * vpair) = lo;
        *reinterpret_cast<unsigned*>(vb + (8 * vcol + 2 * e + 1) * L::vStride + 2 * vpair) = hi;
      }
    }
  };

  f32x16_t acc[2][NDT];
#pragma unroll
  for (int g = 0; g < 2; ++g)
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt) acc[g][dt] = f32x16_t{};
  float m[2] = {-INFINITY, -INFINITY};
  float l[2] = {0.f, 0.f};

  load_block(0);
  store_block(0);
  __syncthreads();

  for (int blk = 0; blk < nb; ++blk) {
    const int cur = blk & 1;
    if (blk + 1 < nb) load_block(blk + 1);

    const uint16_t* kb = reinterpret_cast<const uint16_t*>(smem + cur * L::bufBytes);
    const uint16_t* vb = reinterpret_cast<const uint16_t*>(smem + cur * L::bufBytes + L::kBytes);

    // Column range of each group's query inside this block (block-local).
    int lo[2], hi[2];
    bool act[2];
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      lo[g] = max(qidx[g], -jlo) - 32 * blk;
      hi[g] = min(qidx[g] + w1 - 1, N - 1 - jlo) - 32 * blk;
      act[g] = hi[g] >= 0 && lo[g] <= 31 && lo[g] <= hi[g];
    }

    if (act[0] || act[1]) {
      u32x4_t kf[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t)
        kf[t] = *reinterpret_cast<const u32x4_t*>(kb + c * L::kStride + 16 * t + 8 * h);

      f32x16_t sacc[2];
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        sacc[g] = f32x16_t{};
        if (act[g]) {
#pragma unroll
          for (int t = 0; t < NT; ++t) sacc[g] = mfma32(kf[t], qt[g][t], sacc[g]);
        }
      }

      u32x4_t pf[2][2];
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        if (!act[g]) continue;
        float sv[16];
#pragma unroll
        for (int vv = 0; vv < 16; ++vv) sv[vv] = sacc[g][vv];
        if (lo[g] > 0 || hi[g] < 31) {
#pragma unroll
          for (int vv = 0; vv < 16; ++vv) {
            const int jl = 8 * (vv >> 2) + 4 * h + (vv & 3);
            if (jl < lo[g] || jl > hi[g]) sv[vv] = -INFINITY;
          }
        }
        float mx = sv[0];
#pragma unroll
        for (int vv = 1; vv < 16; ++vv) mx = fmaxf(mx, sv[vv]);
        mx = fmaxf(mx, swap_halves(mx));
        const float mnew = fmaxf(m[g], mx);
        const float alpha = fast_exp2(m[g] - mnew);
        float ps = 0.f;
#pragma unroll
        for (int vv = 0; vv < 16; ++vv) {
          sv[vv] = fast_exp2(sv[vv] - mnew);
          ps += sv[vv];
        }
        l[g] = l[g] * alpha + ps;
        m[g] = mnew;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) acc[g][dt] *= alpha;
#pragma unroll
        for (int u = 0; u < 2; ++u) {
#pragma unroll
          for (int e = 0; e < 4; ++e) pf[g][u][e] = pack_bf16x2(sv[8 * u + 2 * e], sv[8 * u + 2 * e + 1]);
        }
      }

#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const uint16_t* row = vb + (32 * dt + c) * L::vStride + 16 * u + 4 * h;
          const u32x2_t a0 = *reinterpret_cast<const u32x2_t*>(row);
          const u32x2_t a1 = *reinterpret_cast<const u32x2_t*>(row + 8);
          const u32x4_t vf = {a0[0], a0[1], a1[0], a1[1]};
#pragma unroll
          for (int g = 0; g < 2; ++g)
            if (act[g]) acc[g][dt] = mfma32(vf, pf[g][u], acc[g][dt]);
        }
      }
    }

    if (blk + 1 < nb) store_block(cur ^ 1);
    __syncthreads();
  }

  // ---- epilogue: merge the k-rows of each query (log-sum-exp), apply v'_k ----
  float lsum[2], wgt[2];
#pragma unroll
  for (int g = 0; g < 2; ++g) lsum[g] = l[g] + swap_halves(l[g]);
  float* red = reinterpret_cast<float*>(smem) + wave * 32 * L::rStride;
  constexpr int NQ = G == 1 ? 2 : 1;  // queries per wavefront
#pragma unroll
  for (int qq = 0; qq < NQ; ++qq) {
    const int i = i0 + (G == 1 ? qidx[qq] : qidx[0]);
    // row log-sum-exps (log2 units) of the query's rows
    float mq = -INFINITY;
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      if (G == 1 && g != qq) continue;
      const float r2 = rowvalid[g] ? m[g] + fast_log2(lsum[g]) : -INFINITY;
      mq = fmaxf(mq, r2);
    }
    mq = max32(mq);
    float z = 0.f;
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      if (G == 1 && g != qq) continue;
      z += rowvalid[g] ? fast_exp2(m[g] + fast_log2(lsum[g]) - mq) : 0.f;
    }
    z = sum32(z);
    const float lse2 = mq + fast_log2(z);
#pragma unroll
    for (int g = 0; g < 2; ++g) wgt[g] = rowvalid[g] ? fast_exp2(m[g] - lse2) : 0.f;

    float o0 = 0.f, o1 = 0.f;
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      if (G == 1 && g != qq) continue;
      const int kk = i - W2P + 1 + kofs[g] + c;
      const bool ldv = rowvalid[g];
      // red[c][d] = w_r * v'_k[d] * U_r[d] for this lane's row c, then column sums.
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
#pragma unroll
        for (int qd = 0; qd < 4; ++qd) {
          const int d = 32 * dt + 8 * qd + 4 * h;
          u32x2_t vv = {0u, 0u};
          if (ldv) vv = *reinterpret_cast<const u32x2_t*>(vp + base + kk * rs + d);
          float4 val;
          val.x = wgt[g] * bf16_lo(vv[0]) * acc[g][dt][4 * qd + 0];
          val.y = wgt[g] * bf16_hi(vv[0]) * acc[g][dt][4 * qd + 1];
          val.z = wgt[g] * bf16_lo(vv[1]) * acc[g][dt][4 * qd + 2];
          val.w = wgt[g] * bf16_hi(vv[1]) * acc[g][dt][4 * qd + 3];
          *reinterpret_cast<float4*>(red + c * L::rStride + d) = val;
        }
      }
      __syncthreads();
      if (2 * lane < D) {
#pragma unroll 8
        for (int rr = 0; rr < 32; ++rr) {
          const float2 x = *reinterpret_cast<const float2*>(red + rr * L::rStride + 2 * lane);
          o0 += x.x;
          o1 += x.y;
        }
      }
      __syncthreads();
    }
    if (i < N) {
      if (2 * lane < D)
        *reinterpret_cast<unsigned*>(out + base + i * rs + 2 * lane) = pack_bf16x2(o0, o1);
      if (lane == 0) lse[static_cast<size_t>(bh) * N + i] = lse2 * kLn2;
    }
  }
}

template <int D, int G>
hipError_t launch(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                  const void* vp, void* out, float* lse, hipStream_t st) {
  constexpr int QW = 8 / G;
  const long tiles = (s.N + QW - 1) / QW;
  const long total = tiles * s.B * s.H;
  const long grid = ((total + 7) / 8) * 8;
  hipLaunchKernelGGL((fwd_mfma_kernel<D, G>), dim3(static_cast<unsigned>(grid)), dim3(kThreads), 0,
                     st, s, static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                     static_cast<const uint16_t*>(kp), static_cast<const uint16_t*>(v),
                     static_cast<const uint16_t*>(vp), static_cast<uint16_t*>(out), lse);
  return hipGetLastError();
}

}  // namespace

bool mfma_fwd_supported(const Shape& s) {
  return s.dtype == 1 && (s.D == 64 || s.D == 128) && s.w2 <= 64;
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
