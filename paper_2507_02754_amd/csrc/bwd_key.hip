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
//
// Fused backward (FUSED, w2 <= 32). The query-side gradients come from the
// same P and dS, so S and dP are computed once for all five gradients:
//     dQ~_r = sum_j dS_rj k_j,   U~_r = sum_j P_rj v_j   (over this
//     workgroup's 128 keys: a partial sum), then
//     dq_i  += sum_k k'_k o dQ~_r,  dk'_k += q_i o dQ~_r,  dv'_k += dO_i o U~_r
// (scale applied by the reduction). D / 32 more wavefronts (role C) each own
// 32 columns d: they read P and dS of all four key groups from the exchange
// areas with the transposing LDS read (keys along the contraction), multiply
// by their columns of V and K (held in registers), and keep dk' and dv' in
// registers as rings of 32 k-rows. For that the tile rows are ordered by
// k mod 32 (row s holds the k-row k = s mod 32 of the window), so a k-row
// keeps its register from the query that first sees it to the one that last
// does; each row block completes one k-row, whose partial sum is stored.
// Every workgroup stores its partial sums of dq (per query), dk' and dv' (per
// k-row) in the workspace; fused_reduce_kernel adds the partials of the
// workgroups in ascending order, so the result is deterministic. P and dS of
// rows outside the window are set to zero (U~ and dQ~ would otherwise see
// them).
#include "mfma_common.h"

#include <type_traits>

namespace sa {
namespace {

constexpr int kKeyWaves = 8;
constexpr int kKeyThreads = 64 * kKeyWaves;
constexpr int kSlots = 4;  // tile slots in LDS (the loop unroll factor)

// Key groups of 32 keys per workgroup: 4 (128 keys), 2 in the fused backward
// (64 keys, so that roles A and B keep two wavefronts per SIMD with role C).
template <bool FUSED>
constexpr int key_groups() {
  return FUSED ? 2 : 4;
}
// Threads of a workgroup: one role-A and one role-B wavefront per key group,
// plus D / 32 of role C in the fused backward.
template <int D, bool FUSED>
constexpr int key_threads() {
  return 64 * (2 * key_groups<FUSED>() + (FUSED ? D / 32 : 0));
}

template <int D, bool FUSED>
struct KeyLds {
  using T = SwzTile<D>;
  static constexpr int tileBytes = 2 * T::bytes;         // q~ tile, then do~ tile
  static constexpr int NKG = key_groups<FUSED>();
  static constexpr int KW = 32 * NKG;                    // keys of a workgroup
  static constexpr int xOff = kSlots * tileBytes;        // P exchange: [2][NKG groups][2 KB]
  static constexpr int xBuf = NKG * 2048;
  static constexpr int xBytes = 2 * xBuf;
  static constexpr int dsOff = xOff + xBytes;            // fused: dS exchange, same layout
  // fused: K^T and V^T of the workgroup's keys ([D][KW] bf16 each, role C)
  static constexpr int ktRow = 2 * KW;
  static constexpr int ktOff = dsOff + (FUSED ? xBytes : 0);
  static constexpr int mainBytes = ktOff + (FUSED ? 2 * D * ktRow : 0);
  static constexpr int oStride = D + 4;                  // fp32 staging rows of the store
  static constexpr int outBytes = 4 * 32 * oStride * 4;  // one role at a time
  static constexpr int bytes = mainBytes > outBytes ? mainBytes : outBytes;
};

template <int X>
using ic = std::integral_constant<int, X>;

// FORM 1: determinant logits (Section 5): role A forms q~ = k'_k x q_i per
// 3-component chunk (unscaled), so S = q~ K^T is the determinant logit and
// dK = scale sum_r dS_rj q~_r as for the trilinear form.
// GQ: grouped-query attention with fewer K-side heads than query heads (the
// workgroup walks several query heads' row blocks); otherwise one query head
// per K-side head, with no group indexing in the loop.
template <int D, int G, bool BIAS, int FORM, bool FUSED, bool GQ>
__device__ __forceinline__ void key_body(
    Shape s, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ kp, const uint16_t* __restrict__ v, const uint16_t* __restrict__ vp,
    const uint16_t* __restrict__ dout, const float* __restrict__ lse, const float* __restrict__ delta,
    uint16_t* __restrict__ dk, uint16_t* __restrict__ dv, FusedPlan fp, float* __restrict__ part) {
  constexpr int NT = D / 16, NDT = D / 32;
  constexpr int W2P = 32 * G;
  static_assert(!FUSED || (G == 1 && FORM == 0 && !GQ), "fused backward: w2 <= 32, trilinear logits, Hkv = H");
  using L = KeyLds<D, FUSED>;
  using T = typename L::T;
  // tile items (row, 16-byte chunk) per thread of a forming role (64 NKG threads)
  constexpr int IPT = T::CH / (2 * key_groups<FUSED>());
  constexpr int RPI = 32 / IPT;   // rows covered by one pass of a role's threads
  constexpr int NKG = L::NKG, KW = L::KW;
  __shared__ __attribute__((aligned(16))) char smem[L::bytes];

  // Grouped-query attention: a workgroup owns keys of one K-side head hk and
  // walks the row blocks of its QG query heads hk QG .. hk QG + QG - 1 in turn
  // (dK, dV accumulate over all of them).
  const int Hkv = GQ ? s.Hkv : s.H, QG = GQ ? s.H / s.Hkv : 1;
  const int jblocks = (s.N + KW - 1) / KW;
  const int total = jblocks * s.B * Hkv;
  const int per_xcd = (total + 7) / 8;
  const int logical = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (logical >= total) return;
  const int bk = logical / jblocks;
  const int jblk = logical - bk * jblocks;
  const int b = bk / Hkv, hk = bk - b * Hkv;
  const int bh = b * s.H + hk * QG;  // (batch, first query head)

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // Roles by halves: wavefronts w and w + 4 of a 512-thread workgroup run on
  // the same SIMD, so each SIMD holds one role-A and one role-B wavefront
  // (measured faster than alternating roles, which pairs two wavefronts of the
  // same role on a SIMD). Role B's key groups are rotated by two, so the two
  // wavefronts sharing a SIMD belong to different key groups and do not reach
  // their exchange points in lockstep (measured 2.5% faster than pairing the
  // two roles of one key group).
  // Fused (two key groups): wavefronts 0, 1 take role A, 2, 3 role B and
  // 4 .. 4 + D / 32 - 1 role C, so each SIMD holds one wavefront of role C.
  const int role = wave < NKG ? 0 : wave < 2 * NKG ? 1 : 2;
  const bool roleA = role == 0;
  const int kg = roleA ? wave : NKG == 4 ? (wave + 2) & 3 : wave - NKG;  // key group (A, B)
  const int lane = tid & 63, c = lane & 31, h = lane >> 5;
  const int rsb = s.H * D * 2;   // bytes between rows of q, dO
  const int rsbk = Hkv * D * 2;  // bytes between rows of K, K', V, V', dK, dV
  const size_t basek = (static_cast<size_t>(b) * s.N * Hkv + hk) * D;
  // q, dO of the group's first query head; head hg of the group is hg * 2 D bytes further
  const size_t base = (static_cast<size_t>(b) * s.N * s.H + hk * QG) * D;
  const int N = s.N, w1 = s.w1, w2 = s.w2;
  const float qscale = s.scale * kLog2e;
  const size_t stat = static_cast<size_t>(bh) * N;  // LSE / Delta of the group's first query head
  const int j0 = jblk * KW;
  const int jw = j0 + 32 * kg;  // keys jw .. jw + 31 of this wavefront
  const int jme = jw + c;       // key of this lane's accumulator column
  const unsigned hb = head_bytes(N, rsb, D) + (QG - 1) * 2 * D, hbk = head_bytes(N, rsbk, D);

  // K (role A) or V (role B) rows of the group as B operands: lane (h, c) holds
  // key jw + c, d = 16 t + 8 h .. + 7. Keys past the end load as zeros.
  u32x4_t kv[NT];
  if (role < 2) {
    const __amdgpu_buffer_rsrc_t r = make_rsrc((roleA ? k : v) + basek, hbk);
#pragma unroll
    for (int t = 0; t < NT; ++t) kv[t] = ldbuf128(r, jme * rsbk + 32 * t + 16 * h);
  }
  f32x16_t acc[NDT];
#pragma unroll
  for (int dt = 0; dt < NDT; ++dt) acc[dt] = f32x16_t{};

  // Row blocks: (query i, k-chunk g) for i in [j0, min(N, j0 + KW - 1 + w1)),
  // padded to a multiple of the unroll factor (the padding is inactive).
  // The fused kernel runs one more iteration: role C takes the dQ~ products
  // of a row block one iteration after its U~ products.
  const int i_end = min(N, j0 + KW - 1 + w1);
  const int nrb = (i_end - j0) * G;
  const int nrb4 = (nrb + (FUSED ? 1 : 0) + kSlots - 1) / kSlots * kSlots;

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
  // P exchange of this group (and, fused, the dS exchange dsOff - xOff
  // further): [buffer][u] blocks of 1 KB, 16 bytes per lane. In the fused
  // kernel lane (h, c) stores fragment u at slot 32 h + (c ^ (8 h + 4 u)), so
  // that role C's transposing reads of every group are free of bank
  // conflicts.
  int xl[2];
  xl[0] = L::xOff + kg * 2048 + 16 * (FUSED ? 32 * h + (c ^ (8 * h)) : lane);
  xl[1] = FUSED ? L::xOff + kg * 2048 + 1024 + 16 * (32 * h + (c ^ (8 * h + 4))) : xl[0] + 1024;

  // ---- tile formation (role A: q~ = q_i o k'_k, role B: do~ = dO_i o v'_k) ----
  // Thread u of a role forms rows rho + RPI y (y < IPT), 16-byte chunk dc, so
  // the 16 lanes of a store group write 16 consecutive swizzled rows.
  const int u = kg * 64 + lane;  // index of this thread within its role
  const int rho = u % RPI, dc = u / RPI;
  const __amdgpu_buffer_rsrc_t rrow = make_rsrc((roleA ? q : dout) + base, hb);
  const __amdgpu_buffer_rsrc_t rmod = make_rsrc((roleA ? kp : vp) + basek, hbk);
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
  // Row blocks of a workgroup: those of query head 0 of the group, padded to
  // nrb4, then those of head 1, ... (R = hg nrb4 + rb = hgb + rb). The steps
  // take the local rb of head hg; loc / hof map rb + k (k <= 4, possibly past
  // the end of head hg) to its local index and head. Only the guarded steps
  // (cross: std::true_type) reach past the end of a head: the straight-line
  // ones end 4 row blocks before nrb4.
  int hg = 0, hgb = 0;
  auto loc = [&](int r, auto cross) {
    if constexpr (!GQ || !decltype(cross)::value)
      return r;
    else
      return r < nrb4 ? r : r - nrb4;
  };
  auto hof = [&](int r, auto cross) {
    if constexpr (!GQ)
      return 0;
    else if constexpr (!decltype(cross)::value)
      return hg;
    else
      return r < nrb4 ? hg : hg + 1;
  };
  auto fetch = [&](int rb, auto set, auto cross) __attribute__((always_inline)) {
    constexpr int X = decltype(set)::value;
    const int r = loc(rb, cross), hq = hof(rb, cross);  // row block r of query head hq of the group
    const int i = j0 + r / G, g = r % G;
    const int qoff = hq < QG ? i * rsb + hq * 2 * D + 16 * dc : -1;
    fr[X] = ldbuf128(rrow, qoff);
    if constexpr (FORM == 1) {
      if (roleA) {
        frw[X][0] = ldbuf32(rrow, qoff - 4);
        frw[X][1] = ldbuf32(rrow, qoff + 16);
      }
    }
#pragma unroll
    for (int y = 0; y < IPT; ++y) {
      // fused: row rho + RPI y of the tile holds the k-row congruent to it mod 32
      const int kk = FUSED ? i - ((i - rho - RPI * y) & 31) : i - W2P + 1 + 32 * g + rho + RPI * y;
      const bool inwin = kk > i - w2 && (!BIAS || kk >= 0);  // kk < 0 also loads zeros
      fm[X][y] = ldbuf128(rmod, inwin ? kk * rsbk + 16 * dc : -1);
      if constexpr (FORM == 1) {
        if (roleA) {
          fmw[X][y][0] = ldbuf32(rmod, inwin ? kk * rsbk + 16 * dc - 4 : -1);
          fmw[X][y][1] = ldbuf32(rmod, inwin ? kk * rsbk + 16 * dc + 16 : -1);
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
  // of row block (R & ~63) + l (A: -LSE * log2 e, B: Delta), taken with a
  // lane read. The next 64 values are loaded half a window ahead. stat_at
  // must be called for every row block in order (R = hg nrb4 + rb).
  const float* statp = roleA ? lse : delta;
  auto stat_load = [&](int rb0) {  // rb0: R of the first of 64 row blocks
    const int rg = rb0 + lane, hq = GQ ? rg / nrb4 : 0;
    const int ii = min(j0 + (rg - hq * nrb4) / G, N - 1);
    const float x = statp[stat + static_cast<size_t>(min(hq, QG - 1)) * N + ii];
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
  // Fused: K^T and V^T of the KW keys for role C. Row d of K^T holds the keys
  // in KW / 8 chunks of 16 bytes; chunk 4 g + 2 u + h (stored at chunk slot
  // (4 g + 2 u + h) ^ ((d / 2) % 8), free of bank conflicts for the 16 rows a
  // lane group reads) holds keys 32 g + 16 u + 4 h + {0..3} and
  // 32 g + 16 u + 8 + 4 h + {0..3}: the 8 keys, in the order of the P and dS
  // fragments, that lane half h needs for MFMA (g, u).
  if constexpr (FUSED) {
    const __amdgpu_buffer_rsrc_t rk = make_rsrc(k + basek, hbk), rv = make_rsrc(v + basek, hbk);
    constexpr int NTH = key_threads<D, FUSED>();
    for (int x = tid; x < 2 * KW * T::CH; x += NTH) {
      const int tens = x / (KW * T::CH), key = (x / T::CH) % KW, ch = x % T::CH;
      const u32x4_t w = ldbuf128(tens ? rv : rk, (j0 + key) * rsbk + 16 * ch);
      const int r16 = key & 15;
      const int chunk = 4 * (key >> 5) + 2 * ((key >> 4) & 1) + ((r16 >> 2) & 1);
      const int pos = 4 * (r16 >> 3) + (r16 & 3);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int d = 8 * ch + e;
        const unsigned short val = static_cast<unsigned short>((e & 1) ? (w[e >> 1] >> 16) : (w[e >> 1] & 0xffffu));
        *reinterpret_cast<unsigned short*>(smem + L::ktOff + tens * D * L::ktRow + d * L::ktRow +
                                           16 * (chunk ^ ((d >> 1) & 7)) + 2 * pos) = val;
      }
    }
  }
  // tiles 0 and 1 (fused: role B forms the do~ halves, role C the q~ halves)
  if (FUSED ? role == 1 : true) {
    fetch(0, ic<0>{}, std::false_type{});
    form_put(0, ic<0>{});
    fetch(1, ic<0>{}, std::false_type{});
    form_put(L::tileBytes, ic<0>{});
    fetch(2, ic<0>{}, std::false_type{});
    if (roleA) fetch(3, ic<1>{}, std::false_type{});
  }
  // The loops start with every load complete (the wait-count pass would
  // otherwise keep the K/V operand loads pending into every iteration).
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  lds_barrier();

  // Row blocks [rb_lo, rb_hi) have every key group active for rb and rb + 1:
  // there the steps run without the activity tests, as straight-line code
  // the scheduler can interleave. Bounds are multiples of the unroll factor.
  // (the last group starts at key j0 + 32 (NKG - 1); fused: row block rb - 1 too)
  int rb_lo = ((FUSED ? 32 * (NKG - 1) + 1 : 32 * (NKG - 1) * G) + kSlots - 1) / kSlots * kSlots;
  int rb_hi = min((w1 + 30) * G - 1, min(nrb - 1, (N - j0) * G - 1));
  rb_hi = rb_hi / kSlots * kSlots;
  if (j0 + 32 * (NKG - 1) >= N || rb_hi < rb_lo) rb_lo = rb_hi = nrb4;
  auto run_loops = [&](auto& step) __attribute__((always_inline)) {
    auto quad = [&](int rb, auto guard) __attribute__((always_inline)) {
      step(rb, ic<0>{}, guard);
      step(rb + 1, ic<1>{}, guard);
      step(rb + 2, ic<2>{}, guard);
      step(rb + 3, ic<3>{}, guard);
    };
    for (hg = 0, hgb = 0; hg < QG; ++hg, hgb += nrb4) {
      int rb = 0;
      for (; rb < rb_lo; rb += kSlots) quad(rb, ic<1>{});
      for (; rb < rb_hi; rb += kSlots) quad(rb, ic<0>{});
      for (; rb < nrb4; rb += kSlots) quad(rb, ic<1>{});
    }
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
    auto probs = [&](int rb, float nlse2, const f32x16_t& sacc, int xb, u32x4_t* pf, auto cross)
                     __attribute__((always_inline)) {
      const int i = j0 + loc(rb, cross) / G;
      const bool colok = jme <= i && jme > i - w1 && jme < N;
      const float nl = nlse2 - (colok ? 0.f : __builtin_inff());
      // p = 2^min(x, 0): at most 1, so rows formed as zeros (whose statistic
      // may belong to another query) stay finite. Written as a [0, 1] clamp of
      // 2^x, which the compiler folds into the exponential's clamp bit.
      float pr[16];
#pragma unroll
      for (int vv = 0; vv < 16; ++vv)
        pr[vv] = __builtin_amdgcn_fmed3f(fast_exp2(__builtin_fmaf(sacc[vv], qscale, nl)), 0.f, 1.f);
      if constexpr (FUSED) {
        // rows (k-row slots) outside query i's window: P = 0 (U~ and dQ~ read it)
        if (w2 < 32 || i < 31) {
#pragma unroll
          for (int vv = 0; vv < 16; ++vv) {
            const int dd = (i - acc_row(vv, h)) & 31;  // i - k of this row
            if (dd >= w2 || dd > i) pr[vv] = 0.f;
          }
        }
      }
#pragma unroll
      for (int uu = 0; uu < 2; ++uu) {
        pf[uu] = pack_frag(pr, uu);
        lds_st(lds + xl[uu] + xb, pf[uu]);
      }
    };
    u32x4_t pcur[2];  // P of the row block whose dV is next (set only when active)
    if constexpr (FUSED) lds_barrier();  // role C has formed tiles 0 and 1
    {
      const float nl0 = stat_at(0);
      if (is_active(0, j0)) probs(0, nl0, logits(0), 0, pcur, std::false_type{});
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
      const bool act1 = !kGuard || is_active(loc(rb + 1, guard), j0 + loc(rb + 1, guard) / G);
      const float nl1 = stat_at(hgb + rb + 1);
      f32x16_t snext;
      u32x4_t pnext[2];
      if constexpr (!kGuard && FUSED) {
        // Straight-line with the fragment reads spread over the products (the
        // register budget of three wavefronts per SIMD): S products, then the
        // dV products with the probabilities between them.
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
#pragma unroll
        for (int uu = 0; uu < 2; ++uu)
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt) acc[dt] = mfma32(pcur[uu], otr[uu][dt], acc[dt]);
        probs(rb + 1, nl1, snext, (S1 & 1) * L::xBuf, pnext, guard);
#pragma unroll
        for (int x = 0; x < NT; ++x) {
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // q~ row fragment
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // S product
        }
#pragma unroll
        for (int x = 0; x < 2 * NDT; ++x) {
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // do~ transposed fragment
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // dV product
          __builtin_amdgcn_sched_group_barrier(0x002, 7, 0);  // probabilities
        }
      } else if constexpr (!kGuard) {
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
        if constexpr (!FUSED) form_put(S2 * L::tileBytes, ic<S & 1>{});
#pragma unroll
        for (int uu = 0; uu < 2; ++uu)
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt) acc[dt] = mfma32(pcur[uu], otr[uu][dt], acc[dt]);
        probs(rb + 1, nl1, snext, (S1 & 1) * L::xBuf, pnext, guard);
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
        if (act1) probs(rb + 1, nl1, snext, (S1 & 1) * L::xBuf, pnext, guard);
        if constexpr (!FUSED) form_put(S2 * L::tileBytes, ic<S & 1>{});
      }
      if constexpr (!FUSED) fetch(rb + 4, ic<S & 1>{}, guard);
      pcur[0] = pnext[0];
      pcur[1] = pnext[1];
      __builtin_amdgcn_s_setprio(0);
      lds_barrier();
    };
    run_loops(step);
  } else if (role == 1) {
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
    if constexpr (FUSED) lds_barrier();  // role C has formed tiles 0 and 1
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
      const bool act1 = !kGuard || is_active(loc(rb + 1, guard), j0 + loc(rb + 1, guard) / G);
      const float dlt = stat_at(hgb + rb);
      f32x16_t dpnext;
      if constexpr (!kGuard && !FUSED) {
        // Straight-line: reads first, then the dP products of row block rb + 1
        // interleaved with dS of row block rb, then the dK products with the
        // formation of tile rb + 2.
        u32x4_t pf[2], oa[NT], qtr[2][NDT];
#pragma unroll
        for (int uu = 0; uu < 2; ++uu) pf[uu] = lds_ld<u32x4_t>(lds + xl[uu] + (S & 1) * L::xBuf);
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
        if constexpr (FUSED) {
#pragma unroll
          for (int uu = 0; uu < 2; ++uu) lds_st(lds + xl[uu] + (L::dsOff - L::xOff) + (S & 1) * L::xBuf, df[uu]);
        }
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
          for (int uu = 0; uu < 2; ++uu) pf[uu] = lds_ld<u32x4_t>(lds + xl[uu] + (S & 1) * L::xBuf);
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
            if constexpr (FUSED) lds_st(lds + xl[uu] + (L::dsOff - L::xOff) + (S & 1) * L::xBuf, df);
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) acc[dt] = mfma32(df, qtr[uu][dt], acc[dt]);
          }
        }
        form_put(S2 * L::tileBytes, ic<0>{});
      }
      fetch(rb + 3, ic<0>{}, guard);
      dpcur = dpnext;
      __builtin_amdgcn_s_setprio(0);
      lds_barrier();
    };
    run_loops(step);
  } else if constexpr (FUSED) {
    // ---- role C: columns col = 32 xs + c of U~ and dQ~, dk' and dv' rings ----
    const int xs = wave - 2 * NKG;
    const int col = 32 * xs + c;
    // Transposing reads of an exchange area: lane (h, c) receives row (slot) c
    // and keys 32 g + 16 u + 8 (e / 4) + 4 h + e % 4, e = 0..7, of the
    // fragments group g stored (the key order of kx / vx). Within a group of
    // 16 lanes, lane l addresses 4 slots of key 4 h + 8 r + l / 4 (r: first or
    // second read) in the slot 32 (l & 1) + (key ^ (8 (l & 1) + 4 u')) of
    // block u' = (lane / 16) & 1.
    const __amdgpu_buffer_rsrc_t rq = make_rsrc(q + base, hb), rdo = make_rsrc(dout + base, hb),
                                 rkp = make_rsrc(kp + basek, hbk);
    const int grp = lane >> 4, sl = lane & 15;
    const int hp = grp >> 1, uq = grp & 1, hs1 = sl & 1;
    const int xr0 = L::xOff + 1024 * uq + 512 * hs1 + 16 * (8 * hs1 + 4 * (hp ^ uq) + (sl >> 2)) +
                    8 * ((sl >> 1) & 1);
    const int xr1 = xr0 + 128 * (1 - 2 * hs1);
    auto xfrag = [&](int off) __attribute__((always_inline)) {
      const u32x2_t a = lds_tr16(lds + xr0 + off);
      const u32x2_t bb = lds_tr16(lds + xr1 + off);
      return u32x4_t{a[0], a[1], bb[0], bb[1]};
    };
    // B operands of MFMA (g, u) from K^T / V^T (tens 0 / 1): lane (h, c)
    // reads row col, the chunk of lane half h.
    const int ktb = L::ktOff + col * L::ktRow, ktm = h ^ ((col >> 1) & 7);
    auto ktfrag = [&](int tens, int g, int uu) __attribute__((always_inline)) {
      return lds_ld<u32x4_t>(lds + ktb + tens * D * L::ktRow + 16 * ((4 * g + 2 * uu) ^ ktm));
    };
    // q~ half of the tiles for role A (rows in k mod 32 order; role B forms
    // the do~ half): thread fu forms rows frho + RPIC y, chunk fdc, of tile
    // rb + 2 in iteration rb from loads issued two iterations earlier (two
    // register sets).
    constexpr int IPTC = T::CH / 8, RPIC = 32 / IPTC;  // items per thread of role C's 256
    const int fu = xs * 64 + lane;
    const int frho = fu % RPIC, fdc = fu / RPIC;
    const __amdgpu_buffer_rsrc_t rkp_f = make_rsrc(kp + basek, hbk);
    int foff[IPTC];
#pragma unroll
    for (int y = 0; y < IPTC; ++y) foff[y] = T::off(frho + RPIC * y, fdc);
    u32x4_t cq[2], cm[2][IPTC];
    float cbq[2][IPTC];
    auto fetch_rows = [&](int rb, __amdgpu_buffer_rsrc_t rr, __amdgpu_buffer_rsrc_t rm, float bias, u32x4_t& xr,
                          u32x4_t* xm, float* xb) __attribute__((always_inline)) {
      const int i = j0 + rb;
      xr = ldbuf128(rr, i * rsb + 16 * fdc);
#pragma unroll
      for (int y = 0; y < IPTC; ++y) {
        const int kk = i - ((i - frho - RPIC * y) & 31);
        const bool inwin = kk > i - w2 && (!BIAS || kk >= 0);
        xm[y] = ldbuf128(rm, inwin ? kk * rsbk + 16 * fdc : -1);
        xb[y] = inwin ? bias : 0.f;
      }
    };
    auto put_rows = [&](int off, const u32x4_t& xr, const u32x4_t* xm, const float* xb) __attribute__((always_inline)) {
      float lo[4], hi[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        lo[e] = bf16_lo(xr[e]);
        hi[e] = bf16_hi(xr[e]);
      }
#pragma unroll
      for (int y = 0; y < IPTC; ++y) {
        u32x4_t a4;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          a4[e] = pack_bf16x2(lo[e] * plus_bias<BIAS>(bf16_lo(xm[y][e]), xb[y]),
                              hi[e] * plus_bias<BIAS>(bf16_hi(xm[y][e]), xb[y]));
        lds_st(lds + foff[y] + off, a4);
      }
    };
    auto fetchq = [&](int rb, auto set) __attribute__((always_inline)) {
      constexpr int X = decltype(set)::value;
      fetch_rows(rb, rq, rkp_f, s.kp_bias, cq[X], cm[X], cbq[X]);
    };
    // Key group g reaches row block rb (the test of is_active for group g).
    auto gact = [&](int rb, int g) {
      const int i = j0 + rb, jg = j0 + 32 * g;
      return rb < nrb && jg <= i && jg + 31 > i - w1 && jg < N;
    };
    // Ring registers: lane (h, c) holds slot (k mod 32) acc_row(v, h) in v.
    // take: value of slot sr (sr % 4 == S3) in the lanes holding it, cleared.
    auto take = [&](float* r, auto s3c, int sr) __attribute__((always_inline)) {
      constexpr int S3 = decltype(s3c)::value;
      const int q4 = sr >> 3;
      const bool mine = h == ((sr >> 2) & 1);
      float val = r[S3];
#pragma unroll
      for (int qq = 1; qq < 4; ++qq) val = q4 == qq ? r[4 * qq + S3] : val;
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) r[4 * qq + S3] = (mine && q4 == qq) ? 0.f : r[4 * qq + S3];
      return val;
    };
    // The 16 values are live in registers at this point.
    auto pin16 = [](float* r) __attribute__((always_inline)) {
      asm volatile("" : "+v"(r[0]), "+v"(r[1]), "+v"(r[2]), "+v"(r[3]), "+v"(r[4]), "+v"(r[5]), "+v"(r[6]),
                   "+v"(r[7]), "+v"(r[8]), "+v"(r[9]), "+v"(r[10]), "+v"(r[11]), "+v"(r[12]), "+v"(r[13]),
                   "+v"(r[14]), "+v"(r[15]));
    };
    auto put = [&](float* r, auto s3c, int sr, float x) __attribute__((always_inline)) {
      constexpr int S3 = decltype(s3c)::value;
      const int q4 = sr >> 3;
      const bool mine = h == ((sr >> 2) & 1);
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) r[4 * qq + S3] = (mine && q4 == qq) ? x : r[4 * qq + S3];
    };
    // Element col of row `row` (0 outside the sequence).
    auto ld1 = [&](__amdgpu_buffer_rsrc_t r, int row, int stride) {
      return bf16_to_f32(__builtin_amdgcn_raw_buffer_load_b16(r, row * stride + 2 * col, 0, 0));
    };
    float dvr[16], dkr[16], kpr[16];
#pragma unroll
    for (int vv = 0; vv < 16; ++vv) {
      // k' ring for the row block before the first: k-rows j0 - 32 .. j0 - 1
      const int kap = j0 - 32 + acc_row(vv, h);
      kpr[vv] = plus_bias<BIAS>(ld1(rkp, kap, rsbk), kap >= 0 ? s.kp_bias : 0.f);
      dvr[vv] = 0.f;
      dkr[vv] = 0.f;
    }
    const size_t wg = static_cast<size_t>(bh) * fp.njb + jblk;
    float* const pq = part + fp.pq_off + wg * fp.RQ * D + col;            // row i - j0
    float* const pk = part + fp.pk_off + wg * fp.RK * D + col - (j0 - 31) * D;  // row k
    float* const pv = part + fp.pv_off + wg * fp.RK * D + col - (j0 - 31) * D;
    // dO_i of row block rb (its U~), q_i and k'_i of row block rb - 1 (its dQ~),
    // each loaded one iteration ahead.
    float do_c = ld1(rdo, j0, rsb), q_c = 0.f, kp_c = 0.f;
    // q~ halves of tiles 0 and 1, loads for tiles 2 and 3
    fetchq(0, ic<0>{});
    put_rows(0, cq[0], cm[0], cbq[0]);
    fetchq(1, ic<0>{});
    put_rows(L::tileBytes, cq[0], cm[0], cbq[0]);
    fetchq(2, ic<0>{});
    fetchq(3, ic<1>{});
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    lds_barrier();  // tiles 0, 1 and K^T, V^T written (the barrier after the roles' first loads)
    lds_barrier();  // the prologue barrier of roles A and B
    auto step = [&](int rb, auto slot, auto guard) __attribute__((always_inline)) {
      // priority above roles A and B: role C's work bounds the iteration
      __builtin_amdgcn_s_setprio(2);
      constexpr int S = decltype(slot)::value;
      constexpr bool kGuard = decltype(guard)::value != 0;
      const int i = j0 + rb;
      const float do_n = ld1(rdo, i + 1, rsb), q_n = ld1(rq, i, rsb), kp_n = ld1(rkp, i, rsbk);
      constexpr int S2 = (S + 2) % kSlots;
      // dv' from U~ of row block rb; dq and dk' from dQ~ of row block rb - 1
      // (k' ring for query i - 1 first)
      auto dv_update = [&](const f32x16_t& ut) __attribute__((always_inline)) {
#pragma unroll
        for (int vv = 0; vv < 16; ++vv) dvr[vv] = __builtin_fmaf(do_c, ut[vv], dvr[vv]);
        const int sr = (i + 1) & 31;  // k-row i - 31: no later query sees it
        const float val = take(dvr, ic<(S + 1) & 3>{}, sr);
        if (h == ((sr >> 2) & 1) && i >= 31) pv[static_cast<size_t>(i - 31) * D] = val;
      };
      auto dq_update = [&](const f32x16_t& qt) __attribute__((always_inline)) {
        const int i1 = i - 1;
        put(kpr, ic<(S + 3) & 3>{}, i1 & 31, plus_bias<BIAS>(kp_c, s.kp_bias));
        float t = 0.f;
#pragma unroll
        for (int vv = 0; vv < 16; ++vv) t = __builtin_fmaf(kpr[vv], qt[vv], t);
        t += swap_halves(t);
        if (h == 0) pq[static_cast<size_t>(i1 - j0) * D] = t;
#pragma unroll
        for (int vv = 0; vv < 16; ++vv) dkr[vv] = __builtin_fmaf(q_c, qt[vv], dkr[vv]);
        const int sr = i & 31;  // k-row i1 - 31
        const float val = take(dkr, ic<S>{}, sr);
        if (h == ((sr >> 2) & 1) && i1 >= 31) pk[static_cast<size_t>(i1 - 31) * D] = val;
      };
      if constexpr (!kGuard) {
        // U~ (P in exchange buffer rb & 1) and dQ~ (dS in buffer (rb - 1) & 1)
        // products alternate, with the tile formation between them
        f32x16_t ut = {}, qt = {};
#pragma unroll
        for (int g = 0; g < NKG; ++g)
#pragma unroll
          for (int uu = 0; uu < 2; ++uu) {
            ut = mfma32(xfrag((S & 1) * L::xBuf + 2048 * g + 256 * uu), ktfrag(1, g, uu), ut);
            qt = mfma32(xfrag((L::dsOff - L::xOff) + ((S + 1) & 1) * L::xBuf + 2048 * g + 256 * uu),
                        ktfrag(0, g, uu), qt);
          }
        put_rows(S2 * L::tileBytes, cq[S & 1], cm[S & 1], cbq[S & 1]);
#pragma unroll
        for (int x = 0; x < 4 * NKG; ++x) {
          __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);  // operand reads
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // product
          __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);  // formation
        }
        __builtin_amdgcn_sched_barrier(0);
        dv_update(ut);
        dq_update(qt);
      } else {
        if (rb < nrb) {
          f32x16_t ut = {};
#pragma unroll
          for (int g = 0; g < NKG; ++g)
            if (gact(rb, g)) {
#pragma unroll
              for (int uu = 0; uu < 2; ++uu)
                ut = mfma32(xfrag((S & 1) * L::xBuf + 2048 * g + 256 * uu), ktfrag(1, g, uu), ut);
            }
          dv_update(ut);
        }
        if (rb >= 1 && rb <= nrb) {
          f32x16_t qt = {};
#pragma unroll
          for (int g = 0; g < NKG; ++g)
            if (gact(rb - 1, g)) {
#pragma unroll
              for (int uu = 0; uu < 2; ++uu)
                qt = mfma32(xfrag((L::dsOff - L::xOff) + ((S + 1) & 1) * L::xBuf + 2048 * g + 256 * uu),
                            ktfrag(0, g, uu), qt);
            }
          dq_update(qt);
        }
        put_rows(S2 * L::tileBytes, cq[S & 1], cm[S & 1], cbq[S & 1]);
      }
      // the loads for tile rb + 4
      fetchq(rb + 4, ic<S & 1>{});
      do_c = do_n;
      q_c = q_n;
      kp_c = kp_n;
      // keep this row block's ring updates on this side of the barrier (the
      // compiler would otherwise carry the products of several row blocks)
      pin16(dvr);
      pin16(dkr);
      pin16(kpr);
      __builtin_amdgcn_s_setprio(0);
      lds_barrier();
    };
    run_loops(step);
    // k-rows i_end - 31 .. i_end - 1 are still in the rings
#pragma unroll
    for (int vv = 0; vv < 16; ++vv) {
      const int kap = i_end - 32 + ((acc_row(vv, h) - (i_end - 32)) & 31);
      if (kap > i_end - 32 && kap >= 0) {
        pv[static_cast<size_t>(kap) * D] = dvr[vv];
        pk[static_cast<size_t>(kap) * D] = dkr[vv];
      }
    }
    // the barriers of the dK / dV store below, which role C does not take part in
#pragma unroll
    for (int x = 0; x < 4; ++x) lds_barrier();
    return;
  }

  // ---- store: accumulator rows are keys, lanes are columns d; one role at a
  // time through fp32 staging rows ----
  const float oscale = roleA ? 1.f : s.scale;  // q~ is formed unscaled
  uint16_t* dst = roleA ? dv : dk;
#pragma unroll
  for (int pass = 0; pass < 2; ++pass) {
    lds_barrier();
    float* ob = reinterpret_cast<float*>(smem) + kg * 32 * L::oStride;
    const bool mine = role < 2 && (pass == 0) == roleA;
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
          *reinterpret_cast<u32x4_t*>(dst + basek + static_cast<size_t>(j) * Hkv * D + 8 * col) = w;
        }
      }
    }
  }
}

// The split path's key-side kernel and the fused backward kernel (one body).
template <int D, int G, bool BIAS, int FORM, bool GQ>
__global__ __launch_bounds__((key_threads<D, false>()), 1) void bwd_key_kernel(
    Shape s, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ kp, const uint16_t* __restrict__ v, const uint16_t* __restrict__ vp,
    const uint16_t* __restrict__ dout, const float* __restrict__ lse, const float* __restrict__ delta,
    uint16_t* __restrict__ dk, uint16_t* __restrict__ dv, FusedPlan fp, float* __restrict__ part) {
  key_body<D, G, BIAS, FORM, false, GQ>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, fp, part);
}
template <int D, bool BIAS>
__global__ __launch_bounds__((key_threads<D, true>()), 1) void bwd_fused_kernel(
    Shape s, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
    const uint16_t* __restrict__ kp, const uint16_t* __restrict__ v, const uint16_t* __restrict__ vp,
    const uint16_t* __restrict__ dout, const float* __restrict__ lse, const float* __restrict__ delta,
    uint16_t* __restrict__ dk, uint16_t* __restrict__ dv, FusedPlan fp, float* __restrict__ part) {
  key_body<D, 1, BIAS, 0, true, false>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, fp, part);
}

template <int D, int G, bool BIAS, int FORM = 0, bool FUSED = false, bool GQ = false>
hipError_t launch_key(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                      const void* vp, const void* dout, const float* lse, const float* delta, void* dk,
                      void* dv, hipStream_t st, const FusedPlan& fp = FusedPlan{}, float* part = nullptr) {
  constexpr int KW = 32 * key_groups<FUSED>();
  const long tot = static_cast<long>((s.N + KW - 1) / KW) * s.B * s.Hkv;
  auto kern = [] {
    if constexpr (FUSED)
      return bwd_fused_kernel<D, BIAS>;
    else
      return bwd_key_kernel<D, G, BIAS, FORM, GQ>;
  }();
  hipLaunchKernelGGL(kern, dim3(static_cast<unsigned>(((tot + 7) / 8) * 8)), dim3(key_threads<D, FUSED>()), 0,
                     st, s, static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k),
                     static_cast<const uint16_t*>(kp), static_cast<const uint16_t*>(v),
                     static_cast<const uint16_t*>(vp), static_cast<const uint16_t*>(dout), lse, delta,
                     static_cast<uint16_t*>(dk), static_cast<uint16_t*>(dv), fp, part);
  return hipGetLastError();
}

// Sum of the fused kernel's partials: one thread per (query or k-row, 4
// columns). Workgroup jb (keys KW jb .. KW jb + KW - 1) holds dq partials of
// the queries i in [KW jb, KW jb + KW - 1 + w1) and dk' / dv' partials of the
// k-rows in [KW jb - 31, KW jb + KW - 1 + w1), clipped to the sequence; they
// are added in ascending jb, and dq, dk' take the factor scale here.
template <int D>
__global__ __launch_bounds__(256) void fused_reduce_kernel(Shape s, FusedPlan fp, const float* __restrict__ part,
                                                           uint16_t* __restrict__ dq, uint16_t* __restrict__ dkp,
                                                           uint16_t* __restrict__ dvp) {
  constexpr int C4 = D / 4;
  const long idx = static_cast<long>(blockIdx.x) * 256 + threadIdx.x;
  const long total = static_cast<long>(s.B) * s.H * s.N * C4;
  if (idx >= total) return;
  const int d = 4 * static_cast<int>(idx % C4);
  const long row = idx / C4;
  const int n = static_cast<int>(row % s.N);
  const int bh = static_cast<int>(row / s.N);
  const int b = bh / s.H, hh = bh - b * s.H;
  const int w1 = s.w1;
  const int kw = fp.kw;
  // first workgroup whose query range reaches n: kw jb + kw - 2 + w1 >= n
  const int lo = n - (kw - 2) - w1 <= 0 ? 0 : (n - (kw - 2) - w1 + kw - 1) / kw;
  const int hiq = n / kw;
  const int hik = min(fp.njb - 1, (n + 31) / kw);
  const size_t wg0 = static_cast<size_t>(bh) * fp.njb;
  float4 aq = {0.f, 0.f, 0.f, 0.f}, ak = aq, av = aq;
#pragma unroll 4
  for (int jb = lo; jb <= hik; ++jb) {
    const size_t wg = wg0 + jb;
    if (jb <= hiq) {
      const float4 x = *reinterpret_cast<const float4*>(part + fp.pq_off + (wg * fp.RQ + (n - kw * jb)) * D + d);
      aq.x += x.x, aq.y += x.y, aq.z += x.z, aq.w += x.w;
    }
    const size_t kr = wg * fp.RK + (n - kw * jb + 31);
    const float4 y = *reinterpret_cast<const float4*>(part + fp.pk_off + kr * D + d);
    const float4 z = *reinterpret_cast<const float4*>(part + fp.pv_off + kr * D + d);
    ak.x += y.x, ak.y += y.y, ak.z += y.z, ak.w += y.w;
    av.x += z.x, av.y += z.y, av.z += z.z, av.w += z.w;
  }
  const size_t o = ((static_cast<size_t>(b) * s.N + n) * s.H + hh) * D + d;
  const float sc = s.scale;
  auto put4 = [&](uint16_t* dst, float4 a, float f) {
    uint2 w;
    w.x = pack_bf16x2(a.x * f, a.y * f);
    w.y = pack_bf16x2(a.z * f, a.w * f);
    *reinterpret_cast<uint2*>(dst + o) = w;
  };
  put4(dq, aq, sc);
  put4(dkp, ak, sc);
  put4(dvp, av, 1.f);
}

}  // namespace

template <bool BIAS>
hipError_t mfma_bwd_key_b(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                          const void* vp, const void* dout, const float* lse, const float* delta,
                          void* dk, void* dv, hipStream_t st) {
  const int G = s.w2 <= 32 ? 1 : 2;
  if constexpr (!BIAS) {
    if (s.Hkv < s.H) {  // grouped-query attention (no bias constants there)
      if (s.D == 128)
        return G == 1 ? launch_key<128, 1, false, 0, false, true>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st)
                      : launch_key<128, 2, false, 0, false, true>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st);
      if (s.D == 64)
        return G == 1 ? launch_key<64, 1, false, 0, false, true>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st)
                      : launch_key<64, 2, false, 0, false, true>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st);
      return hipErrorInvalidValue;
    }
  }
  if (s.D == 128)
    return G == 1 ? launch_key<128, 1, BIAS>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st)
                  : launch_key<128, 2, BIAS>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st);
  if (s.D == 64)
    return G == 1 ? launch_key<64, 1, BIAS>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st)
                  : launch_key<64, 2, BIAS>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st);
  return hipErrorInvalidValue;
}

FusedPlan mfma_fused_plan(const Shape& s) {
  FusedPlan p{};
  const size_t bh = static_cast<size_t>(s.B) * s.H;
  p.kw = 32 * key_groups<true>();
  p.njb = (s.N + p.kw - 1) / p.kw;
  p.RQ = p.kw - 1 + s.w1;
  p.RK = p.kw + 30 + s.w1;
  auto up = [](size_t x) { return (x + 63) & ~size_t(63); };  // 256-byte alignment, in floats
  const size_t nq = bh * p.njb * static_cast<size_t>(p.RQ) * s.D;
  const size_t nk = bh * p.njb * static_cast<size_t>(p.RK) * s.D;
  p.delta_floats = up(bh * s.N);
  p.pq_off = p.delta_floats;
  p.pk_off = p.pq_off + up(nq);
  p.pv_off = p.pk_off + up(nk);
  p.bytes = (p.pv_off + up(nk)) * 4;
  return p;
}

bool mfma_fused_supported(const Shape& s) {
  return mfma_fwd_supported(s) && s.D == 128 && s.form == 0 && s.w2 <= 32 && s.Hkv == s.H;
}

hipError_t mfma_bwd_fused(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                          const void* vp, const void* dout, const float* lse, void* dk, void* dv,
                          void* workspace, hipStream_t st) {
  if (!mfma_fused_supported(s)) return hipErrorInvalidValue;
  const FusedPlan fp = mfma_fused_plan(s);
  float* ws = static_cast<float*>(workspace);
  const bool bias = s.kp_bias != 0.f || s.vp_bias != 0.f;
  return bias ? launch_key<128, 1, true, 0, true>(s, q, k, kp, v, vp, dout, lse, ws, dk, dv, st, fp, ws)
              : launch_key<128, 1, false, 0, true>(s, q, k, kp, v, vp, dout, lse, ws, dk, dv, st, fp, ws);
}

hipError_t mfma_bwd_fused_reduce(const Shape& s, void* dq, void* dkp, void* dvp, const void* workspace,
                                 hipStream_t st) {
  if (!mfma_fused_supported(s)) return hipErrorInvalidValue;
  const FusedPlan fp = mfma_fused_plan(s);
  const long n = static_cast<long>(s.B) * s.H * s.N * (s.D / 4);
  const dim3 grid(static_cast<unsigned>((n + 255) / 256));
  const float* part = static_cast<const float*>(workspace);
  auto* g0 = static_cast<uint16_t*>(dq);
  auto* g1 = static_cast<uint16_t*>(dkp);
  auto* g2 = static_cast<uint16_t*>(dvp);
  hipLaunchKernelGGL(fused_reduce_kernel<128>, grid, dim3(256), 0, st, s, fp, part, g0, g1, g2);
  return hipGetLastError();
}

hipError_t mfma_bwd_key(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                        const void* vp, const void* dout, const float* lse, const float* delta,
                        void* dk, void* dv, hipStream_t st) {
  const bool bias = s.kp_bias != 0.f || s.vp_bias != 0.f;
  if (s.Hkv < s.H && (s.form != 0 || bias)) return hipErrorInvalidValue;  // grouped-query: trilinear, no constants
  if (s.form == 1) {  // determinant logits: w2 <= 32, no bias constants
    if (s.w2 > 32) return hipErrorInvalidValue;
    return s.D == 128 ? launch_key<128, 1, false, 1>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st)
                      : launch_key<64, 1, false, 1>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st);
  }
  return bias ? mfma_bwd_key_b<true>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st)
             : mfma_bwd_key_b<false>(s, q, k, kp, v, vp, dout, lse, delta, dk, dv, st);
}

}  // namespace sa
