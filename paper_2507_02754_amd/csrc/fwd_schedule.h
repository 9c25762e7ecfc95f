// Load and wait schedule of the forward kernel's K/V block rings.
//
// The forward stages 32-key blocks of K and V through two 4-stage LDS rings
// with buffer loads that write LDS directly. Every wavefront issues an equal
// share of each tile's loads and waits only for its own (vmcnt counts the
// issuing wavefront's loads, completed in issue order); the workgroup barrier
// after the wait then makes the tile visible to all wavefronts. A wait must
// therefore name how many of the wavefront's most recent loads may stay in
// flight, and that number has to match the loads actually issued after the
// tile being waited for: near the end of a tile's window fewer loads follow.
//
// Issue order (w2 <= 32; every block index below nb is a block of the window):
//   prologue      staging rows (k' and q), K0, K1, V0, K2;
//                 wait: staging rows, K0 and K1 complete; barrier;
//                 V1, K3, V2 (after the first logit products are issued)
//   iteration n   wait: K(n+2) and V(n) complete; barrier;
//                 K(n+4) if n+4 < nb, V(n+3) if n+3 < nb;
//                 (n = 0 only) v' rows into the staging tile;
//                 reads V(n), then K(n+2)
// Blocks 0..3 of K and 0..2 of V are loaded in the prologue even when the
// window has fewer blocks (the extra ones are never used).
// With 32 < w2 <= 64 the prologue loads K0..K3 and V0..V2 and waits for all
// of them (vmcnt(0)) before the loop; the loop is the same.
//
// The functions are plain constexpr so that host code (a CPU model of the
// per-wavefront load queues) evaluates the same schedule the kernel runs.
#pragma once

namespace sa {
namespace fwd_schedule {

constexpr int kStages = 4;

// Iteration n issues K(n + 4) into stage n % 4 (K(n) was read at the end of
// iteration n - 2) and V(n + 3) into stage (n + 3) % 4 (V(n - 1) was read in
// iteration n - 1), while those blocks exist.
constexpr bool loads_k(int n, int nb) { return n + 4 < nb; }
constexpr bool loads_v(int n, int nb) { return n + 3 < nb; }

// Whole tiles of loads each wavefront may leave in flight at the wait of
// iteration n so that K(n + 2) and V(n) are complete. In steady state
// V(n+1), K(n+3) and V(n+2) were issued after K(n+2): 3 tiles. In the last
// iterations fewer loads follow:
//   n = nb - 3: K(nb-1) is followed by V(nb-2) and V(nb-1) only -> 2;
//   n = nb - 2: V(nb-2) is followed by V(nb-1) only             -> 1;
//   n = nb - 1: nothing follows V(nb-1)                          -> 0.
// (Blocks loaded in the prologue are followed by more loads than this
// counts, which only makes the wait stricter than necessary.)
constexpr int inflight_tiles(int n, int nb) {
  return n + 3 < nb ? 3 : n + 3 == nb ? 2 : n + 2 == nb ? 1 : 0;
}

// The v' rows issued in iteration 0 are read in the epilogue. When the
// window has at least two blocks, the last iteration (n = nb - 1 >= 1) waits
// for every load and passes a barrier after they were issued; a one-block
// window needs an explicit wait and barrier before the epilogue.
constexpr bool epilogue_waits(int nb) { return nb < 2; }

}  // namespace fwd_schedule
}  // namespace sa
