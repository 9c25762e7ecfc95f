// CPU model of the forward kernel's LDS-DMA load queues, waits and barriers.
//
// Every wavefront of a 4-wavefront workgroup issues its share of each tile's
// loads (buffer loads that write LDS directly) in program order; a wait
// vmcnt(X) guarantees that all but the wavefront's X most recent loads are
// complete; a barrier orders all wavefronts. The model replays the program
// order of the forward kernel (prologue, block iterations, epilogue) for one
// workgroup and checks, for every read of an LDS region (a K or V ring stage
// or a 1 KB chunk of the staging tile):
//   1. every load into that region issued by any wavefront before the barrier
//      that precedes the read was complete at that wavefront's last wait;
//   2. no wavefront issues a load into that region between that barrier and
//      the next one (it could land while another wavefront reads);
//   3. the region holds the block the kernel means to read (K(n+2), V(n), the
//      k' / q rows before q~ is formed, the v' rows in the epilogue).
// The schedule (which loads each iteration issues, how many tiles a wait may
// leave in flight, whether the epilogue waits) comes from the header the
// kernel includes; a second rule set ("steady": always 3 tiles in flight and
// the epilogue wait only for windows under 7 blocks) reproduces the schedule
// before the tail waits were derived from the issued loads.
//
// Usage: fwd_ring_model {kernel|steady}; prints one line per violation and a
// summary "violations: N cases: M"; exit status 0.
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "fwd_schedule.h"

namespace {

struct Load {
  int region;       // LDS region index
  std::string tag;  // what it brings ("K5", "V3", "kp", "q", "vp", "reg")
  int epoch;        // barrier epoch in which it was issued
};

struct Wave {
  std::vector<Load> q;  // issued loads, in order
  size_t done = 0;      // loads [0, done) known complete
};

// Regions: 0-3 K stages, 4-7 V stages, 8 + x staging chunk x, -1 register load.
constexpr int kReg = -1;
int kreg(int s) { return s; }
int vreg(int s) { return 4 + s; }
int sreg(int x) { return 8 + x; }

struct Rules {
  bool steady;
  int inflight(int n, int nb) const {
    return steady ? 3 : sa::fwd_schedule::inflight_tiles(n, nb);
  }
  bool epilogue_waits(int nb) const { return steady ? nb < 7 : sa::fwd_schedule::epilogue_waits(nb); }
};

struct Model {
  int D, G, nb;
  Rules rules;
  int SPW, KI;
  std::vector<Wave> w;
  int epoch = 0;
  // last tag written to each region per wave; regions read in the current epoch
  std::vector<std::vector<std::string>> content;
  std::vector<int> read_epoch;
  std::vector<std::string> errors;

  Model(int D_, int G_, int nb_, Rules r) : D(D_), G(G_), nb(nb_), rules(r), w(4) {
    const int CH = D / 8;
    SPW = (32 * CH / 64) / 4;     // 64-lane loads per tile per wavefront
    KI = (35 * CH + 63) / 64;     // staging loads of k' (or v') rows
    content.assign(8 + KI + 1, std::vector<std::string>(4, ""));
    read_epoch.assign(8 + KI + 1, -1);
  }
  void issue(int wave, int region, const std::string& tag) {
    if (region >= 0 && read_epoch[region] == epoch)
      errors.push_back("load of " + tag + " into a region read in the same barrier interval");
    w[wave].q.push_back({region, tag, epoch});
    if (region >= 0) content[region][wave] = tag;
  }
  void tile(int region, const std::string& tag) {
    for (int x = 0; x < 4; ++x)
      for (int i = 0; i < SPW; ++i) issue(x, region, tag);
  }
  void wait(int tiles_in_flight) {
    for (auto& wv : w) {
      const size_t keep = static_cast<size_t>(tiles_in_flight * SPW);
      const size_t n = wv.q.size() > keep ? wv.q.size() - keep : 0;
      if (n > wv.done) wv.done = n;
    }
  }
  void barrier() { ++epoch; }
  void read(int region, const std::string& want, const std::string& what) {
    read_epoch[region] = epoch;
    for (int x = 0; x < 4; ++x) {
      const Wave& wv = w[x];
      for (size_t i = 0; i < wv.q.size(); ++i) {
        const Load& l = wv.q[i];
        if (l.region != region) continue;
        if (l.epoch >= epoch)
          errors.push_back(what + ": wavefront " + std::to_string(x) + " loads " + l.tag +
                           " into it in the same barrier interval");
        else if (i >= wv.done)
          errors.push_back(what + ": wavefront " + std::to_string(x) + "'s load of " + l.tag +
                           " is not covered by its wait");
      }
      // A tile is loaded in shares by every wavefront, a staging chunk by one.
      if (!want.empty() && !content[region][x].empty() && content[region][x] != want)
        errors.push_back(what + ": holds " + content[region][x] + " from wavefront " +
                         std::to_string(x) + ", expected " + want);
    }
    bool written = false;
    for (int x = 0; x < 4; ++x) written = written || !content[region][x].empty();
    if (!want.empty() && !written) errors.push_back(what + ": nothing was loaded into it");
  }

  void run() {
    const std::string K = "K", V = "V";
    auto kt = [&](int b) { return K + std::to_string(b); };
    auto vt = [&](int b) { return V + std::to_string(b); };
    if (G == 1) {
      for (int x = 0; x < 4; ++x)
        for (int c = x; c < KI + 1; c += 4) issue(x, sreg(c), c < KI ? "kp" : "q");
      tile(kreg(0), kt(0));
      tile(kreg(1), kt(1));
      tile(vreg(0), vt(0));
      tile(kreg(2), kt(2));
      wait(2);
      barrier();
      for (int c = 0; c < KI + 1; ++c) read(sreg(c), c < KI ? "kp" : "q", "q~ formation, staging chunk " + std::to_string(c));
      read(kreg(0), kt(0), "prologue K0");
      tile(vreg(1), vt(1));
      tile(kreg(3), kt(3));
      tile(vreg(2), vt(2));
      read(kreg(1), kt(1), "prologue K1");
    } else {
      for (int b = 0; b < 4; ++b) tile(kreg(b), kt(b));
      for (int b = 0; b < 3; ++b) tile(vreg(b), vt(b));
      const int nreg = 2 * (D / 16);  // q and k' register loads per lane
      for (int x = 0; x < 4; ++x)
        for (int i = 0; i < nreg; ++i) issue(x, kReg, "reg");
      wait(0);
      barrier();
      read(kreg(0), kt(0), "prologue K0");
      read(kreg(1), kt(1), "prologue K1");
    }
    for (int n = 0; n < nb; ++n) {
      wait(rules.inflight(n, nb));
      barrier();
      const int S = n % 4;
      if (sa::fwd_schedule::loads_k(n, nb)) tile(kreg(S), kt(n + 4));
      if (sa::fwd_schedule::loads_v(n, nb)) tile(vreg((S + 3) % 4), vt(n + 3));
      if (G == 1 && n == 0)
        for (int x = 0; x < 4; ++x)
          for (int c = x; c < KI; c += 4) issue(x, sreg(c), "vp");
      read(vreg(S), vt(n), "iteration " + std::to_string(n) + " V" + std::to_string(n));
      read(kreg((S + 2) % 4), n + 2 < nb ? kt(n + 2) : "",
           "iteration " + std::to_string(n) + " K" + std::to_string(n + 2));
    }
    if (G == 1) {
      if (rules.epilogue_waits(nb)) {
        wait(0);
        barrier();
      }
      for (int c = 0; c < KI; ++c) read(sreg(c), "vp", "epilogue v' rows, staging chunk " + std::to_string(c));
    }
  }
};

}  // namespace

int main(int argc, char** argv) {
  Rules r{argc > 1 && std::strcmp(argv[1], "steady") == 0};
  int violations = 0, cases = 0;
  for (int D : {64, 128})
    for (int G : {1, 2})
      for (int nb = 1; nb <= 40; ++nb) {
        Model m(D, G, nb, r);
        m.run();
        ++cases;
        for (const auto& e : m.errors) {
          std::printf("D=%d G=%d nb=%d: %s\n", D, G, nb, e.c_str());
          ++violations;
        }
      }
  std::printf("violations: %d cases: %d\n", violations, cases);
  return 0;
}
