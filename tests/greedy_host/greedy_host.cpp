// Host run of the windowed greedy (App. B.2) with the library's own per-lane
// steps (greedy_window.h), for the tests: the steps of every lane of a
// 64-lane wavefront are executed one lane after another, with the window
// minimum taken over all of them in between, exactly as the kernels
// arrange them. Built for the host only, under AddressSanitizer and
// UndefinedBehaviorSanitizer.
//
// stdin (little-endian u32): E, nslots, cmin, n_records, push, cost[E],
// gofs[E + 1], records[n_records][4]. push = 0: the pull form (a record's
// other slot is the send the chunk arrives by); push = 1: the push form (a
// send waits for every send whose other slot is its own, as in a
// ReduceScatter). stdout: makespan, then the finish time of every slot
// (kGreedyNone for a slot without a send), one a line.
#include <cstdio>
#include <vector>

#include "greedy_window.h"

using taccl::GreedyBest;
using taccl::GreedyLink;
using taccl::kGreedyNone;

namespace {

struct Plain {  // one lane at a time: plain updates
  static void max_into(uint32_t *p, uint32_t v) { *p = *p > v ? *p : v; }
  static uint32_t decrement(uint32_t *p) { return (*p)--; }
  static uint32_t load(uint32_t *p) { return *p; }
};

bool read_u32(uint32_t *out, size_t n) { return fread(out, 4, n, stdin) == n; }

}  // namespace

int main() {
  uint32_t hdr[5];
  if (!read_u32(hdr, 5)) return 2;
  const uint32_t E = hdr[0], nslots = hdr[1], cmin = hdr[2], nrec = hdr[3];
  const bool push = hdr[4] != 0;
  constexpr int kLanes = 64, kSlots = 4;  // a wavefront, four links per lane
  if (E > (uint32_t)kLanes * kSlots || nslots > 65535) return 2;
  std::vector<uint32_t> cost(E), gofs(E + 1);
  std::vector<uint4> grec(nrec);
  if (!read_u32(cost.data(), E) || !read_u32(gofs.data(), E + 1)) return 2;
  for (uint32_t r = 0; r < nrec; r++) {
    uint32_t w[4];
    if (!read_u32(w, 4)) return 2;
    grec[r] = make_uint4(w[0], w[1], w[2], w[3]);
  }
  std::vector<uint32_t> gfin(nslots > 0 ? nslots : 1, kGreedyNone);
  // push form: inputs per send, the latest input finish, and a send without
  // inputs ready at 0
  std::vector<uint32_t> gpend(gfin.size(), 0), grdy(gfin.size(), 0);
  if (push) {
    for (const uint4 &r : grec) {
      const uint32_t other = r.w >> 16;
      if (other != taccl::kGreedyNoPred) {
        if (other >= nslots) return 2;
        gpend[other]++;
      }
    }
    for (const uint4 &r : grec) {
      const uint32_t x = r.w & 0xFFFFu;
      if (x >= nslots) return 2;
      if (gpend[x] == 0) gfin[x] = 0;
    }
  }
  std::vector<GreedyLink> lk((size_t)kLanes * kSlots);
  for (int lane = 0; lane < kLanes; lane++)
    for (int t = 0; t < kSlots; t++) {
      const uint32_t l = lane + kLanes * t;
      GreedyLink &g = lk[(size_t)lane * kSlots + t];
      g.free = 0;
      g.base = l < E ? gofs[l] : 0;
      g.len = l < E ? gofs[l + 1] - gofs[l] : 0;
    }
  uint32_t mk = 0;
  bool fault = false;
  std::vector<GreedyBest> best(lk.size());
  const taccl::RecArray<uint4> view{grec.data()};
  for (uint32_t round = 0;; round++) {
    uint32_t wmin = kGreedyNone;
    for (size_t k = 0; k < lk.size(); k++) {
      best[k] = push ? taccl::greedy_scan_link<true>(lk[k], view, gfin.data())
                     : taccl::greedy_scan_link<false>(lk[k], view, gfin.data());
      const uint32_t st = taccl::greedy_start(best[k]);
      wmin = st < wmin ? st : wmin;
    }
    if (wmin == kGreedyNone) break;
    if (round > nslots) {
      fault = true;
      break;
    }
    const uint64_t wend = (uint64_t)wmin + cmin;
    for (int lane = 0; lane < kLanes; lane++)
      for (int t = 0; t < kSlots; t++) {
        const size_t k = (size_t)lane * kSlots + t;
        const uint32_t st = taccl::greedy_start(best[k]);
        if (st != kGreedyNone && (uint64_t)st < wend)
          fault |= push ? taccl::greedy_commit<true, Plain>(lk[k], best[k], cost[lane + kLanes * t],
                                                            view, gfin.data(), grdy.data(),
                                                            gpend.data(), mk)
                        : taccl::greedy_commit<false, Plain>(lk[k], best[k],
                                                             cost[lane + kLanes * t], view,
                                                             gfin.data(), nullptr, nullptr, mk);
      }
  }
  if (fault) return 3;
  printf("%u\n", mk);
  for (uint32_t s = 0; s < nslots; s++) printf("%u\n", gfin[s]);
  return 0;
}
