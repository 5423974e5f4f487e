// One lane's steps of the windowed time-aware greedy (App. B.2): the scan
// of one link's pending sends for the best ready one, and the commit of a
// window's winner. Shared by the record-based greedy kernels and compiled
// for the host as well (a host harness runs the same steps for every lane
// of a wavefront, under the sanitizers).
//
// A link's pending sends are records {key lo, key hi (~rem << 32 | trav, or
// the mirrored lengths), priority, slot | other slot << 16} in
// grec[base, base + len); the other slot is the send the chunk arrives by
// (its finish, gfin[other], is the ready time; kGreedyNoPred: ready at 0)
// or, in the push form (kRS: a send waits for all its inputs, as in a
// ReduceScatter), the send it is an input of. In the pull form gfin[slot]
// is kGreedyNone while a send is pending; in the push form it is
// kGreedyNone until the send's last input is scheduled and then holds its
// ready time (grdy[slot], the latest input finish; gpend[slot] counts the
// inputs still unscheduled) until the send itself is scheduled.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace taccl {

constexpr uint32_t kGreedyNone = 0xFFFFFFFFu;
constexpr uint32_t kGreedyNoPred = 0xFFFFu;

// a link's busy time and its pending part of the record list
struct GreedyLink {
  uint32_t free, base, len;
};

// The best ready send of a link, as three words compared lexicographically:
// (start, key hi), (key lo, priority), (slot, list index). The winner is
// replaced as a whole, so its list index always belongs to it. w2 ==
// kGreedyNone: no send of the link is ready.
struct GreedyBest {
  uint64_t w0, w1;
  uint32_t w2;
};

__host__ __device__ inline uint32_t greedy_start(const GreedyBest &b) {
  return b.w2 != kGreedyNone ? (uint32_t)(b.w0 >> 32) : kGreedyNone;
}

// Pending-send lists seen through a view: get(i) returns the record at list
// position i ({key lo, key hi, priority, slot | other slot << 16}) and
// swap(i, j) exchanges two positions. RecArray keeps the records
// themselves; other layouts build them from their own arrays.
template <class Rec>
struct RecArray {
  Rec *p;
  __host__ __device__ Rec get(uint32_t i) const { return p[i]; }
  __host__ __device__ void swap(uint32_t i, uint32_t j) const {
    const Rec t = p[i];
    p[i] = p[j];
    p[j] = t;
  }
};

// The best ready send among the link's pending records, two records a step
// (their loads, then their ready times, then the comparisons).
template <bool kRS, class View>
__host__ __device__ inline GreedyBest greedy_scan_link(const GreedyLink &lk, const View &grec,
                                                       const uint32_t *gfin) {
  GreedyBest b{~0ull, ~0ull, kGreedyNone};
  for (uint32_t q0 = 0; q0 < lk.len; q0 += 2) {
    decltype(grec.get(0)) rc[2];
    uint32_t r[2];
    for (int u = 0; u < 2; u++) {
      const uint32_t q = q0 + u < lk.len ? q0 + u : lk.len - 1;
      rc[u] = grec.get(lk.base + q);
    }
    for (int u = 0; u < 2; u++) {
      const uint32_t x = rc[u].w & 0xFFFFu, other = rc[u].w >> 16;
      if (kRS) {
        r[u] = gfin[x];
      } else {
        const uint32_t fo = gfin[other == kGreedyNoPred ? 0u : other];
        r[u] = other == kGreedyNoPred ? 0u : fo;
      }
    }
    for (int u = 0; u < 2; u++) {
      // past the list, or its chunk has not arrived yet
      const bool live = q0 + u < lk.len && r[u] != kGreedyNone;
      const uint32_t st = lk.free > r[u] ? lk.free : r[u];
      const uint64_t w0 = ((uint64_t)st << 32) | rc[u].y;
      const uint64_t w1 = ((uint64_t)rc[u].x << 32) | rc[u].z;
      const uint32_t w2 = ((rc[u].w & 0xFFFFu) << 16) | (q0 + u);
      const bool better = live && (w0 < b.w0 || (w0 == b.w0 && (w1 < b.w1 || (w1 == b.w1 && w2 < b.w2))));
      if (better) b = GreedyBest{w0, w1, w2};
    }
  }
  return b;
}

// Commit the winner b of a link (cost: the link's cost): its finish time,
// the link's busy time and the running makespan; in the push form the send
// it is an input of learns the finish through the Ops hooks (max into grdy,
// one input fewer in gpend; the input that takes the count to zero then
// publishes the ready time in gfin). The committed record is swapped
// to the end of the pending part, so a list ends in reverse service order.
// Returns true if the record at the winner's index is not the winner (never
// the case; reported as a fault).
template <bool kRS, class Ops, class View>
__host__ __device__ inline bool greedy_commit(GreedyLink &lk, const GreedyBest &b, uint32_t cost,
                                              const View &grec, uint32_t *gfin, uint32_t *grdy,
                                              uint32_t *gpend, uint32_t &mk) {
  const uint32_t cs = (uint32_t)(b.w0 >> 32), cq = b.w2 & 0xFFFFu;
  const auto rc = grec.get(lk.base + cq);
  const uint32_t x = rc.w & 0xFFFFu;
  const bool lost = x != (b.w2 >> 16);
  const uint32_t f = cs + cost;
  if (kRS) {
    const uint32_t nxt = rc.w >> 16;
    if (nxt != kGreedyNoPred) {
      Ops::max_into(&grdy[nxt], f);
      if (Ops::decrement(&gpend[nxt]) == 1) gfin[nxt] = Ops::load(&grdy[nxt]);
    }
  }
  gfin[x] = f;
  lk.free = f;
  mk = mk > f ? mk : f;
  grec.swap(lk.base + cq, lk.base + lk.len - 1);
  lk.len--;
  return lost;
}

}  // namespace taccl
