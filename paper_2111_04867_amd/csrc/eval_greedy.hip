// Time-aware greedy orders (App. B.2) for Alltoall plans too large for one
// wavefront's on-chip lists, for gfx950.
//
// One block per candidate at a time, one thread per chunk (CPT chunks per
// thread). The greedy only ever holds one candidate send per chunk: the
// next hop of its routed path (in reverse path order, the hop before the
// last one served). So instead of per-link lists the block keeps per chunk
// its time and next hop in registers, and simulates the greedy exactly in
// windows, as the wavefront kernels do: W = the earliest start any chunk's
// next hop can take (max of its link's busy time and the chunk's time); a
// hop that is not a candidate yet can only become one at least c_min (the
// smallest link latency) after W, so on every link the best candidate by
// (start, Step-2 key, priority, chunk) with start < W + c_min is the
// greedy's next send there. Per window:
//   1. every thread computes its chunks' starts; block minimum -> W;
//   2. per link, an LDS 64-bit atomicMin of start << 32 | key rank (the
//      rank of the hop's (remaining desc, travelled asc) pair among all
//      hops of the plan, from a plan table);
//   3. among the hops that hold that minimum, atomicMin of
//      priority << 16 | chunk;
//   4. the single winner per link commits: finish = start + latency, the
//      link and the chunk advance, and the link's two minima are reset.
// When the whole order fits one 64-bit word the window takes two barriers
// instead of four: every start is at least the previous window's W, and an
// eligible one is below it by less than 2 c_min + c_max (every time so far
// is a finish of a send that started before the previous window's end), so
// (start - previous W, clamped above that bound) | key rank | priority |
// chunk orders exactly; one atomicMin per hop into its link's word and one
// per wavefront of its smallest start, then the holder of each link's
// minimum commits if that start is below W + c_min (two buffers of minima,
// the one for the next window reset while this one is read).
// In reverse path order the greedy serves the mirrored schedule (a chunk's
// hops from its last link back, key ranks of the mirrored lengths) and
// records each send's service position on its link; a link's real order is
// the reverse, and the real times then come from rounds in which, on every
// link, the send at the link's next position goes once its chunk's previous
// hop has ended.
#include <hip/hip_runtime.h>

#include "kernels.h"
#include "wave.h"

namespace taccl {

namespace {

constexpr uint32_t kNone = 0xFFFFFFFFu;

int32_t align16(int32_t x) { return (x + 15) & ~15; }

// Two 1024-thread blocks per CU (8 wavefronts per SIMD, 64 registers) for
// one-word keys; two-word keys would spill there at 4 chunks per thread and
// take up to 128 registers (one block per CU) instead.
template <int CPT, bool kPack>
constexpr int greedy_block_min_waves() {
  return kPack && CPT <= 4 ? 8 : 4;
}

// kStaged: the candidate's priorities are staged in LDS (a.b_sprio >= 0)
template <int CPT, int NT, bool kPack, bool kStaged>
__global__ __launch_bounds__(NT) __attribute__((
    amdgpu_waves_per_eu(greedy_block_min_waves<CPT, kPack>(), 8))) void path_greedy_block(PathGreedyArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int P = a.P, E = a.E, H = a.H;
  constexpr int NW = NT / 64;
  uint32_t *s_cost = (uint32_t *)(lds + a.b_cost);
  uint32_t *lfree = (uint32_t *)(lds + a.b_lfree);
  unsigned long long *best1 = (unsigned long long *)(lds + a.b_best1);
  unsigned long long *best2 = (unsigned long long *)(lds + a.b_best2);
  uint32_t *lserv = (uint32_t *)(lds + a.b_lserv);  // sends served per link
  uint32_t *lnext = (uint32_t *)(lds + a.b_lnext);  // real order: next position
  uint32_t *red = (uint32_t *)(lds + a.b_red);      // [2][NW] window minima
  uint16_t *fpos = (uint16_t *)(lds + a.b_fpos);    // service position per slot
  // the candidate's priorities of its routed hops, chunk after chunk (when
  // the plan's sends fit: a.b_sprio >= 0), so each priority row is read from
  // HBM once instead of hop by hop
  uint32_t *sprio = (uint32_t *)(lds + (kStaged ? a.b_sprio : 0));
  for (int l = tid; l < E; l += NT) s_cost[l] = a.cost[l];

  for (int64_t i = blockIdx.x; i < a.n; i += gridDim.x) {
    const uint8_t *rt = a.routes + (size_t)i * a.route_stride;
    const uint32_t *gpr = a.prio + (size_t)i * a.prio_stride;
    for (int l = tid; l < E; l += NT) {
      lfree[l] = 0;
      lserv[l] = 0;
      lnext[l] = 0;
      best1[l] = ~0ull;
      best2[l] = ~0ull;
    }
    // per chunk: first hop of its option in path_links, hop count, hops
    // served, time, and the current hop's link, key rank and priority (kept
    // as loaded: a one-word key is built from them when the next window
    // needs it, so a commit does not wait for the next hop's loads)
    uint32_t qo[CPT], hops[CPT], cur[CPT], ct[CPT], cl[CPT], kr[CPT], pv[CPT], po[CPT];
    bool bad = false;
    auto load_hop = [&](int j, int c) {
      const uint32_t h = a.mirror ? hops[j] - 1 - cur[j] : cur[j];
      cl[j] = a.path_links[qo[j] + h];
      const uint32_t k = a.gkrank[qo[j] + h];
      // a plain LDS read when staged (a run-time choice made this a generic
      // load that waits for both memory counters)
      pv[j] = kStaged ? sprio[po[j] + h] : gpr[(uint32_t)c * H + h];
      kr[j] = k;
    };
#pragma unroll
    for (int j = 0; j < CPT; j++) {
      const int c = tid + NT * j;
      hops[j] = 0;
      cur[j] = 0;
      ct[j] = 0;
      qo[j] = 0;
      if (c < a.C) {
        const uint32_t sd = (uint32_t)c / (uint32_t)a.cpr;
        const uint32_t s = sd / P, d = sd - s * P;
        if (s != d) {
          const uint32_t k = rt[c];
          if (k < a.npaths[sd]) {
            const uint32_t q = a.pair_base[sd] + k;
            qo[j] = a.path_off[q];
            hops[j] = a.path_off[q + 1] - qo[j];
          } else {
            bad = true;  // the pair is left unrouted
          }
        }
      }
    }
    if (kStaged) {
      // chunk offsets: a block scan of the hop counts
      uint32_t nh = 0;
#pragma unroll
      for (int j = 0; j < CPT; j++) nh += hops[j];
      const uint32_t incl = wave_scan_add(nh);
      if (lane == 63) red[wave] = incl;
      __syncthreads();
      uint32_t off = incl - nh;
      for (int w = 0; w < wave; w++) off += red[w];
#pragma unroll
      for (int j = 0; j < CPT; j++) {
        const int c = tid + NT * j;
        po[j] = off;
        for (uint32_t h = 0; h < hops[j]; h++) sprio[off + h] = gpr[(uint32_t)c * H + h];
        off += hops[j];
      }
      __syncthreads();
    }
#pragma unroll
    for (int j = 0; j < CPT; j++)
      if (hops[j]) load_hop(j, tid + NT * j);
    __syncthreads();

    uint32_t mk = 0;
    bool fault = false;
    // commit hop j of chunk c, which starts at st on link l
    auto commit = [&](int j, int c, uint32_t st, uint32_t l) {
      const uint32_t f = st + s_cost[l];
      ct[j] = f;
      lfree[l] = f;
      mk = max(mk, f);
      if (a.mirror) {  // the reversed order needs each send's service position
        const uint32_t h = hops[j] - 1 - cur[j];
        fpos[(uint32_t)c * H + h] = (uint16_t)lserv[l];
        lserv[l]++;
      }
      if (++cur[j] < hops[j]) load_hop(j, c);
    };
    if (kPack) {
      // best1 / best2 serve as the two buffers of per-link minima (best2 at
      // best1 + bst), red as the two window starts
      const int bst = (a.b_best2 - a.b_best1) / 8;
      if (tid == 0) red[0] = red[1] = kNone;
      __syncthreads();
      uint32_t wp = 0;  // the previous window's W
      for (int round = 0, buf = 0;; round++, buf ^= 1) {
        uint32_t st[CPT];
        uint32_t wmin = kNone;
        // the relative start and the key rank lie in the key's high word
        // (rel_shift, kr_shift >= 32) and the priority straddles the two
        // words: 32-bit shifts only
        const uint32_t rel_hi = (uint32_t)a.rel_shift - 32u, cb = (uint32_t)a.chunk_bits;
        auto key_of = [&](int j) {
          const uint32_t hi = (min(st[j] - wp, a.rel_max) << rel_hi) | (kr[j] << (cb & 31u)) |
                              (cb ? pv[j] >> (32u - cb) : 0u);
          const uint32_t lo = (pv[j] << (cb & 31u)) | (uint32_t)(tid + NT * j);
          return ((uint64_t)hi << 32) | lo;
        };
#pragma unroll
        for (int j = 0; j < CPT; j++) {
          st[j] = kNone;
          if (cur[j] < hops[j]) {
            st[j] = max(ct[j], lfree[cl[j]]);
            wmin = min(wmin, st[j]);
            atomicMin(&best1[buf * bst + cl[j]], key_of(j));
          }
        }
        wmin = ~wave_reduce_max(~wmin);
        if (lane == 0 && wmin != kNone) atomicMin(&red[buf], wmin);
        __syncthreads();
        const uint32_t W = red[buf];
        if (W == kNone) break;  // every chunk is through
        if (round > a.nslots) {  // unreachable: every window serves a send
          fault = true;
          break;
        }
        // a pending start is at least W: st - W < c_min is the window test
        // the link's minimum is this chunk's key exactly when its chunk
        // field (the key's low bits; keys of one window differ in their
        // chunk) is this chunk: the low word of the minimum suffices
        const uint32_t cmask = (1u << a.chunk_bits) - 1u;
        const uint32_t *best1w = (const uint32_t *)best1;
#pragma unroll
        for (int j = 0; j < CPT; j++) {
          const uint32_t c = tid + NT * j;
          if (st[j] != kNone && st[j] - W < a.cmin &&
              (best1w[2 * (buf * bst + cl[j])] & cmask) == c)
            commit(j, (int)c, st[j], cl[j]);
        }
        for (int l = tid; l < E; l += NT) best1[(buf ^ 1) * bst + l] = ~0ull;
        if (tid == 0) red[buf ^ 1] = kNone;
        wp = W;
        __syncthreads();
      }
    }
    for (int round = 0, buf = 0; !kPack; round++, buf ^= 1) {
      // 1. starts and their block minimum
      uint32_t st[CPT];
      uint32_t wmin = kNone;
#pragma unroll
      for (int j = 0; j < CPT; j++) {
        st[j] = kNone;
        if (cur[j] < hops[j]) {
          st[j] = max(ct[j], lfree[cl[j]]);
          wmin = min(wmin, st[j]);
        }
      }
      wmin = ~wave_reduce_max(~wmin);
      if (lane == 0) red[buf * NW + wave] = wmin;
      __syncthreads();
      uint32_t W = kNone;
#pragma unroll
      for (int w = 0; w < NW; w++) W = min(W, red[buf * NW + w]);
      if (W == kNone) break;  // every chunk is through
      if (round > a.nslots) {  // unreachable: every window serves a send
        fault = true;
        break;
      }
      const uint64_t wend = (uint64_t)W + a.cmin;
      // 2. per link the smallest (start, key rank) of the window
      uint64_t k1[CPT];
#pragma unroll
      for (int j = 0; j < CPT; j++) {
        k1[j] = ((uint64_t)st[j] << 32) | kr[j];
        if (st[j] != kNone && (uint64_t)st[j] < wend) atomicMin(&best1[cl[j]], k1[j]);
      }
      __syncthreads();
      // 3. then the smallest (priority, chunk)
#pragma unroll
      for (int j = 0; j < CPT; j++) {
        const int c = tid + NT * j;
        if (st[j] != kNone && (uint64_t)st[j] < wend && best1[cl[j]] == k1[j])
          atomicMin(&best2[cl[j]], ((uint64_t)pv[j] << 16) | (uint32_t)c);
      }
      __syncthreads();
      // 4. the winner of every link commits
#pragma unroll
      for (int j = 0; j < CPT; j++) {
        const int c = tid + NT * j;
        if (st[j] != kNone && (uint64_t)st[j] < wend && best1[cl[j]] == k1[j] &&
            best2[cl[j]] == (((uint64_t)pv[j] << 16) | (uint32_t)c)) {
          const uint32_t l = cl[j];
          best1[l] = ~0ull;
          best2[l] = ~0ull;
          commit(j, c, st[j], l);
        }
      }
      __syncthreads();
    }

    if (a.mirror && !fault) {
      // the real schedule: every link's order is its service order reversed
      mk = 0;
      for (int l = tid; l < E; l += NT) lfree[l] = 0;
#pragma unroll
      for (int j = 0; j < CPT; j++) {
        cur[j] = 0;
        ct[j] = 0;
        if (hops[j]) cl[j] = a.path_links[qo[j]];
      }
      __syncthreads();
      for (int round = 0;; round++) {
        // a chunk's next hop goes when it is at its link's next position
        bool go[CPT], pending = false;
#pragma unroll
        for (int j = 0; j < CPT; j++) {
          const int c = tid + NT * j;
          go[j] = false;
          if (cur[j] < hops[j]) {
            pending = true;
            const uint32_t l = cl[j];
            const uint32_t pos = lserv[l] - 1u - fpos[(uint32_t)c * H + cur[j]];
            go[j] = lnext[l] == pos;
          }
        }
        if (!__syncthreads_or(pending)) break;
        if (round > a.nslots) {  // unreachable: the orders come from a schedule
          fault = true;
          break;
        }
#pragma unroll
        for (int j = 0; j < CPT; j++)
          if (go[j]) {
            const uint32_t l = cl[j];
            const uint32_t f = max(ct[j], lfree[l]) + s_cost[l];
            ct[j] = f;
            lfree[l] = f;
            lnext[l]++;
            mk = max(mk, f);
            if (++cur[j] < hops[j]) cl[j] = a.path_links[qo[j] + cur[j]];
          }
        __syncthreads();
      }
    }

    // makespan and validity (after a barrier: the last window's minima
    // may still be read)
    __syncthreads();
    const uint32_t wm = wave_reduce_max(mk);
    if (lane == 0) red[wave] = wm;
    const bool any_bad = __syncthreads_or(bad);
    const bool any_fault = __syncthreads_or(fault);
    if (tid == 0) {
      uint32_t m = 0;
      for (int w = 0; w < NW; w++) m = max(m, red[w]);
      a.makespan[i] = any_fault ? 0xFFFFFFFFu : m;
      a.valid[i] = (uint8_t)(!any_bad && !any_fault);
    }
    __syncthreads();
  }
}

template <int NT, bool kPack, bool kStaged>
const void *block_fn_ps(int cpt) {
  switch (cpt) {
    case 1: return (const void *)path_greedy_block<1, NT, kPack, kStaged>;
    case 2: return (const void *)path_greedy_block<2, NT, kPack, kStaged>;
    default: return (const void *)path_greedy_block<4, NT, kPack, kStaged>;
  }
}

template <int NT, bool kPack>
const void *block_fn_p(int cpt, bool staged) {
  return staged ? block_fn_ps<NT, kPack, true>(cpt) : block_fn_ps<NT, kPack, false>(cpt);
}

template <int NT>
const void *block_fn(const PathGreedyArgs &a) {
  const bool staged = a.b_sprio >= 0;
  return a.pack ? block_fn_p<NT, true>(a.cpt, staged) : block_fn_p<NT, false>(a.cpt, staged);
}

int bits_for(uint64_t x) {  // bits to hold values 0..x
  int b = 0;
  while (b < 64 && (x >> b) != 0) b++;
  return b;
}

}  // namespace

int32_t path_greedy_block_layout(const taccl_plan &p, PathGreedyArgs &a) {
  const int32_t C = p.coll.C, E = p.topo.E, H = std::max(p.H, 1);
  if (E < 1 || p.gkrank.size() != p.path_links.size() || (int64_t)C * H > 65535) return 0;
  uint32_t cmin = ~0u;
  for (uint32_t c : p.cost) cmin = std::min(cmin, c);
  if (cmin == 0) return 0;
  int cpt = 1;
  while (cpt * kGreedyBlockThreads < C) cpt *= 2;
  // 1024 threads leave at most 128 registers per thread: more than 4
  // chunks per thread would spill the per-chunk state
  if (cpt > 4) return 0;
  a.cmin = cmin;
  a.nslots = C * H;
  a.cpt = cpt;
  // one-word keys: a relative start below 2 c_min + c_max must stay below
  // the clamp value 2^rb - 1
  uint64_t cmax = 0;
  for (uint32_t c : p.cost) cmax = std::max<uint64_t>(cmax, c);
  const int rb = bits_for(2 * (uint64_t)cmin + cmax);
  const int kb = bits_for(p.gk_count > 0 ? (uint64_t)(p.gk_count - 1) : 0);
  const int cb = bits_for(C > 0 ? (uint64_t)(C - 1) : 0);
  a.pack = rb + kb + 32 + cb <= 64 && rb < 32;
  a.chunk_bits = cb;
  a.kr_shift = cb + 32;
  a.rel_shift = cb + 32 + kb;
  a.rel_max = a.pack ? (uint32_t)((1ull << rb) - 1) : 0u;
  int32_t off = 0;
  auto take = [&](int32_t bytes) {
    int32_t o = off;
    off = align16(off + bytes);
    return o;
  };
  a.b_cost = take(4 * E);
  a.b_lfree = take(4 * E);
  a.b_best1 = take(8 * E);
  a.b_best2 = take(8 * E);
  a.b_lserv = take(4 * E);
  a.b_lnext = take(4 * E);
  a.b_red = take(4 * 2 * (kGreedyBlockThreads / 64));
  a.b_fpos = take(p.greedy == 2 ? 2 * a.nslots : 0);
  // staged priorities while two blocks still fit a CU's 160 KB
  a.b_sprio = -1;
  if (off + 4 * p.max_sends <= 80 * 1024) a.b_sprio = take((int32_t)(4 * p.max_sends));
  a.block_bytes = off;
  return off;
}

int path_greedy_block_per_cu(const PathGreedyArgs &a) {
  int nb = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, block_fn<kGreedyBlockThreads>(a),
                                                   kGreedyBlockThreads, a.block_bytes) !=
      hipSuccess)
    return 0;
  return nb;
}

hipError_t launch_path_greedy_block(const PathGreedyArgs &a, int grid, hipStream_t stream) {
  void *args[] = {(void *)&a};
  return hipLaunchKernel(block_fn<kGreedyBlockThreads>(a), dim3(grid),
                         dim3(kGreedyBlockThreads), args, a.block_bytes, stream);
}

}  // namespace taccl
