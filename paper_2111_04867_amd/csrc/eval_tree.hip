// Multicast evaluation kernels for gfx950 (Allgather, explicit, and the
// ReduceScatter / Allreduce built from them), and the time-aware greedy for
// Alltoall plans that fit one wavefront:
//   tree_eval_kernel     general kernel, described below; its kAny variant
//                        adds ReduceScatter, contiguity and greedy orders;
//   tree_layers_kernel   layered kernel for plans within its limits (the
//                        fast path), static orders;
//   tree_greedy_kernel   the layered kernel's trees with greedy orders;
//   path_greedy_kernel   Alltoall greedy orders, one wavefront per candidate.
//
// tree_eval_kernel: persistent blocks of several wavefronts. Each block
// copies the plan's route records and link costs into LDS once; each
// wavefront then evaluates one candidate at a time, its state in LDS, while
// the next candidate's routes and priorities stream from HBM into registers:
//   1. stage the candidate: route choices and priorities go to LDS;
//   2. lane = chunk: the routed paths of the chunk (destinations ascending)
//      are merged into a tree by first reach, one send per reached vertex
//      (one is_sent per chunk and link, App. B.1); distances from the owner
//      (the travelled path of Sec. 5.1) ride along each path in registers;
//   3. same lane, one reverse sweep over the discovery order (children come
//      after their parents): the longest remaining tree path below each
//      vertex (the remaining path of Sec. 5.1), the packed 64-bit Step-2 key
//      of every send (remaining desc, travelled asc) written over the
//      vertex's dead distance slot, and the chunk's bit in its link's mask;
//   4. lane = send: its place in its link's order, by comparing against the
//      other chunks of the link's mask (then priority, then chunk id), four
//      competitors in flight at a time; the send is stored at that place
//      together with the slot of the send that brings its chunk to the link;
//   5. the least schedule of App. B.3 (no contiguity): every link advances
//      through its ordered sends while their chunk has arrived at the link's
//      source; the send with the globally smallest key is always ready, so
//      each round makes progress and a handful of rounds finish;
//   6. postcondition (ballot over chunks) and makespan (wave max).
#include <hip/hip_runtime.h>

#include "greedy_window.h"
#include "kernels.h"
#include "wave.h"

namespace taccl {

namespace {

constexpr uint32_t kNotYet = 0xFFFFFFFFu;
constexpr uint32_t kNoPred = 0xFFFFu;
constexpr int kPfRoute = 4;  // prefetched route words per lane (route_stride <= 1 KiB)
constexpr int kPfPrio = 16;  // prefetched priority words per lane (C*V <= 1024)

// Arrival times are written by one lane and read by others of the same wave
// while links advance; relaxed workgroup-scope atomics keep these accesses
// plain LDS instructions and keep the compiler from caching them.
__device__ __forceinline__ uint32_t lds_get(uint32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void lds_put(uint32_t *p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Phase boundary inside one wavefront. Its lanes run in lockstep and LDS
// serves one wavefront's accesses in order, so this only has to stop the
// compiler from moving LDS accesses across the boundary; it deliberately
// does not wait for outstanding global loads (the prefetch of the next
// candidate stays in flight).
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_wave_barrier();
  asm volatile("" ::: "memory");
}

__device__ __forceinline__ uint32_t wave_max(uint32_t v) { return wave_reduce_max(v); }

// The push-form hooks of the greedy window steps (greedy_window.h) in LDS;
// several lanes of a window may push into the same send's ready time.
struct LdsAtomics {
  __device__ static void max_into(uint32_t *p, uint32_t v) { atomicMax(p, v); }
  __device__ static uint32_t decrement(uint32_t *p) { return atomicSub(p, 1u); }
  __device__ static uint32_t load(uint32_t *p) { return lds_get(p); }
};

// The general variant's per-link orders as greedy lists: chain[] entries
// (slot | the slot on the chunk's other side of the send's source << 16)
// with the Step-2 keys and priorities kept per slot.
struct ChainView {
  uint32_t *chain;
  const uint64_t *key;
  const uint32_t *prio;
  __device__ uint4 get(uint32_t i) const {
    const uint32_t ent = chain[i], s = ent & 0xFFFFu;
    const uint64_t k = key[s];
    return make_uint4((uint32_t)k, (uint32_t)(k >> 32), prio[s], ent);
  }
  __device__ void swap(uint32_t i, uint32_t j) const {
    const uint32_t t = chain[i];
    chain[i] = chain[j];
    chain[j] = t;
  }
};

__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v, int) { return wave_scan_add(v); }

// n / V for n, V < 2^16 with a precomputed m = floor(2^32 / V) + 1
__device__ __forceinline__ uint32_t div_v(uint32_t n, uint32_t m) {
  return (uint32_t)(((uint64_t)n * m) >> 32);
}

// Lane = chunk: the routed paths of the chunk (destinations ascending) are
// merged into a tree by first reach, one send per reached vertex (one
// is_sent per chunk and link, App. B.1); distances from the owner (the
// travelled path of Sec. 5.1) ride along each path in registers. Then one
// reverse sweep over the discovery order (children come after their
// parents) gives the longest remaining tree path below each vertex (the
// remaining path of Sec. 5.1) and writes every send's packed Step-2 key
// (~rem << 32 | trav, ascending = rem desc, trav asc) over the vertex's dead
// distance slot. kMasks also sets the chunk's bit in its link's mask.
// kRS (ReduceScatter; s_cost then holds the cost of every link's reverse):
// the send v -> u has rem = reversed distance from v to the owner and trav =
// longest reversed path up to v, and pend[] counts the sends into each
// vertex other than the owner (the partials its own send waits for).
// par[] (and pend[] for kRS) must be zero on entry; returns whether every
// chunk reached its postcondition ranks.
template <bool kMasks, bool kRS = false>
__device__ __forceinline__ bool build_trees(const TreeArgs &a, const uint32_t *s_rec,
                                            const uint32_t *s_cost, const uint8_t *s_own,
                                            const uint64_t *s_post, const uint8_t *rt,
                                            uint64_t *key, uint16_t *par, uint32_t *ord,
                                            uint32_t *lmask, int lane, uint32_t *pend = nullptr) {
  const int C = a.C, P = a.P, V = a.V, K = a.K, H = a.H, MW = a.mask_words;
  uint32_t *dh = (uint32_t *)key;  // dh[2s] = dist, dh[2s+1] = height
  bool ok = true;
  for (int c = lane; c < C; c += 64) {
    const int o = s_own[c];
    const uint64_t pm = s_post[c];
    const int base = c * V;
    uint64_t reached = 1ull << o;
    int cnt = 0;
    dh[2 * (base + o)] = 0;
    dh[2 * (base + o) + 1] = 0;
    for (int d = 0; d < P; d++) {
      if (d == o || !((pm >> d) & 1)) continue;
      const int k = rt[c * P + d];
      if (k >= K) continue;  // pair left unrouted (no such option)
      const uint32_t *r = s_rec + ((o * P + d) * K + k) * H;
      const uint32_t w0 = r[0];
      const int hops = w0 >> 24;  // 0: the pair has no option k
      int u = o;
      uint32_t du = 0;  // distance of u when `known`
      bool known = true;
      for (int j = 0; j < hops; j++) {
        const uint32_t w = j ? r[j] : w0;
        const int l = w & 0xFFFF;
        const int v = (w >> 16) & 0xFF;
        if (!((reached >> v) & 1)) {
          if (!known) du = dh[2 * (base + u)];
          du += s_cost[l];
          known = true;
          reached |= 1ull << v;
          par[base + v] = (uint16_t)(l + 1);
          dh[2 * (base + v)] = du;
          dh[2 * (base + v) + 1] = 0;
          ord[base + cnt++] = (uint32_t)v | ((uint32_t)u << 8) | ((uint32_t)l << 16);
        } else {
          known = false;
        }
        u = v;
      }
    }
    ok &= (reached & pm) == pm;
    // reverse discovery order visits children before their parents: a
    // vertex's height is final when it is visited, and its parent's
    // distance is still in place
    for (int j = cnt - 1; j >= 0; j--) {
      const uint32_t e = ord[base + j];
      const int v = e & 0xFF, u = (e >> 8) & 0xFF, l = e >> 16;
      const uint32_t hv = dh[2 * (base + v) + 1];
      const uint32_t up = s_cost[l] + hv;  // longest path below u through v
      if (up > dh[2 * (base + u) + 1]) dh[2 * (base + u) + 1] = up;
      if (kRS) {
        key[base + v] = ((uint64_t)(~dh[2 * (base + v)]) << 32) | hv;
        if (u != o) pend[base + u]++;
      } else {
        key[base + v] = ((uint64_t)(~up) << 32) | dh[2 * (base + u)];
      }
      if (kMasks) atomicOr(&lmask[l * MW + (c >> 5)], 1u << (c & 31));
    }
  }
  return ok;
}

// Step 5' of the general variant, one wavefront per candidate. Sends sit
// in chain[] in link order (pred << 16 | slot, pred = the slot whose send
// brings the chunk to the link's source, or kNoPred), fin[] = kNotYet.
// Two dependency forms:
//  * pull (Allgather): a send is ready when the send of slot (c, src) into
//    its source has finished;
//  * push (ReduceScatter): the send of slot (c,v) goes v -> u on the reverse
//    of its tree link and carries v's partial, so it is ready when every
//    send into v has finished: pend[] counts them down and rdy[] keeps the
//    latest finish (the decrement is a release and its read an acquire, so
//    a zero count sees every max before it).
// Timing:
//  * static orders: links advance through chain[] in rounds. Contiguous
//    transfers (a.contig) on links between nodes: the link's next send
//    either joins the open transfer (same remaining length, chunk ready by
//    the transfer's start; m sends cost alpha + ceil(beta*m*S/1000)) or
//    closes it and opens a new one. Finish times of a transfer's sends are
//    published only when it closes, so no dependant reads a time that could
//    still grow; a joiner's pred has a strictly longer remaining path than
//    the transfer, so waiting for it never waits on the transfer;
//  * time-aware greedy (a.greedy == 1, App. B.2): the unserved ready send
//    with the smallest (max(ready, link free), Step-2 key, priority, slot)
//    goes next, simulated exactly in windows (below);
//  * greedy in reverse path order (a.greedy == 2): the same greedy on the
//    mirrored schedule, whose dependencies are the other form (Allgather
//    sends wait for the sends out of their destination, ReduceScatter sends
//    for the send that carries their partial on) and whose keys the caller
//    built with the lengths measured from the other end; a link's real
//    order is the reverse of the order the mirrored greedy served it in,
//    and the real times come from the static rounds over those orders.
// Returns true on a fault (no progress; unreachable for valid orders).
__device__ __forceinline__ bool any_schedule(const TreeArgs &a, bool rs, int lane,
                                          const uint32_t *s_cost, const uint8_t *s_src,
                                          const uint8_t *s_own, const uint64_t *key,
                                          const uint32_t *prio, const uint16_t *par,
                                          uint32_t *chain, const uint32_t *lbase,
                                          uint32_t *lhead, uint32_t *lfree, uint32_t *fin,
                                          uint32_t *pend, uint32_t *rdy, uint32_t *gst,
                                          uint32_t *grem, uint32_t *gcnt, uint32_t *gfirst,
                                          uint32_t &mk) {
  const int V = a.V, E = a.E, CV = a.C * a.V;
  const uint32_t total = lbase[E];
  auto ready_of = [&](uint32_t ent, bool push) -> uint32_t {
    const uint32_t s = ent & 0xFFFFu;
    if (push) {
      if (__hip_atomic_load(&pend[s], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP))
        return kNotYet;
      return lds_get(&rdy[s]);
    }
    const uint32_t p = ent >> 16;
    return p == kNoPred ? 0u : lds_get(&fin[p]);
  };
  auto publish = [&](uint32_t s, uint32_t f, int l, bool push) {
    lds_put(&fin[s], f);
    if (push) {
      const uint32_t c = div_v(s, a.vmagic);
      const int u = s_src[l];
      if (u != s_own[c]) {
        const uint32_t q = c * V + u;
        __hip_atomic_fetch_max(&rdy[q], f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        __hip_atomic_fetch_sub(&pend[q], 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
      }
    }
  };

  if (a.greedy) {
    // plans have no zero-cost link, so c_min > 0 and every window serves
    const bool mirror = a.greedy == 2, push = rs != mirror;
    // windows (as in the record-based greedy kernels, with the same steps,
    // greedy_window.h): W = the earliest start any ready send can take; a
    // send not ready yet can only start c_min or more after W, so on every
    // link the best ready send with start < W + c_min is the greedy's next
    // there. Each link's pending sends are the front of its chain[] segment
    // (count in lhead[]); a served send is swapped to the end of the
    // pending part, so the segment ends up in reverse service order. In the
    // push form a send's ready time appears in fin[] once its last input is
    // served (a send without inputs is ready at 0).
    const ChainView cv{chain, key, prio};
    for (int l = lane; l < E; l += 64) lhead[l] = lbase[l + 1] - lbase[l];
    if (push)
      for (int s = lane; s < CV; s += 64)
        if (par[s] && pend[s] == 0) fin[s] = 0;
    wave_sync();
    uint32_t gmk = 0;
    for (uint32_t round = 0;; round++) {
      uint32_t wmin = kNotYet;
      for (int l = lane; l < E; l += 64) {
        const GreedyLink lk{lfree[l], lbase[l], lhead[l]};
        const GreedyBest b =
            push ? greedy_scan_link<true>(lk, cv, fin) : greedy_scan_link<false>(lk, cv, fin);
        gst[l] = greedy_start(b);
        gfirst[l] = b.w2;
        wmin = min(wmin, gst[l]);
      }
      wmin = ~wave_reduce_max(~wmin);
      if (wmin == kNotYet) break;
      if (round > total) return true;  // unreachable: every window serves a send
      const uint64_t wend = (uint64_t)wmin + a.cmin;
      wave_sync();
      bool lost = false;
      for (int l = lane; l < E; l += 64) {
        const uint32_t cs = gst[l];
        if (cs == kNotYet || (uint64_t)cs >= wend) continue;
        GreedyLink lk{lfree[l], lbase[l], lhead[l]};
        const GreedyBest b{(uint64_t)cs << 32, 0, gfirst[l]};
        lost |= push ? greedy_commit<true, LdsAtomics>(lk, b, s_cost[l], cv, fin, rdy, pend, gmk)
                     : greedy_commit<false, LdsAtomics>(lk, b, s_cost[l], cv, fin, rdy, pend, gmk);
        lfree[l] = lk.free;
        lhead[l] = lk.len;
      }
      if (__ballot(lost)) return true;  // unreachable: the index is the winner's
      wave_sync();
    }
    if (!mirror) mk = max(mk, gmk);
    bool left = false;  // a send that never became ready: unreachable
    for (int l = lane; l < E; l += 64) left |= lhead[l] != 0;
    if (__ballot(left)) return true;
    if (!mirror) return false;
    wave_sync();
    for (int s = lane; s < CV; s += 64) {
      fin[s] = kNotYet;
      pend[s] = 0;
      rdy[s] = 0;
    }
    for (int l = lane; l < E; l += 64) {
      lhead[l] = lbase[l];
      lfree[l] = 0;
      gcnt[l] = 0;
    }
    wave_sync();
    if (rs)  // the real ReduceScatter counts the sends into every vertex
      for (int s = lane; s < CV; s += 64) {
        const int pl = par[s];
        if (!pl) continue;
        const uint32_t c = div_v(s, a.vmagic);
        const int u = s_src[pl - 1];
        if (u != s_own[c]) atomicAdd(&pend[c * V + u], 1u);
      }
    wave_sync();
  }

  for (uint32_t round = 0;; round++) {
    bool pending = false;
    for (int l = lane; l < E; l += 64) {
      uint32_t h = lhead[l];
      const uint32_t e = lbase[l + 1];
      uint32_t f = lfree[l];
      if (!(a.contig && a.lmerge[l])) {
        if (h == e) continue;
        const uint32_t cl = s_cost[l];
        while (h < e) {
          const uint32_t ent = chain[h];
          const uint32_t r = ready_of(ent, rs);
          if (r == kNotYet) break;
          f = max(r, f) + cl;
          publish(ent & 0xFFFFu, f, l, rs);
          h++;
        }
        pending |= h < e;
      } else {
        uint32_t gs = gst[l], gr = grem[l], gm = gcnt[l], g0 = gfirst[l];
        if (h == e && gm == 0) continue;
        const uint32_t le = rs ? a.lrev[l] : (uint32_t)l;  // the link the sends use
        const uint32_t al = a.lalpha[le];
        const uint64_t bsz = a.lbs[le];
        while (true) {
          if (h == e) {
            for (uint32_t j = g0; j < h && gm; j++) publish(chain[j] & 0xFFFFu, f, l, rs);
            gm = 0;
            break;
          }
          const uint32_t ent = chain[h];
          const uint32_t rem = ~(uint32_t)(key[ent & 0xFFFFu] >> 32);
          uint32_t r = kNotYet;
          if (gm && rem == gr) {
            r = ready_of(ent, rs);
            if (r == kNotYet) break;
            if (r <= gs) {  // joins the open transfer
              gm++;
              f = gs + al + (uint32_t)((bsz * gm + 999) / 1000);
              h++;
              continue;
            }
          }
          for (uint32_t j = g0; j < h && gm; j++) publish(chain[j] & 0xFFFFu, f, l, rs);
          gm = 0;
          if (r == kNotYet) r = ready_of(ent, rs);
          if (r == kNotYet) break;
          gs = max(r, f);
          f = gs + al + (uint32_t)((bsz + 999) / 1000);
          gm = 1;
          g0 = h;
          gr = rem;
          h++;
        }
        gst[l] = gs;
        grem[l] = gr;
        gcnt[l] = gm;
        gfirst[l] = g0;
        pending |= h < e || gm;
      }
      lhead[l] = h;
      lfree[l] = f;
      mk = max(mk, f);
    }
    if (__ballot(pending) == 0) return false;
    if (round > 2 * total + 2) return true;  // unreachable: key order is topological
  }
}

// kRecLds: the route records fit in LDS (else they are read from global
// memory, where they stay cache resident). kPrefetch: a candidate's routes
// (whole words) and priorities fit the prefetch registers. kAny: the
// variant for plans outside the layered kernel's limits that also times
// ReduceScatter (a.reduce), contiguous transfers (a.contig) and the
// time-aware greedy (a.greedy); see step 5' below.
template <bool kRecLds, bool kPrefetch, bool kAny>
__global__ __launch_bounds__(kTreeMaxThreads) void tree_eval_kernel(TreeArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int C = a.C, V = a.V, E = a.E, MW = a.mask_words;
  const int CV = C * V;
  const bool rs = kAny && a.reduce;

  // ---- block-wide copy of the plan tables --------------------------------
  uint32_t *s_cost = (uint32_t *)(lds + a.o_cost);
  uint8_t *s_src = lds + a.o_src;
  uint8_t *s_own = lds + a.o_own;
  uint64_t *s_post = (uint64_t *)(lds + a.o_post);
  const uint32_t *s_rec = kRecLds ? (const uint32_t *)(lds + a.o_rec) : a.rec;
  for (int j = threadIdx.x; j < E; j += blockDim.x) {
    uint32_t cj = a.cost[j];
    if (rs) {  // a ReduceScatter send on the reverse of a tree link
      const uint32_t r = a.lrev[j];
      cj = r != 0xFFFFu ? a.cost[r] : 0u;
    }
    s_cost[j] = cj;
    s_src[j] = (uint8_t)a.lsrc[j];
  }
  if (kRecLds)
    for (int j = threadIdx.x; j < a.rec_len; j += blockDim.x)
      ((uint32_t *)(lds + a.o_rec))[j] = a.rec[j];
  for (int j = threadIdx.x; j < C; j += blockDim.x) {
    s_own[j] = a.owner8[j];
    s_post[j] = a.post_mask[j];
  }
  __syncthreads();

  // ---- per-wave state ----------------------------------------------------
  // key[s]: (dist, height) of vertex v = s % V of chunk c = s / V while the
  //         tree is built, then the send's packed Step-2 key;
  // prio[s]: the send's priority, then its finish time (fin);
  // chain[s]: the chunk's discovery order while the tree is built, then the
  //         per-link orders (pred << 16 | slot), one run per link.
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  unsigned char *wl = lds + a.o_wave + wave * a.wave_bytes;
  uint8_t *rt = wl + a.w_rt;
  uint32_t *rt32 = (uint32_t *)rt;
  uint64_t *key = (uint64_t *)(wl + a.w_key);
  uint32_t *prio = (uint32_t *)(wl + a.w_prio);
  uint32_t *fin = prio;
  uint32_t *chain = (uint32_t *)(wl + a.w_chain);
  uint32_t *ord = chain;
  uint16_t *par = (uint16_t *)(wl + a.w_par);     // link+1 into (c,v), 0 = none
  uint32_t *lmask = (uint32_t *)(wl + a.w_mask);  // [E][MW] chunk bits per link
  uint32_t *lbase = (uint32_t *)(wl + a.w_base);  // [E+1]
  uint32_t *lhead = (uint32_t *)(wl + a.w_head);  // [E]
  uint32_t *lfree = (uint32_t *)(wl + a.w_free);  // [E]
  if (kAny) fin = (uint32_t *)(wl + a.w_gfin);     // priorities stay for the greedy
  // kAny: ReduceScatter partials still to come into (c,v) and the latest of
  // them; contiguous transfer open on each link (start, remaining length,
  // sends, first position)
  uint32_t *pend = (uint32_t *)(wl + a.w_gpend);
  uint32_t *rdy = (uint32_t *)(wl + a.w_grdy);
  uint32_t *gst = (uint32_t *)(wl + a.w_gst), *grem = gst + E, *gcnt = grem + E, *gfirst = gcnt + E;

  const int64_t stride = (int64_t)gridDim.x * a.waves_per_block;
  const int64_t first = (int64_t)blockIdx.x * a.waves_per_block + wave;
  // Software pipeline: the next candidate's routes and priorities are
  // loaded into registers while the current one is evaluated, so the HBM
  // latency overlaps the work instead of stalling every candidate.
  const int nrw = kPrefetch ? (a.route_stride >> 2) : 0;  // route words per candidate
  uint32_t pf_r[kPfRoute], pf_p[kPfPrio];
  auto prefetch = [&](int64_t i) {
    if (i >= a.n) return;
    const uint32_t *g32 = (const uint32_t *)(a.routes + (size_t)i * a.route_stride);
    const uint32_t *gpr = a.prio + (size_t)i * a.prio_stride;
#pragma unroll
    for (int k = 0; k < kPfRoute; k++) {
      const int j = lane + 64 * k;
      if (j < nrw) pf_r[k] = __builtin_nontemporal_load(g32 + j);
    }
#pragma unroll
    for (int k = 0; k < kPfPrio; k++) {
      const int j = lane + 64 * k;
      if (j < CV) pf_p[k] = __builtin_nontemporal_load(gpr + j);
    }
  };
  if (kPrefetch) prefetch(first);
  for (int64_t i = first; i < a.n; i += stride) {
    // ---- 1. stage the candidate ----------------------------------------
    if (kPrefetch) {
#pragma unroll
      for (int k = 0; k < kPfRoute; k++) {
        const int j = lane + 64 * k;
        if (j < nrw) rt32[j] = pf_r[k];
      }
#pragma unroll
      for (int k = 0; k < kPfPrio; k++) {
        const int j = lane + 64 * k;
        if (j < CV) prio[j] = pf_p[k];
      }
      prefetch(i + stride);
    } else {
      const uint8_t *grt = a.routes + (size_t)i * a.route_stride;
      const uint32_t *gpr = a.prio + (size_t)i * a.prio_stride;
      for (int j = lane; j < a.route_stride; j += 64) rt[j] = grt[j];
      for (int j = lane; j < CV; j += 64) prio[j] = gpr[j];
    }
    for (int j = lane; j < CV; j += 64) par[j] = 0;
    for (int j = lane; j < E * MW; j += 64) lmask[j] = 0;
    if (kAny) {
      for (int j = lane; j < CV; j += 64) {
        pend[j] = 0;
        rdy[j] = 0;
        fin[j] = kNotYet;
      }
      for (int j = lane; j < E; j += 64) gcnt[j] = 0;
    }
    wave_sync();

    // ---- 2+3. lane = chunk: first-reach tree, then heights and keys -------
    // reverse path order measures the Step-2 lengths from the other end:
    // the keys (and child counts) of the other direction
    const bool up = rs != (kAny && a.greedy == 2);
    const bool ok = up ? build_trees<true, true>(a, s_rec, s_cost, s_own, s_post, rt, key, par,
                                                 ord, lmask, lane, pend)
                       : build_trees<true>(a, s_rec, s_cost, s_own, s_post, rt, key, par, ord,
                                           lmask, lane);
    wave_sync();
    {
      // link bases: exclusive scan of the mask popcounts
      const int per = (E + 63) / 64;
      const int b = min(lane * per, E), e = min(b + per, E);
      uint32_t sum = 0;
      for (int l = b; l < e; l++)
        for (int w = 0; w < MW; w++) sum += __popc(lmask[l * MW + w]);
      const uint32_t incl = wave_incl_scan(sum, lane);
      uint32_t run = incl - sum;
      for (int l = b; l < e; l++) {
        lbase[l] = run;
        lhead[l] = run;
        lfree[l] = 0;
        for (int w = 0; w < MW; w++) run += __popc(lmask[l * MW + w]);
      }
      if (lane == 63) lbase[E] = incl;
    }
    wave_sync();

    // ---- 4. place every send in its link's order --------------------------
    for (int s = lane; s < CV; s += 64) {
      const int pl = par[s];
      if (!pl) continue;
      const int l = pl - 1;
      const uint32_t c = div_v(s, a.vmagic);
      const uint32_t v = s - c * V;
      const uint64_t kx = key[s];
      const uint32_t px = prio[s];
      uint32_t rank = 0;
      for (int w = 0; w < MW; w++) {
        uint32_t m = lmask[l * MW + w];
        while (m) {
          // four competitors at a time (the chunk itself pads, never counts);
          // every send on l enters v, so a competitor's slot is yc*V + v
          uint32_t y[4];
#pragma unroll
          for (int t = 0; t < 4; t++) {
            const uint32_t yc = m ? (w << 5) + __builtin_ctz(m) : c;
            m &= m - 1;
            y[t] = yc * V + v;
          }
          uint64_t ky[4];
          uint32_t py[4];
#pragma unroll
          for (int t = 0; t < 4; t++) {
            ky[t] = key[y[t]];
            py[t] = prio[y[t]];
          }
#pragma unroll
          for (int t = 0; t < 4; t++)
            rank += (ky[t] < kx) || (ky[t] == kx && (py[t] < px || (py[t] == px && y[t] < s)));
        }
      }
      const int u = s_src[l];
      const uint32_t pred = (u == s_own[c]) ? kNoPred : c * V + u;
      chain[lbase[l] + rank] = (pred << 16) | (uint32_t)s;
    }
    wave_sync();
    if (!kAny) {
      for (int s = lane; s < CV; s += 64) lds_put(&fin[s], kNotYet);
      wave_sync();
    }

    // ---- 5. least schedule: links advance through their orders -----------
    const uint32_t total = lbase[E];
    uint32_t mk = 0;
    bool fault = false;
    if (kAny) {
      fault = any_schedule(a, rs, lane, s_cost, s_src, s_own, key, prio, par, chain, lbase, lhead,
                           lfree, fin, pend, rdy, gst, grem, gcnt, gfirst, mk);
    } else {
      for (uint32_t round = 0;; round++) {
        bool pending = false;
        for (int l = lane; l < E; l += 64) {
          uint32_t h = lhead[l];
          const uint32_t e = lbase[l + 1];
          if (h == e) continue;
          uint32_t f = lfree[l];
          const uint32_t cl = s_cost[l];
          uint32_t ent = chain[h];
          while (true) {
            const uint32_t nxt = (h + 1 < e) ? chain[h + 1] : 0u;  // read ahead
            const uint32_t p = ent >> 16;
            const uint32_t ready = (p == kNoPred) ? 0u : lds_get(&fin[p]);
            if (ready == kNotYet) break;
            f = max(ready, f) + cl;
            lds_put(&fin[ent & 0xFFFFu], f);
            if (++h == e) break;
            ent = nxt;
          }
          lhead[l] = h;
          lfree[l] = f;
          mk = max(mk, f);
          pending |= h < e;
        }
        if (__ballot(pending) == 0) break;
        if (round > total) {  // unreachable: the order is acyclic
          fault = true;
          break;
        }
      }
    }

    // ---- 6. postcondition and makespan -----------------------------------
    const bool all_ok = __ballot(!ok) == 0;
    fault = __ballot(fault) != 0;
    mk = wave_max(mk);
    if (lane == 0) {
      if (kAny && a.accumulate) {  // second phase of an Allreduce
        const uint32_t m0 = a.makespan[i];
        a.makespan[i] = (fault || m0 == 0xFFFFFFFFu) ? 0xFFFFFFFFu : m0 + mk;
        a.valid[i] = (uint8_t)(a.valid[i] && all_ok && !fault);
      } else {
        a.makespan[i] = fault ? 0xFFFFFFFFu : mk;
        a.valid[i] = (uint8_t)(all_ok && !fault);
      }
    }
    wave_sync();
  }
}


// Route word j (route bytes of chunk j / PW, destinations 4 (j % PW) ..
// +3) as one-hot option bytes: 1 << choice, 0 for a choice of 8 or more
// (no pair has that many options) and 0 for a destination outside the
// chunk's postcondition (such an entry is never routed).
template <int PW>
__device__ __forceinline__ uint32_t one_hot_word(uint32_t w, uint32_t j, const uint64_t *s_post) {
  const uint32_t pm4 = (uint32_t)(s_post[j / PW] >> (4 * (j % PW))) & 0xFu;
  uint32_t oh = 0;
#pragma unroll
  for (int b = 0; b < 4; b++) {
    const uint32_t kb = (w >> (8 * b)) & 0xFFu;
    oh |= ((kb < 8 && ((pm4 >> b) & 1)) ? (1u << kb) : 0u) << (8 * b);
  }
  return oh;
}

// LDS views that the slot-parallel tree construction reads and writes.
struct TreeLds {
  const uint32_t *cost;
  const uint8_t *own;
  const uint64_t *post;
  const uint4 *rec;
  const uint32_t *opt;
  const uint16_t *rev;
  const uint32_t *rt32;
  uint32_t *dist;
  uint16_t *anc;  // pj_rounds arrays of anc_stride slots: 2^k-th ancestor
};

// Trees, one lane per (chunk c, vertex v) slot (slots lane + 64j). The
// first-reach merge gives v the hop that enters it on the path of the
// smallest destination whose path contains v (found from the one-hot route
// bytes and the per-vertex option bytes, no walk). Distances from the owner
// and the largest distance below every vertex then follow by doubling over
// ancestors (pointer jumping), in ceil(log2 V) rounds each, whatever the
// depth of the trees. On return, per slot with a send: pe = link | parent
// vertex << 16, ps = parent's slot (or kNoPred when the parent is the owner),
// dv = distance from the owner to v; dist[slot] = largest distance below v
// (Allgather) or, for ReduceScatter (kRS: costs of the reverse links), the
// longest reversed path from below up to v. `bad`: a rank of the
// postcondition is unreached; `fault` is never set (parents form a tree).
template <int J, int PW, bool kRS>
__device__ __forceinline__ void slot_trees(const TreeArgs &a, const TreeLds &tl, int lane,
                                           uint32_t (&pe)[J], uint32_t (&ps)[J],
                                           uint32_t (&dv)[J], bool &bad, bool &fault) {
  const int C = a.C, V = a.V, K = a.K;
  constexpr int P = 4 * PW;
  const int CV = C * V;
  const uint32_t *s_cost = tl.cost;
  const uint8_t *s_own = tl.own;
  const uint64_t *s_post = tl.post;
  const uint4 *s_rec = tl.rec;
  const uint32_t *s_opt = tl.opt;
  const uint16_t *s_rev = tl.rev;
  const uint32_t *rt32 = tl.rt32;
  uint32_t *dist = tl.dist;
  uint16_t *anc = tl.anc;
  // The parent hop of every slot, in groups of (up to) four slots and in
  // stages, each stage issuing the LDS loads of the whole group before any
  // is used (selects instead of branches).
  uint32_t ec[J];          // cost of the link into the slot
  uint32_t an[J], acc[J];  // 2^k-th ancestor slot, cost of the path up to it
  constexpr int G = J < 4 ? J : 4;
#pragma unroll
  for (int g0 = 0; g0 < J; g0 += G) {
    uint32_t c[G], v[G], o[G], slc[G];
    uint64_t pm[G];
#pragma unroll
    for (int q = 0; q < G; q++) {
      const uint32_t sl = lane + 64 * (g0 + q);
      slc[q] = sl < (uint32_t)CV ? sl : 0u;
      c[q] = div_v(slc[q], a.vmagic);
      v[q] = slc[q] - c[q] * V;
    }
#pragma unroll
    for (int q = 0; q < G; q++) {
      o[q] = s_own[c[q]];
      pm[q] = s_post[c[q]];
    }
    // (chosen option bit & options through v), one byte per destination
    // (destinations outside the postcondition were zeroed when staged): its
    // lowest set bit is byte 4w + b of the smallest destination d whose
    // drawn path passes through v, and the bit inside the byte is that
    // path's option kd
    uint32_t t[G][PW];
#pragma unroll
    for (int q = 0; q < G; q++)
#pragma unroll
      for (int w = 0; w < PW; w++)
        t[q][w] = rt32[c[q] * PW + w] & s_opt[(o[q] * V + v[q]) * PW + w];
    uint32_t d[G], kd[G];
    bool has[G];
#pragma unroll
    for (int q = 0; q < G; q++) {
      uint32_t tw = t[q][PW - 1], wi = PW - 1;
#pragma unroll
      for (int w = PW - 2; w >= 0; w--)
        if (t[q][w]) {
          tw = t[q][w];
          wi = w;
        }
      const bool in = lane + 64 * (g0 + q) < (uint32_t)CV;
      const bool root = v[q] == o[q];
      has[q] = in && !root && tw != 0;
      bad |= in && !root && tw == 0 && ((pm[q] >> v[q]) & 1);  // a rank is never reached
      const uint32_t bit = tw ? (uint32_t)__builtin_ctz(tw) : 0u;
      d[q] = 4 * wi + (bit >> 3);
      kd[q] = bit & 7;
    }
    uint4 r[G];
#pragma unroll
    for (int q = 0; q < G; q++) r[q] = s_rec[(o[q] * P + d[q]) * K + kd[q]];
    uint32_t l[G], u[G];
#pragma unroll
    for (int q = 0; q < G; q++) {
      // the hop of that path that enters v
      const uint32_t x0 = r[q].x & 0xFFFFFFu, x1 = r[q].y, x2 = r[q].z, x3 = r[q].w;
      uint32_t e = x3, uu = (x2 >> 16) & 0xFFu;
      if (((x2 >> 16) & 0xFFu) == v[q]) {
        e = x2;
        uu = (x1 >> 16) & 0xFFu;
      }
      if (((x1 >> 16) & 0xFFu) == v[q]) {
        e = x1;
        uu = (x0 >> 16) & 0xFFu;
      }
      if ((x0 >> 16) == v[q]) {
        e = x0;
        uu = o[q];
      }
      l[q] = e & 0xFFFFu;
      u[q] = uu;
    }
    // ReduceScatter measures the tree backwards, on reverse links
#pragma unroll
    for (int q = 0; q < G; q++) ec[g0 + q] = s_cost[has[q] ? (kRS ? s_rev[l[q]] : l[q]) : 0u];
#pragma unroll
    for (int q = 0; q < G; q++) {
      const int j = g0 + q;
      const bool top = u[q] == o[q];  // the parent is the chunk's owner
      pe[j] = has[q] ? (l[q] | (u[q] << 16)) : ~0u;
      ps[j] = (has[q] && !top) ? c[q] * V + u[q] : kNoPred;
      // ancestor chain: the parent's slot; the owner's slot (and a slot
      // without a send) is its own ancestor, with distance 0
      an[j] = has[q] ? (top ? c[q] * V + o[q] : c[q] * V + u[q]) : slc[q];
      acc[j] = has[q] ? ec[j] : 0u;
      const uint32_t sl = lane + 64 * j;
      if (sl < (uint32_t)CV) {
        dist[sl] = acc[j];
        anc[sl] = (uint16_t)an[j];
      }
    }
  }
  wave_sync();
  // distances by doubling: acc covers 2^k links up the chain (or reaches the
  // owner, whose slot adds 0 and is its own ancestor); every slot reads its
  // ancestor's pair before any slot writes
  const int R = a.pj_rounds;
  const int AS = a.anc_stride;
  for (int k = 0; k < R; k++) {
    uint32_t ra[J], rn[J];
#pragma unroll
    for (int j = 0; j < J; j++) {
      ra[j] = dist[an[j]];
      rn[j] = anc[k * AS + an[j]];
    }
    wave_sync();
#pragma unroll
    for (int j = 0; j < J; j++) {
      const uint32_t sl = lane + 64 * j;
      acc[j] += ra[j];
      an[j] = rn[j];
      if (sl < (uint32_t)CV) {
        dist[sl] = acc[j];
        if (k + 1 < R) anc[(k + 1) * AS + sl] = (uint16_t)rn[j];
      }
    }
    wave_sync();
  }
  // largest distance below every vertex: in round k each slot pushes the
  // largest distance it knows below it to its 2^k-th ancestor, so after
  // round k a slot knows every descendant less than 2^(k+1) links down
  // (values only ever grow, each is a descendant's distance)
#pragma unroll
  for (int j = 0; j < J; j++) dv[j] = (pe[j] != ~0u) ? acc[j] : kNotYet;
  for (int k = 0; k < R; k++) {
    uint32_t m[J], up[J];
#pragma unroll
    for (int j = 0; j < J; j++) {
      const uint32_t sl = lane + 64 * j;
      const uint32_t slc = sl < (uint32_t)CV ? sl : 0u;
      m[j] = dist[slc];
      up[j] = anc[k * AS + slc];
    }
#pragma unroll
    for (int j = 0; j < J; j++)
      if (pe[j] != ~0u) atomicMax(&dist[up[j]], m[j]);
    wave_sync();
  }
  if (kRS) {
    // ReduceScatter: longest reversed path from a vertex below v up to v =
    // largest reversed distance below v minus v's own
#pragma unroll
    for (int j = 0; j < J; j++)
      if (pe[j] != ~0u) dist[lane + 64 * j] -= acc[j];
    wave_sync();
  }
  (void)fault;
}

// Layered variant for plans with at most 4 hops and 8 options per pair,
// 4 | P <= 32 and C*V <= 1024.
//
// Trees, one lane per (chunk c, vertex v) slot. Merging the destinations'
// paths by first reach in ascending destination order gives v the hop that
// enters it on the path of the smallest destination whose path contains v;
// that destination is found from the route bytes and a plan table of the
// options passing through each vertex, with no walk. Distances from the
// owner follow in rounds (a slot waits for its parent's distance), then the
// largest distance below each vertex is pushed up the tree deepest level
// first; a send into v from u then has trav = dist(u) and
// rem = cost + height(v) = maxdist_below(v) - dist(u) (Sec. 5.1).
//
// Order and timing. A send's layer is floor(rem / c_min) (computed as
// (rem * ceil(2^32 / c_min)) >> 32). Along a tree edge rem grows by at
// least one link cost, so a send's parent send lies in a higher layer; a
// link's Step-2 order sorts by rem first, so the sends of one layer on one
// link are a contiguous run of that link's order. Taking the layers from
// the top down, every dependency inside a layer runs along a link run, and
// the k-th send of a run with ready times r_j, cost c and link busy time F
// finishes at
//     f_k = max(F + (k+1)c, max_{j<=k} r_j + (k-j+1)c),
// the unrolled form of f = max(ready, link free) + c (App. B.3).
// The sends are counting-sorted by (non-empty layer from the top, link)
// with 16-bit counters, each bucket is ordered by the full key
// (rem, trav, priority, chunk), and the layers are timed in turn, one lane
// per send.
template <int J, int PW, bool kContig, bool kRS>
__global__ __launch_bounds__(kTreeMaxThreads)
void tree_layers_kernel(TreeArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int C = a.C, V = a.V, E = a.E, K = a.K;
  constexpr int P = 4 * PW;  // ranks; route bytes per chunk
  const int CV = C * V;

  uint32_t *s_cost = (uint32_t *)(lds + a.o_cost);
  uint8_t *s_src = lds + a.o_src;
  uint8_t *s_own = lds + a.o_own;
  uint64_t *s_post = (uint64_t *)(lds + a.o_post);
  uint4 *s_rec = (uint4 *)(lds + a.o_rec4);       // one 16-byte record per option
  uint32_t *s_opt = (uint32_t *)(lds + a.o_opt);  // option bytes, PW words per (o, v)
  uint8_t *s_merge = lds + a.o_merge;             // links that carry contiguous transfers
  uint16_t *s_rev = (uint16_t *)(lds + a.o_rev);  // ReduceScatter: reverse link
  uint8_t *s_dst = lds + a.o_ldst;
  for (int j = threadIdx.x; j < E; j += blockDim.x) {
    s_cost[j] = a.cost[j];
    s_src[j] = (uint8_t)a.lsrc[j];
    s_merge[j] = a.contig ? a.lmerge[j] : 0;
    if (kRS) {
      s_rev[j] = a.lrev[j];
      s_dst[j] = (uint8_t)a.ldst[j];
    }
  }
  for (int r = threadIdx.x; r < P * P * K; r += blockDim.x) s_rec[r] = a.rec4[r];
  for (int j = threadIdx.x; j < P * V * PW; j += blockDim.x)
    s_opt[j] = ((const uint32_t *)a.topt)[j];
  for (int j = threadIdx.x; j < C; j += blockDim.x) {
    s_own[j] = a.owner8[j];
    s_post[j] = a.post_mask[j];
  }
  __syncthreads();

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  unsigned char *wl = lds + a.o_wave + wave * a.wave_bytes;
  // Regions reused as their contents die. Trees: route words and per-slot
  // distances (later the largest distance below). Bucketing: 16-bit
  // counters, then bucket entries {~rem, trav, priority, slot}. Ordered
  // sends: slot | parent send's slot << 16 and link | index in its run
  // << 16. Timing: finish times per slot and ready times per position.
  uint32_t *rt32 = (uint32_t *)wl;
  uint32_t *dist = (uint32_t *)(wl + a.w_dist);
  uint16_t *anc = (uint16_t *)(wl + a.w_anc);
  uint32_t *cnt = (uint32_t *)(wl + a.w_cnt);
  uint4 *erec = (uint4 *)(wl + a.w_erec);
  uint32_t *ord2 = (uint32_t *)(wl + a.w_ord2);
  uint32_t *info2 = (uint32_t *)(wl + a.w_info2);
  uint32_t *fin = (uint32_t *)(wl + a.w_fin);
  uint32_t *rq = (uint32_t *)(wl + a.w_rq);
  uint32_t *lfree = (uint32_t *)(wl + a.w_free);
  uint64_t *lmask64 = (uint64_t *)(wl + a.w_lmask);
  uint32_t *lst = (uint32_t *)(wl + a.w_lst);  // first ordered position of each layer
  uint32_t *bnd = (uint32_t *)(wl + a.w_bnd);  // bucket start | end << 16 per position
  auto start_of = [&](uint32_t b) -> uint32_t {
    return (cnt[b >> 1] >> ((b & 1) << 4)) & 0xFFFFu;
  };
  // a send (slot | parent or consumer slot << 16) ends at f: Allgather
  // records it for the sends it feeds; ReduceScatter raises the ready time
  // of the send that carries its partial on
  auto finish = [&](uint32_t e, uint32_t f) {
    if (kRS) {
      if ((e >> 16) != kNoPred) atomicMax(&fin[e >> 16], f);
    } else {
      fin[e & 0xFFFFu] = f;
    }
  };

  const int64_t stride = (int64_t)gridDim.x * a.waves_per_block;
  const int64_t first = (int64_t)blockIdx.x * a.waves_per_block + wave;
  const int nrw = a.route_stride >> 2;
  uint32_t pf_r[kPfRoute], pf_p[J];
  // the next candidate's routes and priorities stream into registers while
  // the current one is evaluated
  auto prefetch = [&](int64_t i) {
    if (i >= a.n) return;
    const uint32_t *g32 = (const uint32_t *)(a.routes + (size_t)i * a.route_stride);
    const uint32_t *gpr = a.prio + (size_t)i * a.prio_stride;
#pragma unroll
    for (int k = 0; k < kPfRoute; k++) {
      const int j = lane + 64 * k;
      if (j < nrw) pf_r[k] = __builtin_nontemporal_load(g32 + j);
    }
#pragma unroll
    for (int k = 0; k < J; k++) {
      const int j = lane + 64 * k;
      if (j < CV) pf_p[k] = __builtin_nontemporal_load(gpr + j);
    }
  };
  prefetch(first);
  for (int64_t i = first; i < a.n; i += stride) {
    // ---- stage: routes to LDS, own slots' priorities stay in registers --
    // route bytes become one-hot option bytes (1 << choice, 0 for a choice
    // of 8 or more, which no pair has)
#pragma unroll
    for (int k = 0; k < kPfRoute; k++) {
      const int j = lane + 64 * k;
      if (j < nrw) rt32[j] = one_hot_word<PW>(pf_r[k], j, s_post);
    }
    uint32_t px[J];
#pragma unroll
    for (int k = 0; k < J; k++) px[k] = pf_p[k];
    prefetch(i + stride);
    for (int l = lane; l < E; l += 64) lfree[l] = 0;
    if (lane == 0) *lmask64 = 0;
    wave_sync();

    // ---- trees: the hop into every reached (chunk, vertex) ---------------
    // pe: link | parent vertex << 16 of the send into the slot, ~0 if none
    uint32_t pe[J], ps[J], dv[J];
    bool bad = false, fault = false;
    slot_trees<J, PW, kRS>(a, TreeLds{s_cost, s_own, s_post, s_rec, s_opt, s_rev, rt32, dist, anc},
                           lane, pe, ps, dv, bad, fault);

    // ---- keys and layers of this lane's sends ----------------------------
    uint32_t bl[J];  // link | layer << 16, or ~0 for no send
    uint64_t kk[J];
    uint64_t lm = 0;
    bool clamped = false;
    {
      // Allgather: trav = dist(u), rem = cost + height(v) = maxdist_below(v)
      // - dist(u). ReduceScatter (send v -> u on the reverse link): rem =
      // reversed distance from v to the owner, trav = longest reversed path
      // up to v. The loads of all slots first, then the arithmetic.
      uint32_t lk[J], cl[J], dd[J];
#pragma unroll
      for (int j = 0; j < J; j++) {
        const bool has = pe[j] != ~0u;
        const uint32_t l0 = has ? pe[j] & 0xFFFFu : 0u;
        lk[j] = kRS ? (has ? s_rev[l0] : 0u) : l0;
        const uint32_t sl = lane + 64 * j;
        dd[j] = dist[sl < (uint32_t)CV ? sl : 0u];
      }
#pragma unroll
      for (int j = 0; j < J; j++) cl[j] = kRS ? 0u : s_cost[lk[j]];
#pragma unroll
      for (int j = 0; j < J; j++) {
        bl[j] = ~0u;
        kk[j] = 0;
        if (pe[j] != ~0u) {
          const uint32_t trav = kRS ? dd[j] : dv[j] - cl[j];
          const uint32_t rem = kRS ? dv[j] : dd[j] - trav;
          uint32_t L = (uint32_t)(((uint64_t)rem * a.lmagic) >> 32);
          if (L >= (uint32_t)a.nl_max) {  // unreachable: rem is bounded at plan time
            L = a.nl_max - 1;
            clamped = true;
          }
          bl[j] = lk[j] | (L << 16);
          kk[j] = ((uint64_t)(~rem) << 32) | trav;  // ascending = rem desc, trav asc
          lm |= 1ull << L;
        }
      }
    }
    if (lm) atomicOr((unsigned long long *)lmask64, (unsigned long long)lm);
    wave_sync();
    const uint64_t layers = *lmask64;
    const int nl = __popcll(layers);
    const uint32_t NB = (uint32_t)nl * E;  // buckets (layer from the top, link)
    const int NW = (int)((NB + 2) >> 1);   // u16 counters for NB + 1 starts
    for (int w = lane; w < NW; w += 64) cnt[w] = 0;
    wave_sync();

    // ---- counting sort by (layer from the top, link) ---------------------
    // a slot without a send counts in a per-lane dummy word past the
    // counters, so every slot issues its update without a branch
    uint32_t bb[J], idx[J];
#pragma unroll
    for (int k = 0; k < J; k++) {
      const bool has = bl[k] != ~0u;
      const uint32_t L = (bl[k] >> 16) & 63u;
      const uint32_t above = (uint32_t)__popcll((layers >> L) >> 1);
      const uint32_t b = above * E + (bl[k] & 0xFFFFu);
      const uint32_t sh = (b & 1) << 4;
      const uint32_t old = atomicAdd(&cnt[has ? b >> 1 : (uint32_t)NW + lane], 1u << sh);
      bb[k] = has ? b : 0u;
      idx[k] = (old >> sh) & 0xFFFFu;
    }
    wave_sync();
    {
      // exclusive scan over the 16-bit counters
      const int per = (NW + 63) >> 6;
      const int w0 = min(lane * per, NW), w1 = min(w0 + per, NW);
      uint32_t sum = 0;
      for (int w = w0; w < w1; w++) {
        const uint32_t x = cnt[w];
        sum += (x & 0xFFFFu) + (x >> 16);
      }
      const uint32_t incl = wave_incl_scan(sum, lane);
      uint32_t run = incl - sum;
      for (int w = w0; w < w1; w++) {
        const uint32_t x = cnt[w];
        const uint32_t lo = x & 0xFFFFu;
        cnt[w] = run | ((run + lo) << 16);
        run += lo + (x >> 16);
      }
    }
    wave_sync();
    uint32_t b0[J], b1[J];
#pragma unroll
    for (int k = 0; k < J; k++) {
      b0[k] = start_of(bb[k]);
      b1[k] = start_of(bb[k] + 1);
    }
    for (int ly = lane; ly <= nl; ly += 64) lst[ly] = start_of((uint32_t)ly * E);
    wave_sync();  // the counters are dead from here on
    // bucket entries {key lo, key hi, slot | link << 10, priority}: inside a
    // bucket the link is fixed, so (priority, third word) orders as
    // (priority, slot), and slot order is chunk order (every send of a link
    // enters the same vertex)
#pragma unroll
    for (int k = 0; k < J; k++)
      if (bl[k] != ~0u) {
        const uint32_t pos = b0[k] + idx[k];
        erec[pos] = make_uint4((uint32_t)kk[k], (uint32_t)(kk[k] >> 32),
                               (uint32_t)(lane + 64 * k) | ((bl[k] & 0xFFFFu) << 10), px[k]);
        bnd[pos] = b0[k] | (b1[k] << 16);
      }
    wave_sync();

    // ---- order inside each bucket by (rem, trav, priority, chunk) --------
    // one lane per ordered position, so a pass waits only for the largest
    // bucket among its 64 positions
    const uint32_t total = lst[nl];
    for (uint32_t x = lane; x < total; x += 64) {
      const uint4 rx = erec[x];
      const uint32_t bd = bnd[x];
      const uint32_t bs = bd & 0xFFFFu, be = bd >> 16;
      const uint64_t kx = ((uint64_t)rx.y << 32) | rx.x;
      const uint64_t qx = ((uint64_t)rx.w << 32) | rx.z;
      uint32_t rank = 0, same = 0;
      // four members per step; the array has three spare entries past its
      // end, so the loads need no clamping (entries past the bucket never count)
      for (uint32_t y = bs; y < be; y += 4) {
        uint4 m[4];
#pragma unroll
        for (int t = 0; t < 4; t++) m[t] = erec[y + t];
#pragma unroll
        for (int t = 0; t < 4; t++) {
          const uint64_t ky = ((uint64_t)m[t].y << 32) | m[t].x;
          const uint64_t qy = ((uint64_t)m[t].w << 32) | m[t].z;
          const uint32_t before = (uint32_t)((y + t < be) & ((ky < kx) | ((ky == kx) & (qy < qx))));
          rank += before;
          // an earlier send of the bucket with the same remaining length
          // (the order puts equal remaining lengths next to each other)
          if (kContig) same |= before & (uint32_t)(m[t].y == rx.y);
        }
      }
      const uint32_t sl = rx.z & 0x3FFu, l = rx.z >> 10;
      const uint32_t c = div_v(sl, a.vmagic);
      // Allgather: the send that brings the chunk to the link's source;
      // ReduceScatter: the send out of the link's destination, which waits
      // for this one
      const uint32_t u = kRS ? s_dst[l] : s_src[l];
      const uint32_t pred = (u == s_own[c]) ? kNoPred : c * V + u;
      const uint32_t q = bs + rank;
      ord2[q] = sl | (pred << 16);
      info2[q] = l | (rank << 16) | (same << 31);  // rank < 2^15: at most 1024 sends
    }
    wave_sync();

    // ---- least schedule, layer by layer ----------------------------------
    if (kRS) {  // ready times are raised by the sends that feed each send
      for (int j = lane; j < CV; j += 64) fin[j] = 0;
      wave_sync();
    }
    uint32_t mk = 0;
    for (int ly = 0; ly < nl; ly++) {
      const uint32_t qs = lst[ly], qe = lst[ly + 1];
      if (kContig) {
        // ready times of the layer's sends, for the walkers below (parent
        // sends lie in layers above)
        for (uint32_t q = qs + lane; q < qe; q += 64) {
          if (kRS) {
            rq[q] = fin[ord2[q] & 0xFFFFu];
          } else {
            const uint32_t pj = ord2[q] >> 16;
            rq[q] = (pj == kNoPred) ? 0u : fin[pj];
          }
        }
        wave_sync();
      }
      // Every send's ready time is known (its parent send lies in a layer
      // above), so the k-th send of a link run with cost c and busy time F
      // finishes at (k+1)c + max(F, max_{j<=k}(r_j - j c)). The layer's runs
      // lie in ascending link order, so one plain prefix max over
      // link << 33 | (r_j - j c + 2^32) gives every position the max over the
      // earlier sends of its own run (DPP scan, 64 positions a step). Runs
      // on links that carry contiguous transfers are walked instead.
      uint64_t carry = 0;
      for (uint32_t base = qs; base < qe; base += 64) {
        const uint32_t q = base + lane;
        const bool ok = q < qe;
        const uint32_t qq = ok ? q : qs;
        const uint32_t e = ord2[qq], inf = info2[qq];
        const uint32_t l = inf & 0xFFFFu, k = (inf >> 16) & 0x7FFFu;
        uint32_t r;
        if (kRS) {
          r = fin[e & 0xFFFFu];
        } else {
          const uint32_t pj = e >> 16;
          r = fin[pj == kNoPred ? 0u : pj];
          if (pj == kNoPred) r = 0;
        }
        const uint32_t cl = s_cost[l], F = lfree[l];
        const uint32_t kn = (q + 1 < qe) ? ((info2[q + 1] >> 16) & 0x7FFFu) : 0u;
        const uint64_t comp =
            ok ? (((uint64_t)l << 33) | ((uint64_t)r + (1ull << 32) - (uint64_t)k * cl)) : 0ull;
        const uint64_t incl = max(wave_scan_max64(comp), carry);
        carry = readlane64(incl, 63);
        const int64_t best =
            max((int64_t)F, (int64_t)(incl & ((1ull << 33) - 1)) - (int64_t)(1ull << 32));
        const uint32_t f = (uint32_t)((int64_t)(k + 1) * cl + best);
        const bool merge = kContig && s_merge[l];
        if (ok && !merge) {
          finish(e, f);
          mk = max(mk, f);
          if (kn == 0) lfree[l] = f;  // the run's last send
        }
        if (ok && merge && k == 0) {
          // contiguous transfers: the run's first lane walks the run; a send
          // joins the open transfer when its remaining length equals the
          // previous send's and its chunk was ready when the transfer
          // started
          const uint32_t al = a.lalpha[l];
          const uint64_t bsz = a.lbs[l];
          uint32_t Fw = F, gs = 0, gm = 0, g0 = q;
          bool done = false;
          // the run's entries are read four at a time (clamped to the layer)
          for (uint32_t j0 = q; !done; j0 += 4) {
            uint32_t inf4[4], r4[4];
#pragma unroll
            for (int u = 0; u < 4; u++) {
              const uint32_t jj = min(j0 + u, qe - 1);
              inf4[u] = info2[jj];
              r4[u] = rq[jj];
            }
#pragma unroll
            for (int u = 0; u < 4; u++) {
              if (done) break;
              const uint32_t j = j0 + u;
              const bool end = j >= qe || (j > q && ((inf4[u] >> 16) & 0x7FFFu) == 0);
              const bool join = !end && gm > 0 && (inf4[u] >> 31) && r4[u] <= gs;
              if (gm > 0 && !join) {  // close the open transfer
                const uint32_t fw = gs + al + (uint32_t)((bsz * gm + 999) / 1000);
                for (uint32_t t = g0; t < g0 + gm; t++) finish(ord2[t], fw);
                Fw = fw;
                mk = max(mk, fw);
              }
              if (end) {
                done = true;
              } else if (join) {
                gm++;
              } else {
                gs = max(Fw, r4[u]);
                gm = 1;
                g0 = j;
              }
            }
          }
          lfree[l] = Fw;
        }
      }
      wave_sync();
    }

    // ---- postcondition and makespan ---------------------------------------
    const bool all_ok = __ballot(bad) == 0;
    const bool failed = __ballot(clamped || fault) != 0;
    mk = wave_max(mk);
    if (lane == 0) {
      if (a.accumulate) {  // second phase of an Allreduce
        const uint32_t m0 = a.makespan[i];
        a.makespan[i] = (failed || m0 == 0xFFFFFFFFu) ? 0xFFFFFFFFu : m0 + mk;
        a.valid[i] = (uint8_t)(a.valid[i] && all_ok && !failed);
      } else {
        a.makespan[i] = failed ? 0xFFFFFFFFu : mk;
        a.valid[i] = (uint8_t)(all_ok && !failed);
      }
    }
    wave_sync();
  }
}

constexpr int kGreedyLinkSlots = 4;  // links per lane: at most 256 links

// The time-aware greedy of App. B.2 over per-link lists of pending sends,
// simulated exactly in windows: W = the earliest start any ready send can
// take; a send whose chunk has not arrived can only become ready at least
// c_min (the smallest link cost) after W, so on every link the best ready
// send by (start, Step-2 key, priority, slot) with start < W + c_min is the
// greedy's next send there, and all of them are committed at once. One
// lane holds up to four links; a committed send is swapped to the end of
// its link's pending part. Records: {key lo, key hi (~rem << 32 | trav),
// priority, slot | other slot << 16}, the other slot being the send the
// chunk arrives by (its finish is the ready time; kNoPred: ready at 0) or,
// for ReduceScatter, the send that carries the partial on (ready once every
// input is scheduled). gfin[slot] must be kNotYet for every pending send.
// On return every link's list holds its sends in the reverse of the order
// they were served in. Both record-based greedy kernels use this one loop.
//
// The best send of a link is kept as three packed words compared
// lexicographically, (start, key hi), (key lo, priority), (slot, list
// index), and replaced as a whole, so the list index always belongs to the
// send that won; the commit checks the slot at that index and reports a
// fault if it ever differs. The scan of one link and the commit of its
// winner are plain functions of one lane's data (greedy_window.h), which a
// host build also runs.

template <bool kRS>
__device__ __forceinline__ void greedy_windows(int E, int lane, int nslots, uint32_t cmin,
                                            const uint32_t *s_cost, uint4 *grec,
                                            const uint32_t *gofs, uint32_t *gfin,
                                            uint32_t *grdy, uint32_t *gpend, uint32_t &mk,
                                            bool &fault) {
  GreedyLink lk[kGreedyLinkSlots];
#pragma unroll
  for (int t = 0; t < kGreedyLinkSlots; t++) {
    const int l = lane + 64 * t;
    lk[t].free = 0;
    lk[t].base = l < E ? gofs[l] : 0;
    lk[t].len = l < E ? gofs[l + 1] - gofs[l] : 0;
  }
  for (int round = 0;; round++) {
    GreedyBest best[kGreedyLinkSlots];
    uint32_t wmin = kGreedyNone;
#pragma unroll
    for (int t = 0; t < kGreedyLinkSlots; t++) {
      best[t] = greedy_scan_link<kRS>(lk[t], RecArray<uint4>{grec}, gfin);
      wmin = min(wmin, greedy_start(best[t]));
    }
    wmin = ~wave_reduce_max(~wmin);
    if (wmin == kGreedyNone) break;  // nothing left to schedule
    if (round > nslots) {  // unreachable: every window commits a send
      fault = true;
      break;
    }
    const uint64_t wend = (uint64_t)wmin + cmin;
    wave_sync();
#pragma unroll
    for (int t = 0; t < kGreedyLinkSlots; t++) {
      const int l = lane + 64 * t;
      if (greedy_start(best[t]) != kGreedyNone && (uint64_t)greedy_start(best[t]) < wend)
        fault |= greedy_commit<kRS, LdsAtomics>(lk[t], best[t], s_cost[l], RecArray<uint4>{grec},
                                                gfin, grdy, gpend,
                                                mk);
    }
    wave_sync();
  }
}

// Reverse path order (App. B.2): after the greedy has served the mirrored
// schedule, every link's list holds its sends in the reverse of the mirrored
// service order, which is the real order. The real times then follow the
// App. B.3 rule along those orders: in steps, every link serves the send at
// the front of its list if it is ready (kPush: every send into the source
// is scheduled, the ReduceScatter form; else the send that brings the chunk
// has finished). The orders are acyclic with the chunk dependencies, so
// every step serves a send until all are through.
template <bool kPush>
__device__ __forceinline__ void greedy_real_times(int E, int lane, int nslots,
                                                  const uint32_t *s_cost, const uint4 *grec,
                                                  const uint32_t *gofs, uint32_t *gfin,
                                                  uint32_t *grdy, uint32_t *gpend, uint32_t &mk,
                                                  bool &fault) {
  uint32_t p[kGreedyLinkSlots], e[kGreedyLinkSlots], fr[kGreedyLinkSlots], c[kGreedyLinkSlots];
  uint4 rc[kGreedyLinkSlots];  // the record at the front of each list
#pragma unroll
  for (int t = 0; t < kGreedyLinkSlots; t++) {
    const int l = lane + 64 * t;
    p[t] = l < E ? gofs[l] : 0;
    e[t] = l < E ? gofs[l + 1] : 0;
    c[t] = l < E ? s_cost[l] : 0;
    fr[t] = 0;
    rc[t] = p[t] < e[t] ? grec[p[t]] : make_uint4(0, 0, 0, 0);
  }
  for (int step = 0;; step++) {
    bool pending = false;
#pragma unroll
    for (int t = 0; t < kGreedyLinkSlots; t++) {
      if (p[t] >= e[t]) continue;
      const uint32_t x = rc[t].w & 0xFFFFu, o = rc[t].w >> 16;
      bool ready = true;
      uint32_t r = 0;
      if (kPush) {
        ready = lds_get(&gpend[x]) == 0;
        r = lds_get(&grdy[x]);
      } else if (o != kNoPred) {
        r = lds_get(&gfin[o]);
        ready = r != kNotYet;
      }
      if (ready) {
        const uint32_t f = max(r, fr[t]) + c[t];
        gfin[x] = f;
        fr[t] = f;
        mk = max(mk, f);
        if (kPush && o != kNoPred) {
          atomicMax(&grdy[o], f);
          atomicSub(&gpend[o], 1u);
        }
        if (++p[t] < e[t]) rc[t] = grec[p[t]];
      }
      pending |= p[t] < e[t];
    }
    if (__ballot(pending) == 0) break;
    if (step > nslots) {  // unreachable: the orders come from a schedule
      fault = true;
      break;
    }
    wave_sync();
  }
}

__global__ __launch_bounds__(kTreeMaxThreads) void path_greedy_kernel(PathGreedyArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int C = a.C, P = a.P, E = a.E, H = a.H;
  uint32_t *s_cost = (uint32_t *)lds;
  for (int j = threadIdx.x; j < E; j += blockDim.x) s_cost[j] = a.cost[j];
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  unsigned char *wl = lds + a.o_wave + wave * a.wave_bytes;
  uint32_t *gfin = (uint32_t *)(wl + a.w_gfin);
  uint32_t *gofs = (uint32_t *)(wl + a.w_gofs);  // [E + 1]
  uint32_t *gcur = (uint32_t *)(wl + a.w_gcur);  // [E]
  uint4 *grec = (uint4 *)(wl + a.w_grec);
  const int64_t stride = (int64_t)gridDim.x * a.waves_per_block;
  for (int64_t i = (int64_t)blockIdx.x * a.waves_per_block + wave; i < a.n; i += stride) {
    const uint8_t *rt = a.routes + (size_t)i * a.route_stride;
    const uint32_t *gpr = a.prio + (size_t)i * a.prio_stride;
    for (int l = lane; l <= E; l += 64) gofs[l] = 0;
    for (int sl = lane; sl < a.nslots; sl += 64) gfin[sl] = kNotYet;
    wave_sync();
    // the chosen path of chunk c: global option index, or -1 (no send)
    bool bad = false;
    auto path_of = [&](int c) -> int64_t {
      const uint32_t sd = (uint32_t)c / (uint32_t)a.cpr;
      const uint32_t s = sd / P, d = sd - s * P;
      if (s == d) return -1;
      const uint32_t k = rt[c];
      if (k >= a.npaths[sd]) {
        bad = true;  // the pair is left unrouted
        return -1;
      }
      return (int64_t)a.pair_base[sd] + k;
    };
    for (int c = lane; c < C; c += 64) {
      const int64_t q = path_of(c);
      if (q < 0) continue;
      for (uint32_t j = a.path_off[q]; j < a.path_off[q + 1]; j++)
        atomicAdd(&gofs[a.path_links[j] + 1], 1u);
    }
    wave_sync();
    {
      // exclusive scan of the per-link counts (gofs[0] = 0)
      const int n1 = E + 1;
      const int per = (n1 + 63) >> 6;
      const int b0 = min(lane * per, n1), b1 = min(b0 + per, n1);
      uint32_t sum = 0;
      for (int w = b0; w < b1; w++) sum += gofs[w];
      const uint32_t incl = wave_incl_scan(sum, lane);
      uint32_t run = incl - sum;
      for (int w = b0; w < b1; w++) {
        run += gofs[w];
        gofs[w] = run;
      }
    }
    wave_sync();
    for (int l = lane; l < E; l += 64) gcur[l] = gofs[l];
    wave_sync();
    for (int c = lane; c < C; c += 64) {
      const int64_t q = path_of(c);
      if (q < 0) continue;
      const uint32_t j0 = a.path_off[q], j1 = a.path_off[q + 1];
      uint32_t total = 0;
      for (uint32_t j = j0; j < j1; j++) total += s_cost[a.path_links[j]];
      uint32_t trav = 0;
      for (uint32_t j = j0; j < j1; j++) {
        const uint32_t l = a.path_links[j], h = j - j0;
        const uint32_t rem = total - trav;  // remaining path, this hop included
        const uint32_t sl = (uint32_t)c * H + h;
        const uint32_t cl = s_cost[l];
        const uint32_t pos = atomicAdd(&gcur[l], 1u);
        if (a.mirror) {  // waits for the next hop; lengths from the path's end
          const uint32_t other = (j + 1 < j1) ? sl + 1 : kNoPred;
          grec[pos] = make_uint4(rem - cl, ~(trav + cl), gpr[sl], sl | (other << 16));
        } else {
          const uint32_t other = h ? sl - 1 : kNoPred;  // the hop the chunk arrives by
          grec[pos] = make_uint4(trav, ~rem, gpr[sl], sl | (other << 16));
        }
        trav += cl;
      }
    }
    wave_sync();
    uint32_t mk = 0;
    bool fault = false;
    greedy_windows<false>(E, lane, a.nslots, a.cmin, s_cost, grec, gofs, gfin, nullptr, nullptr,
                          mk, fault);
    if (a.mirror && !__ballot(fault)) {
      // the real schedule: links advance through the lists in rounds, a hop
      // ready when the hop before it (slot - 1) has ended
      mk = 0;
      wave_sync();
      for (int sl = lane; sl < a.nslots; sl += 64) gfin[sl] = kNotYet;
      uint32_t lh[kGreedyLinkSlots], lf[kGreedyLinkSlots];
#pragma unroll
      for (int t = 0; t < kGreedyLinkSlots; t++) {
        const int l = lane + 64 * t;
        lh[t] = l < E ? gofs[l] : 0u;
        lf[t] = 0;
      }
      wave_sync();
      for (int round = 0;; round++) {
        bool pending = false;
#pragma unroll
        for (int t = 0; t < kGreedyLinkSlots; t++) {
          const int l = lane + 64 * t;
          if (l >= E) continue;
          const uint32_t e = gofs[l + 1], cl = s_cost[l];
          while (lh[t] < e) {
            const uint32_t x = grec[lh[t]].w & 0xFFFFu;
            const uint32_t r = (x % (uint32_t)H) ? lds_get(&gfin[x - 1]) : 0u;
            if (r == kNotYet) break;
            lf[t] = max(r, lf[t]) + cl;
            lds_put(&gfin[x], lf[t]);
            mk = max(mk, lf[t]);
            lh[t]++;
          }
          pending |= lh[t] < e;
        }
        if (__ballot(pending) == 0) break;
        if (round > a.nslots) {  // unreachable: the orders come from a schedule
          fault = true;
          break;
        }
      }
    }
    const bool all_ok = __ballot(bad) == 0;
    const bool failed = __ballot(fault) != 0;
    mk = wave_max(mk);
    if (lane == 0) {
      a.makespan[i] = failed ? 0xFFFFFFFFu : mk;
      a.valid[i] = (uint8_t)(all_ok && !failed);
    }
    wave_sync();
  }
}

// Time-aware greedy orders (App. B.2), multicast trees. After the trees and
// Step-2 keys (as in the layered kernel), the greedy is simulated exactly in
// windows: the earliest start W any ready send can take bounds every other
// start, and a send whose chunk is not yet ready can only become ready at
// least one link cost (c_min) after W, so on every link the best ready send
// by (start, Step-2 key) with start < W + c_min is the greedy's next send
// there and all of them can be committed at once. One lane holds up to four
// links and scans each link's pending sends; committed sends are removed by
// swapping in the link's last pending send. In reverse path order
// (a.greedy == 2) the greedy serves the mirrored schedule (lengths measured
// from the other end, every chunk dependency reversed: the Allgather waits
// for the sends out of the destination, the ReduceScatter for the send that
// carries the partial on), and the real times come from the orders it
// leaves (greedy_real_times).
template <int J, int PW, bool kRS>
__global__ __launch_bounds__(kTreeMaxThreads) void tree_greedy_kernel(TreeArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int C = a.C, V = a.V, E = a.E;
  const int CV = C * V;

  uint32_t *s_cost = (uint32_t *)(lds + a.o_cost);
  uint8_t *s_src = lds + a.o_src;
  uint8_t *s_own = lds + a.o_own;
  uint64_t *s_post = (uint64_t *)(lds + a.o_post);
  uint4 *s_rec = (uint4 *)(lds + a.o_rec4);
  uint32_t *s_opt = (uint32_t *)(lds + a.o_opt);
  uint16_t *s_rev = (uint16_t *)(lds + a.o_rev);
  uint8_t *s_dst = lds + a.o_ldst;
  for (int j = threadIdx.x; j < E; j += blockDim.x) {
    s_cost[j] = a.cost[j];
    s_src[j] = (uint8_t)a.lsrc[j];
    if (kRS) {
      s_rev[j] = a.lrev[j];
      s_dst[j] = (uint8_t)a.ldst[j];
    }
  }
  for (int r = threadIdx.x; r < 16 * PW * PW * a.K; r += blockDim.x) s_rec[r] = a.rec4[r];
  for (int j = threadIdx.x; j < 4 * PW * V * PW; j += blockDim.x)
    s_opt[j] = ((const uint32_t *)a.topt)[j];
  for (int j = threadIdx.x; j < C; j += blockDim.x) {
    s_own[j] = a.owner8[j];
    s_post[j] = a.post_mask[j];
  }
  __syncthreads();

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  unsigned char *wl = lds + a.o_wave + wave * a.wave_bytes;
  uint32_t *rt32 = (uint32_t *)(wl + a.w_rt);
  uint32_t *dist = (uint32_t *)(wl + a.w_dist);
  uint16_t *anc = (uint16_t *)(wl + a.w_anc);
  uint32_t *gfin = (uint32_t *)(wl + a.w_gfin);  // per slot: finish, kNotYet before
  uint32_t *grdy = (uint32_t *)(wl + a.w_grdy);  // ReduceScatter: ready so far
  uint32_t *gpend = (uint32_t *)(wl + a.w_gpend);  // ReduceScatter: unscheduled inputs
  // pending sends grouped by link, one 16-byte record each: {key lo, key hi
  // (~rem << 32 | trav), priority, slot | other slot << 16} where the other
  // slot is the send that brings the chunk (Allgather) or carries the partial
  // on (ReduceScatter)
  uint4 *grec = (uint4 *)(wl + a.w_glist);
  uint32_t *gofs = (uint32_t *)(wl + a.w_gofs);  // [E + 1] first list entry per link

  const int64_t stride = (int64_t)gridDim.x * a.waves_per_block;
  const int64_t first = (int64_t)blockIdx.x * a.waves_per_block + wave;
  const int nrw = a.route_stride >> 2;
  uint32_t pf_r[kPfRoute], pf_p[J];
  auto prefetch = [&](int64_t i) {
    if (i >= a.n) return;
    const uint32_t *g32 = (const uint32_t *)(a.routes + (size_t)i * a.route_stride);
    const uint32_t *gpr = a.prio + (size_t)i * a.prio_stride;
#pragma unroll
    for (int k = 0; k < kPfRoute; k++) {
      const int j = lane + 64 * k;
      if (j < nrw) pf_r[k] = __builtin_nontemporal_load(g32 + j);
    }
#pragma unroll
    for (int k = 0; k < J; k++) {
      const int j = lane + 64 * k;
      if (j < CV) pf_p[k] = __builtin_nontemporal_load(gpr + j);
    }
  };
  prefetch(first);
  for (int64_t i = first; i < a.n; i += stride) {
#pragma unroll
    for (int k = 0; k < kPfRoute; k++) {
      const int j = lane + 64 * k;
      if (j < nrw) rt32[j] = one_hot_word<PW>(pf_r[k], j, s_post);
    }
    uint32_t px[J];
#pragma unroll
    for (int k = 0; k < J; k++) px[k] = pf_p[k];
    prefetch(i + stride);
    for (int l = lane; l <= E; l += 64) gofs[l] = 0;
    wave_sync();

    uint32_t pe[J], ps[J], dv[J];
    bool bad = false, fault = false;
    slot_trees<J, PW, kRS>(a, TreeLds{s_cost, s_own, s_post, s_rec, s_opt, s_rev, rt32, dist, anc},
                           lane, pe, ps, dv, bad, fault);

    // ---- per-slot send records; sends counted per link ------------------
    const bool mirror = a.greedy == 2;
    uint32_t lk[J], idx[J];
    uint64_t kk[J];
#pragma unroll
    for (int j = 0; j < J; j++) {
      const uint32_t sl = lane + 64 * j;
      lk[j] = ~0u;
      kk[j] = 0;
      idx[j] = 0;
      if (sl < (uint32_t)CV) {
        gfin[sl] = kNotYet;
        if (kRS || mirror) {
          grdy[sl] = 0;
          gpend[sl] = 0;
        }
      }
      if (pe[j] != ~0u) {
        const uint32_t l0 = pe[j] & 0xFFFFu;
        const uint32_t l = kRS ? s_rev[l0] : l0;
        uint32_t trav = kRS ? lds_get(&dist[sl]) : dv[j] - s_cost[l];
        uint32_t rem = kRS ? dv[j] : lds_get(&dist[sl]) - trav;
        if (mirror) {  // remaining' = travelled + own cost, travelled' = remaining - own cost
          const uint32_t c = s_cost[l], r2 = trav + c;
          trav = rem - c;
          rem = r2;
        }
        lk[j] = l;
        kk[j] = ((uint64_t)(~rem) << 32) | trav;
        idx[j] = atomicAdd(&gofs[l + 1], 1u);
      }
    }
    wave_sync();
    // inputs per send for the push form (the ReduceScatter's schedule, and
    // the mirrored greedy of an Allgather)
    if (kRS || mirror) {
#pragma unroll
      for (int j = 0; j < J; j++)
        if (pe[j] != ~0u && ps[j] != kNoPred) atomicAdd(&gpend[ps[j]], 1u);
    }
    if (kRS != mirror) {
      // push form: a send without inputs is ready at 0
      wave_sync();
#pragma unroll
      for (int j = 0; j < J; j++) {
        const uint32_t sl = lane + 64 * j;
        if (pe[j] != ~0u && gpend[sl] == 0) gfin[sl] = 0;
      }
    }
    {
      // exclusive scan of the per-link counts (gofs[0] = 0)
      const int n1 = E + 1;
      const int per = (n1 + 63) >> 6;
      const int b0 = min(lane * per, n1), b1 = min(b0 + per, n1);
      uint32_t sum = 0;
      for (int w = b0; w < b1; w++) sum += gofs[w];
      const uint32_t incl = wave_incl_scan(sum, lane);
      uint32_t run = incl - sum;
      for (int w = b0; w < b1; w++) {
        run += gofs[w];
        gofs[w] = run;
      }
    }
    wave_sync();
#pragma unroll
    for (int j = 0; j < J; j++)
      if (lk[j] != ~0u)
        grec[gofs[lk[j]] + idx[j]] = make_uint4((uint32_t)kk[j], (uint32_t)(kk[j] >> 32), px[j],
                                                (lane + 64 * j) | (ps[j] << 16));
    wave_sync();

    // ---- the greedy, window by window ------------------------------------
    uint32_t mk = 0;
    if (kRS == mirror) {
      greedy_windows<false>(E, lane, CV, a.cmin, s_cost, grec, gofs, gfin, grdy, gpend, mk, fault);
    } else {
      greedy_windows<true>(E, lane, CV, a.cmin, s_cost, grec, gofs, gfin, grdy, gpend, mk, fault);
    }
    if (mirror && !fault) {
      // the real schedule along the orders the mirrored greedy left
      wave_sync();
#pragma unroll
      for (int j = 0; j < J; j++) {
        const uint32_t sl = lane + 64 * j;
        if (sl < (uint32_t)CV) gfin[sl] = kNotYet;
      }
      wave_sync();
      mk = 0;
      greedy_real_times<kRS>(E, lane, CV, s_cost, grec, gofs, gfin, grdy, gpend, mk, fault);
    }

    const bool all_ok = __ballot(bad) == 0;
    const bool failed = __ballot(fault) != 0;
    mk = wave_max(mk);
    if (lane == 0) {
      if (a.accumulate) {  // second phase of an Allreduce
        const uint32_t m0 = a.makespan[i];
        a.makespan[i] = (failed || m0 == 0xFFFFFFFFu) ? 0xFFFFFFFFu : m0 + mk;
        a.valid[i] = (uint8_t)(a.valid[i] && all_ok && !failed);
      } else {
        a.makespan[i] = failed ? 0xFFFFFFFFu : mk;
        a.valid[i] = (uint8_t)(all_ok && !failed);
      }
    }
    wave_sync();
  }
}

int32_t align16(int32_t x) { return (x + 15) & ~15; }

}  // namespace

int32_t tree_layout(const taccl_plan &p, TreeArgs &a) {
  const int32_t C = p.coll.C, V = p.topo.V, E = p.topo.E, P = p.topo.P;
  const int32_t CV = C * V;
  const int32_t K = std::max(p.max_paths, 1), H = std::max(p.H, 1);
  int32_t off = 0;
  auto take = [&](int32_t bytes) {
    int32_t o = off;
    off = align16(off + bytes);
    return o;
  };
  // shared tables
  a.rec_len = P * P * K * H;
  a.rec_in_lds = 4 * a.rec_len <= kTreeRecLdsMax;
  a.o_cost = take(4 * E);
  a.o_src = take(E);
  a.o_own = take(C);
  a.o_post = take(8 * C);
  a.o_rec = take(a.rec_in_lds ? 4 * a.rec_len : 0);
  a.o_wave = off;
  // one wavefront's state
  a.mask_words = (C + 31) / 32;
  int32_t w = 0;
  auto wtake = [&](int32_t bytes) {
    int32_t o = w;
    w = align16(w + bytes);
    return o;
  };
  a.w_rt = wtake(p.route_stride);
  a.w_key = wtake(8 * CV);
  a.w_prio = wtake(4 * CV);
  a.w_chain = wtake(4 * CV);
  a.w_par = wtake(2 * CV);
  a.w_mask = wtake(4 * E * a.mask_words);
  a.w_base = wtake(4 * (E + 1));
  a.w_head = wtake(4 * E);
  a.w_free = wtake(4 * E);
  a.wave_bytes = w;
  a.K = K;
  a.H = H;
  a.vmagic = (uint32_t)((1ull << 32) / (uint64_t)V + 1);
  return a.o_wave + a.wave_bytes;  // bytes for a one-wave block
}

int32_t tree_any_layout(const taccl_plan &p, TreeArgs &a) {
  if (tree_layout(p, a) <= 0) return 0;
  const int32_t CV = p.coll.C * p.topo.V, E = p.topo.E;
  int32_t w = a.wave_bytes;
  auto wtake = [&](int32_t bytes) {
    int32_t o = w;
    w = align16(w + bytes);
    return o;
  };
  a.w_gfin = wtake(4 * CV);
  a.w_grdy = wtake(4 * CV);
  a.w_gpend = wtake(4 * CV);
  a.w_gst = wtake(16 * E);
  a.wave_bytes = w;
  uint32_t cmin = ~0u;  // the greedy's window (plans have no zero-cost link)
  for (uint32_t c : p.cost) cmin = std::min(cmin, c);
  a.cmin = cmin;
  return a.o_wave + a.wave_bytes;
}

int32_t tree_block_bytes(const TreeArgs &a, int waves) { return a.o_wave + waves * a.wave_bytes; }

template <bool kAny>
static void launch_tree_v(const TreeArgs &a, int grid, hipStream_t stream) {
  const bool pf = a.routes_word_aligned && a.route_stride <= 4 * 64 * kPfRoute &&
                  a.C * a.V <= 64 * kPfPrio;
  const dim3 g(grid), b(64 * a.waves_per_block);
  const int bytes = tree_block_bytes(a, a.waves_per_block);
  if (a.rec_in_lds && pf)
    hipLaunchKernelGGL((tree_eval_kernel<true, true, kAny>), g, b, bytes, stream, a);
  else if (a.rec_in_lds)
    hipLaunchKernelGGL((tree_eval_kernel<true, false, kAny>), g, b, bytes, stream, a);
  else if (pf)
    hipLaunchKernelGGL((tree_eval_kernel<false, true, kAny>), g, b, bytes, stream, a);
  else
    hipLaunchKernelGGL((tree_eval_kernel<false, false, kAny>), g, b, bytes, stream, a);
}

hipError_t launch_tree(const TreeArgs &a, int grid, hipStream_t stream) {
  if (a.any)
    launch_tree_v<true>(a, grid, stream);
  else
    launch_tree_v<false>(a, grid, stream);
  return hipGetLastError();
}

// ancestor doubling: 2^rounds >= V covers the deepest tree (V - 1 links)
static void set_pj(TreeArgs &a, int32_t V, int32_t CV) {
  int r = 0;
  while ((1 << r) < V) r++;
  a.pj_rounds = std::max(r, 1);
  a.anc_stride = align16(2 * CV) / 2;
}

int32_t tree_layers_layout(const taccl_plan &p, TreeArgs &a) {
  if (tree_layout(p, a) <= 0) return 0;
  const int32_t C = p.coll.C, V = p.topo.V, E = p.topo.E, P = p.topo.P;
  const int32_t CV = C * V;
  const int32_t K = std::max(p.max_paths, 1), H = std::max(p.H, 1);
  const int32_t pw = P / 4;  // route words per chunk: 1, 2, 3, 4, 6 or 8
  if (p.topt.empty() || K > 8 || H > 4 || P % 4 ||
      (pw != 1 && pw != 2 && pw != 3 && pw != 4 && pw != 6 && pw != 8) ||
      V > 64 || E < 1 ||
      CV > 64 * kLayerMaxSlotsPerLane || p.route_stride > 4 * 64 * kPfRoute || E > (1 << 22))
    return 0;
  uint64_t cmin = ~0ull, cmax = 0;
  for (uint32_t c : p.cost) {
    cmin = std::min<uint64_t>(cmin, c);
    cmax = std::max<uint64_t>(cmax, c);
  }
  if (cmin == 0) return 0;  // layers need every link cost to be positive
  // rem is at most the cost of a tree path: V - 1 links
  const uint64_t max_rem = (uint64_t)(V - 1) * cmax;
  if (max_rem >= (1ull << 32)) return 0;
  a.lmagic = ((1ull << 32) + cmin - 1) / cmin;  // ceil(2^32 / c_min) <= 2^32
  const uint64_t nl = ((max_rem * a.lmagic) >> 32) + 1;
  if (nl > 64) return 0;
  a.nl_max = (int32_t)nl;
  if (p.tree_rec4.empty()) return 0;
  // shared tables: 16-byte route records and the option bytes, in place of
  // the fixed-stride records
  int32_t off = a.o_rec;
  a.o_rec4 = off;
  off = align16(off + 16 * P * P * K);
  a.o_opt = off;
  off = align16(off + P * V * P);
  a.o_merge = off;
  off = align16(off + E);
  a.o_rev = off;
  off = align16(off + 2 * E);
  a.o_ldst = off;
  off = align16(off + E);
  a.o_wave = off;
  const int32_t S = std::max<int64_t>(std::min<int64_t>(p.max_sends, CV), 1);
  // region X: route words and distances, then bucket entries, then finish
  // and ready times
  set_pj(a, V, CV);
  const int32_t x_tree =
      align16(p.route_stride) + align16(4 * CV) + a.pj_rounds * align16(2 * CV);
  a.w_dist = align16(p.route_stride);
  a.w_anc = a.w_dist + align16(4 * CV);
  a.w_erec = 0;
  a.w_fin = 0;
  a.w_rq = align16(4 * CV);
  const int32_t x = std::max({x_tree, align16(16 * (S + 3)), a.w_rq + align16(4 * S)});
  // region Y: bucket counters, then the ordered sends and bucket bounds
  a.w_cnt = x;
  a.w_ord2 = x;
  a.w_info2 = x + align16(4 * S);
  a.w_bnd = x + 2 * align16(4 * S);
  // counters: u16 pairs for nl_max * E + 1 bucket starts, then one dummy
  // word per lane (slots without a send count there)
  int32_t w = x + std::max(align16(4 * (int32_t)((nl * E + 2) / 2 + 64)), 3 * align16(4 * S));
  a.w_free = w;
  w = align16(w + 4 * E);
  a.w_lmask = w;
  w = align16(w + 8);
  a.w_lst = w;
  w = align16(w + 4 * 65);
  a.wave_bytes = w;
  return a.o_wave + a.wave_bytes;
}

template <int J, bool kC, bool kR>
static const void *layers_fn_j(int pw) {
  switch (pw) {
    case 1: return (const void *)tree_layers_kernel<J, 1, kC, kR>;
    case 2: return (const void *)tree_layers_kernel<J, 2, kC, kR>;
    case 3: return (const void *)tree_layers_kernel<J, 3, kC, kR>;
    case 4: return (const void *)tree_layers_kernel<J, 4, kC, kR>;
    case 6: return (const void *)tree_layers_kernel<J, 6, kC, kR>;
    default: return (const void *)tree_layers_kernel<J, 8, kC, kR>;
  }
}

template <bool kC, bool kR>
static const void *layers_fn_c(const TreeArgs &a) {
  const int J = (a.C * a.V + 63) / 64, pw = a.P / 4;
  if (J <= 1) return layers_fn_j<1, kC, kR>(pw);
  if (J <= 2) return layers_fn_j<2, kC, kR>(pw);
  if (J <= 4) return layers_fn_j<4, kC, kR>(pw);
  return layers_fn_j<8, kC, kR>(pw);
}

// a.reduce selects the ReduceScatter variant (trees run backwards)
static const void *layers_fn(const TreeArgs &a) {
  if (a.reduce) return a.contig ? layers_fn_c<true, true>(a) : layers_fn_c<false, true>(a);
  return a.contig ? layers_fn_c<true, false>(a) : layers_fn_c<false, false>(a);
}

int tree_layers_blocks_per_cu(const TreeArgs &a) {
  int nb = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, layers_fn(a), 64 * a.waves_per_block,
                                                   tree_block_bytes(a, a.waves_per_block)) !=
      hipSuccess)
    return 0;
  return nb;
}

hipError_t launch_tree_layers(const TreeArgs &a, int grid, hipStream_t stream) {
  const int pw = a.P / 4;
  if (a.P % 4 || (pw != 1 && pw != 2 && pw != 3 && pw != 4 && pw != 6 && pw != 8)) return hipErrorInvalidValue;
  const dim3 g(grid), b(64 * a.waves_per_block);
  const int bytes = tree_block_bytes(a, a.waves_per_block);
  void *args[] = {(void *)&a};
  return hipLaunchKernel(layers_fn(a), g, b, args, bytes, stream);
}

int32_t tree_greedy_layout(const taccl_plan &p, TreeArgs &a) {
  if (tree_layers_layout(p, a) <= 0) return 0;
  const int32_t C = p.coll.C, V = p.topo.V, E = p.topo.E;
  const int32_t CV = C * V;
  if (E > 64 * kGreedyLinkSlots) return 0;
  uint32_t cmin = ~0u;
  for (uint32_t c : p.cost) cmin = std::min(cmin, c);
  a.cmin = cmin;
  const int32_t S = std::max<int64_t>(std::min<int64_t>(p.max_sends, CV), 1);
  int32_t w = 0;
  auto wtake = [&](int32_t bytes) {
    int32_t o = w;
    w = align16(w + bytes);
    return o;
  };
  // finish times, and for the push form (ReduceScatter, Allreduce, reverse
  // path order) ready times and unscheduled inputs per send; the pull form
  // never touches the latter two
  const bool push = p.coll.kind == TACCL_REDUCESCATTER || p.coll.kind == TACCL_ALLREDUCE ||
                    p.greedy == 2;
  a.w_gfin = wtake(4 * CV);
  a.w_grdy = push ? wtake(4 * CV) : a.w_gfin;
  a.w_gpend = push ? wtake(4 * CV) : a.w_gfin;
  a.w_gofs = wtake(4 * (E + 1));
  // the trees' arrays (one-hot routes, distances, ancestors) die before the
  // pending-send records are written over them
  set_pj(a, V, CV);
  const int32_t u = w;
  a.w_rt = u;
  a.w_dist = u + align16(p.route_stride);
  a.w_anc = a.w_dist + align16(4 * CV);
  a.w_glist = u;
  a.wave_bytes = std::max(a.w_anc + a.pj_rounds * align16(2 * CV), u + align16(16 * S));
  return a.o_wave + a.wave_bytes;
}

template <int J, bool kR>
static const void *greedy_fn_j(int pw) {
  switch (pw) {
    case 1: return (const void *)tree_greedy_kernel<J, 1, kR>;
    case 2: return (const void *)tree_greedy_kernel<J, 2, kR>;
    case 3: return (const void *)tree_greedy_kernel<J, 3, kR>;
    case 4: return (const void *)tree_greedy_kernel<J, 4, kR>;
    case 6: return (const void *)tree_greedy_kernel<J, 6, kR>;
    default: return (const void *)tree_greedy_kernel<J, 8, kR>;
  }
}

template <bool kR>
static const void *greedy_fn_r(const TreeArgs &a) {
  const int J = (a.C * a.V + 63) / 64, pw = a.P / 4;
  if (J <= 1) return greedy_fn_j<1, kR>(pw);
  if (J <= 2) return greedy_fn_j<2, kR>(pw);
  if (J <= 4) return greedy_fn_j<4, kR>(pw);
  return greedy_fn_j<8, kR>(pw);
}

static const void *greedy_fn(const TreeArgs &a) {
  return a.reduce ? greedy_fn_r<true>(a) : greedy_fn_r<false>(a);
}

int32_t path_greedy_layout(const taccl_plan &p, PathGreedyArgs &a) {
  const int32_t C = p.coll.C, E = p.topo.E, H = std::max(p.H, 1);
  if ((int64_t)C * H > 1024 || E > 64 * kGreedyLinkSlots || E < 1) return 0;
  uint32_t cmin = ~0u;
  for (uint32_t c : p.cost) cmin = std::min(cmin, c);
  if (cmin == 0) return 0;
  a.cmin = cmin;
  a.nslots = C * H;
  const int32_t S = (int32_t)std::max<int64_t>(std::min<int64_t>(p.max_sends, (int64_t)C * H), 1);
  a.o_wave = align16(4 * E);
  int32_t w = 0;
  auto wtake = [&](int32_t bytes) {
    int32_t o = w;
    w = align16(w + bytes);
    return o;
  };
  a.w_gfin = wtake(4 * a.nslots);
  a.w_gofs = wtake(4 * (E + 1));
  a.w_gcur = wtake(4 * E);
  a.w_grec = wtake(16 * S);
  a.wave_bytes = w;
  return a.o_wave + a.wave_bytes;
}

int path_greedy_blocks_per_cu(const PathGreedyArgs &a) {
  int nb = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, (const void *)path_greedy_kernel,
                                                   64 * a.waves_per_block,
                                                   a.o_wave + a.waves_per_block * a.wave_bytes) !=
      hipSuccess)
    return 0;
  return nb;
}

hipError_t launch_path_greedy(const PathGreedyArgs &a, int grid, hipStream_t stream) {
  void *args[] = {(void *)&a};
  return hipLaunchKernel((const void *)path_greedy_kernel, dim3(grid), dim3(64 * a.waves_per_block),
                         args, a.o_wave + a.waves_per_block * a.wave_bytes, stream);
}

int tree_greedy_blocks_per_cu(const TreeArgs &a) {
  int nb = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, greedy_fn(a), 64 * a.waves_per_block,
                                                   tree_block_bytes(a, a.waves_per_block)) !=
      hipSuccess)
    return 0;
  return nb;
}

hipError_t launch_tree_greedy(const TreeArgs &a, int grid, hipStream_t stream) {
  const int pw = a.P / 4;
  if (a.P % 4 || (pw != 1 && pw != 2 && pw != 3 && pw != 4 && pw != 6 && pw != 8)) return hipErrorInvalidValue;
  const dim3 g(grid), b(64 * a.waves_per_block);
  void *args[] = {(void *)&a};
  return hipLaunchKernel(greedy_fn(a), g, b, args, tree_block_bytes(a, a.waves_per_block),
                         stream);
}

}  // namespace taccl
