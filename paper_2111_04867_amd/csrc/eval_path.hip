// Alltoall evaluation kernel for gfx950.
//
// One block evaluates one candidate at a time. Sends are the hops of each
// chunk's routed path. The Step-2 order of Sec. 5.1 puts, on every link,
// longer remaining paths first; along a path the remaining cost strictly
// falls, so grouping sends by remaining cost ("levels", descending) gives a
// topological order in which no send depends on another send of its own
// level. Within a level and a link the order is travelled cost ascending
// (plan-time classes), then priority, then chunk. Each level is:
//   - counted and scattered into its (link, travelled) classes with LDS
//     atomics and a block scan;
//   - ordered inside each class by (priority, chunk) via rank counting;
//   - timed link by link: start = max(chunk's arrival, link free), finish =
//     start + cost (App. B.3 without contiguity), carrying each link's busy
//     time into the next level.
// The postcondition holds iff every off-diagonal chunk is routed (a routed
// path always reaches its destination); the makespan is the latest finish.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "kernels.h"
#include "wave.h"

namespace taccl {

namespace {

constexpr uint32_t kNoOption = 0xFFFFFFFFu;  // a chunk without a send

__device__ __forceinline__ uint32_t wave_max(uint32_t v) {
  for (int o = 32; o > 0; o >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, o));
  return v;
}

__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v, int lane) {
  for (int o = 1; o < 64; o <<= 1) {
    uint32_t t = (uint32_t)__shfl_up((int)v, o);
    if (lane >= o) v += t;
  }
  return v;
}

// out[0..n) = exclusive prefix of in[0..n) (in may alias out), out[n] =
// total, cur[0..n) = copy of out. Called by all threads of the block.
__device__ void block_scan(uint32_t *in_out, uint32_t *cur, int n, uint32_t *wsum) {
  const int tid = threadIdx.x, nt = blockDim.x, lane = tid & 63, wave = tid >> 6;
  const int per = (n + nt - 1) / nt;
  const int b = min(tid * per, n), e = min(b + per, n);
  uint32_t sum = 0;
  for (int j = b; j < e; j++) sum += in_out[j];
  const uint32_t incl = wave_incl_scan(sum, lane);
  if (lane == 63) wsum[wave] = incl;
  __syncthreads();
  uint32_t woff = 0;
  for (int w = 0; w < wave; w++) woff += wsum[w];
  uint32_t run = woff + incl - sum;
  for (int j = b; j < e; j++) {
    const uint32_t x = in_out[j];
    in_out[j] = run;
    cur[j] = run;
    run += x;
  }
  if (tid == nt - 1) in_out[n] = run;
  __syncthreads();
}

// LDS reads and writes of values that other threads update in the same
// pass (relaxed workgroup atomics: plain LDS instructions, never cached)
__device__ __forceinline__ uint32_t lds_get(uint32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void lds_put(uint32_t *p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Rank of entry me among the entries [b, e) of its class, four at a time
// (the staging array has three spare entries past its end; entries past the
// class never count).
__device__ __forceinline__ uint32_t rank_in_class(const uint64_t *e64, uint32_t b, uint32_t e,
                                                  uint64_t me) {
  uint32_t rank = 0;
  for (uint32_t y = b; y < e; y += 4) {
    uint64_t m[4];
#pragma unroll
    for (int t = 0; t < 4; t++) m[t] = e64[y + t];
#pragma unroll
    for (int t = 0; t < 4; t++) rank += (uint32_t)((y + t < e) & (m[t] < me));
  }
  return rank;
}

// Switch ports, one level (App. B.3 switch constraints): a switched send
// holds its send port (its class's link, already ordered in `sorted`) and
// its receive port (the downlink), each port serving its sends in Step-2
// order. The level's switched sends are ordered a second time by receive
// port; then every send port walks its run in order, each switched send
// waiting for the send before it on its receive port. Returns the level's
// latest finish (a block-uniform value is not needed: callers max-reduce);
// updates ctime (arrivals) and lfree (port free times). Sets *fault when a
// wavefront stops making progress (impossible: both ports order the same
// key).
__device__ uint32_t ports_level(const PathArgs &a, int L, const uint32_t *gpr, uint32_t *ctime,
                                uint32_t *lfree, const uint32_t *ccnt, const uint16_t *sorted,
                                uint32_t *red, bool *fault) {
  extern __shared__ __align__(16) unsigned char lds[];
  uint32_t *ccnt2 = (uint32_t *)(lds + a.o_ccnt2);
  uint32_t *ccur2 = (uint32_t *)(lds + a.o_ccur2);
  // the send order is sorted, so its class staging serves the receive-port
  // order: priority << 32 | chunk per scattered send, and its class
  uint64_t *e64 = (uint64_t *)(lds + a.o_e64);
  uint16_t *ecls2 = (uint16_t *)(lds + a.o_ecls);
  uint16_t *sorted2 = (uint16_t *)(lds + a.o_sorted2);
  uint32_t *fcur = (uint32_t *)(lds + a.o_fcur);
  uint16_t *pd = (uint16_t *)(lds + a.o_pd);  // send before it on its receive port
  uint16_t *dl = (uint16_t *)(lds + a.o_dl);  // its receive port (downlink)
  const uint32_t *qc = (const uint32_t *)(lds + a.o_qc);
  const int tid = threadIdx.x, nt = blockDim.x;
  const int C = a.C, E = a.E, nlev = a.nlev;
  const uint32_t lo = a.lvl_cls_begin[L], lo2 = a.lvl_cls2_begin[L];
  const int ncl2 = (int)(a.lvl_cls2_begin[L + 1] - lo2);
  for (int j = tid; j <= ncl2; j += nt) ccnt2[j] = 0;
  for (int c = tid; c < C; c += nt) {
    dl[c] = 0xFFFF;
    fcur[c] = 0;
  }
  __syncthreads();
  // the chunk's send at this level: route option q, first hop h
  auto unit = [&](int c, uint32_t &q, int &h) {
    q = qc[c];
    if (q == kNoOption) return false;
    h = a.path_lvl_hop[(size_t)q * nlev + L];
    return h >= 0;
  };
  // receive-port order of the level's switched sends: count, scan, scatter,
  // rank by (priority, chunk) inside each class
  for (int c = tid; c < C; c += nt) {
    uint32_t q;
    int h;
    if (!unit(c, q, h)) continue;
    const uint32_t k2 = a.hop_class2[a.path_off[q] + h];
    if (k2 != 0xFFFF) atomicAdd(&ccnt2[k2 - lo2], 1u);
  }
  __syncthreads();
  block_scan(ccnt2, ccur2, ncl2, red);
  for (int c = tid; c < C; c += nt) {
    uint32_t q;
    int h;
    if (!unit(c, q, h)) continue;
    const uint32_t k2 = a.hop_class2[a.path_off[q] + h];
    if (k2 == 0xFFFF) continue;
    const uint32_t slot = atomicAdd(&ccur2[k2 - lo2], 1u);
    e64[slot] = ((uint64_t)gpr[(size_t)c * a.H + h] << 32) | (uint32_t)c;
    ecls2[slot] = (uint16_t)(k2 - lo2);
  }
  __syncthreads();
  const uint32_t tot2 = ccnt2[ncl2];
  for (uint32_t x = tid; x < tot2; x += nt) {
    const int k = ecls2[x];
    const uint32_t cx = (uint32_t)e64[x] & 0xFFFFu;
    const uint32_t b = ccnt2[k];
    sorted2[b + rank_in_class(e64, b, ccnt2[k + 1], e64[x])] = (uint16_t)cx;
    dl[cx] = a.cls2_link[lo2 + k];
  }
  __syncthreads();
  // the send before each switched send on its receive port: a port's sends
  // are one contiguous run of the receive-port order
  for (uint32_t x = tid; x < tot2; x += nt) {
    const uint32_t c = sorted2[x], prev = x ? (uint32_t)sorted2[x - 1] : 0u;
    pd[c] = (x && dl[prev] == dl[c]) ? (uint16_t)prev : (uint16_t)0xFFFF;
  }
  __syncthreads();
  // The level's schedule as a dataflow: every send port walks its run in
  // the Step-2 order, and a switched send goes once the send before it on
  // its receive port has finished (the first on a receive port takes the
  // port's busy time instead). Both ports order the same key, so these
  // waits follow one order of the level's sends and every send is reached;
  // each finish is written once, from the finishes it depends on, so it is
  // the least schedule. A wavefront whose lanes make no progress for far
  // longer than the level can take reports a fault instead of waiting on.
  constexpr uint32_t kUnsetF = 0xFFFFFFFFu;
  constexpr int kPortSlots = 4;  // send ports per thread: E <= 4 x threads
  const uint32_t tot = ccnt[a.lvl_cls_begin[L + 1] - lo];
  // per send-order position: chunk | the send before it on its receive
  // port << 16, and its ready time without that send (the receive port's
  // busy time folded in for the first send on a port); the send-order and
  // receive-port staging arrays are dead
  uint32_t *wcp = (uint32_t *)e64, *wr0 = wcp + a.max_lvl;
  for (uint32_t x = tid; x < tot; x += nt) {
    const uint32_t c = sorted[x], d = dl[c];
    const uint32_t pj = d != 0xFFFFu ? (uint32_t)pd[c] : 0xFFFFu;
    uint32_t r0 = ctime[c];
    if (d != 0xFFFFu && pj == 0xFFFFu) r0 = max(r0, lfree[d]);
    wcp[x] = c | (pj << 16);
    wr0[x] = r0;
  }
  for (int c = tid; c < C; c += nt) lds_put(&fcur[c], kUnsetF);
  uint32_t p[kPortSlots], e[kPortSlots], F[kPortSlots], cl[kPortSlots];
#pragma unroll
  for (int t = 0; t < kPortSlots; t++) {
    const int l = tid + nt * t;
    p[t] = e[t] = F[t] = cl[t] = 0;
    if (l < E) {
      const uint32_t cb = a.llc[((size_t)L * E + l) * 2], ce = a.llc[((size_t)L * E + l) * 2 + 1];
      if (cb != ce) {
        p[t] = ccnt[cb - lo];
        e[t] = ccnt[ce - lo];
      }
      F[t] = lfree[l];
      cl[t] = a.cost[l];
    }
  }
  __syncthreads();
  // the send at the front of each owned run
  uint32_t hcp[kPortSlots], hr0[kPortSlots];
#pragma unroll
  for (int t = 0; t < kPortSlots; t++) {
    hcp[t] = p[t] < e[t] ? wcp[p[t]] : 0u;
    hr0[t] = p[t] < e[t] ? wr0[p[t]] : 0u;
  }
  const uint32_t spin_limit = 64u * (tot + 64u);
  for (uint32_t idle = 0;;) {
    bool left = false, moved = false;
#pragma unroll
    for (int t = 0; t < kPortSlots; t++) {
      if (p[t] >= e[t]) continue;
      const uint32_t pj = hcp[t] >> 16;
      uint32_t r = hr0[t];
      bool ready = true;
      if (pj != 0xFFFFu) {
        const uint32_t fp = lds_get(&fcur[pj]);
        ready = fp != kUnsetF;
        r = max(r, fp);
      }
      if (ready) {
        const uint32_t f = max(r, F[t]) + cl[t];
        lds_put(&fcur[hcp[t] & 0xFFFFu], f);
        F[t] = f;
        if (++p[t] < e[t]) {
          hcp[t] = wcp[p[t]];
          hr0[t] = wr0[p[t]];
        }
        moved = true;
      }
      left |= p[t] < e[t];
    }
    if (__ballot(left) == 0) break;
    idle = __ballot(moved) ? 0u : idle + 1u;
    if (idle > spin_limit) {  // unreachable: the waits follow one order
      *fault = true;
      break;
    }
  }
  __syncthreads();
  // arrivals and port free times after the level
  uint32_t mk = 0;
  for (uint32_t x = tid; x < tot; x += nt) {
    const int c = sorted[x];
    ctime[c] = fcur[c];
    mk = max(mk, fcur[c]);
  }
  // a link with classes at this level may still carry no send of this
  // candidate: only a nonempty run moves the port's free time
  for (int l = tid; l < E; l += nt) {
    const uint32_t cb = a.llc[((size_t)L * E + l) * 2], ce = a.llc[((size_t)L * E + l) * 2 + 1];
    if (cb != ce) {
      const uint32_t xb = ccnt[cb - lo], xe = ccnt[ce - lo];
      if (xe > xb) lfree[l] = fcur[sorted[xe - 1]];
    }
    const uint32_t cb2 = a.llc2[((size_t)L * E + l) * 2], ce2 = a.llc2[((size_t)L * E + l) * 2 + 1];
    if (cb2 != ce2) {
      const uint32_t xb = ccnt2[cb2 - lo2], xe = ccnt2[ce2 - lo2];
      if (xe > xb) lfree[l] = fcur[sorted2[xe - 1]];
    }
  }
  __syncthreads();
  return mk;
}

template <int NT>
__global__ __launch_bounds__(NT) void path_eval_kernel(PathArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  // per chunk: its chosen route option (an index into the path tables), or
  // kNoOption when it has no send (its own rank, or left unrouted)
  uint32_t *qc = (uint32_t *)(lds + a.o_qc);
  uint32_t *ctime = (uint32_t *)(lds + a.o_ctime);  // chunk's arrival so far
  uint32_t *lfree = (uint32_t *)(lds + a.o_lfree);
  uint32_t *ccnt = (uint32_t *)(lds + a.o_ccnt);
  uint32_t *ccur = (uint32_t *)(lds + a.o_ccur);
  // per scattered send: priority << 32 | chunk (ascending = the Step-2 tie
  // order), and its class
  uint64_t *e64 = (uint64_t *)(lds + a.o_e64);
  uint16_t *ecls = (uint16_t *)(lds + a.o_ecls);
  uint16_t *sorted = (uint16_t *)(lds + a.o_sorted);
  uint32_t *red = (uint32_t *)(lds + a.o_red);

  const int tid = threadIdx.x, nt = blockDim.x, lane = tid & 63, wave = tid >> 6;
  const int C = a.C, P = a.P, E = a.E, nlev = a.nlev;

  for (int64_t i = blockIdx.x; i < a.n; i += gridDim.x) {
    const uint8_t *grt = a.routes + (size_t)i * a.route_stride;
    const uint32_t *gpr = a.prio + (size_t)i * a.prio_stride;
    bool unrouted = false;
    for (int c = tid; c < C; c += nt) {
      const uint32_t k = grt[c];
      ctime[c] = 0;
      const int pair = c / a.cpr;
      const int s = pair / P, d = pair % P;
      uint32_t q = kNoOption;
      if (s != d) {
        const int pp = s * P + d;
        if (k < a.npaths[pp]) q = a.pair_base[pp] + k;
        else unrouted = true;
      }
      qc[c] = q;
    }
    for (int l = tid; l < E; l += nt) lfree[l] = 0;
    const bool any_unrouted = __syncthreads_or(unrouted);

    uint32_t mk = 0;
    bool fault = false;
    for (int L = 0; L < nlev; L++) {
      const uint32_t lo = a.lvl_cls_begin[L];
      const int ncl = (int)(a.lvl_cls_begin[L + 1] - lo);
      for (int j = tid; j <= ncl; j += nt) ccnt[j] = 0;
      __syncthreads();
      // count the level's sends per class
      for (int c = tid; c < C; c += nt) {
        const uint32_t q = qc[c];
        if (q == kNoOption) continue;
        const int h = a.path_lvl_hop[(size_t)q * nlev + L];
        const uint32_t po = a.path_off[q];
        if (h < 0) continue;
        atomicAdd(&ccnt[a.hop_class[po + h] - lo], 1u);
      }
      __syncthreads();
      block_scan(ccnt, ccur, ncl, red);
      // scatter into classes (arbitrary order inside a class)
      for (int c = tid; c < C; c += nt) {
        const uint32_t q = qc[c];
        if (q == kNoOption) continue;
        const int h = a.path_lvl_hop[(size_t)q * nlev + L];
        const uint32_t po = a.path_off[q];
        if (h < 0) continue;
        const int cls = a.hop_class[po + h] - lo;
        const uint32_t slot = atomicAdd(&ccur[cls], 1u);
        e64[slot] = ((uint64_t)gpr[(size_t)c * a.H + h] << 32) | (uint32_t)c;
        ecls[slot] = (uint16_t)cls;
      }
      __syncthreads();
      // order inside each class: priority, then chunk
      const uint32_t tot = ccnt[ncl];
      for (uint32_t x = tid; x < tot; x += nt) {
        const int k = ecls[x];
        const uint32_t b = ccnt[k];
        sorted[b + rank_in_class(e64, b, ccnt[k + 1], e64[x])] = (uint16_t)e64[x];
      }
      __syncthreads();
      if (a.ports) {
        mk = max(mk, ports_level(a, L, gpr, ctime, lfree, ccnt, sorted, red, &fault));
        continue;
      }
      // time every link's sends of this level in order
      for (int l = tid; l < E; l += nt) {
        const uint32_t cb = a.llc[((size_t)L * E + l) * 2], ce = a.llc[((size_t)L * E + l) * 2 + 1];
        if (cb == ce) continue;
        const uint32_t xb = ccnt[cb - lo], xe = ccnt[ce - lo];
        uint32_t f = lfree[l];
        const uint32_t cl = a.cost[l];
        if (a.contig && a.lmerge[l]) {
          // contiguous transfers (every send of a level has the same
          // remaining length): a send joins the open transfer when its chunk
          // was ready when the transfer started
          const uint32_t al = a.lalpha[l];
          const uint64_t bsz = a.lbs[l];
          uint32_t gs = 0, gm = 0, g0 = xb;
          for (uint32_t x = xb;; x++) {
            const bool end = x == xe;
            const uint32_t r = end ? 0u : ctime[sorted[x]];
            const bool join = !end && gm > 0 && r <= gs;
            if (gm > 0 && !join) {
              f = gs + al + (uint32_t)((bsz * gm + 999) / 1000);
              for (uint32_t t = g0; t < g0 + gm; t++) ctime[sorted[t]] = f;
            }
            if (end) break;
            if (join) {
              gm++;
            } else {
              gs = max(f, r);
              gm = 1;
              g0 = x;
            }
          }
        } else {
          for (uint32_t x = xb; x < xe; x++) {
            const int c = sorted[x];
            f = max(ctime[c], f) + cl;
            ctime[c] = f;
          }
        }
        lfree[l] = f;
        mk = max(mk, f);
      }
      __syncthreads();
    }
    mk = wave_max(mk);
    if (lane == 0) red[wave] = mk;
    __syncthreads();
    const bool failed = __syncthreads_or(fault);
    if (tid == 0) {
      uint32_t m = 0;
      for (int w = 0; w < nt / 64; w++) m = max(m, red[w]);
      a.makespan[i] = failed ? 0xFFFFFFFFu : m;
      a.valid[i] = (uint8_t)(!any_unrouted && !failed);
    }
    __syncthreads();
  }
}

int32_t align16(int32_t x) { return (x + 15) & ~15; }

}  // namespace

int32_t path_layout(const taccl_plan &p, PathArgs &a) {
  const int32_t C = p.coll.C, E = p.topo.E;
  const int32_t M = std::max(p.max_lvl_sends, 1), K = std::max(p.max_lvl_cls, 1);
  int32_t off = 0;
  auto take = [&](int32_t bytes) {
    int32_t o = off;
    off = align16(off + bytes);
    return o;
  };
  a.o_qc = take(4 * C);
  a.o_ctime = take(4 * C);
  a.o_lfree = take(4 * E);
  a.o_ccnt = take(4 * (K + 1));
  a.o_ccur = take(4 * K);
  a.o_e64 = take(8 * (M + 3));
  a.o_ecls = take(2 * M);
  a.o_sorted = take(2 * M);
  a.max_lvl = M;
  a.o_red = take(4 * (kPathPortThreads / 64));
  if (p.ports) {  // receive-port order and per-chunk state
    const int32_t K2 = std::max(p.max_lvl_cls2, 1);
    a.o_ccnt2 = take(4 * (K2 + 1));
    a.o_ccur2 = take(4 * K2);
    a.o_sorted2 = take(2 * M);
    a.o_fcur = take(4 * C);
    a.o_pd = take(2 * C);
    a.o_dl = take(2 * C);
  }
  a.lr_threads = (p.ports && p.max_lvl_sends > 4 * kPathThreads) ? kPathPortThreads : kPathThreads;
  a.lds_bytes = off;
  return off;
}

hipError_t launch_path(const PathArgs &a, int grid, hipStream_t stream) {
  // switch-port plans whose levels hold more sends than four per thread of
  // a 256-thread block run 1024-thread blocks (the port passes keep four
  // positions per thread in registers)
  if (a.lr_threads == kPathPortThreads)
    hipLaunchKernelGGL(path_eval_kernel<kPathPortThreads>, dim3(grid), dim3(kPathPortThreads),
                       a.lds_bytes, stream, a);
  else
    hipLaunchKernelGGL(path_eval_kernel<kPathThreads>, dim3(grid), dim3(kPathThreads),
                       a.lds_bytes, stream, a);
  return hipGetLastError();
}

}  // namespace taccl

// ===========================================================================
// Register-resident Alltoall kernel (paths of <= 6 hops, <= 8 levels,
// <= 4096 chunks). One block of NT threads evaluates one candidate at a
// time. Thread t owns chunks t, t+NT, ...: their route option's record (hop
// count, the hop at each level, the class of every hop) and the priorities
// of their hops are loaded once into registers. Per candidate:
//   A. count every send of every level per (class, top priority bits)
//      bucket (buckets are numbered level by level; within a level classes
//      are ordered by link, then travelled cost, so a link's sends form one
//      contiguous run);
//   B. one block scan of all the bucket counts;
// then per level, O(1) work per send:
//   C. place the level's sends in their buckets (an atomic cursor per
//      bucket: after the level a bucket's cursor is the next one's start);
//   D. order the few sends that share a bucket by (priority, chunk);
//   E. time every link's run at once: with link cost c, carried busy time F
//      and ready times r_j of the run's sends in order, the k-th send
//      finishes at (k+1)c + max(F, max_{j<=k}(r_j - j c)) (App. B.3 without
//      contiguity), so one segmented prefix max over the level gives every
//      finish time.
// ===========================================================================

namespace taccl {
namespace {

constexpr uint32_t kUnset = 0xFFFFFFFFu;

// The top `bits` bits of x (0 for bits = 0): one bit-field extract, whose
// width 0 gives 0
__device__ __forceinline__ uint32_t top_bits(uint32_t x, uint32_t bits) {
  return __builtin_amdgcn_ubfe(x, 32u - bits, bits);
}

// Exclusive scan of cnt[0..n) in place with cnt[n] = total (all threads
// call; cnt 16-byte aligned; cnt[n+1..n+3] are overwritten as well). Each
// wavefront takes a contiguous range of 4-word groups and each lane one
// group per round, so a round reads 1 KB of consecutive words: one pass
// for the wavefront totals, one to write the prefixes.
__device__ void block_excl_scan4(uint32_t *cnt, int n, uint32_t *wsum) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, nw = blockDim.x >> 6;
  const int ng = (n >> 2) + 1;  // groups up to and including index n
  const int gpw = ((ng + nw - 1) / nw + 63) & ~63;
  const int g0 = wave * gpw;
  uint4 *c4 = (uint4 *)cnt;
  auto group = [&](int g) {  // entries from index n on count as 0
    uint4 x = g < ng ? c4[g] : make_uint4(0u, 0u, 0u, 0u);
    const int e = 4 * g;
    x.x = e < n ? x.x : 0u;
    x.y = e + 1 < n ? x.y : 0u;
    x.z = e + 2 < n ? x.z : 0u;
    x.w = e + 3 < n ? x.w : 0u;
    return x;
  };
  uint32_t sum = 0;
  for (int r = 0; r < gpw; r += 64) {
    const uint4 x = group(g0 + r + lane);
    sum += x.x + x.y + x.z + x.w;
  }
  const uint32_t wt = (uint32_t)__builtin_amdgcn_readlane((int)wave_scan_add(sum), 63);
  if (lane == 0) wsum[wave] = wt;
  __syncthreads();
  const uint32_t ws = row_scan_add(lane < nw ? wsum[lane] : 0u);
  const uint32_t w = (uint32_t)__builtin_amdgcn_readfirstlane(wave);
  uint32_t run = w ? (uint32_t)__builtin_amdgcn_readlane((int)ws, w - 1) : 0u;
  for (int r = 0; r < gpw; r += 64) {
    const int g = g0 + r + lane;
    const uint4 x = group(g);
    const uint32_t gs = x.x + x.y + x.z + x.w;
    const uint32_t inc = wave_scan_add(gs);
    const uint32_t e0 = run + inc - gs;
    // the group holding index n receives the total there (later entries
    // count as 0)
    if (g < ng) c4[g] = make_uint4(e0, e0 + x.x, e0 + x.x + x.y, e0 + x.x + x.y + x.z);
    run += (uint32_t)__builtin_amdgcn_readlane((int)inc, 63);
  }
  __syncthreads();
}

template <int CPT, int NT, bool kContig>
__global__ __launch_bounds__(NT) void path_eval_fast(PathArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int C = a.C, E = a.E, H = a.H, nlev = a.nlev;
  const uint32_t NBT = (uint32_t)a.nb_total;

  // per link: {busy time, cost}, one 8-byte read in the timing pass
  uint2 *lfc = (uint2 *)(lds + a.o_flfree);
  uint32_t *lnext = (uint32_t *)(lds + a.o_fnext);  // busy time after this level
  uint32_t *s_cinfo = (uint32_t *)(lds + a.o_fcinfo);
  uint32_t *s_cbkt = (uint32_t *)(lds + a.o_fcbkt);
  uint32_t *s_lfb = (uint32_t *)(lds + a.o_flcb);    // [nlev+1] first bucket of a level
  uint32_t *ctime = (uint32_t *)(lds + a.o_fctime);  // a chunk's arrival so far
  // bucket cursors over all levels: bst[0] = 0 and bst[b + 1] holds bucket
  // b's count, then its start, then (once its level's sends are placed)
  // its end, so bucket b spans [bst[b], bst[b + 1]) from then on; one dummy
  // counter per lane follows at bst[NBT + 2 + lane]. bst + 1 is 16-byte
  // aligned for the scan.
  uint32_t *bst = (uint32_t *)(lds + a.o_fbcnt) + 3;
  // bucket entries: priority << 32 | link << cb | chunk (ascending =
  // Step-2 tie order: a bucket's sends share one link)
  uint64_t *e64 = (uint64_t *)(lds + a.o_fepr);
  // sorted sends, chunk | link << cb | index in its link run << (cb + lb),
  // stored transposed: position t*ept + q of thread t's range at q*NT + t
  uint32_t *pinfo = (uint32_t *)(lds + a.o_fsrt);
  // per bucket-sorted position: its bucket | the first bucket of its link's
  // run << 16
  uint32_t *aux = (uint32_t *)(lds + a.o_faux);
  const uint32_t cb = a.cbits, lb = a.lbits, kb = cb + lb;
  const uint32_t cmask = (1u << cb) - 1, lmask = (1u << lb) - 1;
  uint32_t *red = (uint32_t *)(lds + a.o_fred);      // [2][NT/64] scan scratch
  uint8_t *s_merge = lds + a.o_fmerge;  // links that carry contiguous transfers
  for (int j = tid; j < E; j += NT) {
    lfc[j].y = a.cost[j];
    s_merge[j] = a.contig ? a.lmerge[j] : 0;
  }
  for (int j = tid; j < a.ncls; j += NT) {
    s_cinfo[j] = a.cinfo[j];
    s_cbkt[j] = a.cbkt[j];
  }
  for (int j = tid; j <= nlev; j += NT) {
    // an empty level starts where the next one does
    const uint32_t k = a.lvl_cls_begin[j];
    s_lfb[j] = (j < nlev && k < (uint32_t)a.ncls) ? (a.cbkt[k] & 0xFFFFFFu) : NBT;
  }
  for (uint32_t j = tid; j < NBT + 2; j += NT) bst[j] = 0;
  for (int j = tid; j < NT * CPT; j += NT) pinfo[j] = 0;
  __syncthreads();

  // The candidate's route choices, chunk tables and priorities (one batch
  // of independent loads). The next candidate's batch is issued as soon as
  // the last level has taken what it needs from these registers, so its
  // HBM latency overlaps that level's ordering and timing.
  // kk[j]: the chunk's route byte at bits 8 * (chunk & 3) (the aligned
  // word that holds it, or the byte moved there)
  uint32_t pr[CPT][kFastMaxHops], kk[CPT], cp[CPT];
  // Branch-free loads, so that no loaded value meets a select or a
  // zero-extension before it is used and the batch stays in flight: past
  // the batch the last candidate is read again, past the chunks the last
  // chunk (never used); hops past the plan's longest route are skipped (a
  // uniform branch) and keep stale values, which no route reads.
#pragma unroll
  for (int j = 0; j < CPT; j++)
#pragma unroll
    for (int h = 0; h < kFastMaxHops; h++) pr[j][h] = 0;
  auto load_inputs = [&](int64_t i) {
    const int64_t ii = i < a.n ? i : a.n - 1;
    const uint8_t *grt = a.routes + (size_t)ii * a.route_stride;
    const uint32_t *grw = (const uint32_t *)grt;  // when routes_words
    const uint32_t *gpr = a.prio + (size_t)ii * a.prio_stride;
    // the thread index is hidden from the optimiser, so per-chunk addresses
    // are recomputed instead of being hoisted out of the candidate loop and
    // spilled
    int tv = tid;
    asm volatile("" : "+v"(tv));
#pragma unroll
    for (int j = 0; j < CPT; j++) {
      const uint32_t cc = (uint32_t)min(tv + NT * j, C - 1);
      if (a.routes_words)
        kk[j] = grw[cc >> 2];
      else
        kk[j] = (uint32_t)grt[cc] << (8 * (cc & 3));
      cp[j] = a.cpath[cc];
      // one address per chunk; the hops are immediate offsets from it
      const uint32_t *row = gpr + __umul24(cc, (uint32_t)H);
#pragma unroll
      for (int h = 0; h < kFastMaxHops; h++)
        if (h < H) pr[j][h] = row[h];
    }
  };
  load_inputs(blockIdx.x);
  for (int64_t i = blockIdx.x; i < a.n; i += gridDim.x) {
    // ---- setup: owned chunks' records in registers -----------------------
    int tv = tid;
    asm volatile("" : "+v"(tv));
    // rw0: hop count | level -> hop index << 8 (3 bits per level, 7 = none)
    uint32_t rw0[CPT], rcl[CPT][3];
    bool unrouted = false;
    // second batch: the chosen route records, one unconditional load per
    // chunk (record 0, without hops, for a chunk that has no route or no
    // chunk at all)
#pragma unroll
    for (int j = 0; j < CPT; j++) {
      const int c = tv + NT * j;
      const uint32_t np = cp[j] >> 24;
      const bool live = c < C;
      const uint32_t k = (kk[j] >> (8 * ((uint32_t)c & 3u))) & 0xFFu;  // the route choice
      // no route option at all, or the pair left unrouted: never delivered
      if (live && (cp[j] == kNoRoute || (np && k >= np))) unrouted = true;
      const uint32_t rec = (live && k < np) ? (cp[j] & 0xFFFFFFu) + k : 0u;
      const uint4 r = ((const uint4 *)a.arec)[rec];
      rw0[j] = r.x;
      rcl[j][0] = r.y;
      rcl[j][1] = r.z;
      rcl[j][2] = r.w;
      if (live) ctime[c] = 0;
    }
    for (int l = tid; l < E; l += NT) {
      lfc[l].x = 0;
      lnext[l] = kUnset;
    }
    // ---- A. every send of every level per bucket ----------------------------
    // Straight-line code: a hop past the route counts on the lane's dummy
    // counter, so the counter updates of all hops are in flight together.
#pragma unroll
    for (int j = 0; j < CPT; j++) {
      const uint32_t hops = rw0[j] & 0xFF;
#pragma unroll
      for (int h = 0; h < kFastMaxHops; h++) {
        if (h >= H) break;
        const uint32_t cl = (rcl[j][h >> 1] >> (16 * (h & 1))) & 0xFFFFu;
        const uint32_t cbk = s_cbkt[cl], bits = cbk >> 24;
        const uint32_t b = (cbk & 0xFFFFFF) + top_bits(pr[j][h], bits);
        atomicAdd(&bst[(uint32_t)h < hops ? b + 1 : NBT + 2 + lane], 1u);
      }
    }
    const bool any_unrouted = __syncthreads_or(unrouted);
    // ---- B. bucket starts ----------------------------------------------------
    block_excl_scan4(bst + 1, (int)NBT, red);

    uint32_t mk = 0;
    for (int L = 0; L < nlev; L++) {
      // this level's first position among all levels' sends (the end of the
      // previous level's last bucket, untouched during this level)
      const uint32_t lb0 = bst[s_lfb[L]];
      // busy times after the previous level (a link without a send there
      // keeps its time)
      for (int l = tid; l < E; l += NT) {
        const uint32_t nx = lnext[l];
        if (nx != kUnset) lfc[l].x = nx;
        lnext[l] = kUnset;
      }
      // ---- C. place the level's sends ----------------------------------------
      // Straight-line code (selects, and the lane's dummy counter for a slot
      // without a send here) so that the LDS loads and cursor updates of all
      // slots are in flight together.
#pragma unroll
      for (int j = 0; j < CPT; j++) {
        const uint32_t h = (rw0[j] >> (8 + 3 * L)) & 7;  // 7: no hop at this level
        const bool act = h < (uint32_t)kFastMaxHops;
        // hop h's class and priority. With several chunks per thread: its
        // pair of hops (h >> 1), then the half (h & 1), with three shared
        // conditions; with one, a select per hop (measured faster there)
        static_assert(kFastMaxHops == 6, "three pairs of hops");
        uint32_t cw, pv;
        if constexpr (CPT >= 2) {
          const bool c2 = h >= 2, c4 = h >= 4, odd = (h & 1) != 0;
          cw = c4 ? rcl[j][2] : c2 ? rcl[j][1] : rcl[j][0];
          const uint32_t pe = c4 ? pr[j][4] : c2 ? pr[j][2] : pr[j][0];
          const uint32_t po = c4 ? pr[j][5] : c2 ? pr[j][3] : pr[j][1];
          pv = odd ? po : pe;
        } else {
          cw = rcl[j][0];
          pv = pr[j][0];
#pragma unroll
          for (int t = 1; t < kFastMaxHops; t++)
            if (h == (uint32_t)t) pv = pr[j][t];
          if (h >= 2) cw = rcl[j][1];
          if (h >= 4) cw = rcl[j][2];
        }
        const uint32_t cl = (h & 1) ? (cw >> 16) : (cw & 0xFFFF);
        const uint32_t cbk = s_cbkt[cl], ci = s_cinfo[cl], bits = cbk >> 24;
        const uint32_t b = (cbk & 0xFFFFFF) + top_bits(pv, bits);
        const uint32_t gp = atomicAdd(&bst[act ? b + 1 : NBT + 2 + lane], 1u);
        if (act) {
          e64[gp - lb0] = ((uint64_t)pv << 32) | (uint32_t)(tid + NT * j) | ((ci & 0xFFFFu) << cb);
          aux[gp - lb0] = b | (ci & 0xFFFF0000u);
        }
      }
      if (L == nlev - 1) load_inputs(i + gridDim.x);  // this candidate's inputs are dead
      __syncthreads();
      const uint32_t tot = bst[s_lfb[L + 1]] - lb0;
      const uint32_t ept = (tot + NT - 1) / NT;  // <= CPT: a level has <= C sends
      // pos / ept for pos < 2^16 and ept <= 4 (the same for every thread):
      // a shift, or (pos * 43691) >> 17 for 3 (exact below 2^17); 24-bit
      // multiplies issue at the full VALU rate
      const uint32_t esh = ept >= 4 ? 2u : ept >= 2 ? 1u : 0u;
      auto div_ept = [&](uint32_t pos) -> uint32_t {
        return ept == 3 ? __umul24(pos, 43691u) >> 17 : pos >> esh;
      };
      // the contiguity walker divides with one 64-bit multiply
      // (y / ept = (y * em) >> 32, em = floor((2^32 - 1) / ept) + 1)
      const uint64_t em = (kContig && ept) ? 0xFFFFFFFFull / ept + 1 : 0;
      // The level's ordering and timing passes. Without contiguity the
      // level's ept (the same for every thread) is a compile-time constant
      // EP in each copy of them below; with it, one copy takes EP = CPT and
      // the level's ept at run time (keeping the run walker in one copy).
      auto order_and_time = [&](auto ep_c) {
      constexpr int EP = decltype(ep_c)::value;
      const uint32_t epr = kContig ? ept : (uint32_t)EP;
      // ---- D. order inside buckets by (priority, chunk); record each send's
      //      link and its index in the link's run -------------------------
      // One lane per bucket-sorted position: neighbouring lanes hold
      // neighbouring buckets, so their members are read with few bank
      // conflicts, and a pass waits only for the largest bucket among its
      // 64 positions.
      auto div_e = [&](uint32_t pos) -> uint32_t {
        if constexpr (kContig)
          return div_ept(pos);
        else if constexpr (EP == 3)
          return __umul24(pos, 43691u) >> 17;
        else
          return pos >> (EP == 4 ? 2 : EP == 2 ? 1 : 0);
      };
#pragma unroll
      for (int qq = 0; qq < EP; qq++) {
        const uint32_t x = (uint32_t)tid + (uint32_t)(qq * NT);
        if (x >= tot) break;
        const uint64_t me = e64[x];
        const uint32_t ax = aux[x];
        const uint32_t b = ax & 0xFFFFu;
        const uint32_t b0 = bst[b] - lb0, b1 = bst[b + 1] - lb0, rs = bst[ax >> 16] - lb0;
        // four members a step (three spare entries past the array's end;
        // entries past the bucket never count)
        uint32_t rank = 0;
        for (uint32_t y = b0; y < b1; y += 4) {
          uint64_t m[4];
#pragma unroll
          for (int u = 0; u < 4; u++) m[u] = e64[y + u];
#pragma unroll
          for (int u = 0; u < 4; u++) rank += (uint32_t)((y + u < b1) & (m[u] < me));
        }
        const uint32_t pos = b0 + rank;
        const uint32_t t = div_e(pos), q = pos - __umul24(t, epr);
        pinfo[q * NT + t] = (uint32_t)me | ((pos - rs) << kb);
      }
      __syncthreads();
      // ---- E. finish times of every link run --------------------------------
      // The k-th send of a link run with cost c, ready times r_j and busy
      // time F finishes at (k+1)c + max_{j<=k} a_j with a_0 = max(r_0, F)
      // and a_j = max(r_j - j c, 0) after it (F >= 0 dominates the clipped
      // values): a prefix maximum segmented by runs, which are contiguous
      // along the sorted positions. Thread tid owns sorted positions
      // [tid*ept, tid*ept + ept); every load is issued unmasked (an entry
      // past the level's sends holds a send of an earlier level, or the
      // zero it started with, so its indexes are in range; its values are
      // never used).
      const uint32_t x0 = (uint32_t)tid * epr;
      uint32_t pis[EP], ct[EP], cs[EP], lf[EP];
#pragma unroll
      for (int q = 0; q < EP; q++) pis[q] = pinfo[q * NT + tid];
#pragma unroll
      for (int q = 0; q < EP; q++) {
        const uint32_t l = (pis[q] >> cb) & lmask;
        ct[q] = ctime[pis[q] & cmask];
        const uint2 w = lfc[l];
        cs[q] = w.y;
        lf[q] = w.x;
      }
      // this thread's positions: segmented running maxima s[q]
      const uint32_t nv = tot > x0 ? min(epr, tot - x0) : 0u;  // valid positions
      uint32_t sv[EP];
      uint32_t prev = 0;
#pragma unroll
      for (int q = 0; q < EP; q++) {
        const uint32_t k = pis[q] >> kb, kc = __umul24(k, cs[q]);  // k < 2^16, c < 2^24
        const uint32_t av = k == 0 ? max(ct[q], lf[q]) : __builtin_elementwise_sub_sat(ct[q], kc);
        sv[q] = (k > 0 && q > 0) ? max(prev, av) : av;
        prev = sv[q];
      }
      // the run of the thread's last position: its running maximum, and
      // whether it began before the thread's first position (then the
      // maximum of earlier threads of the same run joins in); a thread
      // without positions passes its predecessors' value on
      const uint32_t kl = nv ? (pis[nv - 1 < EP ? nv - 1 : 0] >> kb) : 0u;
      uint32_t gv = 0, pass = nv == 0 ? 1u : (kl >= nv ? 1u : 0u);
#pragma unroll
      for (int q = 0; q < EP; q++)
        if ((uint32_t)q + 1 == nv) gv = sv[q];
      // inclusive scan of (value, pass) pairs over the lanes: a lane that
      // passes takes the maximum of the lanes before it, up to and
      // including the first one that does not pass
      {
#define TACCL_SEG_STEP(CTRL, RM)                                                         \
  {                                                                                     \
    const uint32_t ov = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)gv, CTRL, RM, 0xf, false); \
    const uint32_t op = (uint32_t)__builtin_amdgcn_update_dpp(1, (int)pass, CTRL, RM, 0xf, false); \
    if (pass) {                                                                         \
      gv = max(gv, ov);                                                                 \
      pass = op;                                                                        \
    }                                                                                   \
  }
        TACCL_SEG_STEP(kRowShr + 1, 0xf)
        TACCL_SEG_STEP(kRowShr + 2, 0xf)
        TACCL_SEG_STEP(kRowShr + 4, 0xf)
        TACCL_SEG_STEP(kRowShr + 8, 0xf)
        TACCL_SEG_STEP(kBcast15, 0xa)
        TACCL_SEG_STEP(kBcast31, 0xc)
#undef TACCL_SEG_STEP
      }
      // across wavefronts: every wavefront combines the totals of the ones
      // before it (value, pass of lane 63)
      if (lane == 63) {
        red[wave] = gv;
        red[NT / 64 + wave] = pass;
      }
      __syncthreads();
      uint32_t cin = 0;  // segmented maximum of the positions before x0
      {
        // exclusive within the wavefront: the lane before (wave_shr:1 gives
        // lane 0 nothing: value 0, pass 1)
        uint32_t ev = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)gv, kWaveShr1, 0xf, 0xf, false);
        uint32_t ep = (uint32_t)__builtin_amdgcn_update_dpp(1, (int)pass, kWaveShr1, 0xf, 0xf, false);
        const uint32_t w = (uint32_t)__builtin_amdgcn_readfirstlane(wave);
        for (int v = (int)w - 1; v >= 0 && ep; v--) {
          ev = max(ev, red[v]);
          ep = red[NT / 64 + v];
        }
        cin = ev;
      }
      // finish times
      const uint32_t nxt0 = (tid + 1 < NT) ? pinfo[tid + 1] : 0u;  // next thread's first
#pragma unroll
      for (int q = 0; q < EP; q++) {
        const uint32_t x = x0 + q;
        if ((uint32_t)q < epr && x < tot) {
          const uint32_t c = pis[q] & cmask, l = (pis[q] >> cb) & lmask, k = pis[q] >> kb;
          if (kContig && s_merge[l]) {
            // contiguous transfers: the run's first position walks the run
            // (every send of a level has the same remaining length); a send
            // joins the open transfer when its chunk was ready at its start
            if (k == 0) {
              const uint32_t al = a.lalpha[l];
              const uint64_t bsz = a.lbs[l];
              uint32_t F = lf[q], gs = 0, gm = 0, g0 = x;
              auto at = [&](uint32_t y) {  // packed send at sorted position y
                const uint32_t ty = (uint32_t)(((uint64_t)y * em) >> 32);
                return pinfo[(y - ty * ept) * NT + ty];
              };
              for (uint32_t y = x;; y++) {
                const uint32_t py = (y < tot) ? at(y) : 0u;
                const bool end = y == tot || (y > x && (py >> kb) == 0);
                const uint32_t ry = end ? 0u : ctime[py & cmask];
                const bool join = !end && gm > 0 && ry <= gs;
                if (gm > 0 && !join) {  // close the open transfer
                  const uint32_t f = gs + al + (uint32_t)((bsz * gm + 999) / 1000);
                  for (uint32_t t = g0; t < g0 + gm; t++) ctime[at(t) & cmask] = f;
                  F = f;
                  mk = max(mk, f);
                }
                if (end) break;
                if (join) {
                  gm++;
                } else {
                  gs = max(F, ry);
                  gm = 1;
                  g0 = y;
                }
              }
              lnext[l] = F;
            }
            continue;
          }
          const uint32_t cl = cs[q];
          // the run began before this thread's first position: k > q
          const uint32_t best = k > (uint32_t)q ? max(sv[q], cin) : sv[q];
          const uint32_t f = __umul24(k + 1, cl) + best;
          ctime[c] = f;
          mk = max(mk, f);
          const uint32_t nk = ((uint32_t)q + 1 < epr ? pis[q < EP - 1 ? q + 1 : q] : nxt0) >> kb;
          if (x + 1 == tot || nk == 0) lnext[l] = f;  // last send of the link's run
        }
      }
      };
      if constexpr (kContig) {
        order_and_time(std::integral_constant<int, CPT>{});
      } else if (ept <= 1) {
        order_and_time(std::integral_constant<int, 1>{});
      } else if constexpr (CPT >= 2) {
        if (ept == 2) {
          order_and_time(std::integral_constant<int, 2>{});
        } else if constexpr (CPT >= 4) {
          if (ept == 3)
            order_and_time(std::integral_constant<int, 3>{});
          else
            order_and_time(std::integral_constant<int, 4>{});
        }
      }
      __syncthreads();
    }
    if (nlev == 0) load_inputs(i + gridDim.x);
    // makespan: block max
    for (int o = 32; o > 0; o >>= 1) mk = max(mk, (uint32_t)__shfl_xor((int)mk, o));
    if (lane == 0) red[wave] = mk;
    __syncthreads();
    if (tid == 0) {
      uint32_t m = 0;
      for (int w = 0; w < NT / 64; w++) m = max(m, red[w]);
      a.makespan[i] = m;
      a.valid[i] = (uint8_t)!any_unrouted;
    }
    // the next candidate's bucket counters (the last level's ordering is done)
    for (uint32_t j = tid; j < (NBT + 4) / 4; j += NT) ((uint4 *)(bst + 1))[j] = make_uint4(0u, 0u, 0u, 0u);
    __syncthreads();
  }
}

}  // namespace

int32_t path_fast_layout(const taccl_plan &p, PathArgs &a) {
  const int32_t C = p.coll.C, E = p.topo.E;
  const int32_t M = std::max(p.max_lvl_sends, 1);
  int32_t off = 0;
  auto take = [&](int32_t bytes) {
    int32_t o = off;
    off = (off + bytes + 15) & ~15;
    return o;
  };
  a.ncls = p.ncls;
  a.nb_total = p.nb_total;
  a.o_fnext = take(4 * E);
  a.o_fmerge = take(E);
  a.o_fcinfo = take(4 * std::max(p.ncls, 1));
  a.o_fcbkt = take(4 * std::max(p.ncls, 1));
  a.o_flcb = take(4 * (p.nlev + 1));
  a.o_fctime = take(4 * C);
  a.o_flfree = take(8 * E);  // {busy time, cost} per link
  // three words of padding, a zero, the bucket cursors of all levels, the
  // total, and one dummy counter per lane of a wavefront (slots without a
  // send count there)
  a.o_fbcnt = take(4 * (3 + p.nb_total + 2 + 64));
  a.o_fepr = take(8 * (M + 3));
  a.o_faux = take(4 * M);
  a.o_fsrt = take(4 * path_fast_threads(p) * path_fast_cpt(p));
  // packed sorted sends: chunk, link and run index in one word
  auto bits = [](uint32_t n) {  // bits to hold 0 .. n-1
    uint32_t b = 0;
    while ((1ull << b) < n) b++;
    return b;
  };
  a.cbits = (int32_t)bits((uint32_t)C);
  a.lbits = (int32_t)bits((uint32_t)E);
  a.o_fred = take(4 * 2 * (kPathFastThreads / 64));  // sized for the largest block
  a.lds_bytes = off;
  return off;
}

int path_fast_threads(const taccl_plan &p) {
  const int C = p.coll.C;
  return C <= 256 ? 256 : C <= 512 ? 512 : kPathFastThreads;
}

int path_fast_cpt(const taccl_plan &p) {
  // a sorted send packs chunk, link and run index (< C) into 32 bits
  auto bits = [](uint32_t n) {
    uint32_t b = 0;
    while ((1ull << b) < n) b++;
    return b;
  };
  if (p.coll.C < 1 || 2 * bits((uint32_t)p.coll.C) + bits((uint32_t)p.topo.E) > 32) return 0;
  // bucket and link fields are packed into 16 bits
  if (p.nb_total > kFastMaxBuckets || p.topo.E > (1 << 16)) return 0;
  // sorted positions below 2^16 and link costs below 2^24 (24-bit multiplies)
  if (p.max_lvl_sends > (1 << 16)) return 0;
  for (uint32_t c : p.cost)
    if (c >= (1u << 24)) return 0;
  const int nt = path_fast_threads(p);
  const int per = (p.coll.C + nt - 1) / nt;
  return per <= 1 ? 1 : per <= 2 ? 2 : per <= 4 ? 4 : 0;
}

template <bool kC>
static const void *path_fast_fn_c(int cpt, int nt) {
  if (nt == 256 && cpt == 1) return (const void *)path_eval_fast<1, 256, kC>;
  if (nt == 512 && cpt == 1) return (const void *)path_eval_fast<1, 512, kC>;
  if (nt == 1024 && cpt == 1) return (const void *)path_eval_fast<1, 1024, kC>;
  if (nt == 1024 && cpt == 2) return (const void *)path_eval_fast<2, 1024, kC>;
  if (nt == 1024 && cpt == 4) return (const void *)path_eval_fast<4, 1024, kC>;
  return nullptr;
}

static const void *path_fast_fn(const PathArgs &a, int cpt, int nt) {
  return a.contig ? path_fast_fn_c<true>(cpt, nt) : path_fast_fn_c<false>(cpt, nt);
}

int path_fast_blocks_per_cu(const PathArgs &a, int cpt, int nt) {
  const void *fn = path_fast_fn(a, cpt, nt);
  int nb = 0;
  if (!fn || hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, fn, nt, a.lds_bytes) != hipSuccess)
    return 0;
  return nb;
}

hipError_t launch_path_fast(const PathArgs &a, int cpt, int nt, int grid, hipStream_t stream) {
  const void *fn = path_fast_fn(a, cpt, nt);
  if (!fn) return hipErrorInvalidValue;
  void *args[] = {(void *)&a};
  return hipLaunchKernel(fn, dim3(grid), dim3(nt), args, a.lds_bytes, stream);
}

}  // namespace taccl
