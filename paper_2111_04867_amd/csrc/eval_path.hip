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

#include "kernels.h"

namespace taccl {

namespace {

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

__global__ __launch_bounds__(kPathThreads) void path_eval_kernel(PathArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  uint8_t *rt = lds + a.o_rt;
  uint32_t *ctime = (uint32_t *)(lds + a.o_ctime);  // chunk's arrival so far
  uint32_t *lfree = (uint32_t *)(lds + a.o_lfree);
  uint32_t *ccnt = (uint32_t *)(lds + a.o_ccnt);
  uint32_t *ccur = (uint32_t *)(lds + a.o_ccur);
  uint16_t *echunk = (uint16_t *)(lds + a.o_echunk);
  uint32_t *eprio = (uint32_t *)(lds + a.o_eprio);
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
      const uint8_t k = grt[c];
      rt[c] = k;
      ctime[c] = 0;
      const int pair = c / a.cpr;
      const int s = pair / P, d = pair % P;
      if (s != d && k >= a.npaths[s * P + d]) unrouted = true;
    }
    for (int l = tid; l < E; l += nt) lfree[l] = 0;
    const bool any_unrouted = __syncthreads_or(unrouted);

    uint32_t mk = 0;
    for (int L = 0; L < nlev; L++) {
      const uint32_t lo = a.lvl_cls_begin[L];
      const int ncl = (int)(a.lvl_cls_begin[L + 1] - lo);
      for (int j = tid; j <= ncl; j += nt) ccnt[j] = 0;
      __syncthreads();
      // count the level's sends per class
      for (int c = tid; c < C; c += nt) {
        const int pair = c / a.cpr;
        const int s = pair / P, d = pair % P;
        if (s == d) continue;
        const int pp = s * P + d;
        const int k = rt[c];
        if (k >= a.npaths[pp]) continue;
        const uint32_t q = a.pair_base[pp] + k;
        const int h = a.path_lvl_hop[(size_t)q * nlev + L];
        if (h < 0) continue;
        atomicAdd(&ccnt[a.hop_class[a.path_off[q] + h] - lo], 1u);
      }
      __syncthreads();
      block_scan(ccnt, ccur, ncl, red);
      // scatter into classes (arbitrary order inside a class)
      for (int c = tid; c < C; c += nt) {
        const int pair = c / a.cpr;
        const int s = pair / P, d = pair % P;
        if (s == d) continue;
        const int pp = s * P + d;
        const int k = rt[c];
        if (k >= a.npaths[pp]) continue;
        const uint32_t q = a.pair_base[pp] + k;
        const int h = a.path_lvl_hop[(size_t)q * nlev + L];
        if (h < 0) continue;
        const int cls = a.hop_class[a.path_off[q] + h] - lo;
        const uint32_t slot = atomicAdd(&ccur[cls], 1u);
        echunk[slot] = (uint16_t)c;
        eprio[slot] = gpr[(size_t)c * a.H + h];
        ecls[slot] = (uint16_t)cls;
      }
      __syncthreads();
      // order inside each class: priority, then chunk
      const uint32_t tot = ccnt[ncl];
      for (uint32_t x = tid; x < tot; x += nt) {
        const int k = ecls[x];
        const uint32_t b = ccnt[k], e = ccnt[k + 1];
        const uint32_t px = eprio[x], cx = echunk[x];
        uint32_t rank = 0;
        for (uint32_t y = b; y < e; y++) {
          const uint32_t py = eprio[y], cy = echunk[y];
          rank += (py < px) || (py == px && cy < cx);
        }
        sorted[b + rank] = (uint16_t)cx;
      }
      __syncthreads();
      // time every link's sends of this level in order
      for (int l = tid; l < E; l += nt) {
        const uint32_t cb = a.llc[((size_t)L * E + l) * 2], ce = a.llc[((size_t)L * E + l) * 2 + 1];
        if (cb == ce) continue;
        const uint32_t xb = ccnt[cb - lo], xe = ccnt[ce - lo];
        uint32_t f = lfree[l];
        const uint32_t cl = a.cost[l];
        for (uint32_t x = xb; x < xe; x++) {
          const int c = sorted[x];
          f = max(ctime[c], f) + cl;
          ctime[c] = f;
        }
        lfree[l] = f;
        mk = max(mk, f);
      }
      __syncthreads();
    }
    mk = wave_max(mk);
    if (lane == 0) red[wave] = mk;
    __syncthreads();
    if (tid == 0) {
      uint32_t m = 0;
      for (int w = 0; w < nt / 64; w++) m = max(m, red[w]);
      a.makespan[i] = m;
      a.valid[i] = (uint8_t)!any_unrouted;
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
  a.o_rt = take(C);
  a.o_ctime = take(4 * C);
  a.o_lfree = take(4 * E);
  a.o_ccnt = take(4 * (K + 1));
  a.o_cbase = a.o_ccnt;
  a.o_ccur = take(4 * K);
  a.o_echunk = take(2 * M);
  a.o_eprio = take(4 * M);
  a.o_ecls = take(2 * M);
  a.o_sorted = take(2 * M);
  a.o_red = take(4 * (kPathThreads / 64));
  a.lds_bytes = off;
  return off;
}

hipError_t launch_path(const PathArgs &a, int grid, hipStream_t stream) {
  hipLaunchKernelGGL(path_eval_kernel, dim3(grid), dim3(kPathThreads), a.lds_bytes, stream, a);
  return hipGetLastError();
}

}  // namespace taccl
