// Multicast (Allgather / explicit) evaluation kernel for gfx950.
//
// One 64-lane wavefront evaluates one candidate at a time, all state in LDS:
//   1. route choices and priorities of the candidate are staged in LDS with
//      coalesced loads;
//   2. lane = chunk: the routed paths of a chunk (destinations ascending)
//      are merged into a tree by first reach, giving one send per reached
//      vertex (one is_sent per chunk and link, App. B.1), with the tree
//      distance travelled so far and the longest remaining tree path below
//      each vertex (the two Step-2 keys of Sec. 5.1);
//   3. sends are bucketed by link (LDS atomics + wave scan) and each send
//      finds its place in the link's order by counting the sends that go
//      before it: remaining path desc, travelled asc, priority asc, chunk asc;
//   4. the least schedule of App. B.3 (no contiguity) is computed by letting
//      every link advance through its ordered sends while their chunk is
//      already present at the link's source; the send with the globally
//      smallest key is always ready, so every round makes progress;
//   5. postcondition (ballot over chunks) and makespan (wave max).
#include <hip/hip_runtime.h>

#include "kernels.h"

namespace taccl {

namespace {

constexpr uint32_t kNotYet = 0xFFFFFFFFu;

// Arrival times are written by one lane and read by others of the same wave
// while links advance; relaxed workgroup-scope atomics keep these accesses
// plain LDS instructions (a volatile pointer would turn them into FLAT ones).
__device__ __forceinline__ uint32_t lds_get(uint32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void lds_put(uint32_t *p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

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

__global__ __launch_bounds__(kTreeThreads) void tree_eval_kernel(TreeArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  uint8_t *rt = lds + a.o_rt;
  uint32_t *pr = (uint32_t *)(lds + a.o_pr);
  uint16_t *par = (uint16_t *)(lds + a.o_par);  // link+1 into (c,v), 0 = none
  uint32_t *dist = (uint32_t *)(lds + a.o_dist);
  uint32_t *hgt = (uint32_t *)(lds + a.o_hgt);
  uint32_t *fin = (uint32_t *)(lds + a.o_fin);
  uint16_t *ord = (uint16_t *)(lds + a.o_ord);
  uint16_t *sidx = (uint16_t *)(lds + a.o_sidx);
  uint16_t *tmp = (uint16_t *)(lds + a.o_tmp);
  uint16_t *chain = (uint16_t *)(lds + a.o_chain);
  uint32_t *krem = (uint32_t *)(lds + a.o_krem);
  uint32_t *ktrav = (uint32_t *)(lds + a.o_ktrav);
  uint32_t *lcnt = (uint32_t *)(lds + a.o_lcnt);
  uint32_t *lhead = (uint32_t *)(lds + a.o_lhead);
  uint32_t *lfree = (uint32_t *)(lds + a.o_lfree);
  uint64_t *reach = (uint64_t *)(lds + a.o_reach);

  const int lane = threadIdx.x;
  const int C = a.C, P = a.P, V = a.V, E = a.E;
  const int CV = C * V;

  for (int64_t i = blockIdx.x; i < a.n; i += gridDim.x) {
    // ---- 1. stage the candidate --------------------------------------
    const uint8_t *grt = a.routes + (size_t)i * a.route_stride;
    const uint32_t *gpr = a.prio + (size_t)i * a.prio_stride;
    for (int j = lane; j < a.route_stride; j += 64) rt[j] = grt[j];
    for (int j = lane; j < CV; j += 64) {
      pr[j] = gpr[j];
      par[j] = 0;
      lds_put(&fin[j], kNotYet);
    }
    for (int l = lane; l <= E; l += 64) lcnt[l] = 0;
    __syncthreads();

    // ---- 2. lane = chunk: first-reach tree, distances, heights ----------
    for (int c = lane; c < C; c += 64) {
      const int o = a.cpr > 0 ? c / a.cpr : a.owner[c];
      const uint64_t pm = a.post_mask[c];
      const int base = c * V;
      uint64_t reached = 1ull << o;
      int cnt = 0;
      dist[base + o] = 0;
      for (int d = 0; d < P; d++) {
        if (d == o || !((pm >> d) & 1)) continue;
        const int pp = o * P + d;
        const int k = rt[c * P + d];
        if (k >= a.npaths[pp]) continue;  // pair left unrouted
        const uint32_t q = a.pair_base[pp] + k;
        for (uint32_t j = a.path_off[q]; j < a.path_off[q + 1]; j++) {
          const int l = a.path_links[j];
          const int v = a.ldst[l];
          if ((reached >> v) & 1) continue;
          reached |= 1ull << v;
          par[base + v] = (uint16_t)(l + 1);
          dist[base + v] = dist[base + a.lsrc[l]] + a.cost[l];
          ord[base + cnt++] = (uint16_t)v;
        }
      }
      reach[c] = reached;
      hgt[base + o] = 0;
      for (int j = 0; j < cnt; j++) hgt[base + ord[base + j]] = 0;
      // children are discovered after their parents: sweep backwards
      for (int j = cnt - 1; j >= 0; j--) {
        const int v = ord[base + j];
        const int l = par[base + v] - 1;
        const int u = a.lsrc[l];
        const uint32_t h = a.cost[l] + hgt[base + v];
        if (h > hgt[base + u]) hgt[base + u] = h;
      }
    }
    __syncthreads();

    // ---- 3. keys and per-link buckets ------------------------------------
    for (int s = lane; s < CV; s += 64) {
      const int pl = par[s];
      if (!pl) continue;
      const int l = pl - 1;
      const int c = s / V;
      krem[s] = a.cost[l] + hgt[s];
      ktrav[s] = dist[c * V + a.lsrc[l]];
      sidx[s] = (uint16_t)atomicAdd(&lcnt[l], 1u);
    }
    __syncthreads();
    {
      const int per = (E + 63) / 64;
      const int b = min(lane * per, E), e = min(b + per, E);
      uint32_t sum = 0;
      for (int j = b; j < e; j++) sum += lcnt[j];
      const uint32_t incl = wave_incl_scan(sum, lane);
      uint32_t run = incl - sum;
      for (int j = b; j < e; j++) {
        const uint32_t x = lcnt[j];
        lcnt[j] = run;
        run += x;
      }
      if (lane == 63) lcnt[E] = incl;
    }
    __syncthreads();
    for (int s = lane; s < CV; s += 64) {
      const int pl = par[s];
      if (pl) tmp[lcnt[pl - 1] + sidx[s]] = (uint16_t)s;
    }
    __syncthreads();
    // place every send in its link's order
    for (int s = lane; s < CV; s += 64) {
      const int pl = par[s];
      if (!pl) continue;
      const int l = pl - 1;
      const uint32_t b = lcnt[l], e = lcnt[l + 1];
      const uint32_t rx = krem[s], tx = ktrav[s], px = pr[s];
      uint32_t rank = 0;
      for (uint32_t j = b; j < e; j++) {
        const int y = tmp[j];
        const uint32_t ry = krem[y], ty = ktrav[y], py = pr[y];
        // every send on l enters the same vertex, so slot order = chunk order
        const bool before = ry > rx || (ry == rx && (ty < tx || (ty == tx && (py < px ||
                                                                             (py == px && y < s)))));
        rank += before;
      }
      chain[b + rank] = (uint16_t)s;
    }
    for (int l = lane; l < E; l += 64) {
      lhead[l] = lcnt[l];
      lfree[l] = 0;
    }
    __syncthreads();

    // ---- 4. least schedule: links advance through their orders -----------
    const uint32_t total = lcnt[E];
    uint32_t mk = 0;
    bool fault = false;
    for (uint32_t round = 0;; round++) {
      bool pending = false;
      for (int l = lane; l < E; l += 64) {
        uint32_t h = lhead[l];
        const uint32_t e = lcnt[l + 1];
        uint32_t f = lfree[l];
        const uint32_t cl = a.cost[l];
        const int u = a.lsrc[l];
        while (h < e) {
          const int s = chain[h];
          const int c = s / V;
          const int o = a.cpr > 0 ? c / a.cpr : a.owner[c];
          const uint32_t ready = (u == o) ? 0u : lds_get(&fin[c * V + u]);
          if (ready == kNotYet) break;
          f = max(ready, f) + cl;
          lds_put(&fin[s], f);
          h++;
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

    // ---- 5. postcondition and makespan -----------------------------------
    bool ok = true;
    for (int c = lane; c < C; c += 64) {
      const uint64_t pm = a.post_mask[c];
      ok &= (reach[c] & pm) == pm;
    }
    const bool all_ok = __ballot(!ok) == 0;
    mk = wave_max(mk);
    if (lane == 0) {
      a.makespan[i] = fault ? 0xFFFFFFFFu : mk;
      a.valid[i] = (uint8_t)(all_ok && !fault);
    }
    __syncthreads();
  }
}

int32_t align16(int32_t x) { return (x + 15) & ~15; }

}  // namespace

int32_t tree_layout(const taccl_plan &p, TreeArgs &a) {
  const int32_t C = p.coll.C, V = p.topo.V, E = p.topo.E;
  const int32_t CV = C * V;
  int32_t off = 0;
  auto take = [&](int32_t bytes) {
    int32_t o = off;
    off = align16(off + bytes);
    return o;
  };
  a.o_rt = take(p.route_stride);
  a.o_pr = take(4 * CV);
  a.o_par = take(2 * CV);
  a.o_dist = take(4 * CV);
  a.o_hgt = take(4 * CV);
  a.o_fin = take(4 * CV);
  a.o_ord = take(2 * CV);
  a.o_sidx = take(2 * CV);
  a.o_tmp = take(2 * CV);
  a.o_chain = take(2 * CV);
  a.o_krem = take(4 * CV);
  a.o_ktrav = take(4 * CV);
  a.o_lcnt = take(4 * (E + 1));
  a.o_lhead = take(4 * E);
  a.o_lfree = take(4 * E);
  a.o_reach = take(8 * C);
  a.lds_bytes = off;
  return off;
}

hipError_t launch_tree(const TreeArgs &a, int grid, hipStream_t stream) {
  hipLaunchKernelGGL(tree_eval_kernel, dim3(grid), dim3(kTreeThreads), a.lds_bytes, stream, a);
  return hipGetLastError();
}

}  // namespace taccl
