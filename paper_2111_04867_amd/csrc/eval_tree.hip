// Multicast (Allgather / explicit) evaluation kernel for gfx950.
//
// Persistent blocks of several wavefronts. Each block copies the plan's
// route records and link costs into LDS once; each wavefront then evaluates
// one candidate at a time, its state in LDS, while the next candidate's
// routes and priorities stream from HBM into registers:
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

#include "kernels.h"

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

// n / V for n, V < 2^16 with a precomputed m = floor(2^32 / V) + 1
__device__ __forceinline__ uint32_t div_v(uint32_t n, uint32_t m) {
  return (uint32_t)(((uint64_t)n * m) >> 32);
}

// kRecLds: the route records fit in LDS (else they are read from global
// memory, where they stay cache resident). kPrefetch: a candidate's routes
// (whole words) and priorities fit the prefetch registers.
template <bool kRecLds, bool kPrefetch>
__global__ __launch_bounds__(kTreeMaxThreads) void tree_eval_kernel(TreeArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int C = a.C, P = a.P, V = a.V, E = a.E, K = a.K, H = a.H, MW = a.mask_words;
  const int CV = C * V;

  // ---- block-wide copy of the plan tables --------------------------------
  uint32_t *s_cost = (uint32_t *)(lds + a.o_cost);
  uint8_t *s_src = lds + a.o_src;
  uint8_t *s_own = lds + a.o_own;
  uint64_t *s_post = (uint64_t *)(lds + a.o_post);
  const uint32_t *s_rec = kRecLds ? (const uint32_t *)(lds + a.o_rec) : a.rec;
  for (int j = threadIdx.x; j < E; j += blockDim.x) {
    s_cost[j] = a.cost[j];
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
  uint32_t *dh = (uint32_t *)key;  // dh[2s] = dist, dh[2s+1] = height
  uint32_t *prio = (uint32_t *)(wl + a.w_prio);
  uint32_t *fin = prio;
  uint32_t *chain = (uint32_t *)(wl + a.w_chain);
  uint32_t *ord = chain;
  uint16_t *par = (uint16_t *)(wl + a.w_par);     // link+1 into (c,v), 0 = none
  uint32_t *lmask = (uint32_t *)(wl + a.w_mask);  // [E][MW] chunk bits per link
  uint32_t *lbase = (uint32_t *)(wl + a.w_base);  // [E+1]
  uint32_t *lhead = (uint32_t *)(wl + a.w_head);  // [E]
  uint32_t *lfree = (uint32_t *)(wl + a.w_free);  // [E]

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
    wave_sync();

    // ---- 2+3. lane = chunk: first-reach tree, then heights and keys -------
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
        const uint32_t rem = s_cost[l] + dh[2 * (base + v) + 1];
        const uint32_t trav = dh[2 * (base + u)];
        if (rem > dh[2 * (base + u) + 1]) dh[2 * (base + u) + 1] = rem;
        key[base + v] = ((uint64_t)(~rem) << 32) | trav;  // ascending = rem desc, trav asc
        atomicOr(&lmask[l * MW + (c >> 5)], 1u << (c & 31));
      }
    }
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
    for (int s = lane; s < CV; s += 64) lds_put(&fin[s], kNotYet);
    wave_sync();

    // ---- 5. least schedule: links advance through their orders -----------
    const uint32_t total = lbase[E];
    uint32_t mk = 0;
    bool fault = false;
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

    // ---- 6. postcondition and makespan -----------------------------------
    const bool all_ok = __ballot(!ok) == 0;
    mk = wave_max(mk);
    if (lane == 0) {
      a.makespan[i] = fault ? 0xFFFFFFFFu : mk;
      a.valid[i] = (uint8_t)(all_ok && !fault);
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

int32_t tree_block_bytes(const TreeArgs &a, int waves) { return a.o_wave + waves * a.wave_bytes; }

hipError_t launch_tree(const TreeArgs &a, int grid, hipStream_t stream) {
  const bool pf = a.routes_word_aligned && a.route_stride <= 4 * 64 * kPfRoute &&
                  a.C * a.V <= 64 * kPfPrio;
  const dim3 g(grid), b(64 * a.waves_per_block);
  const int bytes = tree_block_bytes(a, a.waves_per_block);
  if (a.rec_in_lds && pf)
    hipLaunchKernelGGL((tree_eval_kernel<true, true>), g, b, bytes, stream, a);
  else if (a.rec_in_lds)
    hipLaunchKernelGGL((tree_eval_kernel<true, false>), g, b, bytes, stream, a);
  else if (pf)
    hipLaunchKernelGGL((tree_eval_kernel<false, true>), g, b, bytes, stream, a);
  else
    hipLaunchKernelGGL((tree_eval_kernel<false, false>), g, b, bytes, stream, a);
  return hipGetLastError();
}

}  // namespace taccl
