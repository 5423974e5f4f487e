// Ranked multicast kernel for gfx950: Allgather and explicit multicast with
// the static Step-2 order, one chunk per transfer or contiguous transfers on
// links between nodes (Step 3, Sec. 4.1; also the Allgather phase of an
// Allreduce), for plans whose tree-path lengths take few distinct values.
//
// One wavefront evaluates one candidate at a time (persistent blocks of
// several wavefronts, the next candidate's routes and priorities streaming
// into registers meanwhile), one lane per (chunk c, vertex v) slot:
//   1. trees: the send into v comes from the path of the smallest
//      destination whose drawn route passes v (first-reach merge of the
//      chunk's routes, destinations ascending: one is_sent per chunk and
//      link, App. B.1); found from the one-hot route bytes and per-vertex
//      option bytes, the entering link from a plan table;
//   2. distances and heights together, by doubling over ancestors: in
//      round k every slot reads its 2^k-th ancestor's pointer and distance
//      and pushes the largest depth it knows below itself up to that
//      ancestor, so ceil(log2 V) rounds give every distance from the owner
//      (the travelled length of Sec. 5.1) and every tree height (the
//      remaining length is the link's cost plus the height below v);
//   3. keys: both lengths are sums of at most V - 1 link costs, and a plan
//      constant maps every such sum to an exact 11-bit code that preserves
//      order, so one 64-bit word (remaining code descending, travelled code
//      ascending, priority, slot) orders a link's sends exactly as the
//      Step-2 rule (remaining desc, travelled asc, priority, chunk);
//   4. layers: layer = floor(rem / c_min); a parent send's remaining length
//      exceeds its child's by at least one link cost, so parents lie in
//      higher layers and every dependency inside a layer runs along a link.
//      Counting sort by (layer from the top, link), then each send's rank
//      in its bucket by 64-bit compares against the bucket's members;
//   5. timing layer by layer: the k-th send of a link run with ready times
//      r_j, cost c and link busy time F finishes at
//      (k+1)c + max(F, max_{j<=k}(r_j - jc)) (App. B.3 unrolled), a
//      segmented prefix maximum over the layer's positions (DPP scans inside
//      the wavefront with only the steps the longest run needs);
//   6. postcondition (ballot) and makespan (wave maximum).
// With contiguous transfers, a run on a link between nodes is walked by its
// first lane instead: a send joins the open transfer when its remaining
// length equals the previous send's and its chunk was ready when the
// transfer started; a transfer of g sends takes alpha + ceil(beta bytes g /
// 1000) and all its sends finish together.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "kernels.h"
#include "wave.h"

namespace taccl {

namespace {

constexpr uint32_t kNone = 0xFFFFu;
constexpr int kPfRouteWords = 4;  // route words per lane (route_stride <= 1 KiB)

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_wave_barrier();
  asm volatile("" ::: "memory");
}

// The larger of v and the value of the lane `Ctrl` selects through DPP; a
// lane without one (an out-of-row source, or a row the mask leaves out)
// keeps v (the DPP source reads as 0 there and every value is unsigned), so
// no value from outside the pattern is mixed in. One v_max with a DPP
// operand.
template <int Ctrl, int RowMask = 0xf>
__device__ __forceinline__ uint32_t max_dpp(uint32_t v) {
  return max(v, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, Ctrl, RowMask, 0xf, true));
}

// Route word j (route bytes of chunk j / PW) as one-hot option bytes:
// 1 << choice, 0 for a choice of 8 or more (no pair of these plans has as
// many options, so such a choice leaves the pair unrouted) and 0 for a
// destination outside the chunk's postcondition (never routed).
template <int PW>
__device__ __forceinline__ uint32_t one_hot(uint32_t w, uint32_t j, const uint64_t *s_post) {
  const uint32_t pm4 = (uint32_t)(s_post[j / PW] >> (4 * (j % PW))) & 0xFu;
  uint32_t oh = 0;
#pragma unroll
  for (int b = 0; b < 4; b++) {
    const uint32_t kb = (w >> (8 * b)) & 0xFFu;
    oh |= ((kb < 8 && ((pm4 >> b) & 1)) ? (1u << kb) : 0u) << (8 * b);
  }
  return oh;
}

// kC: contiguous transfers; kR: ReduceScatter (the trees run backwards: a
// send v -> u on the reverse of the link into v, costs of the reverse links,
// remaining length = reversed distance from v to the owner, travelled
// length = longest reversed path from below up to v; a send is ready when
// every send into v has finished)
template <int J, int PW, bool kC, bool kR>
__global__ __launch_bounds__(kRankMaxThreads) void tree_rank_kernel(TreeArgs a) {
  static_assert(!(kC && kR), "contiguous transfers are not combined with ReduceScatter here");
  extern __shared__ __align__(16) unsigned char lds[];
  const int C = a.C, V = a.V, E = a.E, K = a.K;
  constexpr int P = 4 * PW;
  const int CV = C * V;

  uint32_t *s_cost = (uint32_t *)(lds + a.o_cost);
  uint8_t *s_src = lds + a.o_src;
  uint8_t *s_merge = lds + a.o_merge;  // links that carry contiguous transfers
  uint64_t *s_post = (uint64_t *)(lds + a.o_post);
  // option bytes of (o, v), word w, at (o * PW + w) * V + v plus a pad per
  // owner, so that the 16 lanes of a row (one chunk, consecutive vertices)
  // read 16 banks and two owners fall on different halves
  uint32_t *s_opt = (uint32_t *)(lds + a.o_opt);
  uint8_t *s_ent = lds + a.o_ent;  // entering link per (o, v, d, k)
  // per slot: entering-link table base | chunk's first slot << 20 | root <<
  // 30 | in the postcondition << 31, and option base | route word base << 16
  // | owner << 24
  uint2 *s_slot = (uint2 *)(lds + a.o_slot);
  const int OS = a.opt_ostride;
  for (int j = threadIdx.x; j < E; j += blockDim.x) {
    // ReduceScatter: every link's entry holds its reverse's cost (a tree
    // link always has a reverse, checked at plan time)
    s_cost[j] = kR ? a.cost[a.lrev[j] != 0xFFFFu ? a.lrev[j] : j] : a.cost[j];
    s_src[j] = (uint8_t)a.lsrc[j];
    if (kC) s_merge[j] = a.lmerge[j];
  }
  for (int j = threadIdx.x; j < P * V * PW; j += blockDim.x) {
    const int w = j % PW, ov = j / PW, o = ov / V, v = ov - o * V;
    s_opt[o * OS + w * V + v] = ((const uint32_t *)a.topt)[j];
  }
  for (int j = threadIdx.x; j < P * V * P * K; j += blockDim.x) s_ent[j] = a.ent[j];
  for (int j = threadIdx.x; j < C; j += blockDim.x) {
    s_post[j] = a.post_mask[j];
  }
  for (int j = threadIdx.x; j < CV; j += blockDim.x) {
    const int c = j / V, v = j - c * V, o = a.owner8[c];
    const uint32_t post = (uint32_t)((a.post_mask[c] >> v) & 1);
    s_slot[j] = make_uint2((uint32_t)((o * V + v) * P * K) | ((uint32_t)(c * V) << 20) |
                               ((uint32_t)(v == o) << 30) | (post << 31),
                           (uint32_t)(o * OS + v) | ((uint32_t)(c * PW) << 16) |
                               ((uint32_t)o << 24));
  }
  __syncthreads();

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  unsigned char *wl = lds + a.o_wave + wave * a.wave_bytes;
  // Region A: one-hot routes, distances, ancestors and heights per slot;
  // then the bucket counters; then bucket entries, bounds and parent sends
  // per position; then finish times per slot. Region B: the ordered sends.
  // (distance, ancestor) and height per slot are padded to 64 J slots, so
  // lanes past the last slot store without a guard
  uint32_t *rt32 = (uint32_t *)wl;
  uint2 *da = (uint2 *)(wl + a.w_dist);
  uint32_t *hgt = (uint32_t *)(wl + a.w_h);
  uint32_t *cnt = (uint32_t *)wl;
  uint64_t *erec = (uint64_t *)wl;
  uint32_t *bnd = (uint32_t *)(wl + a.w_bnd);
  uint16_t *pjs = (uint16_t *)(wl + a.w_pj);  // parent send per position
  uint32_t *fin = (uint32_t *)wl;
  uint32_t *rq = (uint32_t *)(wl + a.w_rq);  // ready times per position (contiguity)
  uint32_t *ord = (uint32_t *)(wl + a.w_ord2);
  uint32_t *info = (uint32_t *)(wl + a.w_info2);
  uint32_t *lfree = (uint32_t *)(wl + a.w_free);
  uint64_t *lmask64 = (uint64_t *)(wl + a.w_lmask);
  uint32_t *lst = (uint32_t *)(wl + a.w_lst);  // first ordered position of each layer
  auto start_of = [&](uint32_t b) -> uint32_t {
    return (cnt[b >> 1] >> ((b & 1) << 4)) & 0xFFFFu;
  };

  const int64_t stride = (int64_t)gridDim.x * a.waves_per_block;
  const int64_t first = (int64_t)blockIdx.x * a.waves_per_block + wave;
  const int nrw = a.route_stride >> 2;
  // The next candidate's route words are loaded as soon as this one's are
  // staged, and its priorities as soon as this one's are folded into keys,
  // so both arrive while this candidate is evaluated and only one set of
  // each is held at a time.
  uint32_t pf_r[kPfRouteWords], px[J];
  auto load_routes = [&](int64_t i, int ln) {
    if (i >= a.n) return;
    const uint32_t *g32 = (const uint32_t *)(a.routes + (size_t)i * a.route_stride);
#pragma unroll
    for (int k = 0; k < kPfRouteWords; k++) {
      const int j = ln + 64 * k;
      if (j < nrw) pf_r[k] = __builtin_nontemporal_load(g32 + j);
    }
  };
  auto load_prio = [&](int64_t i, int ln) {
    if (i >= a.n) return;
    const uint32_t *gpr = a.prio + (size_t)i * a.prio_stride;
#pragma unroll
    for (int k = 0; k < J; k++) {
      const int j = ln + 64 * k;
      if (j < CV) px[k] = __builtin_nontemporal_load(gpr + j);
    }
  };
  // per-lane constants of the cross-row steps of the segmented scans: a
  // lane of rows 1 and 3 takes the previous row's last lane when its run
  // reaches back that far, a lane of rows 2 and 3 takes lane 31 likewise
  const uint32_t reach15 = (lane & 16) ? (uint32_t)(lane & 15) + 1 : 0xFFFFu;
  const uint32_t reach31 = lane >= 32 ? (uint32_t)lane - 31 : 0xFFFFu;
  const int R = a.pj_rounds;

  load_routes(first, lane);
  load_prio(first, lane);
  for (int64_t i = first; i < a.n; i += stride) {
    // The lane index is hidden from the optimiser once per candidate, so
    // per-slot LDS addresses are recomputed where used instead of being
    // hoisted out of the loop into registers.
    int lane = threadIdx.x & 63;
    asm volatile("" : "+v"(lane));
    // ---- stage: one-hot routes to LDS ------------------------------------
#pragma unroll
    for (int k = 0; k < kPfRouteWords; k++) {
      const int j = lane + 64 * k;
      if (j < nrw) rt32[j] = one_hot<PW>(pf_r[k], j, s_post);
    }
    load_routes(i + stride, lane);
    for (int l = lane; l < E; l += 64) lfree[l] = 0;
    if (lane == 0) *lmask64 = 0;
    wave_sync();

    // ---- trees: the hop into every reached (chunk, vertex) slot ------------
    // pl: link | parent vertex << 8 | owner vertex << 14 | the owner's slot
    // << 20 for a slot with a send (V <= 64, C * V <= 1024), ~0 otherwise;
    // an / acc: the slot's 2^k-th ancestor and the cost of the path up to it
    uint32_t pl[J], an[J], acc[J];
    uint32_t bad = 0, fault = 0;
#pragma unroll
    for (int g0 = 0; g0 < J; g0 += 2) {
      constexpr int G = J < 2 ? J : 2;
      uint32_t slc[G], pos[G];
      uint2 si[G];
#pragma unroll
      for (int q = 0; q < G; q++) {
        const uint32_t sl = lane + 64 * (g0 + q);
        slc[q] = sl < (uint32_t)CV ? sl : 0u;
        si[q] = s_slot[slc[q]];
      }
      // (chosen option bit & options through v), one byte per destination:
      // its lowest set bit, over the words in destination order, is byte
      // 4w + b of the smallest destination d whose drawn route passes v,
      // and the bit inside the byte is that route's option kd (all ones when
      // no word has a set bit; a later word's bits all lie above an earlier
      // word's, so the minimum over the words that have one is the first)
#pragma unroll
      for (int q = 0; q < G; q++) {
        const uint32_t ob = si[q].y & 0xFFFFu, rb = (si[q].y >> 16) & 0xFFu;
        uint32_t best = ~0u;
#pragma unroll
        for (int w = 0; w < PW; w++) {
          const uint32_t t = rt32[rb + w] & s_opt[ob + w * V];
          // lowest set bit, all ones for none (v_ffbl_b32 gives that for
          // 0; written as an instruction, so the compiler does not turn the
          // minimum back into compares and selects), then the word's
          // offset (all ones stay all ones)
          uint32_t f;
          asm("v_ffbl_b32 %0, %1" : "=v"(f) : "v"(t));
          best = min(best, f | (32u * w));
        }
        pos[q] = best;
      }
      uint32_t l[G];
#pragma unroll
      for (int q = 0; q < G; q++) {
        // a slot with a send: in range, not the owner, and some route
        // passes it; a rank of the postcondition without one is never reached
        const uint32_t in = (lane + 64 * (g0 + q) < (uint32_t)CV) ? 1u : 0u;
        const uint32_t live = in & ~(si[q].x >> 30) & 1u;
        const uint32_t has = live & (pos[q] != ~0u ? 1u : 0u);
        bad |= live & ~has & (si[q].x >> 31);
        const uint32_t d = pos[q] >> 3, kd = pos[q] & 7;
        // entry 0 for a slot without a send (a mask, not a select, so that
        // no lane-masked block is formed here); read for every lane (the
        // empty asm keeps the compiler from moving the read into a branch of
        // its own), then selected
        // 24-bit multiplies (d < 64, K <= 8) issue at the full VALU rate
        const uint32_t ei = ((si[q].x & 0xFFFFFu) + __umul24(d, (uint32_t)K) + kd) & (0u - has);
        uint32_t le = s_ent[ei];
        asm volatile("" : "+v"(le));
        l[q] = has ? le : 0xFFu;
        pos[q] = has;
      }
#pragma unroll
      for (int q = 0; q < G; q++) {
        const int jj = g0 + q;
        const bool has = pos[q] != 0;
        const uint32_t lq = l[q] < (uint32_t)E ? l[q] : 0u;
        fault |= has && l[q] >= (uint32_t)E;  // unreachable: the option passes v
        uint32_t u = s_src[lq], ec = s_cost[lq];
        asm volatile("" : "+v"(u), "+v"(ec));
        const uint32_t cbase = (si[q].x >> 20) & 0x3FFu;
        const uint32_t sl = lane + 64 * jj;
        const uint32_t own = si[q].y >> 24;
        pl[jj] = has ? (lq | (u << 8) | (own << 14) | ((cbase + own) << 20)) : ~0u;
        // the owner's slot (and a slot without a send, or past the last
        // slot) is its own ancestor, at distance 0
        an[jj] = has ? cbase + u : sl;
        acc[jj] = has ? ec : 0u;
        da[sl] = make_uint2(acc[jj], an[jj]);
        hgt[sl] = 0;
      }
    }
    wave_sync();
    // ---- distances and heights by doubling over ancestors -----------------
    // Before round k a slot knows its 2^k-th ancestor an and the cost acc of
    // the path up to it, and hgt[slot] is the largest distance down to a
    // descendant fewer than 2^k links below. The slot pushes hgt + acc to
    // its 2^k-th ancestor (so that one learns descendants fewer than 2^(k+1)
    // links below) and then doubles. Values only grow and each is a real
    // descendant's depth, so reading one that another push already raised
    // is harmless. Once every slot's ancestor is its chunk's owner (no tree
    // is 2^k links deep), distances and heights are complete.
    for (int k = 0; k < R; k++) {
      uint32_t ra[J], rn[J], hv[J];
      uint32_t open = 0;
#pragma unroll
      for (int j = 0; j < J; j++) {
        const uint2 r = da[an[j]];
        ra[j] = r.x;
        rn[j] = r.y;
        hv[j] = hgt[lane + 64 * j];
        open |= (pl[j] != ~0u && an[j] != (pl[j] >> 20)) ? 1u : 0u;
      }
      if (__ballot(open) == 0) break;
      wave_sync();
#pragma unroll
      for (int j = 0; j < J; j++) {
        const uint32_t sl = lane + 64 * j;
        // no push into the owner's slot: it has no send and its height is
        // never read, and every chain ends there, so the pushes of a whole
        // chunk would queue on one LDS word
        if (pl[j] != ~0u && an[j] != (pl[j] >> 20)) atomicMax(&hgt[an[j]], hv[j] + acc[j]);
        acc[j] += ra[j];
        an[j] = rn[j];
        da[sl] = make_uint2(acc[j], an[j]);
      }
      wave_sync();
    }
    wave_sync();

    // ---- keys and layers -----------------------------------------------
    // trav = dist(u) = dist(v) - cost, rem = cost + height(v); the key
    // orders (rem desc, trav asc, priority, slot); within a link every send
    // enters the same vertex, so slot order is chunk order
    // link | layer << 8 | parent send << 16 (the parent vertex's slot, kNone
    // when the parent is the owner), or ~0 for no send
    uint32_t bl[J];
    uint64_t key[J];
    uint64_t lm = 0;
    {
      uint32_t hh[J], cl[J];
#pragma unroll
      for (int j = 0; j < J; j++) {
        hh[j] = hgt[lane + 64 * j];
        cl[j] = s_cost[pl[j] != ~0u ? pl[j] & 0xFFu : 0u];
      }
      const uint32_t top = (uint32_t)a.qrange - 1;
      const uint32_t lmag = (uint32_t)a.lmagic, qmag = (uint32_t)a.qmagic;
#pragma unroll
      for (int j = 0; j < J; j++) {
        bl[j] = ~0u;
        key[j] = 0;
        if (pl[j] != ~0u) {
          const uint32_t trav = kR ? hh[j] : acc[j] - cl[j];
          const uint32_t rem = kR ? acc[j] : cl[j] + hh[j];
          uint32_t L = __umulhi(rem, lmag);
          const uint32_t rq = __umulhi(rem, qmag);
          const uint32_t tq = __umulhi(trav, qmag);
          if (L >= (uint32_t)a.nl_max || rq > top || tq > top) {  // unreachable (plan bounds)
            L = 0;
            fault = 1;
          }
          const uint32_t u = (pl[j] >> 8) & 63u, own = (pl[j] >> 14) & 63u;
          const uint32_t pjs_v = u == own ? kNone : (pl[j] >> 20) - own + u;
          bl[j] = (pl[j] & 0xFFu) | (L << 8) | (pjs_v << 16);
          const uint32_t hi = ((top - rq) << 21) | (tq << 10) | (px[j] >> 22);
          const uint32_t lo = (px[j] << 10) | (uint32_t)(lane + 64 * j);
          key[j] = ((uint64_t)hi << 32) | lo;
          lm |= 1ull << L;
        }
      }
    }
    load_prio(i + stride, lane);  // this candidate's priorities are in the keys
    if (lm) atomicOr((unsigned long long *)lmask64, (unsigned long long)lm);
    wave_sync();  // also: every read of the tree arrays is done
    const uint64_t layers = *lmask64;
    const int nl = __popcll(layers);
    const uint32_t NB = (uint32_t)nl * E;  // buckets (layer from the top, link)
    const int NW = (int)((NB + 2) >> 1);   // u16 counters for NB + 1 starts
    for (int w = lane; w < NW + 64; w += 64) cnt[w] = 0;
    wave_sync();

    // ---- counting sort by (layer from the top, link) ---------------------
    // a slot without a send counts in a per-lane dummy word past the
    // counters, so every slot issues its update without a branch
    uint32_t bb[J], idx[J];
#pragma unroll
    for (int k = 0; k < J; k++) {
      const bool has = bl[k] != ~0u;
      const uint32_t L = (bl[k] >> 8) & 63u;
      const uint32_t above = (uint32_t)__popcll((layers >> L) >> 1);
      const uint32_t b = __umul24(above, (uint32_t)E) + (bl[k] & 0xFFu);
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
      const uint32_t incl = wave_scan_add(sum);
      uint32_t run = incl - sum;
      for (int w = w0; w < w1; w++) {
        const uint32_t x = cnt[w];
        const uint32_t lo = x & 0xFFFFu;
        cnt[w] = run | ((run + lo) << 16);
        run += lo + (x >> 16);
      }
    }
    wave_sync();
    // a bucket's start and end: two neighbouring u16 counters, read as the
    // two words that hold them (one LDS read of a word pair)
    uint32_t b0[J], b1[J];
#pragma unroll
    for (int k = 0; k < J; k++) {
      const uint32_t w = bb[k] >> 1, x0 = cnt[w], x1 = cnt[w + 1];
      const bool odd = (bb[k] & 1) != 0;
      b0[k] = odd ? x0 >> 16 : x0 & 0xFFFFu;
      b1[k] = odd ? x1 & 0xFFFFu : x0 >> 16;
    }
    for (int ly = lane; ly <= nl; ly += 64) lst[ly] = start_of((uint32_t)ly * E);
    wave_sync();  // the counters are dead from here on (entries overwrite them)
#pragma unroll
    for (int k = 0; k < J; k++)
      if (bl[k] != ~0u) {
        const uint32_t pos = b0[k] + idx[k];
        erec[pos] = key[k];
        bnd[pos] = b0[k] | (b1[k] << 10) | ((bl[k] & 0xFFu) << 20);
        pjs[pos] = (uint16_t)(bl[k] >> 16);
      }
    wave_sync();

    // ---- rank inside each bucket -----------------------------------------
    // one lane per ordered position; the entry array has three spare
    // entries past its end, so four members load without clamping (entries
    // past the bucket never count)
    // The next pass's entry, bounds and parent send are loaded while this
    // pass ranks, so a pass waits only for its bucket's members.
    const uint32_t total = lst[nl];
    uint64_t kx_n = 0;
    uint32_t bd_n = 0, pj_n = 0;
    if (total > 0) {
      const uint32_t x0 = min((uint32_t)lane, total - 1u);
      kx_n = erec[x0];
      bd_n = bnd[x0];
      pj_n = pjs[x0];
    }
    for (uint32_t x = lane; x < total; x += 64) {
      const uint64_t kx = kx_n;
      const uint32_t bd = bd_n, pred = pj_n;
      {
        const uint32_t xn = min(x + 64u, total - 1u);
        kx_n = erec[xn];
        bd_n = bnd[xn];
        pj_n = pjs[xn];
      }
      const uint32_t bs = bd & 0x3FFu, be = (bd >> 10) & 0x3FFu, l = bd >> 20;
      const uint32_t sl = (uint32_t)kx & 0x3FFu;
      uint32_t rank = 0, same = 0;
      for (uint32_t y = bs; y < be; y += 4) {
        uint64_t m[4];
#pragma unroll
        for (int t = 0; t < 4; t++) m[t] = erec[y + t];
#pragma unroll
        for (int t = 0; t < 4; t++) {
          const uint32_t before = (uint32_t)((y + t < be) & (m[t] < kx));
          rank += before;
          // an earlier send of the bucket with the same remaining length
          // (the code in the key's top 11 bits; equal lengths sort next to
          // each other)
          if (kC) same |= before & (uint32_t)((m[t] >> 53) == (kx >> 53));
        }
      }
      const uint32_t q = bs + rank;
      ord[q] = sl | (pred << 16);
      // link | index in the run << 16 | same remaining length as the
      // previous send << 30 | the run's last send << 31
      info[q] = l | (rank << 16) | (same << 30) | ((uint32_t)(rank + 1 == be - bs) << 31);
    }
    wave_sync();

    // ---- least schedule, layer by layer ----------------------------------
    // a_j = max(r_0, F) for the run's first send, max(r_j - j c, 0) after
    // it (F >= 0 dominates the clipped values), and f_k = (k+1)c + max_{j<=k}
    // a_j: a prefix maximum segmented by runs, which are contiguous (runs
    // are buckets). kk = how many earlier sends of the lane's run lie in
    // this pass of 64 positions; the scan takes only the steps some lane
    // needs.
    // The ordered sends of the next pass (the layer's next 64 positions, or
    // the next layer's first) are loaded while the current pass is timed, so
    // a pass waits for one round of LDS reads (ready time, cost, busy time);
    // layer starts come from a register (lane ly holds layer ly's).
    if (kR) {  // ready times start at 0 and are raised by the inputs
      for (int j = lane; j < CV; j += 64) fin[j] = 0;
      wave_sync();
    }
    uint32_t mk = 0;
    const uint32_t lst_r = lane < nl ? lst[lane] : total;
    auto layer_start = [&](int ly) -> uint32_t {
      return ly < nl ? (uint32_t)__builtin_amdgcn_readlane((int)lst_r, ly) : total;
    };
    uint32_t e_n = 0, inf_n = 0;
    auto prefetch = [&](uint32_t start) {  // positions past the end: the last one
      const uint32_t q = min(start + (uint32_t)lane, total - 1u);
      e_n = ord[q];
      inf_n = info[q];
    };
    if (nl > 0) prefetch(0);
    for (int ly = 0; ly < nl; ly++) {
      const uint32_t qs = layer_start(ly), qe = layer_start(ly + 1);
      if (kC) {
        // ready times of the layer's sends, for the walkers below (parent
        // sends lie in layers above)
        for (uint32_t q = qs + lane; q < qe; q += 64) {
          const uint32_t pj = ord[q] >> 16;
          rq[q] = pj == kNone ? 0u : fin[pj];
        }
        wave_sync();
      }
      uint32_t carry = 0;
      for (uint32_t base = qs; base < qe; base += 64) {
        const uint32_t q = base + lane;
        const bool ok = q < qe;
        // a lane past the layer holds a valid send of a later one: its link
        // and parent index valid reads, and it neither counts nor writes
        const uint32_t e = e_n, inf = inf_n;
        prefetch(min(base + 64u, qe));
        const uint32_t l = inf & 0xFFFFu, k = ok ? (inf >> 16) & 0x3FFFu : 0u;
        const uint32_t pj = e >> 16;
        // Allgather: the finish of the send that brings the chunk;
        // ReduceScatter: the slot's own ready time, raised by its inputs
        uint32_t r0 = fin[kR ? e & 0xFFFFu : (pj == kNone ? 0u : pj)];
        uint32_t c = s_cost[l], F = lfree[l];
        // all three reads issued together (the compiler would otherwise
        // move the busy time's into the branch of a run's first send)
        asm volatile("" : "+v"(r0), "+v"(c), "+v"(F));
        const uint32_t r = (!kR && pj == kNone) ? 0u : r0;
        const uint32_t kc = __umul24(k, c);  // k < 2^15, c < 2^24 (plan bound)
        uint32_t v = k == 0 ? max(r, F) : (r > kc ? r - kc : 0u);
        if (!ok) v = 0;
        const uint32_t kk = min(k, (uint32_t)lane);
        {
          const bool c1 = kk >= 1;
          if (__ballot(c1)) {
            const uint32_t t1 = max_dpp<kRowShr + 1>(v);
            v = c1 ? t1 : v;
            const bool c2 = kk >= 2;
            if (__ballot(c2)) {
              const uint32_t t2 = max_dpp<kRowShr + 2>(v);
              v = c2 ? t2 : v;
              const bool c4 = kk >= 4;
              if (__ballot(c4)) {
                const uint32_t t4 = max_dpp<kRowShr + 4>(v);
                v = c4 ? t4 : v;
                const bool c8 = kk >= 8;
                if (__ballot(c8)) {
                  const uint32_t t8 = max_dpp<kRowShr + 8>(v);
                  v = c8 ? t8 : v;
                }
              }
            }
            // runs that reach back across a row boundary
            const bool x15 = kk >= reach15;
            if (__ballot(x15)) {
              const uint32_t t15 = max_dpp<kBcast15, 0xa>(v);
              v = x15 ? t15 : v;
            }
            const bool x31 = kk >= reach31;
            if (__ballot(x31)) {
              const uint32_t t31 = max_dpp<kBcast31, 0xc>(v);
              v = x31 ? t31 : v;
            }
          }
        }
        // runs that began in an earlier pass of this layer
        if (k > (uint32_t)lane) v = max(v, carry);
        carry = (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
        const uint32_t f = kc + c + v;
        const bool merge = kC && s_merge[l] != 0;
        if (ok && !merge) {
          if (kR) {  // the send out of u waits for this one
            if (pj != kNone) atomicMax(&fin[pj], f);
          } else {
            fin[e & 0xFFFFu] = f;
          }
          mk = max(mk, f);
          if (inf >> 31) lfree[l] = f;  // the run's last send
        }
        if (kC && ok && merge && k == 0) {
          // contiguous transfers: the run's first lane walks the run; a send
          // joins the open transfer when its remaining length equals the
          // previous send's and its chunk was ready when the transfer
          // started, and a transfer of g sends takes alpha + ceil(beta
          // bytes g / 1000)
          const uint32_t al = a.lalpha[l];
          const uint64_t bsz = a.lbs[l];
          uint32_t Fw = F, gs = 0, gm = 0, g0 = q;
          for (uint32_t j = q;; j++) {
            const uint32_t ij = info[min(j, qe - 1u)];
            const bool end = j >= qe || (j > q && ((ij >> 16) & 0x3FFFu) == 0);
            const uint32_t rj = end ? 0u : rq[j];
            const bool join = !end && gm > 0 && (ij >> 30 & 1u) && rj <= gs;
            if (gm > 0 && !join) {  // close the open transfer
              const uint32_t fw = gs + al + (uint32_t)((bsz * gm + 999) / 1000);
              for (uint32_t t = g0; t < g0 + gm; t++) fin[ord[t] & 0xFFFFu] = fw;
              Fw = fw;
              mk = max(mk, fw);
            }
            if (end) break;
            if (join) {
              gm++;
            } else {
              gs = max(Fw, rj);
              gm = 1;
              g0 = j;
            }
          }
          lfree[l] = Fw;
        }
      }
      wave_sync();
    }

    // ---- postcondition and makespan ---------------------------------------
    const bool all_ok = __ballot(bad != 0) == 0;
    const bool failed = __ballot(fault != 0) != 0;
    mk = wave_reduce_max(mk);
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

template <int J, bool kC, bool kR>
const void *rank_fn_jc(int pw) {
  switch (pw) {
    case 1: return (const void *)tree_rank_kernel<J, 1, kC, kR>;
    case 2: return (const void *)tree_rank_kernel<J, 2, kC, kR>;
    case 3: return (const void *)tree_rank_kernel<J, 3, kC, kR>;
    case 4: return (const void *)tree_rank_kernel<J, 4, kC, kR>;
    case 6: return (const void *)tree_rank_kernel<J, 6, kC, kR>;
    default: return (const void *)tree_rank_kernel<J, 8, kC, kR>;
  }
}

// ReduceScatter never runs with contiguous transfers here
template <int J>
const void *rank_fn_j(int pw, bool contig, bool reduce) {
  if (reduce) return rank_fn_jc<J, false, true>(pw);
  return contig ? rank_fn_jc<J, true, false>(pw) : rank_fn_jc<J, false, false>(pw);
}

// slots per lane of the instantiation that runs C * V <= 512 slots
int rank_slots_per_lane(int cv) {
  const int j = (cv + 63) / 64;
  return j <= 1 ? 1 : j <= 2 ? 2 : j <= 4 ? 4 : 8;
}

const void *rank_fn(const TreeArgs &a) {
  const int pw = a.P / 4;
  switch (rank_slots_per_lane(a.C * a.V)) {
    case 1: return rank_fn_j<1>(pw, a.contig != 0, a.reduce != 0);
    case 2: return rank_fn_j<2>(pw, a.contig != 0, a.reduce != 0);
    case 4: return rank_fn_j<4>(pw, a.contig != 0, a.reduce != 0);
    default: return rank_fn_j<8>(pw, a.contig != 0, a.reduce != 0);
  }
}

}  // namespace

int32_t tree_rank_layout(const taccl_plan &p, TreeArgs &a) {
  const int32_t C = p.coll.C, V = p.topo.V, E = p.topo.E, P = p.topo.P;
  const int32_t CV = C * V;
  const int32_t K = std::max(p.max_paths, 1), H = std::max(p.H, 1);
  const int32_t pw = P / 4;
  if (p.coll.kind == TACCL_ALLTOALL || p.topt.empty() || p.tent.empty() || p.pq_range <= 0 ||
      K > 8 || H > 4 || P % 4 || (pw != 1 && pw != 2 && pw != 3 && pw != 4 && pw != 6 && pw != 8) ||
      V > 64 || E < 1 || E > 255 || CV > 64 * kLayerMaxSlotsPerLane || p.route_stride > 4 * 64 * kPfRouteWords ||
      p.route_stride % 4)
    return 0;
  uint64_t cmin = ~0ull, cmax = 0;
  for (uint32_t c : p.cost) {
    cmin = std::min<uint64_t>(cmin, c);
    cmax = std::max<uint64_t>(cmax, c);
  }
  if (cmin == 0 || cmax >= (1u << 24)) return 0;  // link costs: 24-bit multiplies
  const uint64_t max_rem = (uint64_t)(V - 1) * cmax;
  if (max_rem >= (1ull << 32)) return 0;
  a.lmagic = ((1ull << 32) + cmin - 1) / cmin;  // ceil(2^32 / c_min)
  if (a.lmagic >= (1ull << 32) || p.pq_magic >= (1ull << 32)) return 0;  // 32-bit multiply-high
  const uint64_t nl = ((max_rem * a.lmagic) >> 32) + 1;
  if (nl > 64) return 0;
  a.nl_max = (int32_t)nl;
  a.qmagic = p.pq_magic;
  a.qrange = p.pq_range;
  a.K = K;
  a.H = H;
  int32_t off = 0;
  auto take = [&](int32_t bytes) {
    const int32_t o = off;
    off = align16(off + bytes);
    return o;
  };
  a.o_cost = take(4 * E);
  a.o_src = take(E);
  a.o_merge = take(E);
  a.o_post = take(8 * C);
  // owner stride of the transposed option words: PW * V rounded up to 16
  // mod 32 (two owners' rows fall on different bank halves)
  a.opt_ostride = pw * V + ((16 - (pw * V) % 32) + 32) % 32;
  a.o_opt = take(4 * P * a.opt_ostride);
  a.o_ent = take(P * V * P * K);
  a.o_slot = take(8 * CV);
  if ((int64_t)P * V * P * K >= (1 << 20)) return 0;  // entering-link base: 20 bits
  a.o_wave = off;
  const int32_t S = std::max<int64_t>(std::min<int64_t>(p.max_sends, CV), 1);
  int r = 0;
  while ((1 << r) < V) r++;
  a.pj_rounds = std::max(r, 1);
  // region A: one-hot routes, (distance, ancestor) pairs and heights for
  // every slot a lane holds (64 J, J of the instantiation that runs); then
  // u16 counters for nl_max * E + 1 starts plus one dummy word per lane;
  // then 8-byte entries (three spare), bounds and u16 parent sends per
  // position; then finish times
  const int32_t CVp = 64 * rank_slots_per_lane(CV);
  const int32_t tree_bytes = align16(p.route_stride) + align16(8 * CVp) + align16(4 * CVp);
  a.w_dist = align16(p.route_stride);
  a.w_anc = a.w_dist;
  a.w_h = a.w_dist + align16(8 * CVp);
  const int32_t cnt_bytes = align16(4 * (int32_t)((nl * E + 2) / 2 + 64));
  a.w_bnd = align16(8 * (S + 3));
  a.w_pj = a.w_bnd + align16(4 * S);
  const int32_t ent_bytes = a.w_pj + align16(2 * S);
  // finish times per slot, then (contiguous transfers) ready times per
  // position
  a.w_rq = align16(4 * CVp);
  const int32_t region_a = std::max({tree_bytes, cnt_bytes, ent_bytes, a.w_rq + align16(4 * S)});
  // region B: the ordered sends (slot | parent send, link | rank | last)
  a.w_ord2 = region_a;
  a.w_info2 = a.w_ord2 + align16(4 * S);
  int32_t w = a.w_info2 + align16(4 * S);
  a.w_free = w;
  w = align16(w + 4 * E);
  a.w_lmask = w;
  w = align16(w + 8);
  a.w_lst = w;
  w = align16(w + 4 * 65);
  a.wave_bytes = w;
  return a.o_wave + a.wave_bytes;
}

bool tree_rank_reverse_ok(const taccl_plan &p) {
  // the reverse of every route hop exists and costs the same, so reversed
  // path sums are sums of the same costs and the path codes stay exact
  if (p.contig || p.lrev.size() != (size_t)p.topo.E) return false;
  for (uint16_t l : p.path_links) {
    const uint16_t r = p.lrev[l];
    if (r == 0xFFFFu || p.cost[r] != p.cost[l]) return false;
  }
  return true;
}

int tree_rank_blocks_per_cu(const TreeArgs &a) {
  int nb = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, rank_fn(a), 64 * a.waves_per_block,
                                                   tree_block_bytes(a, a.waves_per_block)) !=
      hipSuccess)
    return 0;
  return nb;
}

hipError_t launch_tree_rank(const TreeArgs &a, int grid, hipStream_t stream) {
  const int pw = a.P / 4;
  if (a.P % 4 || (pw != 1 && pw != 2 && pw != 3 && pw != 4 && pw != 6 && pw != 8) ||
      a.C * a.V > 1024 || a.E > 255 || a.qrange <= 0)
    return hipErrorInvalidValue;
  const dim3 g(grid), b(64 * a.waves_per_block);
  const int bytes = tree_block_bytes(a, a.waves_per_block);
  void *args[] = {(void *)&a};
  return hipLaunchKernel(rank_fn(a), g, b, args, bytes, stream);
}

}  // namespace taccl
