// C ABI: plan upload and batched evaluation.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstring>
#include <vector>

#include "kernels.h"
#include "plan.h"

namespace taccl {
namespace {

struct Packer {
  std::vector<unsigned char> bytes;
  template <class T>
  size_t add(const std::vector<T> &v) {
    size_t off = (bytes.size() + 255) & ~size_t(255);
    bytes.resize(off + std::max<size_t>(v.size() * sizeof(T), 1), 0);
    if (!v.empty()) std::memcpy(bytes.data() + off, v.data(), v.size() * sizeof(T));
    return off;
  }
};

taccl_status_t hip_fail(hipError_t e, const char *what) {
  return fail(TACCL_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

// Upload the read-only tables of `p` to the current device (once).
taccl_status_t ensure_device(taccl_plan *p, DeviceTables **out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  std::lock_guard<std::mutex> lock(p->mu);
  auto it = p->dev.find(dev);
  if (it != p->dev.end()) {
    *out = &it->second;
    return TACCL_OK;
  }
  hipDeviceProp_t prop;
  e = hipGetDeviceProperties(&prop, dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDeviceProperties");
  Packer pk;
  size_t o_cost = pk.add(p->cost), o_lsrc = pk.add(p->lsrc), o_ldst = pk.add(p->ldst),
         o_pb = pk.add(p->pair_base), o_np = pk.add(p->npaths), o_po = pk.add(p->path_off),
         o_pl = pk.add(p->path_links), o_own = pk.add(p->coll.owner),
         o_pm = pk.add(p->post_mask), o_hc = pk.add(p->hop_class),
         o_plh = pk.add(p->path_lvl_hop), o_lcb = pk.add(p->lvl_cls_begin),
         o_llc = pk.add(p->llc), o_trec = pk.add(p->tree_rec), o_own8 = pk.add(p->owner8),
         o_arec = pk.add(p->arec), o_cpath = pk.add(p->cpath), o_cinfo = pk.add(p->cinfo),
         o_cbkt = pk.add(p->cbkt), o_topt = pk.add(p->topt), o_trec4 = pk.add(p->tree_rec4),
         o_lal = pk.add(p->lalpha), o_lbs = pk.add(p->lbs), o_lmg = pk.add(p->lmerge),
         o_lrev = pk.add(p->lrev), o_hc2 = pk.add(p->hop_class2),
         o_lcb2 = pk.add(p->lvl_cls2_begin), o_llc2 = pk.add(p->llc2),
         o_gkr = pk.add(p->gkrank), o_tent = pk.add(p->tent), o_c2l = pk.add(p->cls2_link);
  void *blk = nullptr;
  e = hipMalloc(&blk, pk.bytes.size());
  if (e != hipSuccess) return fail(TACCL_ERR_NO_MEMORY, "hipMalloc of plan tables failed");
  e = hipMemcpy(blk, pk.bytes.data(), pk.bytes.size(), hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(blk);
    return hip_fail(e, "hipMemcpy of plan tables");
  }
  DeviceTables t;
  auto at = [&](size_t off) { return (const unsigned char *)blk + off; };
  t.block = blk;
  t.cost = (const uint32_t *)at(o_cost);
  t.lsrc = (const uint16_t *)at(o_lsrc);
  t.ldst = (const uint16_t *)at(o_ldst);
  t.pair_base = (const uint32_t *)at(o_pb);
  t.npaths = (const uint8_t *)at(o_np);
  t.path_off = (const uint32_t *)at(o_po);
  t.path_links = (const uint16_t *)at(o_pl);
  t.owner = (const int32_t *)at(o_own);
  t.post_mask = (const uint64_t *)at(o_pm);
  t.hop_class = (const uint16_t *)at(o_hc);
  t.path_lvl_hop = (const int8_t *)at(o_plh);
  t.lvl_cls_begin = (const uint32_t *)at(o_lcb);
  t.llc = (const uint32_t *)at(o_llc);
  t.tree_rec = (const uint32_t *)at(o_trec);
  t.owner8 = (const uint8_t *)at(o_own8);
  t.topt = p->topt.empty() ? nullptr : (const uint8_t *)at(o_topt);
  t.tree_rec4 = p->tree_rec4.empty() ? nullptr : (const uint32_t *)at(o_trec4);
  t.lalpha = (const uint32_t *)at(o_lal);
  t.lbs = (const uint64_t *)at(o_lbs);
  t.lmerge = (const uint8_t *)at(o_lmg);
  t.lrev = (const uint16_t *)at(o_lrev);
  t.hop_class2 = (const uint16_t *)at(o_hc2);
  t.lvl_cls2_begin = (const uint32_t *)at(o_lcb2);
  t.llc2 = (const uint32_t *)at(o_llc2);
  t.cls2_link = (const uint16_t *)at(o_c2l);
  t.arec = (const uint32_t *)at(o_arec);
  t.cpath = (const uint32_t *)at(o_cpath);
  t.cinfo = (const uint32_t *)at(o_cinfo);
  t.cbkt = (const uint32_t *)at(o_cbkt);
  t.gkrank = (const uint32_t *)at(o_gkr);
  t.tent = p->tent.empty() ? nullptr : (const uint8_t *)at(o_tent);
  t.max_lds = (int)prop.sharedMemPerBlock;
  t.lds_per_cu = (int)std::max<size_t>(prop.maxSharedMemoryPerMultiProcessor, prop.sharedMemPerBlock);
  t.num_cus = prop.multiProcessorCount;
  *out = &(p->dev[dev] = t);
  return TACCL_OK;
}

}  // namespace
}  // namespace taccl

using namespace taccl;

extern "C" {

void taccl_plan_destroy(taccl_plan_t p) {
  if (!p) return;
  int cur = -1;
  (void)hipGetDevice(&cur);
  for (auto &kv : p->dev) {
    if (hipSetDevice(kv.first) == hipSuccess) (void)hipFree(kv.second.block);
  }
  if (cur >= 0) (void)hipSetDevice(cur);
  delete p;
}

taccl_status_t taccl_plan_upload(taccl_plan_t p) {
  if (!p) return fail(TACCL_ERR_INVALID_ARGUMENT, "null plan");
  DeviceTables *t = nullptr;
  return ensure_device(p, &t);
}

taccl_status_t taccl_eval_batch(taccl_plan_t p, int64_t n, const uint8_t *d_routes,
                                const uint32_t *d_prio, uint32_t *d_makespan, uint8_t *d_valid,
                                taccl_stream_t stream) {
  if (!p) return fail(TACCL_ERR_INVALID_ARGUMENT, "null plan");
  if (n < 0) return fail(TACCL_ERR_INVALID_ARGUMENT, "negative candidate count");
  if (n == 0) return TACCL_OK;
  if (!d_routes || !d_prio || !d_makespan || !d_valid)
    return fail(TACCL_ERR_INVALID_ARGUMENT, "null device pointer");
  if (((uintptr_t)d_prio & 3) || ((uintptr_t)d_makespan & 3))
    return fail(TACCL_ERR_INVALID_ARGUMENT, "d_prio and d_makespan must be 4-byte aligned");
  DeviceTables *t = nullptr;
  taccl_status_t st = ensure_device(p, &t);
  if (st) return st;
  hipStream_t s = (hipStream_t)stream;
  // enough blocks to fill every CU several times over; each block loops
  const int64_t cap = (int64_t)std::max(t->num_cus, 1) * 64;
  const int grid = (int)std::min<int64_t>(n, cap);
  hipError_t e;
  if (p->coll.kind == TACCL_ALLTOALL && p->greedy) {
    PathGreedyArgs g{};
    // one wavefront per candidate while its lists fit, else one block
    const bool wave =
        path_greedy_layout(*p, g) > 0 && g.o_wave + g.wave_bytes <= t->max_lds;
    if (!wave && (path_greedy_block_layout(*p, g) <= 0 || g.block_bytes > t->max_lds))
      return fail(TACCL_ERR_UNSUPPORTED,
                  "time-aware greedy orders for Alltoall need at most 65535 send slots "
                  "(chunks x longest path), 4096 chunks and no zero-cost link");
    g.mirror = p->greedy == 2;
    g.gkrank = t->gkrank;
    g.C = p->coll.C;
    g.P = p->topo.P;
    g.E = p->topo.E;
    g.H = std::max(p->H, 1);
    g.cpr = std::max(p->coll.cpr, 1);
    g.route_stride = p->route_stride;
    g.prio_stride = p->prio_stride;
    g.cost = t->cost;
    g.pair_base = t->pair_base;
    g.npaths = t->npaths;
    g.path_off = t->path_off;
    g.path_links = t->path_links;
    g.routes = d_routes;
    g.prio = d_prio;
    g.makespan = d_makespan;
    g.valid = d_valid;
    g.n = n;
    if (!wave) {
      const int nb = std::max(1, path_greedy_block_per_cu(g));
      const int bgrid = (int)std::min<int64_t>(n, (int64_t)std::max(t->num_cus, 1) * nb);
      e = launch_path_greedy_block(g, bgrid, s);
      if (e != hipSuccess) return hip_fail(e, "kernel launch");
      return TACCL_OK;
    }
    // wavefronts per block: most resident wavefronts per CU
    int best_w = 1, best_res = 0, best_bpc = 1;
    for (int w = 1; w <= kTreeMaxThreads / 64; w++) {
      const int bytes = g.o_wave + w * g.wave_bytes;
      if (bytes > t->max_lds) break;
      g.waves_per_block = w;
      int bpc = std::min(t->lds_per_cu / bytes, 32 / w);
      const int nb = path_greedy_blocks_per_cu(g);
      if (nb > 0) bpc = std::min(bpc, nb);
      if (bpc * w > best_res) {
        best_res = bpc * w;
        best_w = w;
        best_bpc = bpc;
      }
    }
    g.waves_per_block = best_w;
    const int64_t want = (n + best_w - 1) / best_w;
    const int ggrid = (int)std::min<int64_t>(want, (int64_t)std::max(t->num_cus, 1) * best_bpc);
    e = launch_path_greedy(g, ggrid, s);
    if (e != hipSuccess) return hip_fail(e, "kernel launch");
    return TACCL_OK;
  }
  if (p->coll.kind == TACCL_ALLTOALL) {
    PathArgs a{};
    a.C = p->coll.C;
    a.P = p->topo.P;
    a.E = p->topo.E;
    a.H = std::max(p->H, 1);
    a.cpr = p->coll.cpr;
    a.nlev = p->nlev;
    a.route_stride = p->route_stride;
    a.prio_stride = p->prio_stride;
    a.cost = t->cost;
    a.pair_base = t->pair_base;
    a.npaths = t->npaths;
    a.path_off = t->path_off;
    a.hop_class = t->hop_class;
    a.path_lvl_hop = t->path_lvl_hop;
    a.lvl_cls_begin = t->lvl_cls_begin;
    a.llc = t->llc;
    a.routes = d_routes;
    a.prio = d_prio;
    a.makespan = d_makespan;
    a.valid = d_valid;
    a.n = n;
    a.contig = p->contig;
    a.lalpha = t->lalpha;
    a.lbs = t->lbs;
    a.lmerge = t->lmerge;
    a.ports = p->ports;
    a.hop_class2 = t->hop_class2;
    a.lvl_cls2_begin = t->lvl_cls2_begin;
    a.llc2 = t->llc2;
    a.cls2_link = t->cls2_link;
    a.arec = t->arec;
    a.cpath = t->cpath;
    a.routes_words = (p->route_stride % 4 == 0) && (((uintptr_t)d_routes & 3) == 0);
    a.cinfo = t->cinfo;
    a.cbkt = t->cbkt;
    const int cpt = p->path_fast ? path_fast_cpt(*p) : 0;
    if (cpt && path_fast_layout(*p, a) <= t->max_lds) {
      const int nt = path_fast_threads(*p);
      int bpc = std::max(1, std::min(t->lds_per_cu / a.lds_bytes, 4));
      const int nb = path_fast_blocks_per_cu(a, cpt, nt);
      if (nb > 0) bpc = std::min(bpc, nb);
      const int fgrid = (int)std::min<int64_t>(n, (int64_t)std::max(t->num_cus, 1) * bpc);
      e = launch_path_fast(a, cpt, nt, fgrid, s);
    } else {
      if (path_layout(*p, a) > t->max_lds)
        return fail(TACCL_ERR_UNSUPPORTED, "Alltoall plan needs more LDS than a block has");
      if (a.ports && a.E > 4 * a.lr_threads)
        return fail(TACCL_ERR_UNSUPPORTED, "switch ports take at most four links per thread");
      e = launch_path(a, grid, s);
    }
  } else {
    TreeArgs a{};
    a.C = p->coll.C;
    a.P = p->topo.P;
    a.V = p->topo.V;
    a.E = p->topo.E;
    a.route_stride = p->route_stride;
    a.prio_stride = p->prio_stride;
    a.routes_word_aligned = (p->route_stride % 4 == 0) && (((uintptr_t)d_routes & 3) == 0);
    a.cost = t->cost;
    a.lsrc = t->lsrc;
    a.ldst = t->ldst;
    a.rec = t->tree_rec;
    a.npaths = t->npaths;
    a.owner8 = t->owner8;
    a.topt = t->topt;
    a.contig = p->contig;
    a.lalpha = t->lalpha;
    a.lbs = t->lbs;
    a.lmerge = t->lmerge;
    a.rec4 = (const uint4 *)t->tree_rec4;
    a.post_mask = t->post_mask;
    a.routes = d_routes;
    a.prio = d_prio;
    a.makespan = d_makespan;
    a.valid = d_valid;
    a.n = n;
    // the layered kernel needs whole route words and priorities in registers
    const bool greedy = p->greedy != 0;
    const bool layered =
        a.routes_word_aligned &&
        (greedy ? tree_greedy_layout(*p, a) : tree_layers_layout(*p, a)) > 0 &&
        tree_block_bytes(a, 1) <= t->max_lds;
    const int kind = p->coll.kind;
    const bool reduction = kind == TACCL_REDUCESCATTER || kind == TACCL_ALLREDUCE;
    // plans outside the layered kernel's limits: the general kernel, whose
    // variant with reductions, contiguity and greedy orders keeps more state
    a.any = !layered && (reduction || p->contig || greedy);
    a.greedy = p->greedy;
    if (!layered && (a.any ? tree_any_layout(*p, a) : tree_layout(*p, a)) > t->max_lds)
      return fail(TACCL_ERR_UNSUPPORTED, "multicast plan needs more LDS than a block has");
    a.lrev = t->lrev;
    // wavefronts per block: most resident wavefronts per CU (LDS, and for
    // the layered kernel registers too, by the runtime's occupancy query)
    auto launch = [&](TreeArgs &x) {
      int best_w = 1, best_res = 0, best_bpc = 1;
      for (int w = 1; w <= kTreeMaxThreads / 64; w++) {
        const int bytes = tree_block_bytes(x, w);
        if (bytes > t->max_lds) break;
        int bpc = std::min(t->lds_per_cu / bytes, 32 / w);
        if (layered) {
          x.waves_per_block = w;
          const int nb = greedy ? tree_greedy_blocks_per_cu(x) : tree_layers_blocks_per_cu(x);
          if (nb > 0) bpc = std::min(bpc, nb);
        }
        const int res = std::min(bpc * w, 32);
        if (res > best_res) {
          best_res = res;
          best_w = w;
          best_bpc = bpc;
        }
      }
      x.waves_per_block = best_w;
      const int64_t want = (n + best_w - 1) / best_w;
      const int tgrid =
          (int)std::min<int64_t>(want, (int64_t)std::max(t->num_cus, 1) * best_bpc);
      if (!layered) return launch_tree(x, tgrid, s);
      return greedy ? launch_tree_greedy(x, tgrid, s) : launch_tree_layers(x, tgrid, s);
    };
    // The static order on the ranked kernel, when the plan's path lengths
    // have exact short codes: Allgather, explicit multicast and the
    // Allgather phase of an Allreduce (contiguous transfers included), and
    // the ReduceScatter (alone or as an Allreduce's first phase) when every
    // route hop has a reverse link of equal cost and there is no contiguity
    TreeArgs ra = a;
    const bool ranked = !greedy && a.routes_word_aligned && t->tent &&
                        tree_rank_layout(*p, ra) > 0 && tree_block_bytes(ra, 1) <= t->max_lds;
    ra.ent = t->tent;
    const bool ranked_rs = ranked && tree_rank_reverse_ok(*p);
    auto launch_ranked = [&](TreeArgs &x) {
      int best_w = 1, best_res = 0, best_bpc = 1;
      for (int w = 1; w <= kRankMaxThreads / 64; w++) {
        const int bytes = tree_block_bytes(x, w);
        if (bytes > t->max_lds) break;
        int bpc = std::min(t->lds_per_cu / bytes, 32 / w);
        x.waves_per_block = w;
        const int nb = tree_rank_blocks_per_cu(x);
        if (nb > 0) bpc = std::min(bpc, nb);
        const int res = std::min(bpc * w, 32);
        if (res > best_res) {
          best_res = res;
          best_w = w;
          best_bpc = bpc;
        }
      }
      x.waves_per_block = best_w;
      const int64_t want = (n + best_w - 1) / best_w;
      const int tgrid =
          (int)std::min<int64_t>(want, (int64_t)std::max(t->num_cus, 1) * best_bpc);
      return launch_tree_rank(x, tgrid, s);
    };
    if (kind == TACCL_ALLREDUCE) {
      // ReduceScatter on the first priority row, then Allgather on the
      // second, adding its makespan (same stream, so in order)
      a.reduce = 1;
      a.accumulate = 0;
      if (ranked_rs) {
        TreeArgs r = ra;
        r.reduce = 1;
        r.accumulate = 0;
        e = launch_ranked(r);
      } else {
        e = launch(a);
      }
      if (e == hipSuccess) {
        TreeArgs b = ranked ? ra : a;
        b.reduce = 0;
        b.accumulate = 1;
        b.prio = d_prio + (size_t)p->coll.C * p->topo.V;
        e = ranked ? launch_ranked(b) : launch(b);
      }
    } else if (kind == TACCL_REDUCESCATTER ? ranked_rs : ranked) {
      ra.reduce = kind == TACCL_REDUCESCATTER;
      ra.accumulate = 0;
      e = launch_ranked(ra);
    } else {
      a.reduce = kind == TACCL_REDUCESCATTER;
      a.accumulate = 0;
      e = launch(a);
    }
  }
  if (e != hipSuccess) return hip_fail(e, "kernel launch");
  return TACCL_OK;
}

taccl_status_t taccl_count_faults(int64_t n, const uint32_t *makespan, int64_t *faults) {
  if (!faults) return fail(TACCL_ERR_INVALID_ARGUMENT, "null output");
  if (n < 0) return fail(TACCL_ERR_INVALID_ARGUMENT, "negative candidate count");
  if (n > 0 && !makespan) return fail(TACCL_ERR_INVALID_ARGUMENT, "null makespan array");
  int64_t k = 0;
  for (int64_t i = 0; i < n; i++) k += makespan[i] == TACCL_MAKESPAN_FAULT;
  *faults = k;
  return TACCL_OK;
}

// the seeded input generator shared with the tests (workloads/candgen.c)
extern "C" int candgen_fill(uint64_t seed, int64_t first, int64_t count, int route_stride,
                            const int32_t *options, int prio_stride, uint8_t *routes,
                            uint32_t *prio);

taccl_status_t taccl_generate_host(taccl_plan_t p, uint64_t seed, int64_t first, int64_t count,
                                   uint8_t *routes, uint32_t *prio) {
  if (!p) return fail(TACCL_ERR_INVALID_ARGUMENT, "null plan");
  if (first < 0 || count < 0)
    return fail(TACCL_ERR_INVALID_ARGUMENT, "negative first candidate or count");
  if (count == 0) return TACCL_OK;
  if (!routes || !prio) return fail(TACCL_ERR_INVALID_ARGUMENT, "null output buffer");
  if (candgen_fill(seed, first, count, p->route_stride, p->route_options.data(), p->prio_stride,
                   routes, prio) != 0)
    return fail(TACCL_ERR_INVALID_ARGUMENT, "candidate range beyond 2^32");
  return TACCL_OK;
}

taccl_status_t taccl_connections_batch(taccl_plan_t p, int64_t n, const uint8_t *d_routes,
                                       uint32_t *d_connections, taccl_stream_t stream) {
  if (!p) return fail(TACCL_ERR_INVALID_ARGUMENT, "null plan");
  if (n < 0) return fail(TACCL_ERR_INVALID_ARGUMENT, "negative candidate count");
  if (n == 0) return TACCL_OK;
  if (!d_routes || !d_connections) return fail(TACCL_ERR_INVALID_ARGUMENT, "null device pointer");
  if ((uintptr_t)d_connections & 3)
    return fail(TACCL_ERR_INVALID_ARGUMENT, "d_connections must be 4-byte aligned");
  const int32_t P = p->topo.P, V = p->topo.V;
  const bool tree = p->coll.kind != TACCL_ALLTOALL;
  if (P > 256 || (tree && (P > 64 || V > 255)))
    return fail(TACCL_ERR_UNSUPPORTED, "connection counts need at most 256 ranks (multicast: "
                                       "64 ranks and 255 vertices)");
  DeviceTables *t = nullptr;
  taccl_status_t st = ensure_device(p, &t);
  if (st) return st;
  ConnArgs a{};
  a.C = p->coll.C;
  a.P = P;
  a.V = V;
  a.cpr = std::max(p->coll.cpr, 1);
  a.kind = p->coll.kind;
  a.tree = tree ? 1 : 0;
  a.mask_words = (P * P + 31) / 32;
  a.route_stride = p->route_stride;
  a.ldst = t->ldst;
  a.pair_base = t->pair_base;
  a.npaths = t->npaths;
  a.path_off = t->path_off;
  a.path_links = t->path_links;
  a.owner = t->owner;
  a.post_mask = t->post_mask;
  a.routes = d_routes;
  a.out = d_connections;
  a.n = n;
  // one chunk per thread at a time; multicast blocks keep a parent byte per
  // vertex and thread in LDS
  int threads = std::min(kConnMaxThreads, std::max(64, (a.C + 63) / 64 * 64));
  while (threads > 64 && connections_lds_bytes(a, threads) > t->max_lds) threads -= 64;
  if (connections_lds_bytes(a, threads) > t->max_lds)
    return fail(TACCL_ERR_UNSUPPORTED, "connection count needs more LDS than a block has");
  const int per_cu = std::max(1, std::min(t->lds_per_cu / std::max(connections_lds_bytes(a, threads), 1),
                                          2048 / threads));
  const int grid = (int)std::min<int64_t>(n, (int64_t)std::max(t->num_cus, 1) * per_cu);
  hipError_t e = launch_connections(a, threads, grid, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "kernel launch");
  return TACCL_OK;
}

}  // extern "C"
