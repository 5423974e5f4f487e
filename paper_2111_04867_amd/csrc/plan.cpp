// Host-side plan builder: topology, collective, sketch -> evaluation plan.
//
// Route options follow the sketch (Sec. 3.1) and the shortest-path
// restriction of routing (Sec. 5.1, Step 1): the k best simple paths by
// (cost, hops, vertex sequence). They are found by a best-first search over
// partial paths ordered by cost so far plus a lower bound of the cost still
// to go (the distance to the destination over the usable links, ignoring
// the simple-path and crossing rules). Complete paths then leave the queue
// in nondecreasing cost, and every path of cost <= C is out before a
// partial path whose bound exceeds C; so once k complete paths are out, the
// search goes on only while the bound is at most the k-th cost (to collect
// its ties), and the collected paths sorted by (cost, hops, vertex
// sequence) give the k best exactly.
#include <algorithm>
#include <unordered_map>
#include <cstring>
#include <memory>
#include <queue>
#include <set>
#include <tuple>

#include "kernels.h"
#include "plan.h"

namespace taccl {

static thread_local std::string g_err;

taccl_status_t fail(taccl_status_t st, const std::string &msg) {
  g_err = msg;
  return st;
}

const char *last_error() { return g_err.c_str(); }
void clear_error() { g_err.clear(); }

namespace {

struct Path {
  std::vector<int32_t> verts;  // hops+1 vertices
  std::vector<int32_t> links;  // hops links
  uint64_t cost = 0;
};

struct Partial {
  uint64_t bound;  // cost + lower bound of the cost still to go
  uint64_t cost;
  int32_t cross;
  std::vector<int32_t> verts;
  std::vector<int32_t> links;
};

// priority_queue keeps the largest on top; invert (bound, hops, verts)
struct PartialAfter {
  bool operator()(const Partial &a, const Partial &b) const {
    if (a.bound != b.bound) return a.bound > b.bound;
    if (a.links.size() != b.links.size()) return a.links.size() > b.links.size();
    return a.verts > b.verts;
  }
};

bool path_before(const Path &a, const Path &b) {
  if (a.cost != b.cost) return a.cost < b.cost;
  if (a.links.size() != b.links.size()) return a.links.size() < b.links.size();
  return a.verts < b.verts;
}

class Router {
 public:
  Router(const taccl_topology &t, const std::vector<uint32_t> &cost, const uint8_t *allowed,
         const uint8_t *relay)
      : t_(t), cost_(cost), allowed_(allowed), relay_(relay), in_(t.V) {
    for (int32_t e = 0; e < t.E; e++) in_[t.col[e]].push_back(e);
  }

  // Up to k best simple paths s -> d with at most max_cross node crossings.
  // only_min keeps just the minimal-cost ones. Returns false if the search
  // exceeded its expansion budget.
  bool k_best(int32_t s, int32_t d, int32_t k, int32_t max_cross, bool only_min,
              std::vector<Path> &out) const {
    out.clear();
    const std::vector<uint64_t> &h = to_go(d);
    if (h[s] == kFar) return true;  // no path at all
    std::priority_queue<Partial, std::vector<Partial>, PartialAfter> q;
    q.push(Partial{h[s], 0, 0, {s}, {}});
    int64_t budget = 20000000;
    while (!q.empty()) {
      Partial cur = q.top();
      q.pop();
      // enough paths, and no cheaper or equally cheap one can follow
      if (!out.empty() && (int32_t)out.size() >= (only_min ? 1 : k) &&
          cur.bound > out[only_min ? 0 : k - 1].cost)
        break;
      if (--budget < 0) return false;
      int32_t u = cur.verts.back();
      if (u == d) {
        out.push_back(Path{cur.verts, cur.links, cur.cost});
        continue;
      }
      for (int32_t e = t_.row_ptr[u]; e < t_.row_ptr[u + 1]; e++) {
        if (allowed_ && !allowed_[e]) continue;
        int32_t v = t_.col[e];
        if (h[v] == kFar) continue;
        if (std::find(cur.verts.begin(), cur.verts.end(), v) != cur.verts.end()) continue;
        int32_t cross = cur.cross;
        if (t_.node[u] != t_.node[v]) {
          cross++;
          if (max_cross >= 0 && cross > max_cross) continue;
          if (relay_ && !(relay_[u] && relay_[v])) continue;
        }
        const uint64_t c = cur.cost + cost_[e];
        Partial nxt{c + h[v], c, cross, cur.verts, cur.links};
        nxt.verts.push_back(v);
        nxt.links.push_back(e);
        q.push(std::move(nxt));
      }
    }
    std::sort(out.begin(), out.end(), path_before);
    if (only_min)
      while (!out.empty() && out.back().cost != out[0].cost) out.pop_back();
    if ((int32_t)out.size() > k) out.resize(k);
    return true;
  }

  // Best single path (empty path when s == d); false if none exists.
  bool best(int32_t s, int32_t d, int32_t max_cross, Path &out, bool &budget_ok) const {
    if (s == d) {
      out = Path{{s}, {}, 0};
      return true;
    }
    std::vector<Path> v;
    budget_ok = k_best(s, d, 1, max_cross, false, v) && budget_ok;
    if (v.empty()) return false;
    out = v[0];
    return true;
  }

  Path join(const Path &a, int32_t mid, const Path &b) const {
    Path p = a;
    if (mid >= 0) {
      p.links.push_back(mid);
      p.verts.push_back(t_.col[mid]);
      p.cost += cost_[mid];
    }
    for (size_t i = 0; i < b.links.size(); i++) {
      p.links.push_back(b.links[i]);
      p.verts.push_back(b.verts[i + 1]);
      p.cost += cost_[b.links[i]];
    }
    return p;
  }

  int32_t link(int32_t u, int32_t v) const {
    for (int32_t e = t_.row_ptr[u]; e < t_.row_ptr[u + 1]; e++)
      if (t_.col[e] == v && (!allowed_ || allowed_[e])) return e;
    return -1;
  }

 private:
  static constexpr uint64_t kFar = ~0ull;
  // cost of the cheapest walk from every vertex to d over the usable links
  // (allowed, and between nodes only between relays): a lower bound of any
  // simple path's remaining cost, cached per destination
  const std::vector<uint64_t> &to_go(int32_t d) const {
    auto it = h_.find(d);
    if (it != h_.end()) return it->second;
    std::vector<uint64_t> dist(t_.V, kFar);
    using Item = std::pair<uint64_t, int32_t>;
    std::priority_queue<Item, std::vector<Item>, std::greater<Item>> q;
    dist[d] = 0;
    q.push({0, d});
    while (!q.empty()) {
      auto [du, v] = q.top();
      q.pop();
      if (du != dist[v]) continue;
      // links u -> v: scan every link whose head is v
      for (int32_t e : in_[v]) {
        const int32_t u = t_.src[e];
        if (allowed_ && !allowed_[e]) continue;
        if (t_.node[u] != t_.node[v] && relay_ && !(relay_[u] && relay_[v])) continue;
        const uint64_t nd = du + cost_[e];
        if (nd < dist[u]) {
          dist[u] = nd;
          q.push({nd, u});
        }
      }
    }
    return h_.emplace(d, std::move(dist)).first->second;
  }

  const taccl_topology &t_;
  const std::vector<uint32_t> &cost_;
  const uint8_t *allowed_;
  const uint8_t *relay_;
  std::vector<std::vector<int32_t>> in_;  // links into every vertex
  mutable std::unordered_map<int32_t, std::vector<uint64_t>> h_;
};

}  // namespace

// -------------------------------------------------------------------------
// route options, layouts and kernel tables
// -------------------------------------------------------------------------

static taccl_status_t build_routes(taccl_plan *p, const uint8_t *allowed, const uint8_t *relay) {
  const taccl_topology &t = p->topo;
  const int32_t P = t.P;
  Router R(t, p->cost, allowed, relay);
  // relay routes join best single paths, and the same legs recur for many
  // pairs: each (s, d, crossing limit) is searched once
  std::unordered_map<uint64_t, int32_t> memo;  // -> index into legs, -1 = none
  std::vector<Path> legs;
  auto best = [&](int32_t s, int32_t d, int32_t mc, Path &out, bool &ok) {
    const uint64_t key = ((uint64_t)(uint32_t)s << 32 | (uint32_t)d) * 4 + (uint64_t)(mc + 1);
    auto it = memo.find(key);
    if (it == memo.end()) {
      Path q;
      const int32_t idx = R.best(s, d, mc, q, ok) ? (int32_t)legs.size() : -1;
      if (idx >= 0) legs.push_back(std::move(q));
      it = memo.emplace(key, idx).first;
    }
    if (it->second < 0) return false;
    out = legs[it->second];
    return true;
  };
  p->pair_base.assign((size_t)P * P, 0);
  p->npaths.assign((size_t)P * P, 0);
  p->path_off.assign(1, 0);
  bool budget_ok = true;
  std::vector<std::vector<int32_t>> relays_of_node;
  if (p->mode == TACCL_ROUTE_HIER_RELAY) {
    int32_t nn = 0;
    for (int32_t v = 0; v < t.V; v++) nn = std::max(nn, t.node[v] + 1);
    relays_of_node.assign(nn, {});
    for (int32_t r = 0; r < P; r++)
      if (relay && relay[r]) relays_of_node[t.node[r]].push_back(r);
  }
  for (int32_t s = 0; s < P; s++) {
    for (int32_t d = 0; d < P; d++) {
      std::vector<Path> opts;
      if (s != d) {
        switch (p->mode) {
          case TACCL_ROUTE_SHORTEST_ONLY:
          case TACCL_ROUTE_KSHORTEST:
            budget_ok = R.k_best(s, d, p->k, p->max_cross, p->mode == TACCL_ROUTE_SHORTEST_ONLY,
                                 opts) && budget_ok;
            break;
          case TACCL_ROUTE_RELAY1: {
            Path q;
            if (best(s, d, p->max_cross, q, budget_ok)) opts.push_back(q);
            for (int32_t m = 0; m < P; m++) {
              if (m == s || m == d || (relay && !relay[m])) continue;
              Path a, b;
              if (!best(s, m, p->max_cross, a, budget_ok)) continue;
              if (!best(m, d, p->max_cross, b, budget_ok)) continue;
              opts.push_back(R.join(a, -1, b));
            }
            break;
          }
          case TACCL_ROUTE_HIER_RELAY: {
            if (t.node[s] == t.node[d]) {
              Path q;
              if (best(s, d, 0, q, budget_ok)) opts.push_back(q);
            } else {
              const auto &rs = relays_of_node[t.node[s]];
              const auto &rd = relays_of_node[t.node[d]];
              size_t nr = std::min(rs.size(), rd.size());
              for (size_t i = 0; i < nr; i++) {
                int32_t mid = R.link(rs[i], rd[i]);
                if (mid < 0) continue;
                Path a, b;
                if (!best(s, rs[i], 0, a, budget_ok)) continue;
                if (!best(rd[i], d, 0, b, budget_ok)) continue;
                opts.push_back(R.join(a, mid, b));
              }
            }
            break;
          }
          default:
            return fail(TACCL_ERR_INVALID_ARGUMENT, "unknown route mode");
        }
      }
      if (!budget_ok)
        return fail(TACCL_ERR_UNSUPPORTED, "path search exceeded its expansion budget");
      if (opts.size() > 255)
        return fail(TACCL_ERR_LIMIT, "more than 255 route options for one pair");
      size_t pp = (size_t)s * P + d;
      p->pair_base[pp] = (uint32_t)(p->path_off.size() - 1);
      p->npaths[pp] = (uint8_t)opts.size();
      p->max_paths = std::max<int32_t>(p->max_paths, (int32_t)opts.size());
      for (const Path &q : opts) {
        std::set<int32_t> uniq(q.links.begin(), q.links.end());
        if (uniq.size() != q.links.size())
          return fail(TACCL_ERR_UNSUPPORTED, "a route option uses one link twice");
        for (int32_t l : q.links) p->path_links.push_back((uint16_t)l);
        p->path_off.push_back((uint32_t)p->path_links.size());
        p->path_cost.push_back(q.cost);
        p->H = std::max<int32_t>(p->H, (int32_t)q.links.size());
      }
    }
  }
  return TACCL_OK;
}

// Remaining-cost levels and (level, link, travelled) classes of every hop of
// every Alltoall route option. A chunk's remaining cost strictly decreases
// along its path, so a path has at most one hop per level and, within one
// level, no send depends on another send of the same level.
static taccl_status_t build_levels(taccl_plan *p) {
  const int32_t P = p->topo.P, E = p->topo.E;
  const size_t npath = p->path_cost.size();
  std::vector<uint8_t> used_path(npath, 0);
  for (int32_t s = 0; s < P; s++)
    for (int32_t d = 0; d < P; d++) {
      if (s == d) continue;
      size_t pp = (size_t)s * P + d;
      for (int32_t k = 0; k < p->npaths[pp]; k++) used_path[p->pair_base[pp] + k] = 1;
    }
  // sends of every path: one per hop, or with switch ports one per hop pair
  // rank -> switch -> rank (first hop j, send-port link, receive-port link,
  // cost of the uplink)
  struct Unit {
    uint32_t j;
    int32_t link, link2;
    uint64_t cost;
  };
  std::vector<std::vector<Unit>> units(npath);
  std::vector<uint64_t> ucost(npath, 0);
  for (size_t q = 0; q < npath; q++) {
    if (!used_path[q]) continue;
    for (uint32_t j = p->path_off[q]; j < p->path_off[q + 1]; j++) {
      const int32_t l = p->path_links[j];
      Unit x{j - p->path_off[q], l, -1, p->cost[l]};
      if (p->ports && p->topo.col[l] >= P && j + 1 < p->path_off[q + 1]) {
        x.link2 = p->path_links[j + 1];
        j++;
      }
      units[q].push_back(x);
      ucost[q] += x.cost;
    }
  }
  std::set<uint64_t, std::greater<uint64_t>> rems;
  for (size_t q = 0; q < npath; q++) {
    uint64_t rem = ucost[q];
    for (const Unit &x : units[q]) {
      rems.insert(rem);
      rem -= x.cost;
    }
  }
  std::vector<uint64_t> lv(rems.begin(), rems.end());  // descending
  p->nlev = (int32_t)lv.size();
  // the level tables hold a signed byte per (route option, level) and a
  // class range per (level, link)
  if (p->H > 127) return fail(TACCL_ERR_UNSUPPORTED, "Alltoall paths of more than 127 hops");
  if ((double)npath * p->nlev + 8.0 * p->nlev * E > (double)(256u << 20))
    return fail(TACCL_ERR_UNSUPPORTED, "remaining-cost level tables beyond 256 MiB");
  auto level_of = [&](uint64_t rem) {
    return (int32_t)(std::lower_bound(lv.begin(), lv.end(), rem, std::greater<uint64_t>()) -
                     lv.begin());
  };
  // classes sorted by (level, link, travelled): the send-port link; with
  // switch ports also receive-port classes (level, downlink, travelled)
  std::set<std::tuple<int32_t, int32_t, uint64_t>> cls, cls2;
  for (size_t q = 0; q < npath; q++) {
    uint64_t rem = ucost[q], trav = 0;
    for (const Unit &x : units[q]) {
      cls.insert({level_of(rem), x.link, trav});
      if (x.link2 >= 0) cls2.insert({level_of(rem), x.link2, trav});
      rem -= x.cost;
      trav += x.cost;
    }
  }
  if (cls.size() > 65535 || cls2.size() > 65535)
    return fail(TACCL_ERR_UNSUPPORTED, "more than 65535 send classes");
  if (p->ports) {
    // the kernel keeps a link's send-port and receive-port orders apart, so
    // no link may serve as both (only a switch-to-switch link could)
    std::vector<uint8_t> role((size_t)E, 0);
    for (const auto &x : cls) role[std::get<1>(x)] |= 1;
    for (const auto &x : cls2) role[std::get<1>(x)] |= 2;
    for (int32_t l = 0; l < E; l++)
      if (role[l] == 3)
        return fail(TACCL_ERR_UNSUPPORTED,
                    "switch ports: a link is both a send port and a receive port");
  }
  std::vector<std::tuple<int32_t, int32_t, uint64_t>> cv(cls.begin(), cls.end());
  std::vector<std::tuple<int32_t, int32_t, uint64_t>> cv2(cls2.begin(), cls2.end());
  p->ncls = (int32_t)cv.size();
  p->cls_link.resize(cv.size());
  auto class_tables = [&](const std::vector<std::tuple<int32_t, int32_t, uint64_t>> &v,
                          std::vector<uint32_t> &begin, std::vector<uint32_t> &llc,
                          int32_t &maxcls) {
    begin.assign((size_t)p->nlev + 1, 0);
    llc.assign((size_t)p->nlev * E * 2, 0);
    for (size_t i = 0; i < v.size(); i++) {
      int32_t L = std::get<0>(v[i]), l = std::get<1>(v[i]);
      begin[L + 1] = (uint32_t)(i + 1);
      uint32_t *r = &llc[((size_t)L * E + l) * 2];
      if (r[0] == r[1]) r[0] = (uint32_t)i;
      r[1] = (uint32_t)(i + 1);
    }
    maxcls = 0;
    for (int32_t L = 0; L < p->nlev; L++) {
      begin[L + 1] = std::max(begin[L + 1], begin[L]);
      maxcls = std::max<int32_t>(maxcls, (int32_t)(begin[L + 1] - begin[L]));
    }
  };
  for (size_t i = 0; i < cv.size(); i++) p->cls_link[i] = (uint16_t)std::get<1>(cv[i]);
  p->cls2_link.resize(cv2.size());
  for (size_t i = 0; i < cv2.size(); i++) p->cls2_link[i] = (uint16_t)std::get<1>(cv2[i]);
  class_tables(cv, p->lvl_cls_begin, p->llc, p->max_lvl_cls);
  if (p->ports) class_tables(cv2, p->lvl_cls2_begin, p->llc2, p->max_lvl_cls2);
  // per hop: its send's class (first hop of a unit; 0xFFFF for the second
  // hop of a switched send) and receive-port class (0xFFFF if none)
  p->hop_class.assign(p->path_links.size(), 0xFFFF);
  p->hop_class2.assign(p->ports ? p->path_links.size() : 0, 0xFFFF);
  p->path_lvl_hop.assign(npath * (size_t)std::max(p->nlev, 1), (int8_t)-1);
  for (size_t q = 0; q < npath; q++) {
    uint64_t rem = ucost[q], trav = 0;
    for (const Unit &x : units[q]) {
      int32_t L = level_of(rem);
      const uint32_t j = p->path_off[q] + x.j;
      auto it = std::lower_bound(cv.begin(), cv.end(), std::make_tuple(L, x.link, trav));
      p->hop_class[j] = (uint16_t)(it - cv.begin());
      if (x.link2 >= 0) {
        auto it2 = std::lower_bound(cv2.begin(), cv2.end(), std::make_tuple(L, x.link2, trav));
        p->hop_class2[j] = (uint16_t)(it2 - cv2.begin());
      }
      p->path_lvl_hop[q * p->nlev + L] = (int8_t)x.j;
      rem -= x.cost;
      trav += x.cost;
    }
  }
  // sends a level can hold: pairs with some option having a hop there
  std::vector<int64_t> per_level(p->nlev, 0);
  for (int32_t s = 0; s < P; s++)
    for (int32_t d = 0; d < P; d++) {
      if (s == d) continue;
      size_t pp = (size_t)s * P + d;
      std::vector<uint8_t> has(p->nlev, 0);
      for (int32_t k = 0; k < p->npaths[pp]; k++)
        for (int32_t L = 0; L < p->nlev; L++)
          if (p->path_lvl_hop[(size_t)(p->pair_base[pp] + k) * p->nlev + L] >= 0) has[L] = 1;
      // an ordered rank pair stands for chunks_per_rank chunks
      for (int32_t L = 0; L < p->nlev; L++) per_level[L] += has[L] ? p->coll.cpr : 0;
    }
  for (int32_t L = 0; L < p->nlev; L++)
    p->max_lvl_sends = std::max<int32_t>(p->max_lvl_sends, (int32_t)per_level[L]);

  // greedy orders: rank of every hop's Step-2 key (remaining desc,
  // travelled asc; in reverse path order the mirrored lengths, remaining' =
  // travelled + latency and travelled' = remaining - latency)
  p->gkrank.clear();
  p->gk_count = 0;
  if (p->greedy) {
    std::vector<std::pair<uint64_t, uint64_t>> keys(p->path_links.size());
    for (size_t q = 0; q < npath; q++) {
      const uint64_t total = p->path_cost[q];
      uint64_t trav = 0;
      for (uint32_t j = p->path_off[q]; j < p->path_off[q + 1]; j++) {
        const uint64_t c = p->cost[p->path_links[j]], rem = total - trav;
        // ascending pair order = Step-2 order: (~remaining, travelled)
        keys[j] = p->greedy == 2 ? std::make_pair(~(trav + c), rem - c)
                                 : std::make_pair(~rem, trav);
        trav += c;
      }
    }
    std::vector<std::pair<uint64_t, uint64_t>> uniq(keys);
    std::sort(uniq.begin(), uniq.end());
    uniq.erase(std::unique(uniq.begin(), uniq.end()), uniq.end());
    p->gkrank.resize(keys.size());
    for (size_t j = 0; j < keys.size(); j++)
      p->gkrank[j] = (uint32_t)(std::lower_bound(uniq.begin(), uniq.end(), keys[j]) - uniq.begin());
    p->gk_count = (int32_t)uniq.size();
  }

  // compact tables of the register-resident kernel (paths of <= 6 hops,
  // <= 8 levels, fewer than 2^24 - 2 route options)
  p->path_fast = !p->ports && p->H <= kFastMaxHops && p->nlev <= 8 && npath + 1 < kNoRoute &&
                 p->coll.C <= kFastMaxChunks;
  if (p->path_fast) {
    // record 0 has no hops (what a chunk without a route loads); option q's
    // record is record q + 1
    p->arec.assign((npath + 1) * 4, 0);
    p->arec[0] = 0xFFFFFFu << 8;
    for (size_t q = 0; q < npath; q++) {
      if (!used_path[q]) continue;
      uint32_t *r = &p->arec[(q + 1) * 4];
      uint64_t rem = p->path_cost[q];
      int32_t h = 0;
      uint32_t hm = 0xFFFFFFu;  // level -> hop, 3 bits per level (7: none)
      for (uint32_t j = p->path_off[q]; j < p->path_off[q + 1]; j++, h++) {
        const uint32_t lv = (uint32_t)level_of(rem);
        hm = (hm & ~(7u << (3 * lv))) | ((uint32_t)h << (3 * lv));
        r[1 + h / 2] |= (uint32_t)p->hop_class[j] << (16 * (h & 1));
        rem -= p->cost[p->path_links[j]];
      }
      r[0] = (uint32_t)h | (hm << 8);
    }
    const int32_t C = p->coll.C, cpr = p->coll.cpr;
    p->cpath.assign(C, 0);
    for (int32_t ch = 0; ch < C; ch++) {
      const int32_t pair = ch / cpr, s = pair / P, d = pair % P;
      if (s == d) continue;
      const size_t pp = (size_t)s * P + d;
      // a pair without any route option can never be delivered: marked by
      // an all-ones option index and no options
      p->cpath[ch] = p->npaths[pp] ? (p->pair_base[pp] + 1) | ((uint32_t)p->npaths[pp] << 24)
                                   : kNoRoute;
    }
    // priority sub-buckets per class, sized from the class's expected
    // membership under uniform route choice so a bucket holds 1-2 sends
    // (any input stays exact: a crowded bucket is only slower to order),
    // then halved all over until every level's buckets together fit the
    // kernel's counters
    std::vector<double> expect(p->ncls, 0.0);
    for (int32_t s2 = 0; s2 < P; s2++)
      for (int32_t d2 = 0; d2 < P; d2++) {
        if (s2 == d2) continue;
        const size_t pp = (size_t)s2 * P + d2;
        const int32_t np = p->npaths[pp];
        for (int32_t k = 0; k < np; k++) {
          const uint32_t q = p->pair_base[pp] + k;
          for (uint32_t j = p->path_off[q]; j < p->path_off[q + 1]; j++)
            expect[p->hop_class[j]] += (double)cpr / np;
        }
      }
    std::vector<int> cbits(p->ncls, 0);
    for (int32_t k = 0; k < p->ncls; k++)
      while (cbits[k] < 10 && (double)(2u << cbits[k]) <= expect[k]) cbits[k]++;
    p->cbkt.assign(p->ncls, 0);
    for (;;) {
      // classes are numbered level by level, so one running count numbers
      // every level's buckets in level order
      uint64_t nb = 0;
      for (int32_t k = 0; k < p->ncls; k++) {
        p->cbkt[k] = (uint32_t)nb | ((uint32_t)cbits[k] << 24);
        nb += 1u << cbits[k];
      }
      p->nb_total = (int32_t)std::min<uint64_t>(nb, INT32_MAX);
      if (nb <= (uint64_t)kFastMaxBuckets || p->ncls > kFastMaxBuckets) break;
      for (int &b : cbits) b = std::max(b - 1, 0);
    }
    p->cinfo.assign(p->ncls, 0);
    for (int32_t L = 0; L < p->nlev; L++)
      for (uint32_t k = p->lvl_cls_begin[L]; k < p->lvl_cls_begin[L + 1]; k++) {
        const uint32_t l = p->cls_link[k];
        const uint32_t first = p->llc[((size_t)L * E + l) * 2];
        p->cinfo[k] = l | ((p->cbkt[first] & 0xFFFFFFu) << 16);
      }
  }
  return TACCL_OK;
}

// Codes for the remaining and travelled lengths of multicast sends. Each is
// the cost of a path of a chunk's tree (at most V - 1 links, every one a
// hop of some route option), so it lies in S, the set of sums of at most
// V - 1 costs of such links. With g the smallest gap between two elements
// of S and m = ceil(2^32 / g), x -> floor(x * m / 2^32) is nondecreasing
// everywhere and gains at least 1 per step of S (g * m >= 2^32), so it
// orders and separates S exactly. Left at range 0 when S exceeds 16384
// elements or the codes need more than 11 bits.
static void path_sum_codes(taccl_plan *p) {
  p->pq_magic = 0;
  p->pq_range = 0;
  std::vector<uint64_t> costs;
  for (uint16_t l : p->path_links) costs.push_back(p->cost[l]);
  std::sort(costs.begin(), costs.end());
  costs.erase(std::unique(costs.begin(), costs.end()), costs.end());
  if (costs.empty() || costs[0] == 0) return;
  std::vector<uint64_t> S{0}, next;
  for (int32_t step = 0; step < p->topo.V - 1; step++) {
    next = S;
    for (uint64_t s : S)
      for (uint64_t c : costs) next.push_back(s + c);
    std::sort(next.begin(), next.end());
    next.erase(std::unique(next.begin(), next.end()), next.end());
    if (next.size() > 16384) return;
    if (next.size() == S.size()) break;  // closed: no longer sums appear
    S.swap(next);
  }
  if (S.back() >= (1ull << 32)) return;
  uint64_t gap = ~0ull;
  for (size_t i = 1; i < S.size(); i++) gap = std::min(gap, S[i] - S[i - 1]);
  if (S.size() == 1) gap = S[0] ? S[0] : 1;
  const uint64_t m = ((1ull << 32) + gap - 1) / gap;  // <= 2^32
  auto code = [&](uint64_t x) { return (x * m) >> 32; };
  for (size_t i = 1; i < S.size(); i++)
    if (code(S[i]) <= code(S[i - 1])) return;  // cannot happen (see above)
  const uint64_t range = code(S.back()) + 1;
  if (range > 2048) return;
  p->pq_magic = m;
  p->pq_range = (int32_t)range;
}

static taccl_status_t build_layout(taccl_plan *p) {
  const taccl_topology &t = p->topo;
  const taccl_collective &c = p->coll;
  const int32_t P = t.P, V = t.V, C = c.C;
  if (c.kind == TACCL_ALLTOALL) {
    p->route_stride = C;
    p->prio_stride = C * std::max(p->H, 1);
    p->route_options.assign(C, 0);
    int64_t sends = 0;
    for (int32_t ch = 0; ch < C; ch++) {
      int32_t s = c.owner[ch], d = c.post[c.post_ptr[ch]];
      if (s == d) continue;
      size_t pp = (size_t)s * P + d;
      p->route_options[ch] = p->npaths[pp];
      p->num_pairs++;
      int32_t longest = 0;
      for (int32_t k = 0; k < p->npaths[pp]; k++) {
        uint32_t q = p->pair_base[pp] + k;
        longest = std::max<int32_t>(longest, (int32_t)(p->path_off[q + 1] - p->path_off[q]));
      }
      sends += longest;
    }
    p->max_sends = sends;
  } else {
    p->route_stride = C * P;
    // Allreduce: the ReduceScatter row, then the Allgather row
    p->prio_stride = C * V * (c.kind == TACCL_ALLREDUCE ? 2 : 1);
    p->route_options.assign((size_t)C * P, 0);
    p->post_mask.assign(C, 0);
    std::vector<uint8_t> used((size_t)C * P, 0);
    for (int32_t ch = 0; ch < C; ch++) {
      for (int32_t j = c.post_ptr[ch]; j < c.post_ptr[ch + 1]; j++) {
        int32_t d = c.post[j];
        if (P <= 64) p->post_mask[ch] |= 1ull << d;
        if (d == c.owner[ch] || used[(size_t)ch * P + d]) continue;
        used[(size_t)ch * P + d] = 1;
        p->num_pairs++;
        p->route_options[(size_t)ch * P + d] = p->npaths[(size_t)c.owner[ch] * P + d];
      }
    }
    p->max_sends = (int64_t)C * (V - 1);
    // fixed-stride copy of the route options for on-chip lookup
    const int32_t K = std::max(p->max_paths, 1), H = std::max(p->H, 1);
    p->tree_rec.assign((size_t)P * P * K * H, 0);
    for (int32_t pp = 0; pp < P * P; pp++)
      for (int32_t k = 0; k < p->npaths[pp]; k++) {
        uint32_t q = p->pair_base[pp] + k;
        uint32_t *r = &p->tree_rec[((size_t)pp * K + k) * H];
        const uint32_t hops = p->path_off[q + 1] - p->path_off[q];
        for (uint32_t j = 0; j < hops; j++) {
          const uint32_t l = p->path_links[p->path_off[q] + j];
          r[j] = l | ((uint32_t)p->ldst[l] << 16);
        }
        r[0] |= hops << 24;
      }
    p->owner8.resize(C);
    for (int32_t ch = 0; ch < C; ch++) p->owner8[ch] = (uint8_t)c.owner[ch];
    p->tree_rec4.clear();
    if (H <= 4) {
      p->tree_rec4.assign((size_t)P * P * K * 4, 0);
      for (size_t r = 0; r < (size_t)P * P * K; r++)
        for (int32_t j = 0; j < H; j++) p->tree_rec4[r * 4 + j] = p->tree_rec[r * H + j];
    }
    p->tent.clear();
    if (t.E <= 255) {
      p->tent.assign((size_t)P * V * P * K, 0xFF);
      for (int32_t o = 0; o < P; o++)
        for (int32_t d = 0; d < P; d++) {
          const int32_t pp = o * P + d;
          for (int32_t k = 0; k < p->npaths[pp]; k++) {
            const uint32_t q = p->pair_base[pp] + k;
            // a relay route may enter a vertex twice (a switch on both
            // legs); the first-reach merge takes the first entry
            for (uint32_t j = p->path_off[q]; j < p->path_off[q + 1]; j++) {
              const uint16_t l = p->path_links[j];
              uint8_t &slot = p->tent[(((size_t)o * V + p->ldst[l]) * P + d) * K + k];
              if (slot == 0xFF) slot = (uint8_t)l;
            }
          }
        }
    }
    path_sum_codes(p);
    p->topt.clear();
    if (K <= 8) {
      p->topt.assign((size_t)P * V * P, 0);
      for (int32_t o = 0; o < P; o++)
        for (int32_t d = 0; d < P; d++) {
          const int32_t pp = o * P + d;
          for (int32_t k = 0; k < p->npaths[pp]; k++) {
            const uint32_t q = p->pair_base[pp] + k;
            for (uint32_t j = p->path_off[q]; j < p->path_off[q + 1]; j++) {
              const int32_t v = p->ldst[p->path_links[j]];
              p->topt[((size_t)o * V + v) * P + d] |= (uint8_t)(1u << k);
            }
          }
        }
    }
  }
  return TACCL_OK;
}

}  // namespace taccl

using namespace taccl;

extern "C" {

taccl_status_t taccl_topology_create(int32_t V, int32_t P, const int32_t *row_ptr,
                                     const int32_t *col, const uint32_t *alpha_ns,
                                     const uint32_t *beta_ps_per_byte,
                                     const int32_t *node_of_vertex, taccl_topology_t *out) {
  if (!out) return fail(TACCL_ERR_INVALID_ARGUMENT, "out is null");
  *out = nullptr;
  if (V <= 0 || P <= 0 || P > V || !row_ptr)
    return fail(TACCL_ERR_INVALID_ARGUMENT, "need 0 < num_ranks <= num_vertices and row_ptr");
  if (V > 65535) return fail(TACCL_ERR_LIMIT, "more than 65535 vertices");
  if (row_ptr[0] != 0) return fail(TACCL_ERR_INVALID_ARGUMENT, "row_ptr[0] must be 0");
  for (int32_t u = 0; u < V; u++)
    if (row_ptr[u + 1] < row_ptr[u]) return fail(TACCL_ERR_INVALID_ARGUMENT, "row_ptr decreases");
  const int32_t E = row_ptr[V];
  if (E > 65535) return fail(TACCL_ERR_LIMIT, "more than 65535 links");
  if (E > 0 && (!col || !alpha_ns || !beta_ps_per_byte))
    return fail(TACCL_ERR_INVALID_ARGUMENT, "col, alpha_ns and beta_ps_per_byte are required");
  auto *t = new (std::nothrow) taccl_topology();
  if (!t) return fail(TACCL_ERR_NO_MEMORY, "topology allocation failed");
  t->V = V;
  t->P = P;
  t->E = E;
  t->row_ptr.assign(row_ptr, row_ptr + V + 1);
  t->col.assign(col, col + E);
  t->alpha.assign(alpha_ns, alpha_ns + E);
  t->beta.assign(beta_ps_per_byte, beta_ps_per_byte + E);
  t->src.resize(E);
  t->node.assign(V, 0);
  if (node_of_vertex) t->node.assign(node_of_vertex, node_of_vertex + V);
  std::set<std::pair<int32_t, int32_t>> seen;
  for (int32_t u = 0; u < V; u++)
    for (int32_t e = row_ptr[u]; e < row_ptr[u + 1]; e++) {
      int32_t v = col[e];
      if (v < 0 || v >= V || v == u || !seen.insert({u, v}).second) {
        delete t;
        return fail(TACCL_ERR_INVALID_ARGUMENT,
                    "link " + std::to_string(e) + " is a self loop, duplicate or out of range");
      }
      t->src[e] = u;
    }
  *out = t;
  return TACCL_OK;
}

void taccl_topology_destroy(taccl_topology_t t) { delete t; }

taccl_status_t taccl_collective_create(taccl_kind_t kind, int32_t P, int32_t cpr,
                                       uint64_t chunk_bytes, taccl_collective_t *out) {
  if (!out) return fail(TACCL_ERR_INVALID_ARGUMENT, "out is null");
  *out = nullptr;
  if (P <= 0 || cpr <= 0 || chunk_bytes == 0)
    return fail(TACCL_ERR_INVALID_ARGUMENT, "need num_ranks, chunks_per_rank, chunk_bytes > 0");
  const bool tree = kind == TACCL_ALLGATHER || kind == TACCL_REDUCESCATTER ||
                    kind == TACCL_ALLREDUCE;
  int64_t C = tree ? (int64_t)P * cpr : kind == TACCL_ALLTOALL ? (int64_t)P * P * cpr : -1;
  if (C < 0)
    return fail(TACCL_ERR_INVALID_ARGUMENT,
                "kind must be ALLGATHER, ALLTOALL, REDUCESCATTER or ALLREDUCE");
  if (C > 65536) return fail(TACCL_ERR_LIMIT, "more than 65536 chunks");
  auto *c = new (std::nothrow) taccl_collective();
  if (!c) return fail(TACCL_ERR_NO_MEMORY, "collective allocation failed");
  c->kind = kind;
  c->P = P;
  c->cpr = cpr;
  c->C = (int32_t)C;
  c->S = chunk_bytes;
  c->owner.resize(C);
  c->post_ptr.resize(C + 1);
  for (int32_t ch = 0; ch < C; ch++) {
    c->post_ptr[ch] = (int32_t)c->post.size();
    if (tree) {
      c->owner[ch] = ch / cpr;
      for (int32_t r = 0; r < P; r++) c->post.push_back(r);
    } else {
      int32_t pair = ch / cpr;
      c->owner[ch] = pair / P;
      c->post.push_back(pair % P);
    }
  }
  c->post_ptr[C] = (int32_t)c->post.size();
  *out = c;
  return TACCL_OK;
}

taccl_status_t taccl_collective_create_explicit(int32_t C, int32_t P, uint64_t chunk_bytes,
                                                const int32_t *owner, const int32_t *post_ptr,
                                                const int32_t *post, taccl_collective_t *out) {
  if (!out) return fail(TACCL_ERR_INVALID_ARGUMENT, "out is null");
  *out = nullptr;
  if (C <= 0 || P <= 0 || chunk_bytes == 0 || !owner || !post_ptr || (post_ptr[C] > 0 && !post))
    return fail(TACCL_ERR_INVALID_ARGUMENT, "bad explicit collective arguments");
  if (C > 65536) return fail(TACCL_ERR_LIMIT, "more than 65536 chunks");
  if (post_ptr[0] != 0) return fail(TACCL_ERR_INVALID_ARGUMENT, "post_ptr[0] must be 0");
  for (int32_t ch = 0; ch < C; ch++) {
    if (owner[ch] < 0 || owner[ch] >= P || post_ptr[ch + 1] < post_ptr[ch])
      return fail(TACCL_ERR_INVALID_ARGUMENT, "bad owner or post_ptr");
    for (int32_t j = post_ptr[ch]; j < post_ptr[ch + 1]; j++)
      if (post[j] < 0 || post[j] >= P) return fail(TACCL_ERR_INVALID_ARGUMENT, "bad post rank");
  }
  auto *c = new (std::nothrow) taccl_collective();
  if (!c) return fail(TACCL_ERR_NO_MEMORY, "collective allocation failed");
  c->kind = TACCL_EXPLICIT;
  c->P = P;
  c->cpr = 0;
  c->C = C;
  c->S = chunk_bytes;
  c->owner.assign(owner, owner + C);
  c->post_ptr.assign(post_ptr, post_ptr + C + 1);
  c->post.assign(post, post + post_ptr[C]);
  *out = c;
  return TACCL_OK;
}

void taccl_collective_destroy(taccl_collective_t c) { delete c; }

taccl_status_t taccl_sketch_apply(taccl_topology_t topo, taccl_collective_t coll,
                                  const taccl_sketch_desc_t *sk, taccl_plan_t *out) {
  if (!out) return fail(TACCL_ERR_INVALID_ARGUMENT, "out is null");
  *out = nullptr;
  if (!topo || !coll || !sk) return fail(TACCL_ERR_INVALID_ARGUMENT, "null handle or sketch");
  if (coll->P != topo->P)
    return fail(TACCL_ERR_INVALID_ARGUMENT, "collective and topology disagree on rank count");
  if (sk->route_mode < 0 || sk->route_mode > 3)
    return fail(TACCL_ERR_INVALID_ARGUMENT, "unknown route mode");
  if ((sk->route_mode == TACCL_ROUTE_SHORTEST_ONLY || sk->route_mode == TACCL_ROUTE_KSHORTEST) &&
      (sk->k <= 0 || sk->k > 255))
    return fail(TACCL_ERR_INVALID_ARGUMENT, "k must be in [1, 255]");
  auto *p = new (std::nothrow) taccl_plan();
  if (!p) return fail(TACCL_ERR_NO_MEMORY, "plan allocation failed");
  std::unique_ptr<taccl_plan> guard(p);
  p->topo = *topo;
  p->coll = *coll;
  p->mode = sk->route_mode;
  p->k = sk->k;
  p->max_cross = sk->max_node_crossings;
  if (sk->contiguity < 0 || sk->contiguity > 1)
    return fail(TACCL_ERR_INVALID_ARGUMENT, "contiguity must be 0 or 1");
  p->contig = sk->contiguity;
  if (sk->order < 0 || sk->order > 2)
    return fail(TACCL_ERR_INVALID_ARGUMENT, "order must be 0, 1 or 2");
  if (sk->switch_ports < 0 || sk->switch_ports > 1)
    return fail(TACCL_ERR_INVALID_ARGUMENT, "switch_ports must be 0 or 1");
  if (sk->switch_ports && (sk->order || sk->contiguity))
    return fail(TACCL_ERR_INVALID_ARGUMENT,
                "switch ports are not combined with greedy orders or contiguity");
  if (sk->switch_ports && coll->kind != TACCL_ALLTOALL)
    return fail(TACCL_ERR_UNSUPPORTED, "switch ports are modelled for Alltoall");
  p->ports = sk->switch_ports;
  if (sk->order && sk->contiguity)
    return fail(TACCL_ERR_INVALID_ARGUMENT, "greedy orders are not combined with contiguity");
  p->greedy = sk->order;
  const int32_t E = topo->E;
  // integer alpha-beta cost of one chunk on every link (Sec. 4.1)
  p->cost.resize(E);
  p->lsrc.resize(E);
  p->ldst.resize(E);
  uint64_t max_cost = 0;
  for (int32_t e = 0; e < E; e++) {
    uint64_t bs = (uint64_t)topo->beta[e] * coll->S;
    if (topo->beta[e] != 0 && bs / topo->beta[e] != coll->S)
      return fail(TACCL_ERR_LIMIT, "beta * chunk_bytes overflows 64 bits");
    uint64_t c = (uint64_t)topo->alpha[e] + bs / 1000 + (bs % 1000 != 0);
    if (c == 0) return fail(TACCL_ERR_INVALID_ARGUMENT, "a link has zero cost");
    if (c > 0xFFFFFFFFull) return fail(TACCL_ERR_LIMIT, "a link cost does not fit 32 bits");
    p->cost[e] = (uint32_t)c;
    max_cost = std::max(max_cost, c);
    p->lsrc[e] = (uint16_t)topo->src[e];
    p->ldst[e] = (uint16_t)topo->col[e];
  }
  p->lalpha.assign(topo->alpha.begin(), topo->alpha.end());
  p->lbs.resize(E);
  p->lmerge.assign(E, 0);
  for (int32_t e = 0; e < E; e++) {
    p->lbs[e] = (uint64_t)topo->beta[e] * coll->S;
    p->lmerge[e] = p->contig && topo->node[topo->src[e]] != topo->node[topo->col[e]];
    // a transfer of up to C chunks: beta * S * C must fit 64 bits
    if (p->lmerge[e] && (unsigned __int128)p->lbs[e] * (uint64_t)coll->C >= ((unsigned __int128)1 << 64))
      return fail(TACCL_ERR_LIMIT, "beta * chunk_bytes * chunks overflows 64 bits");
  }
  taccl_status_t st = build_routes(p, sk->allowed_link, sk->is_relay);
  if (st) return st;
  // reverse of every link (reductions run the trees backwards)
  p->lrev.assign(E, 0xFFFF);
  for (int32_t e = 0; e < E; e++)
    for (int32_t f = topo->row_ptr[topo->col[e]]; f < topo->row_ptr[topo->col[e] + 1]; f++)
      if (topo->col[f] == topo->src[e]) p->lrev[e] = (uint16_t)f;
  if (coll->kind == TACCL_REDUCESCATTER || coll->kind == TACCL_ALLREDUCE)
    for (uint16_t l : p->path_links)
      if (p->lrev[l] == 0xFFFF)
        return fail(TACCL_ERR_INVALID_ARGUMENT, "a routed link has no reverse link");
  st = build_layout(p);
  if (st) return st;
  // every time is at most the sum of all send costs (both phases of an
  // Allreduce); it must stay below 0xFFFFFFFF, the value the kernels write
  // for a candidate whose evaluation exceeded an internal bound
  const unsigned __int128 phases = coll->kind == TACCL_ALLREDUCE ? 2 : 1;
  if ((unsigned __int128)p->max_sends * max_cost * phases >= (unsigned __int128)0xFFFFFFFFu)
    return fail(TACCL_ERR_LIMIT, "worst-case makespan does not fit below 2^32 - 1");
  if (coll->kind == TACCL_ALLTOALL) {
    st = build_levels(p);
    if (st) return st;
  } else {
    if (topo->V > 64)
      return fail(TACCL_ERR_UNSUPPORTED, "multicast evaluation holds at most 64 vertices");
    if ((int64_t)coll->C * topo->V > 65535)
      return fail(TACCL_ERR_UNSUPPORTED, "multicast evaluation holds at most 65535 send slots");
    if (topo->E > 65534)
      return fail(TACCL_ERR_UNSUPPORTED, "multicast evaluation holds at most 65534 links");
    if (p->H > 255)
      return fail(TACCL_ERR_UNSUPPORTED, "multicast evaluation holds paths of at most 255 hops");
  }
  // on-chip bytes of one block (of one wavefront, where blocks hold
  // several) of the kernel the plan runs on, as the launch picks it
  if (coll->kind == TACCL_ALLTOALL) {
    PathArgs a{};
    PathGreedyArgs g{};
    if (p->greedy)
      p->path_lds = path_greedy_layout(*p, g) > 0 ? g.o_wave + g.wave_bytes
                                                  : path_greedy_block_layout(*p, g);
    else
      p->path_lds =
          (p->path_fast && path_fast_cpt(*p)) ? path_fast_layout(*p, a) : path_layout(*p, a);
  } else {
    TreeArgs a{};
    const bool any = coll->kind == TACCL_REDUCESCATTER || coll->kind == TACCL_ALLREDUCE ||
                     p->contig || p->greedy;
    const int32_t layered =
        p->greedy == 2 ? 0 : (p->greedy ? tree_greedy_layout(*p, a) : tree_layers_layout(*p, a));
    p->tree_lds = layered > 0 ? layered : any ? tree_any_layout(*p, a) : tree_layout(*p, a);
  }
  *out = guard.release();
  clear_error();
  return TACCL_OK;
}

taccl_status_t taccl_plan_info(taccl_plan_t p, taccl_plan_info_t *o) {
  if (!p || !o) return fail(TACCL_ERR_INVALID_ARGUMENT, "null plan or out");
  std::memset(o, 0, sizeof *o);
  o->num_vertices = p->topo.V;
  o->num_ranks = p->topo.P;
  o->num_links = p->topo.E;
  o->num_chunks = p->coll.C;
  o->kind = p->coll.kind;
  o->route_stride = p->route_stride;
  o->prio_stride = p->prio_stride;
  o->max_hops = p->H;
  o->max_paths = p->max_paths;
  o->num_pairs = p->num_pairs;
  o->num_levels = p->nlev;
  o->max_sends = p->max_sends;
  o->bytes_per_candidate = (uint64_t)p->route_stride + 4ull * p->prio_stride + 5ull;
  o->num_classes = p->ncls;
  o->lds_bytes = p->coll.kind == TACCL_ALLTOALL ? p->path_lds : p->tree_lds;
  return TACCL_OK;
}

taccl_status_t taccl_plan_route_options(taccl_plan_t p, int32_t *options) {
  if (!p || !options) return fail(TACCL_ERR_INVALID_ARGUMENT, "null plan or options");
  std::memcpy(options, p->route_options.data(), sizeof(int32_t) * p->route_options.size());
  return TACCL_OK;
}

taccl_status_t taccl_plan_path(taccl_plan_t p, int32_t s, int32_t d, int32_t i, int32_t *links,
                               int32_t cap, int32_t *hops) {
  if (!p || !hops || (cap > 0 && !links)) return fail(TACCL_ERR_INVALID_ARGUMENT, "null argument");
  const int32_t P = p->topo.P;
  if (s < 0 || d < 0 || s >= P || d >= P) return fail(TACCL_ERR_INVALID_ARGUMENT, "bad pair");
  size_t pp = (size_t)s * P + d;
  if (i < 0 || i >= p->npaths[pp]) return fail(TACCL_ERR_INVALID_ARGUMENT, "no such option");
  uint32_t q = p->pair_base[pp] + i;
  int32_t n = (int32_t)(p->path_off[q + 1] - p->path_off[q]);
  *hops = n;
  if (n > cap) return fail(TACCL_ERR_INVALID_ARGUMENT, "links buffer too small");
  for (int32_t j = 0; j < n; j++) links[j] = p->path_links[p->path_off[q] + j];
  return TACCL_OK;
}

taccl_status_t taccl_plan_link_costs(taccl_plan_t p, uint32_t *cost_ns) {
  if (!p || !cost_ns) return fail(TACCL_ERR_INVALID_ARGUMENT, "null argument");
  std::memcpy(cost_ns, p->cost.data(), sizeof(uint32_t) * p->cost.size());
  return TACCL_OK;
}

const char *taccl_last_error(void) { return taccl::last_error(); }

int32_t taccl_version(void) { return 100; }

}  // extern "C"
