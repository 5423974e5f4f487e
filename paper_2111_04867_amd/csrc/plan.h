// Internal plan structures of the evaluator library (not part of the ABI).
#pragma once

#include <cstdint>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "taccl.h"

namespace taccl {

// Limits of the register-resident Alltoall kernel.
constexpr int kFastMaxHops = 6;
constexpr int kFastMaxChunks = 4096;
// priority sub-buckets of all levels together in the register-resident
// Alltoall kernel (one LDS counter each)
constexpr int kFastMaxBuckets = 16384;
// chunk table entry of a pair that has no route option at all
constexpr uint32_t kNoRoute = 0x00FFFFFFu;

// Set the thread-local error message and return the status.
taccl_status_t fail(taccl_status_t st, const std::string &msg);

}  // namespace taccl

struct taccl_topology {
  int32_t V = 0, P = 0, E = 0;
  std::vector<int32_t> row_ptr, col, src, node;
  std::vector<uint32_t> alpha, beta;
};

struct taccl_collective {
  int32_t kind = 0, P = 0, cpr = 0, C = 0;
  uint64_t S = 0;
  std::vector<int32_t> owner;     // [C]
  std::vector<int32_t> post_ptr;  // [C+1]
  std::vector<int32_t> post;      // ranks to reach
};

namespace taccl {

// Device copies of the read-only plan tables (one set per device).
struct DeviceTables {
  void *block = nullptr;  // one allocation holding every table
  const uint32_t *cost = nullptr;
  const uint16_t *lsrc = nullptr, *ldst = nullptr;
  const uint32_t *pair_base = nullptr;
  const uint8_t *npaths = nullptr;
  const uint32_t *path_off = nullptr;
  const uint16_t *path_links = nullptr;
  const int32_t *owner = nullptr;
  const uint64_t *post_mask = nullptr;
  const uint32_t *tree_rec = nullptr;
  const uint8_t *owner8 = nullptr;
  const uint8_t *topt = nullptr;
  const uint32_t *tree_rec4 = nullptr;
  const uint8_t *tent = nullptr;
  const uint32_t *lalpha = nullptr;
  const uint64_t *lbs = nullptr;
  const uint8_t *lmerge = nullptr;
  const uint16_t *lrev = nullptr;
  const uint16_t *hop_class2 = nullptr, *cls2_link = nullptr;
  const uint32_t *lvl_cls2_begin = nullptr, *llc2 = nullptr;
  const uint16_t *hop_class = nullptr;
  const int8_t *path_lvl_hop = nullptr;
  const uint32_t *lvl_cls_begin = nullptr;
  const uint32_t *llc = nullptr;
  const uint32_t *arec = nullptr, *cpath = nullptr, *cinfo = nullptr, *cbkt = nullptr;
  const uint32_t *gkrank = nullptr;
  int max_lds = 0;  // bytes of LDS a block may use on this device
  int lds_per_cu = 0;
  int num_cus = 0;
};

}  // namespace taccl

struct taccl_plan {
  taccl_topology topo;
  taccl_collective coll;
  int32_t mode = 0, k = 0, max_cross = -1;

  // link tables
  std::vector<uint32_t> cost;  // [E] integer alpha-beta cost in ns
  std::vector<uint16_t> lsrc, ldst;
  // contiguous transfers: per link alpha, beta * chunk_bytes and whether the
  // link joins two nodes (only those merge)
  int32_t contig = 0;
  int32_t greedy = 0;  // link orders from the time-aware greedy
  int32_t ports = 0;   // Alltoall: switched sends hold a send and a receive port
  std::vector<uint32_t> lalpha;
  std::vector<uint64_t> lbs;
  std::vector<uint8_t> lmerge;
  std::vector<uint16_t> lrev;  // link in the opposite direction, 0xFFFF if none

  // route options per ordered rank pair (s, d), pair index s*P + d
  std::vector<uint32_t> pair_base;  // [P*P] first option's global path index
  std::vector<uint8_t> npaths;      // [P*P]
  std::vector<uint32_t> path_off;   // [NPATH+1] into path_links
  std::vector<uint16_t> path_links;
  std::vector<uint64_t> path_cost;  // [NPATH]

  int32_t H = 0, max_paths = 0, num_pairs = 0;
  int32_t route_stride = 0, prio_stride = 0;
  int64_t max_sends = 0;
  std::vector<int32_t> route_options;  // [route_stride]

  // multicast (tree) evaluation
  std::vector<uint64_t> post_mask;  // [C], ranks a chunk must reach
  // fixed-stride route records, one word per hop of option k of pair (s,d)
  // at [((s*P+d)*max_paths + k)*H + j]: link | dst << 16 | (hops << 24 on
  // the first word); options a pair does not have are all zero (no hops)
  std::vector<uint32_t> tree_rec;
  std::vector<uint8_t> owner8;      // [C] owner rank of every chunk
  // [(o*V + v)*P + d]: bit k set when option k of pair (o, d) passes
  // through vertex v (v != o); empty unless every pair has at most 8 options
  std::vector<uint8_t> topt;
  // the route records again with 4 words per option (zero padded), for
  // plans with at most 4 hops
  std::vector<uint32_t> tree_rec4;
  // [((o*V + v)*P + d)*max_paths + k]: the link by which option k of pair
  // (o, d) enters vertex v (0xFF where it does not pass v); empty unless
  // every link id fits 8 bits
  std::vector<uint8_t> tent;
  // Exact order-preserving compression of tree-path lengths: every
  // remaining or travelled length of a multicast send is a sum of at most
  // V - 1 link costs, and x -> (x * pq_magic) >> 32 is strictly increasing
  // on the set of such sums, with values below pq_range (0: the set is too
  // large or too dense for 11-bit codes)
  uint64_t pq_magic = 0;
  int32_t pq_range = 0;

  // Alltoall (path) evaluation: levels of equal remaining cost
  int32_t nlev = 0, ncls = 0, max_lvl_cls = 0, max_lvl_sends = 0;
  std::vector<uint16_t> hop_class;     // [path_links.size()] class of each hop's send
  // switch ports: receive-port class of each switched send's first hop
  std::vector<uint16_t> hop_class2;
  std::vector<uint16_t> cls2_link;  // [receive-port classes]: the downlink
  std::vector<uint32_t> lvl_cls2_begin, llc2;
  int32_t max_lvl_cls2 = 0;
  std::vector<int8_t> path_lvl_hop;    // [NPATH*nlev] hop at each level or -1
  std::vector<uint32_t> lvl_cls_begin; // [nlev+1]
  std::vector<uint32_t> llc;           // [nlev*E*2] class range of a link at a level
  std::vector<uint16_t> cls_link;      // [ncls]
  // register-resident Alltoall kernel: per route option {hops | the hop at
  // each level (3 bits per level, 7: none) << 8, classes of hops 0..5 as u16
  // pairs}, option q at record q + 1 after an empty record 0; per chunk its
  // pair's first record | option count << 24 (kNoRoute: the pair has no
  // option);
  // per class link | (first bucket of the same level and link) << 16
  bool path_fast = false;
  std::vector<uint32_t> arec, cpath, cinfo;
  // per class: first priority sub-bucket | bits << 24. Buckets are numbered
  // over all levels at once (level by level, class by class), nb_total of
  // them.
  std::vector<uint32_t> cbkt;
  int32_t nb_total = 0;
  // Alltoall greedy orders: per hop (index into path_links) the rank of its
  // Step-2 key (remaining desc, travelled asc) among all hops of the plan,
  // with the lengths of the greedy's direction (mirrored in reverse path
  // order), and the number of distinct ranks
  std::vector<uint32_t> gkrank;
  int32_t gk_count = 0;

  // launch shape
  int32_t tree_lds = 0, path_lds = 0;

  std::mutex mu;
  std::map<int, taccl::DeviceTables> dev;
};
