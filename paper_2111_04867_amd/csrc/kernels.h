// Launch interface between the C ABI layer and the evaluation kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "plan.h"

namespace taccl {

// Multicast (Allgather / explicit) evaluation: persistent blocks of
// wavefronts, one candidate per wavefront at a time.
struct TreeArgs {
  int32_t C, P, V, E, K, H, mask_words;
  int32_t route_stride, prio_stride, routes_word_aligned;
  uint32_t vmagic;  // floor(2^32 / V) + 1
  const uint32_t *cost;
  const uint16_t *lsrc, *ldst;
  const uint32_t *rec;  // fixed-stride route records (one word per hop)
  int32_t rec_len, rec_in_lds;
  const uint8_t *npaths;
  const uint8_t *owner8;
  const uint64_t *post_mask;
  const uint8_t *routes;
  const uint32_t *prio;
  uint32_t *makespan;
  uint8_t *valid;
  int64_t n;
  int32_t waves_per_block;
  // LDS carve-up: shared tables (byte offsets from the block's base)
  int32_t o_cost, o_src, o_rec, o_own, o_post, o_wave;
  // per-wavefront state (byte offsets from the wavefront's base)
  int32_t w_rt, w_key, w_prio, w_chain, w_par, w_mask, w_base, w_head, w_free;
  int32_t wave_bytes;
  // layered variant: layer of a send = (rem * lmagic) >> 32, below nl_max
  uint64_t lmagic;
  int32_t nl_max;
  // contiguous transfers on links between nodes (contig != 0)
  int32_t contig;
  const uint32_t *lalpha;
  const uint64_t *lbs;    // beta * chunk_bytes per link
  const uint8_t *lmerge;  // 1: the link joins two nodes
  int32_t o_merge;
  // reductions: reverse of every link; 1 = add makespan to the output and
  // and valid into it (the Allgather phase of an Allreduce)
  const uint16_t *lrev;
  int32_t o_rev, o_ldst, accumulate, reduce;
  // time-aware greedy orders: smallest link cost (the simulation's
  // lookahead) and per-wavefront arrays
  uint32_t cmin;
  int32_t w_gfin, w_grdy, w_gpend, w_glist, w_gofs;
  const uint8_t *topt;  // options of (o, d) through vertex v, one byte per d
  const uint4 *rec4;    // route records, one 16-byte record per option
  int32_t o_rec4, o_opt;
  int32_t w_dist, w_cnt, w_erec, w_rq, w_lst, w_bnd, w_ord2, w_info2, w_fin, w_lmask;
  // ancestor doubling of the slot-parallel trees: rounds (2^rounds >= V) and
  // the per-round arrays of 16-bit slots (anc_stride slots apart)
  int32_t w_anc, pj_rounds, anc_stride;
  // general variant (any != 0): time-aware greedy instead of the static
  // order, and the per-link state of open contiguous transfers
  int32_t any, greedy, w_gst;
  // ranked variant: exact order-preserving codes of path lengths
  // (code = (x * qmagic) >> 32 < qrange), the entering-link table, the
  // per-slot heights and the parent send of each bucket-sorted position
  uint64_t qmagic;
  int32_t qrange;
  const uint8_t *ent;
  int32_t o_ent, w_h, o_slot, opt_ostride, w_pj;
};

// Alltoall evaluation: one block per candidate, level by level.
struct PathArgs {
  int32_t C, P, E, H, cpr, nlev;
  int32_t route_stride, prio_stride;
  const uint32_t *cost;
  const uint32_t *pair_base;
  const uint8_t *npaths;
  const uint32_t *path_off;
  const uint16_t *hop_class;
  const int8_t *path_lvl_hop;
  const uint32_t *lvl_cls_begin;
  const uint32_t *llc;
  const uint8_t *routes;
  const uint32_t *prio;
  uint32_t *makespan;
  uint8_t *valid;
  int64_t n;
  int32_t o_qc, o_ctime, o_lfree, o_ccnt, o_ccur, o_e64, o_ecls, o_sorted, o_red, max_lvl;
  // register-resident kernel
  int32_t ncls, nb_total;
  // route_stride a multiple of 4 and the routes 4-byte aligned: a chunk's
  // route byte is read with the aligned word that holds it
  int32_t routes_words;
  const uint32_t *arec, *cpath, *cinfo, *cbkt;
  int32_t o_faux;
  int32_t o_fnext, o_fcinfo, o_fcbkt, o_flcb, o_fctime, o_flfree, o_fbcnt, o_fepr, o_fsrt, o_fred;
  int32_t lds_bytes;
  int32_t cbits, lbits;  // chunk and link fields of a packed sorted send
  // contiguous transfers on links between nodes (contig != 0)
  int32_t contig;
  const uint32_t *lalpha;
  const uint64_t *lbs;    // beta * chunk_bytes per link
  const uint8_t *lmerge;  // 1: the link joins two nodes
  int32_t o_fmerge;
  // switch ports (LDS-record kernel): receive-port classes and state
  int32_t ports;
  const uint16_t *hop_class2, *cls2_link;
  const uint32_t *lvl_cls2_begin, *llc2;
  int32_t o_ccnt2, o_ccur2, o_sorted2, o_fcur, o_pd, o_dl;
  int32_t lr_threads;  // block size of the LDS-record kernel for this plan
};

// Time-aware greedy orders for Alltoall: persistent blocks of wavefronts,
// one candidate per wavefront at a time (send slots c*H + h).
struct PathGreedyArgs {
  int32_t C, P, E, H, cpr, nslots;
  int32_t route_stride, prio_stride;
  uint32_t cmin;
  const uint32_t *cost;
  const uint32_t *pair_base;
  const uint8_t *npaths;
  const uint32_t *path_off;
  const uint16_t *path_links;
  const uint8_t *routes;
  const uint32_t *prio;
  uint32_t *makespan;
  uint8_t *valid;
  int64_t n;
  int32_t waves_per_block;
  // LDS: link costs, then per wavefront finish times per slot, list
  // offsets and fill pointers per link, pending-send records
  int32_t o_wave, wave_bytes, w_gfin, w_gofs, w_gcur, w_grec;
  int32_t mirror;  // greedy in reverse path order
  // block-per-candidate variant for larger plans: Step-2 key rank of every
  // hop (plan table), chunks per thread and the LDS carve-up
  const uint32_t *gkrank;
  int32_t cpt, block_bytes;
  int32_t b_cost, b_lfree, b_best1, b_best2, b_lserv, b_lnext, b_red, b_fpos, b_sprio;
  // one-word window keys: start - previous window start (clamped to
  // rel_max) << rel_shift | key rank << kr_shift | priority << chunk_bits |
  // chunk, when they fit 64 bits (pack != 0)
  int32_t pack, rel_shift, kr_shift, chunk_bits;
  uint32_t rel_max;
};

// Switch-hyperedge connection count: one block per candidate at a time.
struct ConnArgs {
  int32_t C, P, V, cpr, kind, tree, mask_words;  // mask_words: ceil(P*P / 32)
  int32_t route_stride;
  const uint16_t *ldst;
  const uint32_t *pair_base;
  const uint8_t *npaths;
  const uint32_t *path_off;
  const uint16_t *path_links;
  const int32_t *owner;
  const uint64_t *post_mask;
  const uint8_t *routes;
  uint32_t *out;
  int64_t n;
};

constexpr int kConnMaxThreads = 256;

constexpr int kTreeMaxThreads = 512;  // up to 8 wavefronts per block
// (chunk, vertex) slots per lane of the layered, greedy and ranked multicast
// kernels: at most 8, i.e. C x V <= 512 (beyond that their register state
// would spill to scratch; larger plans run on the general kernel)
constexpr int kLayerMaxSlotsPerLane = 8;
constexpr int kRankMaxThreads = 768;  // ranked multicast kernel: up to 12
constexpr int kTreeRecLdsMax = 32768;  // route records kept in LDS up to this size
constexpr int kPathThreads = 256;
constexpr int kPathPortThreads = 1024;  // LDS-record kernel on switch-port plans
constexpr int kPathFastThreads = 1024;  // largest block of the register-resident kernel

// Fill the LDS layout; returns the bytes needed by a one-wavefront block.
int32_t tree_layout(const taccl_plan &p, TreeArgs &a);
// The same for the general variant (ReduceScatter, contiguous transfers and
// greedy orders on plans outside the layered kernel's limits).
int32_t tree_any_layout(const taccl_plan &p, TreeArgs &a);
int32_t tree_block_bytes(const TreeArgs &a, int waves);
// Ranked multicast kernel (static orders, no contiguity, trees forwards):
// fills the layout and returns the bytes of a one-wavefront block, or 0
// when the plan does not meet its conditions.
int32_t tree_rank_layout(const taccl_plan &p, TreeArgs &a);
// the ranked kernel may run the plan's ReduceScatter (reverse links with
// equal costs, no contiguity)
bool tree_rank_reverse_ok(const taccl_plan &p);
int tree_rank_blocks_per_cu(const TreeArgs &a);
hipError_t launch_tree_rank(const TreeArgs &a, int grid, hipStream_t stream);
// Layered multicast kernel: fills the layout and returns the bytes of a
// one-wavefront block, or 0 when the plan does not meet its conditions.
int32_t tree_layers_layout(const taccl_plan &p, TreeArgs &a);
// Time-aware greedy variant (same shared tables, own per-wavefront arrays):
// bytes of a one-wavefront block, or 0 when the plan does not fit it.
int32_t tree_greedy_layout(const taccl_plan &p, TreeArgs &a);
hipError_t launch_tree_greedy(const TreeArgs &a, int grid, hipStream_t stream);
int tree_greedy_blocks_per_cu(const TreeArgs &a);
int32_t path_layout(const taccl_plan &p, PathArgs &a);
int32_t path_fast_layout(const taccl_plan &p, PathArgs &a);
int path_fast_cpt(const taccl_plan &p);      // chunks per thread, 0 = not eligible
int path_fast_threads(const taccl_plan &p);  // threads per block: 256, 512 or 1024
int path_fast_blocks_per_cu(const PathArgs &a, int cpt, int nt);

hipError_t launch_tree(const TreeArgs &a, int grid, hipStream_t stream);
// Alltoall greedy: fills the layout; returns the bytes of a one-wavefront
// block, or 0 when the plan has more than 1024 send slots or 256 links
int32_t path_greedy_layout(const taccl_plan &p, PathGreedyArgs &a);
int path_greedy_blocks_per_cu(const PathGreedyArgs &a);
hipError_t launch_path_greedy(const PathGreedyArgs &a, int grid, hipStream_t stream);
// Alltoall greedy, one block per candidate (plans beyond the wavefront
// kernel): fills the layout; returns the block's LDS bytes, or 0 when the
// plan has more than 8 chunks per thread (8192 chunks), 65535 send slots or
// a zero-cost link
constexpr int kGreedyBlockThreads = 1024;
int32_t path_greedy_block_layout(const taccl_plan &p, PathGreedyArgs &a);
int path_greedy_block_per_cu(const PathGreedyArgs &a);
hipError_t launch_path_greedy_block(const PathGreedyArgs &a, int grid, hipStream_t stream);
// connection count: LDS bytes of a block of `threads`, and the launch
int32_t connections_lds_bytes(const ConnArgs &a, int threads);
hipError_t launch_connections(const ConnArgs &a, int threads, int grid, hipStream_t stream);
hipError_t launch_tree_layers(const TreeArgs &a, int grid, hipStream_t stream);
// resident blocks per CU of the layered kernel at a.waves_per_block
int tree_layers_blocks_per_cu(const TreeArgs &a);
hipError_t launch_path(const PathArgs &a, int grid, hipStream_t stream);
hipError_t launch_path_fast(const PathArgs &a, int cpt, int nt, int grid, hipStream_t stream);

}  // namespace taccl
