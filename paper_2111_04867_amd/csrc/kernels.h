// Launch interface between the C ABI layer and the evaluation kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "plan.h"

namespace taccl {

// Multicast (Allgather / explicit) evaluation: one wavefront per candidate.
struct TreeArgs {
  int32_t C, P, V, E, cpr;  // cpr > 0: owner = c / cpr; else owner table
  int32_t route_stride, prio_stride;
  const uint32_t *cost;
  const uint16_t *lsrc, *ldst;
  const uint32_t *pair_base;
  const uint8_t *npaths;
  const uint32_t *path_off;
  const uint16_t *path_links;
  const int32_t *owner;
  const uint64_t *post_mask;
  const uint8_t *routes;
  const uint32_t *prio;
  uint32_t *makespan;
  uint8_t *valid;
  int64_t n;
  // LDS carve-up (byte offsets)
  int32_t o_rt, o_pr, o_par, o_dist, o_hgt, o_fin, o_ord, o_sidx, o_tmp, o_chain, o_krem,
      o_ktrav, o_lcnt, o_lhead, o_lfree, o_reach;
  int32_t lds_bytes;
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
  int32_t o_rt, o_ctime, o_lfree, o_ccnt, o_cbase, o_ccur, o_echunk, o_eprio, o_ecls, o_sorted,
      o_red;
  int32_t lds_bytes;
};

constexpr int kTreeThreads = 64;
constexpr int kPathThreads = 256;

// Fill the LDS layout; returns the bytes needed per block.
int32_t tree_layout(const taccl_plan &p, TreeArgs &a);
int32_t path_layout(const taccl_plan &p, PathArgs &a);

hipError_t launch_tree(const TreeArgs &a, int grid, hipStream_t stream);
hipError_t launch_path(const PathArgs &a, int grid, hipStream_t stream);

}  // namespace taccl
