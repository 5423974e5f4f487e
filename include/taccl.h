/*
 * taccl.h - C ABI of the MI355X evaluator of candidate collective schedules
 * (TACCL: Guiding Collective Algorithm Synthesis using Communication
 * Sketches, arXiv 2111.04867).
 *
 * The library evaluates, for many candidates at once, the part of TACCL's
 * synthesizer that follows routing: given one route per (chunk, destination)
 * pair through a sketch-restricted topology, it
 *   - orders the sends on every link with the Step-2 heuristic (Sec. 5.1,
 *     App. B.2): longest remaining path first, then shortest path already
 *     travelled, then a per-send 32-bit priority, then chunk id;
 *   - times every send under the alpha-beta model (Sec. 4.1) with strict
 *     per-link bandwidth (App. B.3), in integer nanoseconds: by default every
 *     send carries one chunk; optionally sends on links between nodes merge
 *     into contiguous transfers (taccl_sketch_desc_t.contiguity);
 *   - checks the collective's postcondition (App. B) and returns the
 *     makespan (the objective of App. B.1).
 *
 * Conventions
 *   - All functions return a taccl_status_t; on failure a message is kept per
 *     thread and returned by taccl_last_error().
 *   - Handles are opaque. create/apply deep-copy every host array they are
 *     given; the caller may free its arrays when the call returns.
 *   - Handles are immutable once built and may be used from several threads
 *     and streams at once. Each destroy function accepts NULL.
 *   - Device arrays passed to taccl_eval_batch belong to the caller.
 *   - Nothing here allocates device memory except the first evaluation of a
 *     plan on a device (or taccl_plan_upload), which uploads the plan's
 *     read-only tables to that device once; they are freed by
 *     taccl_plan_destroy.
 */
#ifndef TACCL_H
#define TACCL_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TACCL_OK = 0,
  TACCL_ERR_INVALID_ARGUMENT = 1, /* null/negative/out-of-range argument */
  TACCL_ERR_UNSUPPORTED = 2,      /* valid input the evaluator cannot handle */
  TACCL_ERR_LIMIT = 3,            /* an integer width would overflow */
  TACCL_ERR_NO_MEMORY = 4,        /* host or device allocation failed */
  TACCL_ERR_HIP = 5               /* a HIP runtime call failed */
} taccl_status_t;

/* Collectives (App. B: pre- and postcondition as (chunk, rank) pairs). */
typedef enum {
  /* chunk c = r*chunks_per_rank + j starts at rank r, must reach every rank */
  TACCL_ALLGATHER = 0,
  /* chunk c = (s*P + d)*chunks_per_rank + j starts at s, must reach d */
  TACCL_ALLTOALL = 1,
  /* one owner per chunk and an explicit list of ranks to reach (multicast) */
  TACCL_EXPLICIT = 2,
  /* chunk c = r*chunks_per_rank + j is reduced from every rank into rank r
   * along its Allgather tree run backwards (Sec. 5.2 builds ReduceScatter
   * from an Allgather algorithm): the send from v to its tree parent carries
   * v's partial, waits for every send into v and uses the reverse of the
   * tree link (every routed link needs one); Step-2 lengths are measured on
   * the reversed tree. Routes and priorities are indexed as for Allgather. */
  TACCL_REDUCESCATTER = 3,
  /* ReduceScatter then Allgather on the same trees, timed back to back; the
   * priority row is two Allgather rows, ReduceScatter's first (prio_stride
   * = 2*C*V). The makespan is the sum of the two phases. */
  TACCL_ALLREDUCE = 4
} taccl_kind_t;

/* How the candidate route options of a (source, destination) pair are
 * built from the logical topology (Sec. 3.1, Sec. 5.1 Step 1). Paths are
 * ordered by (cost, hops, lexicographic vertex sequence). */
typedef enum {
  TACCL_ROUTE_SHORTEST_ONLY = 0, /* minimal-cost simple paths, at most k */
  TACCL_ROUTE_KSHORTEST = 1,     /* the first k simple paths */
  TACCL_ROUTE_RELAY1 = 2,        /* best path, then best(s,m)+best(m,d) for
                                    relay ranks m (ascending, m != s,d) */
  TACCL_ROUTE_HIER_RELAY = 3     /* same node: best path; other node: for the
                                    i-th relay R_i of each node,
                                    best(s,R_i) + link(R_i,R'_i) + best(R'_i,d) */
} taccl_route_mode_t;

typedef struct taccl_topology *taccl_topology_t;
typedef struct taccl_collective *taccl_collective_t;
typedef struct taccl_plan *taccl_plan_t;

/* A hipStream_t, passed as an opaque pointer (NULL = the null stream). */
typedef void *taccl_stream_t;

/*
 * Physical topology (Sec. 4; alpha and beta per link, Table 1).
 *   num_vertices V: vertices [0, num_ranks) are GPU ranks, the rest are
 *     switch vertices (a store-and-forward switch with one link per port);
 *   row_ptr[V+1], col[E]: directed links in CSR form; link id = CSR index;
 *     no self loops, no duplicate (u, v);
 *   alpha_ns[E]: latency in ns; beta_ps_per_byte[E]: inverse bandwidth in
 *     ps per byte (= us per MB with MB = 10^6 B);
 *   node_of_vertex[V]: machine of every vertex, or NULL (all on one node).
 * Errors: INVALID_ARGUMENT for malformed CSR, LIMIT for more than 65535
 * links or vertices.
 */
taccl_status_t taccl_topology_create(int32_t num_vertices, int32_t num_ranks,
                                     const int32_t *row_ptr, const int32_t *col,
                                     const uint32_t *alpha_ns, const uint32_t *beta_ps_per_byte,
                                     const int32_t *node_of_vertex, taccl_topology_t *out);
void taccl_topology_destroy(taccl_topology_t topo);

/*
 * Allgather, Alltoall, ReduceScatter or Allreduce over num_ranks ranks with
 * chunks_per_rank chunks per rank (Allgather, ReduceScatter, Allreduce) or
 * per ordered rank pair (Alltoall), each chunk_bytes long (Sec. 5.2, buffer
 * size and chunk partitioning).
 */
taccl_status_t taccl_collective_create(taccl_kind_t kind, int32_t num_ranks,
                                       int32_t chunks_per_rank, uint64_t chunk_bytes,
                                       taccl_collective_t *out);

/*
 * Explicit multicast collective: chunk c starts at owner[c] and must reach
 * every rank in post[post_ptr[c] .. post_ptr[c+1]) (App. B). Evaluated like
 * Allgather (routes merge into one tree per chunk).
 */
taccl_status_t taccl_collective_create_explicit(int32_t num_chunks, int32_t num_ranks,
                                                uint64_t chunk_bytes, const int32_t *owner,
                                                const int32_t *post_ptr, const int32_t *post,
                                                taccl_collective_t *out);
void taccl_collective_destroy(taccl_collective_t coll);

/*
 * Communication sketch (Sec. 3, App. A) reduced to what routing needs.
 *   allowed_link[E]: 1 = the link is in the logical topology, or NULL;
 *   is_relay[V]: ranks allowed to send or receive across nodes (and the
 *     relay set of RELAY1 / HIER_RELAY), or NULL (every rank);
 *   max_node_crossings: node-boundary crossings allowed per path, -1 = any.
 *     With 1, a path between nodes crosses exactly once and a path inside a
 *     node never leaves it (App. B.1, inter-node constraint);
 *   route_mode, k: see taccl_route_mode_t;
 *   contiguity: 0 = every send is its own transfer (App. B.3 without
 *     contiguity); 1 = contiguous transfers on links whose endpoints lie in
 *     different nodes (the IB links of Sec. 4.1 and Step 3 of Sec. 5.1): a
 *     transfer carries the next send of the link's order and every following
 *     send of that order with the same remaining path length whose chunk is
 *     already at the link's source when the transfer starts; m chunks cost
 *     alpha + ceil(beta * m * chunk_bytes / 1000) ns and all of them arrive
 *     when the transfer ends;
 *   order: 0 = static Step-2 order per link (Sec. 5.1: remaining path desc,
 *     travelled path asc, priority, chunk); 1 = the time-aware greedy of
 *     App. B.2: round by round, among the sends whose chunk has arrived, the
 *     one that can start earliest (max of link time and chunk time) goes
 *     next, ties broken by the Step-2 key; 2 = the same greedy in reverse
 *     path order (App. B.2): it serves the mirrored schedule (every chunk
 *     dependency reversed, remaining and travelled lengths measured from
 *     the other end), each link's order is the reverse of the order it was
 *     served in, and those orders are timed as for 0. Greedy orders are not
 *     combined with contiguity (INVALID_ARGUMENT). On the GPU they are
 *     evaluated for every multicast
 *     plan (Allgather, explicit, ReduceScatter, Allreduce) and for Alltoall
 *     plans with at most 4096 chunks and 65535 send slots (chunks x longest
 *     route option) and no zero-cost link; larger Alltoall plans are
 *     refused at evaluation (UNSUPPORTED);
 *   switch_ports (Alltoall only): 0 = a switch vertex stores and forwards
 *     (uplink, then downlink, each one latency); 1 = the switch model of
 *     App. B.3: a hop pair rank -> switch -> rank is one send costing one
 *     latency (the uplink's alpha and beta) that holds the sender's send
 *     port (uplink) and the receiver's receive port (downlink) for its whole
 *     duration, each port serving its sends in Step-2 order (App. B.2's
 *     switch send and receive orders). Not combined with contiguity or
 *     greedy orders (INVALID_ARGUMENT); other kinds, and topologies where a
 *     link would be a send port of some switched sends and a receive port
 *     of others (a switch-to-switch link), are refused (UNSUPPORTED).
 */
typedef struct {
  const uint8_t *allowed_link;
  const uint8_t *is_relay;
  int32_t max_node_crossings;
  int32_t route_mode;
  int32_t k;
  int32_t contiguity;
  int32_t order;
  int32_t switch_ports;
} taccl_sketch_desc_t;

/*
 * Build an evaluation plan: link costs alpha + ceil(beta*chunk_bytes/1000)
 * ns, route options per pair, layouts and the per-level tables the kernels
 * read. Host only; device tables are uploaded on first use.
 * Errors: INVALID_ARGUMENT (mismatched ranks, bad mode), LIMIT (a link cost
 * or the worst-case makespan does not fit 32 bits, more than 255 options
 * per pair), UNSUPPORTED (sizes beyond what the kernels hold on chip).
 */
taccl_status_t taccl_sketch_apply(taccl_topology_t topo, taccl_collective_t coll,
                                  const taccl_sketch_desc_t *sketch, taccl_plan_t *out);
void taccl_plan_destroy(taccl_plan_t plan);

typedef struct {
  int32_t num_vertices, num_ranks, num_links, num_chunks;
  int32_t kind;         /* taccl_kind_t */
  int32_t route_stride; /* bytes of routes per candidate */
  int32_t prio_stride;  /* uint32 priorities per candidate */
  int32_t max_hops;     /* longest route option, in links */
  int32_t max_paths;    /* most route options of any pair */
  int32_t num_pairs;    /* route entries that carry a choice */
  int32_t num_levels;   /* Alltoall: distinct remaining-path costs */
  int64_t max_sends;    /* most sends one candidate can have */
  uint64_t bytes_per_candidate; /* routes + priorities + 5 output bytes */
  int32_t num_classes;  /* Alltoall: (level, link, travelled) send classes */
  int32_t lds_bytes;    /* LDS of one block (one wavefront's, where blocks
                           hold several) of the kernel the plan runs on;
                           above the device's limit, evaluation refuses */
} taccl_plan_info_t;

/*
 * Candidate layout, per candidate i (rows are contiguous):
 *   routes[i*route_stride + e], uint8: route option chosen for entry e.
 *     Allgather/explicit: e = c*P + d (chunk c to rank d); Alltoall: e = c.
 *     A value >= the entry's option count leaves the pair unrouted, which
 *     is not an error (the candidate may then fail its postcondition).
 *   prio[i*prio_stride + q], uint32: tie-break priority of send slot q.
 *     Allgather/explicit: q = c*V + v (the send that brings c into v);
 *     Alltoall: q = c*max_hops + h (hop h of chunk c's path).
 */
taccl_status_t taccl_plan_info(taccl_plan_t plan, taccl_plan_info_t *out);

/* options[route_stride]: number of route options of every route entry
 * (0 for entries no pair uses). */
taccl_status_t taccl_plan_route_options(taccl_plan_t plan, int32_t *options);

/* Links of option `index` of pair (src, dst), hop order, into links[cap];
 * *hops = its length. INVALID_ARGUMENT if the option does not exist. */
taccl_status_t taccl_plan_path(taccl_plan_t plan, int32_t src, int32_t dst, int32_t index,
                               int32_t *links, int32_t cap, int32_t *hops);

/* cost_ns[num_links]: integer alpha-beta cost of one chunk on every link. */
taccl_status_t taccl_plan_link_costs(taccl_plan_t plan, uint32_t *cost_ns);

/* Upload the plan's read-only tables to the current device now (otherwise
 * done by the first taccl_eval_batch on that device). Allocates. */
taccl_status_t taccl_plan_upload(taccl_plan_t plan);

/*
 * Evaluate n candidates on the current device, asynchronously on `stream`.
 *   d_routes: device, n*route_stride bytes;
 *   d_prio: device, n*prio_stride uint32, 4-byte aligned;
 *   d_makespan: device, n uint32: latest finish over all sends in ns (0 if
 *     the candidate sends nothing);
 *   d_valid: device, n uint8: 1 if every (chunk, rank) pair of the
 *     postcondition holds at the end, else 0.
 * Each candidate is evaluated independently; results are exact (integer).
 * Every real makespan is below TACCL_MAKESPAN_FAULT (taccl_sketch_apply
 * refuses plans whose worst case, the sum of all send costs over both
 * phases of an Allreduce, could reach it). A candidate whose evaluation
 * exceeded a bound the kernel relies on (a round limit of an iterative
 * schedule, a layer index past the plan's bound, a switch-port walk that
 * stops making progress; none is reachable for a plan that
 * taccl_sketch_apply accepted) comes back as makespan ==
 * TACCL_MAKESPAN_FAULT with valid == 0, so such an internal fault is never
 * mistaken for a bad candidate; taccl_count_faults counts them.
 * Errors (synchronous): INVALID_ARGUMENT for null pointers with n > 0,
 * n < 0 or a misaligned d_prio; UNSUPPORTED when a candidate's state does
 * not fit one block's LDS, an Alltoall greedy plan exceeds its limits, or a
 * switch-port plan has more than four links per thread of its block; HIP if
 * the plan upload or the launch fails.
 * Faults inside the kernel surface at the caller's next synchronisation.
 * n == 0 is a no-op.
 */
taccl_status_t taccl_eval_batch(taccl_plan_t plan, int64_t n, const uint8_t *d_routes,
                                const uint32_t *d_prio, uint32_t *d_makespan, uint8_t *d_valid,
                                taccl_stream_t stream);

/* Makespan written for a candidate whose evaluation hit an internal fault. */
#define TACCL_MAKESPAN_FAULT 0xFFFFFFFFu

/*
 * Host check of a batch's results after synchronisation: the number of
 * candidates i < n with makespan[i] == TACCL_MAKESPAN_FAULT (host arrays,
 * owned by the caller). A nonzero count means a kernel fault, not a bad
 * candidate. Errors: INVALID_ARGUMENT for a null array with n > 0 or n < 0.
 */
taccl_status_t taccl_count_faults(int64_t n, const uint32_t *makespan, int64_t *faults);

/*
 * Switch-hyperedge connections of n candidates on the current device,
 * asynchronously on `stream` (Sec. 3.2; Sec. 5.1, switch-hyperedge policy;
 * App. B.3: is_util[src, r] = 1 when some chunk goes from GPU src to GPU r
 * over switched links, and the uc-max / uc-min policies minimise
 * time + gamma * sum(is_util) with gamma < 0 for uc-max and gamma > 0 for
 * uc-min).
 *   d_routes: device, n*route_stride bytes, laid out as for taccl_eval_batch
 *     (priorities play no part in the count);
 *   d_connections: device, n uint32, 4-byte aligned: the number of ordered
 *     rank pairs (a, b) that exchange a chunk through switch vertices only.
 *     Alltoall: two ranks of a chunk's routed path with only switch
 *     vertices between them. Multicast (Allgather, explicit): a rank whose
 *     tree parent is a switch vertex, paired with the nearest rank above it
 *     in the chunk's tree (first-reach merge of its routed paths,
 *     destinations ascending); ReduceScatter reverses every pair and
 *     Allreduce counts both directions. 0 on topologies without switch
 *     vertices. Unrouted pairs contribute nothing.
 * A caller ranks candidates under a policy by makespan + gamma * count.
 * Errors (synchronous): INVALID_ARGUMENT for null pointers with n > 0,
 * n < 0 or a misaligned d_connections; UNSUPPORTED for more than 256 ranks
 * (multicast: more than 64 ranks or 255 vertices); HIP if the plan upload or
 * the launch fails. n == 0 is a no-op.
 */
taccl_status_t taccl_connections_batch(taccl_plan_t plan, int64_t n, const uint8_t *d_routes,
                                       uint32_t *d_connections, taccl_stream_t stream);

/*
 * Seeded synthetic candidates on the host: the counter-based generator the
 * tests and the benchmark feed to taccl_eval_batch (SplitMix64 of a counter
 * keyed by stream, candidate and entry, so any candidate range comes out the
 * same on its own). For candidates first .. first+count-1 it writes
 *   routes[count][route_stride]: per route entry a uniform choice among its
 *     route options (Sec. 5.1 Step 1 leaves each chunk a set of shortest
 *     paths), 0 for entries without options;
 *   prio[count][prio_stride]: uniform 32-bit priorities (the final tie-break
 *     of the Step-2 order).
 * Host buffers, owned by the caller. Errors: INVALID_ARGUMENT for a null
 * plan, null buffers with count > 0, first < 0, count < 0 or
 * first + count > 2^32. count == 0 is a no-op.
 */
taccl_status_t taccl_generate_host(taccl_plan_t plan, uint64_t seed, int64_t first, int64_t count,
                                   uint8_t *routes, uint32_t *prio);

/* Message of the last failed call on this thread ("" if none). */
const char *taccl_last_error(void);

/* Library version: major*10000 + minor*100 + patch. */
int32_t taccl_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TACCL_H */
