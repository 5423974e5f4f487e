/*
 * CPU oracle for batched evaluation of candidate collective schedules
 * (TACCL, arXiv 2111.04867).
 *
 * TEST INFRASTRUCTURE ONLY. This file is the plain, slow, sequential
 * definition against which the GPU evaluator is checked. Only the tests,
 * the smoke check and the CPU-baseline leg of the benchmark may load it.
 * It shares no code, header, table or constant with the GPU library.
 *
 * What it computes, per candidate (a route choice per (chunk, destination)
 * pair plus one 32-bit priority per send slot):
 *   1. link cost under the alpha-beta model of Sec. 4.1 (Table 1), in
 *      integer ns: alpha + ceil(beta_ps_per_byte * chunk_bytes / 1000);
 *   2. the send set: Allgather chunks are multicast, so the routed paths of
 *      one chunk are merged into a tree by first reach (destinations in
 *      ascending rank order); this gives one is_sent per (chunk, link) as in
 *      the routing encoding of App. B.1. Alltoall chunks follow their path;
 *   3. the Step-2 ordering heuristic of Sec. 5.1 / App. B.2 as a static
 *      per-link total order: longest remaining path first, then shortest
 *      path already travelled, then the candidate's priority, then chunk id;
 *   4. the exact schedule of App. B.3 with no contiguity (every send carries
 *      one chunk): send >= start at the source, start = send + lat, and the
 *      strict per-link order. The least solution of these difference
 *      constraints is found by a topological sweep (Kahn's algorithm).
 *      Optionally (orc_set_contiguity), sends on links between nodes are
 *      merged into contiguous transfers (Sec. 4.1, Step 3 of Sec. 5.1, the
 *      is_together constraints of App. B.3): a transfer carries the next
 *      send of the link's order and every following send of that order with
 *      the same remaining length that is ready when it starts; it costs
 *      alpha + ceil(beta * m * S / 1000) for m chunks and all of them
 *      arrive when it ends;
 *   5. the postcondition of App. B (every (chunk, rank) pair it lists holds)
 *      and the makespan, the objective of App. B.1 (latest finishing send).
 *
 * Optionally (orc_set_order), the per-link orders come from the time-aware
 * greedy of App. B.2 instead of the static rule: round by round, among the
 * sends whose chunk has arrived at their source, the one that can start
 * earliest (max of its link's time and its chunk's time) is scheduled next,
 * ties broken by the Step-2 heuristics, then priority, then chunk id; its
 * link and chunk times advance by the link latency. The orders it produces
 * are timed by the same rule as above (the greedy's own times). Mode 2 runs
 * the greedy in reverse path order (see reverse_greedy_orders).
 *
 * Optionally (orc_set_switch_ports), Alltoall hops through a switch vertex
 * follow the switch model of App. B.3: the pair rank -> switch -> rank is one
 * switched send costing one latency (the uplink's alpha and beta) that holds
 * the sender's send port (its uplink) and the receiver's receive port (its
 * downlink) for its whole duration; each port serves its sends in Step-2
 * order (switch_send_order / switch_recv_order of App. B.2).
 *
 * ReduceScatter and Allreduce (Sec. 5.2, which builds them from an
 * Allgather algorithm): ReduceScatter runs every chunk's Allgather tree
 * backwards. The send from v to its tree parent carries v's partial
 * reduction, so it waits for every send into v; Step 2 measures remaining
 * and travelled lengths on the reversed tree (remaining: reversed distance
 * from v to the owner; travelled: longest reversed path from a vertex below
 * v up to v). Allreduce is ReduceScatter then Allgather on the same trees,
 * timed back to back, with a separate priority row for each phase.
 *
 * Operation count (orc_eval_ops): per candidate, the algorithmic integer
 * operations of the op model described at phase_ops, for pricing the
 * evaluation against an integer-issue roofline.
 *
 * Connections (orc_connections): per candidate, the number of ordered rank
 * pairs that exchange a chunk through switch vertices only, the is_util
 * count that the uc-max / uc-min switch-hyperedge policies weigh in the
 * objective (Sec. 5.1, App. B.3).
 *
 * Paths: the sketch of Sec. 3.1 restricts links; routes are limited to
 * shortest paths in the logical topology (Sec. 5.1, Step 1). Paths are found
 * here by exhaustive depth-first search with cost pruning and sorted by
 * (cost, hops, lexicographic vertex sequence).
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

enum { ORC_ALLGATHER = 0, ORC_ALLTOALL = 1, ORC_EXPLICIT = 2, ORC_REDUCESCATTER = 3,
       ORC_ALLREDUCE = 4 };
enum { ORC_SHORTEST_ONLY = 0, ORC_KSHORTEST = 1, ORC_RELAY1 = 2, ORC_HIER_RELAY = 3 };

#define ORC_OK 0
#define ORC_EINVAL 1
#define ORC_ELIMIT 2
#define ORC_ENOMEM 3

typedef struct {
  int hops;
  int *link; /* [hops] */
  int *vert; /* [hops+1] */
  uint64_t cost;
} opath;

typedef struct {
  int n;
  opath *p;
} oplist;

typedef struct orc_plan {
  /* topology (CSR, link id = CSR edge index) */
  int V, P, E;
  int *row_ptr, *col, *lsrc, *node;
  uint32_t *alpha, *beta;
  /* collective */
  int kind, cpr, C;
  uint64_t S;
  int *owner;    /* [C] */
  int *post_ptr; /* [C+1] */
  int *post;     /* ranks that must hold the chunk at the end */
  /* sketch */
  uint8_t *allowed, *relay;
  int max_cross, mode, k;
  /* derived */
  uint64_t *cost; /* [E] */
  oplist *paths;  /* [P*P], by (source rank, destination rank) */
  int H;          /* longest path in hops */
  int route_stride, prio_stride;
  int max_sends;
  int contig; /* merge contiguous sends on links between nodes */
  int greedy; /* per-link orders from the time-aware greedy (App. B.2) */
  int ports;  /* Alltoall: switched sends hold a send and a receive port */
  int *rev;   /* [E] link in the opposite direction, or -1 */
  char err[256];
} orc_plan;

/* ------------------------------------------------------------------ */
/* paths                                                               */
/* ------------------------------------------------------------------ */

/* Order of Sec. 5.1's shortest-path restriction, made total:
 * cost, then hop count, then vertex sequence. */
static int path_cmp(const opath *a, const opath *b) {
  if (a->cost != b->cost) return a->cost < b->cost ? -1 : 1;
  if (a->hops != b->hops) return a->hops < b->hops ? -1 : 1;
  for (int i = 0; i <= a->hops; i++)
    if (a->vert[i] != b->vert[i]) return a->vert[i] < b->vert[i] ? -1 : 1;
  return 0;
}

static opath path_make(int hops, const int *link, const int *vert, uint64_t cost) {
  opath p;
  p.hops = hops;
  p.cost = cost;
  p.link = (int *)malloc(sizeof(int) * (hops > 0 ? hops : 1));
  p.vert = (int *)malloc(sizeof(int) * (hops + 1));
  if (hops > 0) memcpy(p.link, link, sizeof(int) * hops);
  memcpy(p.vert, vert, sizeof(int) * (hops + 1));
  return p;
}

static void path_free(opath *p) {
  free(p->link);
  free(p->vert);
}

/* k best complete paths found so far, kept sorted */
typedef struct {
  int k, n;
  opath *p;
} kbest;

static void kbest_offer(kbest *kb, int hops, const int *link, const int *vert, uint64_t cost) {
  opath cand;
  cand.hops = hops;
  cand.cost = cost;
  cand.link = (int *)link;
  cand.vert = (int *)vert;
  if (kb->n == kb->k && path_cmp(&cand, &kb->p[kb->n - 1]) >= 0) return;
  opath keep = path_make(hops, link, vert, cost);
  if (kb->n == kb->k) {
    path_free(&kb->p[kb->n - 1]);
    kb->n--;
  }
  int i = kb->n;
  while (i > 0 && path_cmp(&keep, &kb->p[i - 1]) < 0) {
    kb->p[i] = kb->p[i - 1];
    i--;
  }
  kb->p[i] = keep;
  kb->n++;
}

typedef struct {
  const orc_plan *pl;
  int dst;
  int max_cross;
  int *vs, *ls;
  uint8_t *seen;
  kbest *kb;
} dfs_ctx;

/* A link may be used if the sketch allows it; a link between two nodes
 * counts as a crossing and, when relays are named, must join two relays
 * (Sec. 3.1, Example 2; App. A internode sketch). */
static void dfs(dfs_ctx *x, int u, int depth, uint64_t cost, int cross) {
  const orc_plan *p = x->pl;
  if (u == x->dst) {
    kbest_offer(x->kb, depth, x->ls, x->vs, cost);
    return;
  }
  /* every extension adds at least one link of positive cost */
  if (x->kb->n == x->kb->k && cost >= x->kb->p[x->kb->n - 1].cost) return;
  for (int e = p->row_ptr[u]; e < p->row_ptr[u + 1]; e++) {
    if (p->allowed && !p->allowed[e]) continue;
    int v = p->col[e];
    if (x->seen[v]) continue;
    int c2 = cross;
    if (p->node[u] != p->node[v]) {
      c2++;
      if (x->max_cross >= 0 && c2 > x->max_cross) continue;
      if (p->relay && !(p->relay[u] && p->relay[v])) continue;
    }
    x->seen[v] = 1;
    x->vs[depth + 1] = v;
    x->ls[depth] = e;
    dfs(x, v, depth + 1, cost + p->cost[e], c2);
    x->seen[v] = 0;
  }
}

/* the k best simple paths s -> d (fills kb, caller frees) */
static void k_best_paths(const orc_plan *p, int s, int d, int k, int max_cross, kbest *kb) {
  kb->k = k;
  kb->n = 0;
  kb->p = (opath *)calloc((size_t)k + 1, sizeof(opath));
  dfs_ctx x;
  x.pl = p;
  x.dst = d;
  x.max_cross = max_cross;
  x.vs = (int *)calloc((size_t)p->V + 1, sizeof(int));
  x.ls = (int *)calloc((size_t)p->V + 1, sizeof(int));
  x.seen = (uint8_t *)calloc((size_t)p->V, 1);
  x.kb = kb;
  x.vs[0] = s;
  x.seen[s] = 1;
  dfs(&x, s, 0, 0, 0);
  free(x.vs);
  free(x.ls);
  free(x.seen);
}

/* Join a, one optional link, and b into one path. */
static int join3(const orc_plan *p, const opath *a, int mid_link, const opath *b, opath *out) {
  int h = a->hops + (mid_link >= 0 ? 1 : 0) + b->hops;
  int *ls = (int *)malloc(sizeof(int) * (h > 0 ? h : 1));
  int *vs = (int *)malloc(sizeof(int) * (h + 1));
  int n = 0;
  uint64_t cost = 0;
  vs[0] = a->vert[0];
  for (int i = 0; i < a->hops; i++) {
    ls[n] = a->link[i];
    vs[n + 1] = a->vert[i + 1];
    cost += p->cost[a->link[i]];
    n++;
  }
  if (mid_link >= 0) {
    ls[n] = mid_link;
    vs[n + 1] = p->col[mid_link];
    cost += p->cost[mid_link];
    n++;
  }
  for (int i = 0; i < b->hops; i++) {
    ls[n] = b->link[i];
    vs[n + 1] = b->vert[i + 1];
    cost += p->cost[b->link[i]];
    n++;
  }
  *out = path_make(n, ls, vs, cost);
  free(ls);
  free(vs);
  return 0;
}

static int find_link(const orc_plan *p, int u, int v) {
  for (int e = p->row_ptr[u]; e < p->row_ptr[u + 1]; e++)
    if (p->col[e] == v && (!p->allowed || p->allowed[e])) return e;
  return -1;
}

static void push_path(oplist *L, opath q) {
  L->p = (opath *)realloc(L->p, sizeof(opath) * (size_t)(L->n + 1));
  L->p[L->n++] = q;
}

/* the single best path s -> d under a crossing limit; 0 if none */
static int best_path(const orc_plan *p, int s, int d, int max_cross, opath *out) {
  if (s == d) {
    int v = s;
    *out = path_make(0, NULL, &v, 0);
    return 1;
  }
  kbest kb;
  k_best_paths(p, s, d, 1, max_cross, &kb);
  int ok = kb.n == 1;
  if (ok) *out = kb.p[0];
  free(kb.p);
  return ok;
}

static int build_paths(orc_plan *p) {
  int P = p->P;
  p->paths = (oplist *)calloc((size_t)P * P, sizeof(oplist));
  for (int s = 0; s < P; s++) {
    for (int d = 0; d < P; d++) {
      if (s == d) continue;
      oplist *L = &p->paths[s * P + d];
      if (p->mode == ORC_SHORTEST_ONLY || p->mode == ORC_KSHORTEST) {
        kbest kb;
        k_best_paths(p, s, d, p->k, p->max_cross, &kb);
        for (int i = 0; i < kb.n; i++) {
          /* "the <=k shortest" keeps only minimal-cost paths */
          if (p->mode == ORC_SHORTEST_ONLY && kb.p[i].cost != kb.p[0].cost) {
            path_free(&kb.p[i]);
            continue;
          }
          push_path(L, kb.p[i]);
        }
        free(kb.p);
      } else if (p->mode == ORC_RELAY1) {
        /* option 0: the best direct path; then one relay rank m, ascending */
        opath q;
        if (best_path(p, s, d, p->max_cross, &q)) push_path(L, q);
        for (int m = 0; m < P; m++) {
          if (m == s || m == d) continue;
          if (p->relay && !p->relay[m]) continue;
          opath a, b, j;
          if (!best_path(p, s, m, p->max_cross, &a)) continue;
          if (!best_path(p, m, d, p->max_cross, &b)) {
            path_free(&a);
            continue;
          }
          join3(p, &a, -1, &b, &j);
          path_free(&a);
          path_free(&b);
          push_path(L, j);
        }
      } else if (p->mode == ORC_HIER_RELAY) {
        if (p->node[s] == p->node[d]) {
          opath q;
          if (best_path(p, s, d, 0, &q)) push_path(L, q);
        } else {
          /* i-th relay of the source node -> i-th relay of the destination node */
          int rs[4096], rd[4096], ns = 0, nd = 0;
          for (int r = 0; r < P; r++) {
            if (!p->relay || !p->relay[r]) continue;
            if (p->node[r] == p->node[s] && ns < 4096) rs[ns++] = r;
            if (p->node[r] == p->node[d] && nd < 4096) rd[nd++] = r;
          }
          int nr = ns < nd ? ns : nd;
          for (int i = 0; i < nr; i++) {
            int mid = find_link(p, rs[i], rd[i]);
            if (mid < 0) continue;
            opath a, b, j;
            if (!best_path(p, s, rs[i], 0, &a)) continue;
            if (!best_path(p, rd[i], d, 0, &b)) {
              path_free(&a);
              continue;
            }
            join3(p, &a, mid, &b, &j);
            path_free(&a);
            path_free(&b);
            push_path(L, j);
          }
        }
      }
      if (L->n > 255) {
        snprintf(p->err, sizeof p->err, "more than 255 paths for pair (%d,%d)", s, d);
        return ORC_ELIMIT;
      }
      for (int i = 0; i < L->n; i++) {
        if (L->p[i].hops > p->H) p->H = L->p[i].hops;
        /* a path never uses a link twice, so a chunk crosses a link once */
        for (int a = 0; a < L->p[i].hops; a++)
          for (int b = a + 1; b < L->p[i].hops; b++)
            if (L->p[i].link[a] == L->p[i].link[b]) {
              snprintf(p->err, sizeof p->err, "path reuses a link (pair %d,%d)", s, d);
              return ORC_EINVAL;
            }
      }
    }
  }
  return ORC_OK;
}

/* ------------------------------------------------------------------ */
/* plan                                                                */
/* ------------------------------------------------------------------ */

void orc_destroy(orc_plan *p) {
  if (p) free(p->rev);
  if (!p) return;
  if (p->paths) {
    for (int i = 0; i < p->P * p->P; i++) {
      for (int j = 0; j < p->paths[i].n; j++) path_free(&p->paths[i].p[j]);
      free(p->paths[i].p);
    }
    free(p->paths);
  }
  free(p->row_ptr);
  free(p->col);
  free(p->lsrc);
  free(p->node);
  free(p->alpha);
  free(p->beta);
  free(p->owner);
  free(p->post_ptr);
  free(p->post);
  free(p->allowed);
  free(p->relay);
  free(p->cost);
  free(p);
}

const char *orc_error(const orc_plan *p) { return p ? p->err : "null plan"; }

/* 0: switch vertices store and forward; 1: switched sends hold ports. */
int orc_set_switch_ports(orc_plan *p, int mode) {
  if (!p || mode < 0 || mode > 1) return ORC_EINVAL;
  p->ports = mode;
  return ORC_OK;
}

/* 0: static Step-2 orders (Sec. 5.1); 1: time-aware greedy (App. B.2) in
 * path order; 2: the same greedy in reverse path order. */
int orc_set_order(orc_plan *p, int mode) {
  if (!p || mode < 0 || mode > 2) return ORC_EINVAL;
  p->greedy = mode;
  return ORC_OK;
}

/* 0: every send is its own transfer (App. B.3 without contiguity);
 * 1: contiguous transfers on links whose endpoints lie in different nodes. */
int orc_set_contiguity(orc_plan *p, int mode) {
  if (!p || mode < 0 || mode > 1) return ORC_EINVAL;
  p->contig = mode;
  return ORC_OK;
}

/*
 * Build a plan.
 *   V, P, row_ptr[V+1], col[E], alpha_ns[E], beta_ps_per_byte[E]: topology,
 *     vertices [0,P) are ranks, the rest are switch vertices;
 *   node_of[V] or NULL;
 *   kind, cpr, chunk_bytes: collective; for ORC_EXPLICIT, C, owner[C],
 *     post_ptr[C+1], post[] give the pre/postcondition (one owner per chunk);
 *   allowed[E] or NULL, relay[V] or NULL, max_cross (-1 = no limit),
 *     mode, k: sketch.
 */
int orc_create(int V, int P, const int *row_ptr, const int *col, const uint32_t *alpha,
               const uint32_t *beta, const int *node_of, int kind, int cpr, uint64_t chunk_bytes,
               int C_explicit, const int *owner_explicit, const int *post_ptr_explicit,
               const int *post_explicit, const uint8_t *allowed, const uint8_t *relay,
               int max_cross, int mode, int k, orc_plan **out) {
  *out = NULL;
  orc_plan *p = (orc_plan *)calloc(1, sizeof(orc_plan));
  if (!p) return ORC_ENOMEM;
  *out = p;
  if (V <= 0 || P <= 0 || P > V || !row_ptr || !col || !alpha || !beta) {
    snprintf(p->err, sizeof p->err, "bad topology arguments");
    return ORC_EINVAL;
  }
  p->V = V;
  p->P = P;
  p->E = row_ptr[V];
  p->row_ptr = (int *)malloc(sizeof(int) * (V + 1));
  memcpy(p->row_ptr, row_ptr, sizeof(int) * (V + 1));
  p->col = (int *)malloc(sizeof(int) * (p->E > 0 ? p->E : 1));
  p->lsrc = (int *)malloc(sizeof(int) * (p->E > 0 ? p->E : 1));
  p->alpha = (uint32_t *)malloc(sizeof(uint32_t) * (p->E > 0 ? p->E : 1));
  p->beta = (uint32_t *)malloc(sizeof(uint32_t) * (p->E > 0 ? p->E : 1));
  p->cost = (uint64_t *)malloc(sizeof(uint64_t) * (p->E > 0 ? p->E : 1));
  p->node = (int *)calloc((size_t)V, sizeof(int));
  for (int u = 0; u < V; u++) {
    if (row_ptr[u + 1] < row_ptr[u]) {
      snprintf(p->err, sizeof p->err, "row_ptr not monotone");
      return ORC_EINVAL;
    }
    for (int e = row_ptr[u]; e < row_ptr[u + 1]; e++) {
      if (col[e] < 0 || col[e] >= V || col[e] == u) {
        snprintf(p->err, sizeof p->err, "bad link %d", e);
        return ORC_EINVAL;
      }
      p->col[e] = col[e];
      p->lsrc[e] = u;
    }
  }
  memcpy(p->alpha, alpha, sizeof(uint32_t) * p->E);
  memcpy(p->beta, beta, sizeof(uint32_t) * p->E);
  if (node_of) memcpy(p->node, node_of, sizeof(int) * V);
  p->S = chunk_bytes;
  /* alpha-beta cost of one chunk on one link (Sec. 4.1), integer ns */
  for (int e = 0; e < p->E; e++) {
    uint64_t c = (uint64_t)alpha[e] + ((uint64_t)beta[e] * chunk_bytes + 999u) / 1000u;
    if (c == 0 || c >= (1ull << 32)) {
      snprintf(p->err, sizeof p->err, "link %d cost out of range", e);
      return ORC_ELIMIT;
    }
    p->cost[e] = c;
  }
  /* collective */
  p->kind = kind;
  p->cpr = cpr;
  if (kind == ORC_ALLGATHER || kind == ORC_REDUCESCATTER || kind == ORC_ALLREDUCE) {
    if (cpr <= 0) return ORC_EINVAL;
    p->C = P * cpr;
    p->owner = (int *)malloc(sizeof(int) * p->C);
    p->post_ptr = (int *)malloc(sizeof(int) * (p->C + 1));
    p->post = (int *)malloc(sizeof(int) * p->C * P);
    for (int c = 0; c < p->C; c++) {
      p->owner[c] = c / cpr;
      p->post_ptr[c] = c * P;
      for (int r = 0; r < P; r++) p->post[c * P + r] = r;
    }
    p->post_ptr[p->C] = p->C * P;
  } else if (kind == ORC_ALLTOALL) {
    if (cpr <= 0) return ORC_EINVAL;
    p->C = P * P * cpr;
    p->owner = (int *)malloc(sizeof(int) * p->C);
    p->post_ptr = (int *)malloc(sizeof(int) * (p->C + 1));
    p->post = (int *)malloc(sizeof(int) * p->C);
    for (int c = 0; c < p->C; c++) {
      int pair = c / cpr;
      p->owner[c] = pair / P;
      p->post_ptr[c] = c;
      p->post[c] = pair % P;
    }
    p->post_ptr[p->C] = p->C;
  } else if (kind == ORC_EXPLICIT) {
    if (C_explicit <= 0 || !owner_explicit || !post_ptr_explicit || !post_explicit)
      return ORC_EINVAL;
    p->C = C_explicit;
    p->owner = (int *)malloc(sizeof(int) * p->C);
    p->post_ptr = (int *)malloc(sizeof(int) * (p->C + 1));
    int np = post_ptr_explicit[p->C];
    p->post = (int *)malloc(sizeof(int) * (np > 0 ? np : 1));
    memcpy(p->owner, owner_explicit, sizeof(int) * p->C);
    memcpy(p->post_ptr, post_ptr_explicit, sizeof(int) * (p->C + 1));
    memcpy(p->post, post_explicit, sizeof(int) * (np > 0 ? np : 0));
    for (int c = 0; c < p->C; c++) {
      if (p->owner[c] < 0 || p->owner[c] >= P) return ORC_EINVAL;
      for (int j = p->post_ptr[c]; j < p->post_ptr[c + 1]; j++)
        if (p->post[j] < 0 || p->post[j] >= P) return ORC_EINVAL;
    }
  } else {
    snprintf(p->err, sizeof p->err, "bad collective kind");
    return ORC_EINVAL;
  }
  /* sketch */
  if (allowed) {
    p->allowed = (uint8_t *)malloc(p->E > 0 ? p->E : 1);
    memcpy(p->allowed, allowed, p->E);
  }
  if (relay) {
    p->relay = (uint8_t *)malloc(V);
    memcpy(p->relay, relay, V);
  }
  p->max_cross = max_cross;
  p->mode = mode;
  p->k = k;
  if (mode < 0 || mode > 3 || ((mode == ORC_SHORTEST_ONLY || mode == ORC_KSHORTEST) && k <= 0)) {
    snprintf(p->err, sizeof p->err, "bad route mode");
    return ORC_EINVAL;
  }
  int rc = build_paths(p);
  if (rc) return rc;
  /* reductions run the trees backwards: every routed link needs a reverse */
  p->rev = (int *)malloc(sizeof(int) * (p->E > 0 ? p->E : 1));
  for (int e = 0; e < p->E; e++) {
    p->rev[e] = -1;
    for (int f = p->row_ptr[p->col[e]]; f < p->row_ptr[p->col[e] + 1]; f++)
      if (p->col[f] == p->lsrc[e]) p->rev[e] = f;
  }
  if (kind == ORC_REDUCESCATTER || kind == ORC_ALLREDUCE)
    for (int pp = 0; pp < P * P; pp++)
      for (int i = 0; i < p->paths[pp].n; i++)
        for (int j = 0; j < p->paths[pp].p[i].hops; j++)
          if (p->rev[p->paths[pp].p[i].link[j]] < 0) {
            snprintf(p->err, sizeof p->err, "a routed link has no reverse link");
            return ORC_EINVAL;
          }
  /* layouts: Allgather-like (tree) chunks read route c*P+d and priority
   * c*V+v; Alltoall chunks read route c and priority c*H+h */
  if (kind == ORC_ALLTOALL) {
    p->route_stride = p->C;
    p->prio_stride = p->C * (p->H > 0 ? p->H : 1);
    p->max_sends = p->C * p->H;
  } else {
    p->route_stride = p->C * P;
    /* Allreduce: the ReduceScatter row, then the Allgather row */
    p->prio_stride = p->C * V * (kind == ORC_ALLREDUCE ? 2 : 1);
    p->max_sends = p->C * (V - 1);
  }
  return ORC_OK;
}

int orc_route_stride(const orc_plan *p) { return p->route_stride; }
int orc_prio_stride(const orc_plan *p) { return p->prio_stride; }
int orc_max_hops(const orc_plan *p) { return p->H; }
int orc_num_chunks(const orc_plan *p) { return p->C; }
int orc_max_sends(const orc_plan *p) { return p->max_sends; }
uint64_t orc_link_cost(const orc_plan *p, int e) { return (e >= 0 && e < p->E) ? p->cost[e] : 0; }
int orc_npaths(const orc_plan *p, int s, int d) {
  if (s < 0 || d < 0 || s >= p->P || d >= p->P) return 0;
  return p->paths[s * p->P + d].n;
}
/* copies the links of path (s,d,i) into out; returns hop count or -1 */
int orc_path(const orc_plan *p, int s, int d, int i, int *out_links, int cap) {
  if (s < 0 || d < 0 || s >= p->P || d >= p->P) return -1;
  const oplist *L = &p->paths[s * p->P + d];
  if (i < 0 || i >= L->n) return -1;
  if (L->p[i].hops > cap) return -1;
  for (int j = 0; j < L->p[i].hops; j++) out_links[j] = L->p[i].link[j];
  return L->p[i].hops;
}

/* number of route options of route entry e (0 for entries no pair uses) */
int orc_route_options(const orc_plan *p, int e) {
  if (e < 0 || e >= p->route_stride) return 0;
  if (p->kind == ORC_ALLTOALL) {
    int s = p->owner[e], d = p->post[p->post_ptr[e]];
    return s == d ? 0 : p->paths[s * p->P + d].n;
  }
  int c = e / p->P, d = e % p->P, s = p->owner[c];
  if (d == s) return 0;
  for (int j = p->post_ptr[c]; j < p->post_ptr[c + 1]; j++)
    if (p->post[j] == d) return p->paths[s * p->P + d].n;
  return 0;
}

/* ------------------------------------------------------------------ */
/* evaluation of one candidate                                         */
/* ------------------------------------------------------------------ */

typedef struct {
  int chunk, link, from, to, hop;
  uint64_t rem, trav;
  uint32_t prio;
  int cpred;   /* send that brings the chunk to `from`, or -1 */
  int csucc;   /* reduction: the send that carries this partial on, or -1 */
  int lpred;   /* previous send on the same link, or -1 */
  int link2;   /* switched send: the receive port (downlink), else -1 */
  int lpred2;  /* previous send on link2, or -1 */
  int pos;     /* position in the link's order */
  uint64_t start, finish;
} osend;

static _Thread_local const osend *g_sort_base;

/* Step-2 order (Sec. 5.1): longer remaining path first, then shorter
 * travelled path, then the priority, then the chunk id. */
static int send_order_cmp(const void *a, const void *b) {
  const osend *x = &g_sort_base[*(const int *)a];
  const osend *y = &g_sort_base[*(const int *)b];
  if (x->rem != y->rem) return x->rem > y->rem ? -1 : 1;
  if (x->trav != y->trav) return x->trav < y->trav ? -1 : 1;
  if (x->prio != y->prio) return x->prio < y->prio ? -1 : 1;
  if (x->chunk != y->chunk) return x->chunk < y->chunk ? -1 : 1;
  return 0;
}

typedef struct {
  osend *s;
  int n;
  int *tree_parent; /* [C*V] link into (c,v), -1 if none */
  int *send_of;     /* [C*V] send index that brings c into v */
  uint8_t *present; /* [C*V] */
  int *idx, *succ_ptr, *succ, *indeg, *queue;
  int *pred_ptr, *pred; /* chunk predecessors of every send (CSR) */
  uint64_t *dist, *height;
} oscratch;

static void scratch_init(const orc_plan *p, oscratch *w) {
  size_t cv = (size_t)p->C * p->V;
  size_t ms = (size_t)(p->max_sends > 0 ? p->max_sends : 1);
  w->s = (osend *)malloc(sizeof(osend) * ms);
  w->tree_parent = (int *)malloc(sizeof(int) * cv);
  w->send_of = (int *)malloc(sizeof(int) * cv);
  w->present = (uint8_t *)malloc(cv);
  w->idx = (int *)malloc(sizeof(int) * ms);
  w->succ_ptr = (int *)malloc(sizeof(int) * (ms + 1));
  w->succ = (int *)malloc(sizeof(int) * 2 * ms);
  w->indeg = (int *)malloc(sizeof(int) * ms);
  w->queue = (int *)malloc(sizeof(int) * ms);
  w->pred_ptr = (int *)malloc(sizeof(int) * (ms + 1));
  w->pred = (int *)malloc(sizeof(int) * ms);
  w->dist = (uint64_t *)malloc(sizeof(uint64_t) * p->V);
  w->height = (uint64_t *)malloc(sizeof(uint64_t) * p->V);
}

static void scratch_free(oscratch *w) {
  free(w->s);
  free(w->tree_parent);
  free(w->send_of);
  free(w->present);
  free(w->idx);
  free(w->succ_ptr);
  free(w->succ);
  free(w->indeg);
  free(w->queue);
  free(w->pred_ptr);
  free(w->pred);
  free(w->dist);
  free(w->height);
}

/* is d one of the ranks chunk c must reach? */
static int in_post(const orc_plan *p, int c, int d) {
  for (int j = p->post_ptr[c]; j < p->post_ptr[c + 1]; j++)
    if (p->post[j] == d) return 1;
  return 0;
}

/* Multicast sends of one chunk: walk the routed path of every destination
 * in ascending rank order and keep the first link that reaches each vertex
 * (one is_sent per chunk and link, App. B.1; a GPU may forward a chunk it
 * received once over several links, Sec. 8). Keys follow the resulting tree. */
static void build_tree_sends(const orc_plan *p, const uint8_t *rt, const uint32_t *pr,
                             oscratch *w) {
  int V = p->V, P = p->P;
  for (int c = 0; c < p->C; c++) {
    int o = p->owner[c];
    int *par = &w->tree_parent[(size_t)c * V];
    uint8_t *pres = &w->present[(size_t)c * V];
    for (int v = 0; v < V; v++) {
      par[v] = -1;
      pres[v] = 0;
    }
    pres[o] = 1;
    for (int d = 0; d < P; d++) {
      if (d == o || !in_post(p, c, d)) continue;
      int ch = rt[(size_t)c * P + d];
      const oplist *L = &p->paths[o * P + d];
      if (ch >= L->n) continue; /* this pair is left unrouted */
      const opath *q = &L->p[ch];
      for (int j = 0; j < q->hops; j++) {
        int v = q->vert[j + 1];
        if (!pres[v]) {
          pres[v] = 1;
          par[v] = q->link[j];
        }
      }
    }
    /* distance from the owner along the tree (the path travelled so far) */
    for (int v = 0; v < V; v++) {
      uint64_t t = 0;
      int x = v;
      if (!pres[v]) {
        w->dist[v] = 0;
        continue;
      }
      while (x != o) {
        int l = par[x];
        t += p->cost[l];
        x = p->lsrc[l];
      }
      w->dist[v] = t;
    }
    /* height: longest tree distance from v down to any vertex below it */
    for (int v = 0; v < V; v++) w->height[v] = 0;
    for (int v = 0; v < V; v++) {
      if (!pres[v]) continue;
      int x = v;
      while (x != o) {
        int a = p->lsrc[par[x]];
        uint64_t h = w->dist[v] - w->dist[a];
        if (h > w->height[a]) w->height[a] = h;
        x = a;
      }
    }
    for (int v = 0; v < V; v++) {
      w->send_of[(size_t)c * V + v] = -1;
      if (par[v] < 0) continue;
      osend *s = &w->s[w->n];
      s->chunk = c;
      s->link = par[v];
      s->from = p->lsrc[par[v]];
      s->to = v;
      s->hop = -1;
      s->trav = w->dist[s->from];
      s->rem = p->cost[par[v]] + w->height[v];
      s->prio = pr[(size_t)c * V + v];
      w->send_of[(size_t)c * V + v] = w->n;
      w->n++;
    }
  }
  for (int i = 0; i < w->n; i++) {
    osend *s = &w->s[i];
    s->cpred = (s->from == p->owner[s->chunk]) ? -1 : w->send_of[(size_t)s->chunk * V + s->from];
    s->csucc = -1;
    s->link2 = -1;
  }
}

/* ReduceScatter sends: the Allgather tree of every chunk backwards. The
 * Allgather send u -> v (link l) becomes v -> u on the reverse of l and
 * carries the partial reduction of v's subtree: it waits for every send into
 * v, and the send out of u waits for it. Keys on the reversed tree:
 * remaining = reversed distance from v to the owner (this send included),
 * travelled = longest reversed path from a vertex below v up to v. */
static void reverse_tree_sends(const orc_plan *p, oscratch *w) {
  int V = p->V;
  for (int c = 0; c < p->C; c++) {
    int o = p->owner[c];
    const int *par = &w->tree_parent[(size_t)c * V];
    const uint8_t *pres = &w->present[(size_t)c * V];
    /* up[v]: reversed distance from v to the owner */
    for (int v = 0; v < V; v++) {
      uint64_t t = 0;
      int x = v;
      if (pres[v])
        while (x != o) {
          t += p->cost[p->rev[par[x]]];
          x = p->lsrc[par[x]];
        }
      w->dist[v] = t;
    }
    /* below[a]: longest reversed path from a vertex of a's subtree up to a */
    for (int v = 0; v < V; v++) w->height[v] = 0;
    for (int v = 0; v < V; v++) {
      if (!pres[v]) continue;
      int x = v;
      while (x != o) {
        int a = p->lsrc[par[x]];
        uint64_t h = w->dist[v] - w->dist[a];
        if (h > w->height[a]) w->height[a] = h;
        x = a;
      }
    }
    for (int v = 0; v < V; v++) {
      int i = w->send_of[(size_t)c * V + v];
      if (i < 0) continue;
      osend *s = &w->s[i];
      int u = s->from;
      s->link = p->rev[par[v]];
      s->from = v;
      s->to = u;
      s->rem = w->dist[v];
      s->trav = w->height[v];
      s->cpred = -1;
      s->csucc = (u == o) ? -1 : w->send_of[(size_t)c * V + u];
    }
  }
}

/* Alltoall sends: each hop of the chunk's routed path. */
static void build_path_sends(const orc_plan *p, const uint8_t *rt, const uint32_t *pr,
                             oscratch *w) {
  int V = p->V, P = p->P, H = p->H;
  for (int c = 0; c < p->C; c++) {
    uint8_t *pres = &w->present[(size_t)c * V];
    for (int v = 0; v < V; v++) pres[v] = 0;
    int s0 = p->owner[c], d = p->post[p->post_ptr[c]];
    pres[s0] = 1;
    if (s0 == d) continue;
    int ch = rt[c];
    const oplist *L = &p->paths[s0 * P + d];
    if (ch >= L->n) continue; /* unrouted */
    const opath *q = &L->p[ch];
    /* sends: one per hop, or with switch ports one per hop pair through a
     * switch vertex (rank -> switch -> rank), costing the uplink's latency */
    uint64_t total = 0, before = 0;
    for (int j = 0; j < q->hops; j++) {
      total += p->cost[q->link[j]];
      if (p->ports && q->vert[j + 1] >= P && j + 1 < q->hops) j++;
    }
    for (int j = 0; j < q->hops; j++) {
      const int switched = p->ports && q->vert[j + 1] >= P && j + 1 < q->hops;
      osend *s = &w->s[w->n];
      s->chunk = c;
      s->link = q->link[j];
      s->link2 = switched ? q->link[j + 1] : -1;
      s->from = q->vert[j];
      s->to = q->vert[j + 1 + switched];
      s->hop = j;
      s->trav = before;
      s->rem = total - before;
      s->prio = pr[(size_t)c * H + j];
      s->cpred = (j == 0) ? -1 : w->n - 1;
      s->csucc = -1;
      before += p->cost[q->link[j]];
      w->n++;
      j += switched;
    }
    pres[d] = 1;
  }
}

/* Evaluate one candidate. If detail is non-NULL the sends are copied there
 * (at most cap of them) and *nsends is set. Returns ORC_OK. */
/* every (chunk, rank) pair of the postcondition holds the chunk (App. B) */
static int postcondition(const orc_plan *p, const oscratch *w) {
  for (int c = 0; c < p->C; c++)
    for (int j = p->post_ptr[c]; j < p->post_ptr[c + 1]; j++)
      if (!w->present[(size_t)c * p->V + p->post[j]]) return 0;
  return 1;
}

/* cost of one transfer of m chunks on link e: alpha + ceil(beta * m * S / 1000) */
static uint64_t transfer_cost(const orc_plan *p, int e, uint64_t m) {
  unsigned __int128 b = (unsigned __int128)p->beta[e] * m * p->S;
  return (uint64_t)p->alpha[e] + (uint64_t)((b + 999) / 1000);
}

/* Chunk predecessors of every send: the send that brings the chunk to its
 * source (cpred), or, in a reduction, every send whose partial it carries on
 * (the sends whose csucc it is). A send is ready when all of them ended. */
static void chunk_preds(oscratch *w) {
  int n = w->n;
  for (int i = 0; i <= n; i++) w->pred_ptr[i] = 0;
  for (int i = 0; i < n; i++) {
    if (w->s[i].cpred >= 0) w->pred_ptr[i + 1]++;
    if (w->s[i].csucc >= 0) w->pred_ptr[w->s[i].csucc + 1]++;
  }
  for (int i = 0; i < n; i++) w->pred_ptr[i + 1] += w->pred_ptr[i];
  int *fill = w->indeg; /* cursor, before the sweep uses it */
  for (int i = 0; i < n; i++) fill[i] = w->pred_ptr[i];
  for (int i = 0; i < n; i++) {
    if (w->s[i].cpred >= 0) w->pred[fill[i]++] = w->s[i].cpred;
    if (w->s[i].csucc >= 0) w->pred[fill[w->s[i].csucc]++] = i;
  }
}

static uint64_t ready_time(const oscratch *w, int i) {
  uint64_t r = 0;
  for (int j = w->pred_ptr[i]; j < w->pred_ptr[i + 1]; j++)
    if (w->s[w->pred[j]].finish > r) r = w->s[w->pred[j]].finish;
  return r;
}

/* Schedule with contiguous transfers. Sends are taken in the global Step-2
 * key order, which is a topological order of the schedule: a send's chunk
 * arrives by a send with a strictly longer remaining path, and a link's
 * order is the key order. A send joins the link's open transfer when the
 * link is between nodes, its remaining length equals the transfer's and its
 * chunk was ready when the transfer started; the transfer then ends later
 * and so do all of its sends. Every send that could still join a transfer
 * precedes, in key order, every send that depends on it (shorter remaining
 * path), so finish times are final when they are read. */
static int contig_sweep(const orc_plan *p, oscratch *w, uint32_t *makespan, uint8_t *valid) {
  int n = w->n, E = p->E;
  int *order = w->queue;
  for (int i = 0; i < n; i++) order[i] = i;
  g_sort_base = w->s;
  if (n > 1) qsort(order, (size_t)n, sizeof(int), send_order_cmp);
  uint64_t *busy = (uint64_t *)calloc((size_t)(E > 0 ? E : 1), sizeof(uint64_t));
  uint64_t *g_start = (uint64_t *)calloc((size_t)(E > 0 ? E : 1), sizeof(uint64_t));
  uint64_t *g_rem = (uint64_t *)calloc((size_t)(E > 0 ? E : 1), sizeof(uint64_t));
  int *g_m = (int *)calloc((size_t)(E > 0 ? E : 1), sizeof(int));
  uint64_t span = 0;
  for (int t = 0; t < n; t++) {
    int i = order[t];
    osend *s = &w->s[i];
    int e = s->link;
    uint64_t ready = ready_time(w, i);
    int between_nodes = p->node[p->lsrc[e]] != p->node[p->col[e]];
    if (between_nodes && g_m[e] > 0 && s->rem == g_rem[e] && ready <= g_start[e]) {
      g_m[e]++;
      uint64_t f = g_start[e] + transfer_cost(p, e, (uint64_t)g_m[e]);
      s->start = g_start[e];
      /* this send and the g_m - 1 sends before it on the link */
      int j = i;
      for (int q = 0; q < g_m[e]; q++) {
        w->s[j].finish = f;
        j = w->s[j].lpred;
      }
      busy[e] = f;
      if (f > span) span = f;
    } else {
      uint64_t start = ready > busy[e] ? ready : busy[e];
      s->start = start;
      s->finish = start + transfer_cost(p, e, 1);
      g_start[e] = start;
      g_rem[e] = s->rem;
      g_m[e] = 1;
      busy[e] = s->finish;
      if (s->finish > span) span = s->finish;
    }
  }
  free(busy);
  free(g_start);
  free(g_rem);
  free(g_m);
  if (span >= (1ull << 32)) return ORC_ELIMIT;
  *makespan = (uint32_t)span;
  *valid = (uint8_t)postcondition(p, w);
  return ORC_OK;
}

/* Time-aware greedy (App. B.2): repeatedly schedule, among the sends whose
 * chunk predecessors are all scheduled, the one with the smallest
 * (max(link time, ready time), Step-2 key); it starts there and ends one
 * link latency later. Writes start/finish and each send's position in its
 * link's order. Plain O(n^2) scan. */
static int greedy_sweep(const orc_plan *p, oscratch *w, uint32_t *makespan, uint8_t *valid) {
  int n = w->n, E = p->E;
  uint64_t *busy = (uint64_t *)calloc((size_t)(E > 0 ? E : 1), sizeof(uint64_t));
  int *count = (int *)calloc((size_t)(E > 0 ? E : 1), sizeof(int));
  int *waiting = w->indeg; /* unscheduled chunk predecessors */
  uint8_t *done = (uint8_t *)calloc((size_t)(n > 0 ? n : 1), 1);
  for (int i = 0; i < n; i++) waiting[i] = w->pred_ptr[i + 1] - w->pred_ptr[i];
  g_sort_base = w->s;
  uint64_t span = 0;
  for (int step = 0; step < n; step++) {
    int best = -1;
    uint64_t best_t = 0;
    for (int i = 0; i < n; i++) {
      if (done[i] || waiting[i]) continue;
      uint64_t r = ready_time(w, i), b = busy[w->s[i].link];
      uint64_t t = r > b ? r : b;
      if (best < 0 || t < best_t || (t == best_t && send_order_cmp(&i, &best) < 0)) {
        best = i;
        best_t = t;
      }
    }
    if (best < 0) {
      free(busy);
      free(count);
      free(done);
      return ORC_EINVAL; /* nothing schedulable: cannot happen */
    }
    osend *s = &w->s[best];
    s->start = best_t;
    s->finish = best_t + p->cost[s->link];
    s->pos = count[s->link]++;
    busy[s->link] = s->finish;
    done[best] = 1;
    if (s->finish > span) span = s->finish;
    /* its chunk successors lose one unscheduled predecessor */
    if (s->csucc >= 0) waiting[s->csucc]--;
    for (int j = 0; j < n; j++)
      if (w->s[j].cpred == best) waiting[j]--;
  }
  free(busy);
  free(count);
  free(done);
  if (span >= (1ull << 32)) return ORC_ELIMIT;
  *makespan = (uint32_t)span;
  *valid = (uint8_t)postcondition(p, w);
  return ORC_OK;
}

/* Greedy in reverse path order. App. B.2 notes that the greedy may start
 * from the first link of every path or from the last one. Reading: the
 * greedy of greedy_sweep runs on the mirrored schedule, in which every
 * chunk dependency points the other way (a send waits for every send that
 * waited for it) and the two Step-2 lengths trade places (remaining' =
 * travelled + the send's own latency, travelled' = remaining - that
 * latency); links and latencies stay. The mirrored greedy serves every link
 * in some order; the link's order in the real schedule is the reverse, and
 * the real times then come from the App. B.3 rule with these orders (the
 * caller's DAG sweep). Sets pos and lpred of every send. */
static int reverse_greedy_orders(const orc_plan *p, oscratch *w) {
  int n = w->n, E = p->E;
  int *waiting = w->indeg; /* mirrored: forward successors not yet served */
  uint64_t *ready = (uint64_t *)calloc((size_t)(n > 0 ? n : 1), sizeof(uint64_t));
  uint64_t *busy = (uint64_t *)calloc((size_t)(E > 0 ? E : 1), sizeof(uint64_t));
  int *count = (int *)calloc((size_t)(E > 0 ? E : 1) + 1, sizeof(int));
  uint8_t *done = (uint8_t *)calloc((size_t)(n > 0 ? n : 1), 1);
  for (int i = 0; i < n; i++) waiting[i] = 0;
  for (int i = 0; i < n; i++)
    for (int j = w->pred_ptr[i]; j < w->pred_ptr[i + 1]; j++) waiting[w->pred[j]]++;
  for (int i = 0; i < n; i++) { /* mirrored lengths */
    osend *s = &w->s[i];
    uint64_t c = p->cost[s->link], rem = s->rem;
    s->rem = s->trav + c;
    s->trav = rem - c;
  }
  g_sort_base = w->s;
  int rc = ORC_OK;
  for (int step = 0; step < n; step++) {
    int best = -1;
    uint64_t best_t = 0;
    for (int i = 0; i < n; i++) {
      if (done[i] || waiting[i]) continue;
      uint64_t b = busy[w->s[i].link];
      uint64_t t = ready[i] > b ? ready[i] : b;
      if (best < 0 || t < best_t || (t == best_t && send_order_cmp(&i, &best) < 0)) {
        best = i;
        best_t = t;
      }
    }
    if (best < 0) {
      rc = ORC_EINVAL; /* nothing servable: cannot happen */
      break;
    }
    osend *s = &w->s[best];
    uint64_t f = best_t + p->cost[s->link];
    busy[s->link] = f;
    s->pos = count[s->link]++;
    done[best] = 1;
    /* the sends it waited for in the real schedule may now be served */
    for (int j = w->pred_ptr[best]; j < w->pred_ptr[best + 1]; j++) {
      int q = w->pred[j];
      waiting[q]--;
      if (f > ready[q]) ready[q] = f;
    }
  }
  for (int i = 0; i < n; i++) { /* lengths back */
    osend *s = &w->s[i];
    uint64_t c = p->cost[s->link], trav = s->rem - c;
    s->rem = s->trav + c;
    s->trav = trav;
  }
  if (rc == ORC_OK) {
    /* the real order of each link is the reverse of the mirrored one */
    int *off = (int *)calloc((size_t)(E > 0 ? E : 1) + 1, sizeof(int));
    for (int e = 0; e < E; e++) off[e + 1] = off[e] + count[e];
    for (int i = 0; i < n; i++) {
      osend *s = &w->s[i];
      s->pos = count[s->link] - 1 - s->pos;
      w->idx[off[s->link] + s->pos] = i;
    }
    for (int i = 0; i < n; i++) {
      osend *s = &w->s[i];
      s->lpred = s->pos > 0 ? w->idx[off[s->link] + s->pos - 1] : -1;
      s->lpred2 = -1;
    }
    free(off);
  }
  free(ready);
  free(busy);
  free(count);
  free(done);
  return rc;
}

/* One schedule: `phase` is ORC_ALLGATHER, ORC_ALLTOALL, ORC_EXPLICIT or
 * ORC_REDUCESCATTER (the send sets differ; ordering and timing do not). */
static int eval_phase(const orc_plan *p, int phase, const uint8_t *rt, const uint32_t *pr,
                      oscratch *w, uint32_t *makespan, uint8_t *valid) {
  w->n = 0;
  if (phase == ORC_ALLTOALL)
    build_path_sends(p, rt, pr, w);
  else
    build_tree_sends(p, rt, pr, w);
  if (phase == ORC_REDUCESCATTER) reverse_tree_sends(p, w);
  int n = w->n;
  /* per-link total order chunk_order(l) (App. B.2) */
  for (int i = 0; i < n; i++) w->idx[i] = i;
  g_sort_base = w->s;
  /* sort by link first, then by the Step-2 key inside each link */
  for (int i = 0; i < n; i++) w->s[i].lpred = -1;
  {
    /* bucket the send indices by resource: its link, and for a switched
     * send also its receive port (link2) */
    int E = p->E;
    int *cnt = (int *)calloc((size_t)E + 1, sizeof(int));
    for (int i = 0; i < n; i++) {
      w->s[i].lpred2 = -1;
      cnt[w->s[i].link + 1]++;
      if (w->s[i].link2 >= 0) cnt[w->s[i].link2 + 1]++;
    }
    for (int e = 0; e < E; e++) cnt[e + 1] += cnt[e];
    int *fill = (int *)malloc(sizeof(int) * (E > 0 ? E : 1));
    for (int e = 0; e < E; e++) fill[e] = cnt[e];
    for (int i = 0; i < n; i++) {
      w->idx[fill[w->s[i].link]++] = i;
      if (w->s[i].link2 >= 0) w->idx[fill[w->s[i].link2]++] = i;
    }
    for (int e = 0; e < E; e++) {
      int a = cnt[e], b = cnt[e + 1];
      if (b - a > 1) qsort(&w->idx[a], (size_t)(b - a), sizeof(int), send_order_cmp);
      for (int j = a; j < b; j++) {
        osend *s = &w->s[w->idx[j]];
        int prev = j > a ? w->idx[j - 1] : -1;
        if (s->link == e) {
          s->pos = j - a;
          s->lpred = prev;
        } else {
          s->lpred2 = prev;
        }
        if (j > a && send_order_cmp(&w->idx[j - 1], &w->idx[j]) == 0) {
          free(cnt);
          free(fill);
          return ORC_EINVAL; /* two sends of one chunk on one link */
        }
      }
    }
    free(cnt);
    free(fill);
  }
  chunk_preds(w);
  if (p->greedy && p->contig) return ORC_EINVAL; /* not combined */
  if (p->ports && (p->greedy || p->contig)) return ORC_EINVAL;
  if (p->greedy == 1) return greedy_sweep(p, w, makespan, valid);
  if (p->greedy == 2) {
    int rc = reverse_greedy_orders(p, w);
    if (rc) return rc;
  }
  if (p->contig) return contig_sweep(p, w, makespan, valid);
  /* the difference constraints of App. B.3 without contiguity form a DAG
   * (chunk edges and link-order edges); sweep it in topological order */
  for (int i = 0; i <= n; i++) w->succ_ptr[i] = 0;
  for (int i = 0; i < n; i++) {
    w->indeg[i] = w->pred_ptr[i + 1] - w->pred_ptr[i];
    for (int j = w->pred_ptr[i]; j < w->pred_ptr[i + 1]; j++) w->succ_ptr[w->pred[j] + 1]++;
    if (w->s[i].lpred >= 0) {
      w->succ_ptr[w->s[i].lpred + 1]++;
      w->indeg[i]++;
    }
    if (w->s[i].lpred2 >= 0) {
      w->succ_ptr[w->s[i].lpred2 + 1]++;
      w->indeg[i]++;
    }
  }
  for (int i = 0; i < n; i++) w->succ_ptr[i + 1] += w->succ_ptr[i];
  {
    int *fill = w->queue; /* reuse as a cursor array before the sweep */
    for (int i = 0; i < n; i++) fill[i] = w->succ_ptr[i];
    for (int i = 0; i < n; i++) {
      for (int j = w->pred_ptr[i]; j < w->pred_ptr[i + 1]; j++) w->succ[fill[w->pred[j]]++] = i;
      if (w->s[i].lpred >= 0) w->succ[fill[w->s[i].lpred]++] = i;
      if (w->s[i].lpred2 >= 0) w->succ[fill[w->s[i].lpred2]++] = i;
    }
  }
  int head = 0, tail = 0;
  for (int i = 0; i < n; i++)
    if (w->indeg[i] == 0) w->queue[tail++] = i;
  uint64_t span = 0;
  while (head < tail) {
    int i = w->queue[head++];
    osend *s = &w->s[i];
    uint64_t ready = ready_time(w, i);
    uint64_t busy = s->lpred >= 0 ? w->s[s->lpred].finish : 0;
    if (s->lpred2 >= 0 && w->s[s->lpred2].finish > busy) busy = w->s[s->lpred2].finish;
    s->start = ready > busy ? ready : busy;
    s->finish = s->start + p->cost[s->link];
    if (s->finish > span) span = s->finish;
    for (int j = w->succ_ptr[i]; j < w->succ_ptr[i + 1]; j++)
      if (--w->indeg[w->succ[j]] == 0) w->queue[tail++] = w->succ[j];
  }
  if (tail != n) return ORC_EINVAL; /* a cycle: cannot happen under this order */
  if (span >= (1ull << 32)) return ORC_ELIMIT;
  *makespan = (uint32_t)span;
  *valid = (uint8_t)postcondition(p, w);
  return ORC_OK;
}

static int eval_one(const orc_plan *p, const uint8_t *rt, const uint32_t *pr, oscratch *w,
                    uint32_t *makespan, uint8_t *valid) {
  if (p->kind != ORC_ALLREDUCE) return eval_phase(p, p->kind, rt, pr, w, makespan, valid);
  /* Allreduce: ReduceScatter, then Allgather starting when it has ended */
  uint32_t m1, m2;
  uint8_t v1, v2;
  int rc = eval_phase(p, ORC_REDUCESCATTER, rt, pr, w, &m1, &v1);
  if (rc) return rc;
  rc = eval_phase(p, ORC_ALLGATHER, rt, pr + (size_t)p->C * p->V, w, &m2, &v2);
  if (rc) return rc;
  if ((uint64_t)m1 + m2 >= (1ull << 32)) return ORC_ELIMIT;
  *makespan = m1 + m2;
  *valid = (uint8_t)(v1 && v2);
  return ORC_OK;
}

/* Switch-hyperedge connections: the count that the uc-max and uc-min
 * policies (Sec. 5.1, switch-hyperedge policy; App. B.3, is_util with the
 * objective time + gamma * sum of is_util) weigh. A connection is an ordered
 * rank pair (a, b) that carries some chunk through switch vertices only.
 * Alltoall: along each routed path, two ranks with only switch vertices
 * between them. Multicast: a rank b whose tree parent is a switch, paired
 * with the nearest rank above it in the tree. ReduceScatter runs the trees
 * backwards, so each pair is (b, a); Allreduce has both directions. The
 * count does not depend on priorities. */
static uint32_t connections_one(const orc_plan *p, const uint8_t *rt, oscratch *w,
                                const uint32_t *zero_prio, uint8_t *mark) {
  const int P = p->P, V = p->V;
  memset(mark, 0, (size_t)P * P);
  if (p->kind == ORC_ALLTOALL) {
    for (int c = 0; c < p->C; c++) {
      int s0 = p->owner[c], d = p->post[p->post_ptr[c]];
      if (s0 == d) continue;
      const oplist *L = &p->paths[s0 * P + d];
      int ch = rt[c];
      if (ch >= L->n) continue;
      const opath *q = &L->p[ch];
      int last = 0; /* index of the latest rank on the path */
      for (int j = 1; j <= q->hops; j++) {
        int v = q->vert[j];
        if (v >= P) continue;
        if (j - last > 1) mark[q->vert[last] * P + v] = 1;
        last = j;
      }
    }
  } else {
    w->n = 0;
    build_tree_sends(p, rt, zero_prio, w);
    for (int c = 0; c < p->C; c++) {
      const int *par = &w->tree_parent[(size_t)c * V];
      for (int b = 0; b < P; b++) {
        if (par[b] < 0) continue;
        int x = p->lsrc[par[b]];
        if (x < P) continue;
        while (x >= P) x = p->lsrc[par[x]]; /* the owner is a rank */
        if (p->kind != ORC_REDUCESCATTER) mark[x * P + b] = 1;
        if (p->kind == ORC_REDUCESCATTER || p->kind == ORC_ALLREDUCE) mark[b * P + x] = 1;
      }
    }
  }
  uint32_t n = 0;
  for (int i = 0; i < P * P; i++) n += mark[i];
  return n;
}

int orc_connections(const orc_plan *p, int64_t n, const uint8_t *routes, uint32_t *out) {
  oscratch w;
  scratch_init(p, &w);
  uint32_t *zero = (uint32_t *)calloc((size_t)p->C * p->V + 1, sizeof(uint32_t));
  uint8_t *mark = (uint8_t *)malloc((size_t)p->P * p->P);
  if (!zero || !mark) {
    free(zero);
    free(mark);
    scratch_free(&w);
    return ORC_ENOMEM;
  }
  for (int64_t i = 0; i < n; i++)
    out[i] = connections_one(p, routes + (size_t)i * p->route_stride, &w, zero, mark);
  free(zero);
  free(mark);
  scratch_free(&w);
  return ORC_OK;
}

/* Evaluate n candidates; routes row stride route_stride bytes, priorities
 * row stride prio_stride words. */
int orc_eval(const orc_plan *p, int64_t n, const uint8_t *routes, const uint32_t *prio,
             uint32_t *makespan, uint8_t *valid) {
  oscratch w;
  scratch_init(p, &w);
  int rc = ORC_OK;
  for (int64_t i = 0; i < n && rc == ORC_OK; i++)
    rc = eval_one(p, routes + (size_t)i * p->route_stride, prio + (size_t)i * p->prio_stride, &w,
                  &makespan[i], &valid[i]);
  scratch_free(&w);
  return rc;
}

/* Algorithmic integer operations of one schedule, the op model that prices
 * the evaluation against the chip's integer issue rate:
 *   one per link of every routed path walked while building the send set
 *     (route decode and tree merge, or the path hops of an Alltoall);
 *   three per send for its Step-2 keys (remaining, travelled, priority);
 *   n_l * ceil(log2 n_l) comparisons to order the n_l sends of each link
 *     (the per-link total order of Sec. 5.1 / App. B.2);
 *   four per send for the timing sweep of App. B.3 (max of ready and link
 *     free, add the latency, update the link, fold into the makespan);
 *   two per word of the presence bitmasks the postcondition reads (App. B):
 *     one bit per chunk at every vertex for multicast, one bit per source
 *     chunk at every rank for Alltoall.
 * Called after eval_phase, whose sends it reads. */
static uint64_t ceil_log2(uint64_t n) {
  uint64_t b = 0;
  while ((1ull << b) < n) b++;
  return b;
}

static uint64_t phase_ops(const orc_plan *p, int phase, const uint8_t *rt, const oscratch *w) {
  const int P = p->P;
  uint64_t visits = 0;
  for (int c = 0; c < p->C; c++) {
    const int o = p->owner[c];
    if (phase == ORC_ALLTOALL) {
      const int d = p->post[p->post_ptr[c]];
      if (d == o) continue;
      const oplist *L = &p->paths[o * P + d];
      if (rt[c] < L->n) visits += (uint64_t)L->p[rt[c]].hops;
      continue;
    }
    for (int d = 0; d < P; d++) {
      if (d == o || !in_post(p, c, d)) continue;
      const oplist *L = &p->paths[o * P + d];
      const int ch = rt[(size_t)c * P + d];
      if (ch < L->n) visits += (uint64_t)L->p[ch].hops;
    }
  }
  uint64_t *per_link = (uint64_t *)calloc((size_t)p->E + 1, sizeof(uint64_t));
  uint64_t order = 0;
  if (per_link) {
    for (int i = 0; i < w->n; i++) per_link[w->s[i].link]++;
    for (int e = 0; e < p->E; e++) order += per_link[e] * ceil_log2(per_link[e]);
    free(per_link);
  }
  uint64_t words;
  if (phase == ORC_ALLTOALL)
    words = (uint64_t)P * (((uint64_t)P * (uint64_t)p->cpr + 31) / 32);
  else
    words = (uint64_t)p->V * (((uint64_t)p->C + 31) / 32);
  return visits + 3 * (uint64_t)w->n + order + 4 * (uint64_t)w->n + 2 * words;
}

/* Evaluate n candidates like orc_eval and also write ops[i], the algorithmic
 * operation count of candidate i (both phases of an Allreduce). */
int orc_eval_ops(const orc_plan *p, int64_t n, const uint8_t *routes, const uint32_t *prio,
                 uint32_t *makespan, uint8_t *valid, uint64_t *ops) {
  oscratch w;
  scratch_init(p, &w);
  int rc = ORC_OK;
  for (int64_t i = 0; i < n && rc == ORC_OK; i++) {
    const uint8_t *rt = routes + (size_t)i * p->route_stride;
    const uint32_t *pr = prio + (size_t)i * p->prio_stride;
    if (p->kind != ORC_ALLREDUCE) {
      rc = eval_phase(p, p->kind, rt, pr, &w, &makespan[i], &valid[i]);
      if (rc == ORC_OK) ops[i] = phase_ops(p, p->kind, rt, &w);
      continue;
    }
    uint32_t m1, m2;
    uint8_t v1, v2;
    rc = eval_phase(p, ORC_REDUCESCATTER, rt, pr, &w, &m1, &v1);
    if (rc) break;
    const uint64_t o1 = phase_ops(p, ORC_REDUCESCATTER, rt, &w);
    rc = eval_phase(p, ORC_ALLGATHER, rt, pr + (size_t)p->C * p->V, &w, &m2, &v2);
    if (rc) break;
    if ((uint64_t)m1 + m2 >= (1ull << 32)) {
      rc = ORC_ELIMIT;
      break;
    }
    makespan[i] = m1 + m2;
    valid[i] = (uint8_t)(v1 && v2);
    ops[i] = o1 + phase_ops(p, ORC_ALLGATHER, rt, &w);
  }
  scratch_free(&w);
  return rc;
}

/* One candidate with every send reported: chunk, link, from, to, hop,
 * rem, trav, prio, position in its link's order, start, finish. For
 * Allreduce the ReduceScatter sends come first, then the Allgather sends
 * with their times shifted by the ReduceScatter makespan. */
typedef struct {
  int *chunk, *link, *from, *to, *hop, *pos;
  uint64_t *rem, *trav, *start, *finish;
  uint32_t *pr;
} odetail;

static void copy_detail(const oscratch *w, const odetail *o, int at, int cap, uint64_t shift) {
  for (int i = 0; i < w->n && at + i < cap; i++) {
    const osend *s = &w->s[i];
    o->chunk[at + i] = s->chunk;
    o->link[at + i] = s->link;
    o->from[at + i] = s->from;
    o->to[at + i] = s->to;
    o->hop[at + i] = s->hop;
    o->rem[at + i] = s->rem;
    o->trav[at + i] = s->trav;
    o->pr[at + i] = s->prio;
    o->pos[at + i] = s->pos;
    o->start[at + i] = s->start + shift;
    o->finish[at + i] = s->finish + shift;
  }
}

int orc_eval_detail(const orc_plan *p, const uint8_t *routes, const uint32_t *prio, int cap,
                    int *nsends, int *chunk, int *link, int *from, int *to, int *hop,
                    uint64_t *rem, uint64_t *trav, uint32_t *pr, int *pos, uint64_t *start,
                    uint64_t *finish, uint32_t *makespan, uint8_t *valid) {
  odetail o = {chunk, link, from, to, hop, pos, rem, trav, start, finish, pr};
  oscratch w;
  scratch_init(p, &w);
  int rc;
  if (p->kind != ORC_ALLREDUCE) {
    rc = eval_phase(p, p->kind, routes, prio, &w, makespan, valid);
    if (rc == ORC_OK) {
      *nsends = w.n;
      if (w.n > cap) rc = ORC_ELIMIT;
      copy_detail(&w, &o, 0, cap, 0);
    }
  } else {
    uint32_t m1, m2;
    uint8_t v1, v2;
    rc = eval_phase(p, ORC_REDUCESCATTER, routes, prio, &w, &m1, &v1);
    int n1 = w.n;
    if (rc == ORC_OK) copy_detail(&w, &o, 0, cap, 0);
    if (rc == ORC_OK)
      rc = eval_phase(p, ORC_ALLGATHER, routes, prio + (size_t)p->C * p->V, &w, &m2, &v2);
    if (rc == ORC_OK) {
      copy_detail(&w, &o, n1, cap, m1);
      *nsends = n1 + w.n;
      if (n1 + w.n > cap) rc = ORC_ELIMIT;
      *makespan = m1 + m2;
      *valid = (uint8_t)(v1 && v2);
    }
  }
  scratch_free(&w);
  return rc;
}
