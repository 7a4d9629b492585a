/*
 * CPU oracle for one multi-signal iteration of a growing self-organizing network
 * (Parigi, Stramieri, Pau, Piastra: "A Multi-signal Variant for the GPU-based
 * Parallelization of Growing Self-Organizing Networks").
 *
 * TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  These routines define the results the
 * HIP path must reproduce.  They share no source, header, table or helper with the HIP
 * path.  Only the test suite, the smoke check and the CPU-baseline leg of the benchmark
 * load this library.
 *
 * Every step is a plain sequential loop written in the order the paper states the
 * iteration (Sec. 2.1 "basic iteration", Sec. 2.2 "multi-signal variant"):
 *
 *   find winners   Sec. 2.1 step 2 / Sec. 2.2 step 2: exhaustive k = 2 nearest search.
 *   resolve        Sec. 2.2, collision kinds and the implicit lock: among signals whose
 *                  updates would touch a common unit, one survivor, the others discarded.
 *   adapt          Sec. 2.1 step 3, Eq. (adaptation), with eta(i,b) = 1 iff connected.
 *   update edges   Sec. 2.1 step 3: create or reset the winner-second connection, age
 *                  the winner's connections (footnote: GNG aging), drop old ones.
 *   grow           Sec. 2.1, insertion near the unit of largest accumulated error (GNG);
 *                  removal of units left without connections.
 *
 * Readings of points the paper leaves open (all fixed here, the HIP path follows them):
 *   - distance: squared Euclidean distance in IEEE binary32, computed exactly as
 *       dx = sx - wx; dy = sy - wy; dz = sz - wz; d = (dx*dx + dy*dy) + dz*dz
 *     with every operation rounded to nearest even, no fused multiply-add, no sqrt
 *     (the square root is monotone, so the order of units is the same, but rounding
 *     it could merge distinct values into ties);
 *   - ties: the order is lexicographic on (d, unit index); the second winner is the
 *     minimum over all units other than the winner;
 *   - snapshot: all winners, all neighbourhoods and all conflicts are taken from the
 *     state before the iteration;
 *   - lock scope: a signal j claims L_j = {b_j, s_j} plus the pre-iteration neighbours
 *     of b_j; its key is (bits(d1_j) << 32) | j; j survives iff no other signal with a
 *     smaller key claims a unit of L_j (one round, no re-admission);
 *   - adaptation step (the equation prints a norm where a vector is meant):
 *       t = xi - w;  t = eps * t;  w = w + t   per component, binary32;
 *     eps_b for b_j, eps_n for each unit of N(b_j) plus s_j (s_j moved once);
 *   - order inside one accepted signal: age every edge at b_j by one, then set the
 *     edge {b_j, s_j} to age 0 (creating it if absent), then remove the edges at b_j
 *     whose age exceeds max_age;
 *   - error: err[b_j] += d1_j for accepted signals, then err[i] *= beta for every unit
 *     once per iteration;
 *   - removal: a unit is removed (stable compaction) only if its last edge was removed
 *     by aging since the last grow call; units that never had edges stay;
 *   - insertion: q = argmax err, f = argmax err over N(q) (ties to the lower index),
 *     w_r = (w_q + w_f) * 0.5, edge {q,f} replaced by {q,r} and {r,f} at age 0,
 *     err_q *= alpha, err_f *= alpha, err_r = err_q; skipped when N(q) is empty.
 *
 * The paper's own collision rule is a second mode (lock_mode = 1, key_mode = 1 for its
 * arrival order): the lock covers the winner only (Sec. 2.2, "implicit lock on the winner
 * unit"), so the survivor of each winner unit is its signal of smallest key and all other
 * signals with that winner are discarded; the survivors then update the network one after
 * another in ascending key order, each with the complete single-signal step of Sec. 2.1
 * (age, connect, move the winner and its neighbours as they are at that moment plus the
 * second, drop old edges, err[b] += d1) on the network left by the survivors before it;
 * winners and seconds stay those of the snapshot.  err *= beta once after all survivors.
 * In this mode adapt performs the whole update and update_edges has nothing left to do.
 * key_mode 1 keys a signal by its index alone (arrival order), 0 by (bits(d1) << 32) | j.
 *
 * The growing-network schedule (orc_run_schedule) drives whole iterations the way the
 * paper's runs do (Sec. 3.1): starting from the current network, the level of parallelism
 * of every iteration is the smallest power of two greater than the number of units, capped;
 * units are inserted GNG-style every insert_every signals (Sec. 2.1: insertion at regular
 * intervals near the unit of largest error), several in one iteration when it drew that
 * many signals; the run stops on a threshold on the quantization error, the mean squared
 * distance between the signals and their winners (Sec. 2.1, convergence criterion).
 * Readings: signals are drawn from a point cloud by SplitMix64 (a counter-based generator
 * with a published definition: output c of seed s mixes s + c * 0x9E3779B97F4A7C15), the
 * c-th signal of the run (c = 1, 2, ...) takes point ((output_c >> 32) * P) >> 32; the
 * error is tested on windows of at least qe_window signals (whole iterations), each d1
 * counted as the integer floor(d1 * 2^32) (capped at 2^44 for d1 >= 4096) so that the sum
 * is exact and does not depend on its order; a window's mean is
 * (double)sum * 2^-32 / (double)count.  Per iteration: draw, find, resolve, adapt, update
 * edges, accumulate, remove orphaned units, insert, then the window test and the signal cap.
 *
 * A third collision rule (lock_mode = 2) keeps the lock sets of lock_mode 0 but takes the
 * signals greedily in key order: a signal is accepted iff its lock set is disjoint from the
 * lock set of every signal accepted before it (signals whose blockers were themselves
 * rejected are re-admitted); accepted lock sets are still pairwise disjoint, so adapt and
 * the edge update are those of lock_mode 0.
 *
 * Indexed find winners (orc_find_winners_grid) is the hash index of the paper's "Indexed"
 * implementation (Sec. 3.1) applied to every signal of the batch: a grid of cubes of side h
 * over an axis-parallel box that holds the input signals; the winner and the second are
 * searched among the units of the signal's cube and its 26 neighbours, and the exhaustive
 * search is used when that search fails (fewer than two units there).  Readings: the cell
 * of a point p is c_a = floor((p_a - lo_a) * inv_h) per axis, inv_h = 1 / h rounded to
 * binary32 and every operation in binary32, clamped to [0, dims_a - 1] (so points outside
 * the box fall into its border cells); candidates are the units whose cell differs from
 * the signal's by at most one on every axis; among them the order is the same (d, index)
 * order as the exhaustive search.  The result can differ from the exhaustive one when a
 * unit outside the 27 cubes is nearer than the second found inside, as the paper notes.
 *
 * Build: gcc -O2 -ffp-contract=off -fopenmp -shared -fPIC (no -ffast-math, no -march).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>

#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_OK 0
#define ORC_E_INVAL -1
#define ORC_E_CAPACITY -2
#define ORC_E_STATE -4

typedef struct {
  float eps_b;
  float eps_n;
  int32_t max_age;
  float err_alpha;
  float err_beta;
  int32_t n_max;
  int32_t e_max;
  int32_t m_max;
  int32_t lock_mode;  /* 0: lock set {b, s} + N(b), one round; 1: the winner only,
                         sequential update; 2: lock set, greedy in key order */
  int32_t key_mode;   /* 0: (bits(d1) << 32) | j; 1: j */
} orc_params;

typedef struct {
  orc_params p;
  int32_t n;        /* live units */
  int64_t n_edges;  /* undirected edges */
  float *x, *y, *z, *err;
  int32_t *deg;     /* neighbours per unit */
  int32_t *cap;     /* allocated length of nb[u] / ag[u] */
  int32_t **nb;     /* neighbour ids of u, ascending */
  int32_t **ag;     /* age of edge {u, nb[u][k]} */
  uint8_t *orphan;  /* 1: last edge removed by aging since the last grow call */
  int32_t status;   /* sticky error */
} orc_net;

/* ------------------------------------------------------------------ adjacency --- */

static int32_t edge_pos(const orc_net* g, int32_t u, int32_t v) {
  for (int32_t k = 0; k < g->deg[u]; ++k)
    if (g->nb[u][k] == v) return k;
  return -1;
}

static int half_insert(orc_net* g, int32_t u, int32_t v, int32_t age) {
  if (g->deg[u] == g->cap[u]) {
    int32_t nc = g->cap[u] ? 2 * g->cap[u] : 8;
    int32_t* nb = (int32_t*)realloc(g->nb[u], sizeof(int32_t) * (size_t)nc);
    if (!nb) return ORC_E_CAPACITY;
    g->nb[u] = nb;
    int32_t* ag = (int32_t*)realloc(g->ag[u], sizeof(int32_t) * (size_t)nc);
    if (!ag) return ORC_E_CAPACITY;
    g->ag[u] = ag;
    g->cap[u] = nc;
  }
  /* keep the row ascending by neighbour id */
  int32_t k = g->deg[u];
  while (k > 0 && g->nb[u][k - 1] > v) {
    g->nb[u][k] = g->nb[u][k - 1];
    g->ag[u][k] = g->ag[u][k - 1];
    --k;
  }
  g->nb[u][k] = v;
  g->ag[u][k] = age;
  g->deg[u] += 1;
  return ORC_OK;
}

static void half_remove(orc_net* g, int32_t u, int32_t v) {
  int32_t k = edge_pos(g, u, v);
  if (k < 0) return;
  for (; k + 1 < g->deg[u]; ++k) {
    g->nb[u][k] = g->nb[u][k + 1];
    g->ag[u][k] = g->ag[u][k + 1];
  }
  g->deg[u] -= 1;
}

static int add_edge(orc_net* g, int32_t u, int32_t v, int32_t age) {
  int rc = half_insert(g, u, v, age);
  if (rc) return rc;
  rc = half_insert(g, v, u, age);
  if (rc) return rc;
  g->n_edges += 1;
  return ORC_OK;
}

static void remove_edge(orc_net* g, int32_t u, int32_t v) {
  half_remove(g, u, v);
  half_remove(g, v, u);
  g->n_edges -= 1;
}

static void set_age(orc_net* g, int32_t u, int32_t v, int32_t age) {
  int32_t k = edge_pos(g, u, v);
  if (k >= 0) g->ag[u][k] = age;
  k = edge_pos(g, v, u);
  if (k >= 0) g->ag[v][k] = age;
}

static int32_t get_age(const orc_net* g, int32_t u, int32_t v) {
  int32_t k = edge_pos(g, u, v);
  return k >= 0 ? g->ag[u][k] : -1;
}

/* ------------------------------------------------------------- create/destroy --- */

void orc_destroy(orc_net* g) {
  if (!g) return;
  if (g->nb)
    for (int32_t u = 0; u < g->p.n_max; ++u) free(g->nb[u]);
  if (g->ag)
    for (int32_t u = 0; u < g->p.n_max; ++u) free(g->ag[u]);
  free(g->nb); free(g->ag); free(g->deg); free(g->cap);
  free(g->x); free(g->y); free(g->z); free(g->err); free(g->orphan);
  free(g);
}

static int params_ok(const orc_params* p) {
  if (!p) return 0;
  if (!(p->eps_b >= 0.0f && p->eps_b <= 1.0f)) return 0;
  if (!(p->eps_n >= 0.0f && p->eps_n <= 1.0f)) return 0;
  if (p->max_age < 0) return 0;
  if (p->n_max < 2 || p->e_max < 0 || p->m_max < 1) return 0;
  if (p->lock_mode < 0 || p->lock_mode > 2 || p->key_mode < 0 || p->key_mode > 1) return 0;
  return 1;
}

/* xyz: SoA [3][n0] binary32 (all x, then all y, then all z). */
int orc_create(const orc_params* p, int32_t n0, const float* xyz, orc_net** out) {
  if (!out) return ORC_E_INVAL;
  *out = NULL;
  if (!params_ok(p) || n0 < 0 || n0 > p->n_max || (n0 > 0 && !xyz)) return ORC_E_INVAL;
  orc_net* g = (orc_net*)calloc(1, sizeof(orc_net));
  if (!g) return ORC_E_CAPACITY;
  g->p = *p;
  size_t nm = (size_t)p->n_max;
  g->x = (float*)calloc(nm, sizeof(float));
  g->y = (float*)calloc(nm, sizeof(float));
  g->z = (float*)calloc(nm, sizeof(float));
  g->err = (float*)calloc(nm, sizeof(float));
  g->deg = (int32_t*)calloc(nm, sizeof(int32_t));
  g->cap = (int32_t*)calloc(nm, sizeof(int32_t));
  g->nb = (int32_t**)calloc(nm, sizeof(int32_t*));
  g->ag = (int32_t**)calloc(nm, sizeof(int32_t*));
  g->orphan = (uint8_t*)calloc(nm, 1);
  if (!g->x || !g->y || !g->z || !g->err || !g->deg || !g->cap || !g->nb || !g->ag ||
      !g->orphan) {
    orc_destroy(g);
    return ORC_E_CAPACITY;
  }
  g->n = n0;
  for (int32_t i = 0; i < n0; ++i) {
    g->x[i] = xyz[i];
    g->y[i] = xyz[(size_t)n0 + i];
    g->z[i] = xyz[2 * (size_t)n0 + i];
  }
  *out = g;
  return ORC_OK;
}

/* ---------------------------------------------------------------- find winners --- */

/* (da, ia) < (db, ib) in the lexicographic order on (distance, unit index). */
static int key_less(float da, int32_t ia, float db, int32_t ib) {
  return da < db || (da == db && ia < ib);
}

/*
 * For every signal j: b_j = the unit of smallest (d, index), s_j = the unit of smallest
 * (d, index) among the others; d1_j, d2_j their distances.  sig: SoA [3][m].
 * Signals are independent, so they may be shared out over threads; each signal's scan
 * is the same sequential loop whatever the thread count.
 */
int orc_find_winners(const orc_net* g, const float* sig, int32_t m, int32_t* winner,
                     int32_t* second, float* d1, float* d2, int32_t nthreads) {
  if (!g || m < 0 || m > g->p.m_max) return ORC_E_INVAL;
  if (g->n < 2) return ORC_E_INVAL;
  if (m == 0) return ORC_OK;
  if (!sig || !winner || !second || !d1 || !d2) return ORC_E_INVAL;
  const int32_t n = g->n;
  const float *x = g->x, *y = g->y, *z = g->z;
#ifdef _OPENMP
  if (nthreads < 1) nthreads = 1;
#pragma omp parallel for num_threads(nthreads) schedule(dynamic, 16)
#endif
  for (int32_t j = 0; j < m; ++j) {
    const float sx = sig[j], sy = sig[(size_t)m + j], sz = sig[2 * (size_t)m + j];
    float bd = INFINITY, sd = INFINITY;
    int32_t bi = -1, si = -1;
    for (int32_t i = 0; i < n; ++i) {
      float dx = sx - x[i];
      float dy = sy - y[i];
      float dz = sz - z[i];
      float d = (dx * dx + dy * dy) + dz * dz;
      if (bi < 0 || key_less(d, i, bd, bi)) {
        sd = bd; si = bi;
        bd = d; bi = i;
      } else if (si < 0 || key_less(d, i, sd, si)) {
        sd = d; si = i;
      }
    }
    winner[j] = bi; second[j] = si; d1[j] = bd; d2[j] = sd;
  }
  (void)nthreads;
  return ORC_OK;
}

/* ------------------------------------------------------------- resolve conflicts --- */

static uint64_t signal_key(const orc_net* g, float d1, int32_t j) {
  if (g->p.key_mode == 1) return (uint64_t)(uint32_t)j;
  uint32_t bits;
  memcpy(&bits, &d1, sizeof bits);
  return ((uint64_t)bits << 32) | (uint32_t)j;
}

static int check_pair(const orc_net* g, int32_t b, int32_t s) {
  return b >= 0 && b < g->n && s >= 0 && s < g->n && b != s;
}

/*
 * L_j = {b_j, s_j} + N(b_j) on the pre-iteration graph (lock_mode 0) or {b_j} (lock_mode
 * 1).  owner[u] = the smallest key among the signals that claim u; j is accepted iff it
 * owns every unit of L_j.
 */
static int resolve_greedy(const orc_net* g, int32_t m, const int32_t* winner,
                          const int32_t* second, const float* d1, uint8_t* accepted);

int orc_resolve_conflicts(const orc_net* g, int32_t m, const int32_t* winner,
                          const int32_t* second, const float* d1, uint8_t* accepted) {
  if (!g || m < 0 || m > g->p.m_max) return ORC_E_INVAL;
  if (m == 0) return ORC_OK;
  if (!winner || !second || !d1 || !accepted) return ORC_E_INVAL;
  for (int32_t j = 0; j < m; ++j)
    if (!check_pair(g, winner[j], second[j])) return ORC_E_INVAL;
  if (g->p.lock_mode == 2) return resolve_greedy(g, m, winner, second, d1, accepted);
  uint64_t* owner = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)(g->n > 0 ? g->n : 1));
  if (!owner) return ORC_E_CAPACITY;
  for (int32_t u = 0; u < g->n; ++u) owner[u] = UINT64_MAX;
  const int whole = g->p.lock_mode == 0;
  for (int32_t j = 0; j < m; ++j) {
    const uint64_t key = signal_key(g, d1[j], j);
    const int32_t b = winner[j], s = second[j];
    if (key < owner[b]) owner[b] = key;
    if (!whole) continue;
    if (key < owner[s]) owner[s] = key;
    for (int32_t k = 0; k < g->deg[b]; ++k) {
      int32_t u = g->nb[b][k];
      if (key < owner[u]) owner[u] = key;
    }
  }
  for (int32_t j = 0; j < m; ++j) {
    const uint64_t key = signal_key(g, d1[j], j);
    const int32_t b = winner[j], s = second[j];
    int ok = owner[b] == key;
    if (whole) {
      ok = ok && owner[s] == key;
      for (int32_t k = 0; ok && k < g->deg[b]; ++k) ok = owner[g->nb[b][k]] == key;
    }
    accepted[j] = (uint8_t)ok;
  }
  free(owner);
  return ORC_OK;
}

/* ---------------------------------------------------------------------- adapt --- */

/* w <- w + eps * (xi - w), one rounding per operation, per component. */
static void move_unit(orc_net* g, int32_t u, float eps, float sx, float sy, float sz) {
  float t;
  t = sx - g->x[u]; t = eps * t; g->x[u] = g->x[u] + t;
  t = sy - g->y[u]; t = eps * t; g->y[u] = g->y[u] + t;
  t = sz - g->z[u]; t = eps * t; g->z[u] = g->z[u] + t;
}

static int sequential_update(orc_net* g, const float* sig, int32_t m, const int32_t* winner,
                             const int32_t* second, const float* d1, const uint8_t* accepted);

int orc_adapt(orc_net* g, const float* sig, int32_t m, const int32_t* winner,
              const int32_t* second, const float* d1, const uint8_t* accepted) {
  if (!g || m < 0 || m > g->p.m_max) return ORC_E_INVAL;
  if (m > 0 && (!sig || !winner || !second || !d1 || !accepted)) return ORC_E_INVAL;
  for (int32_t j = 0; j < m; ++j)
    if (accepted[j] && !check_pair(g, winner[j], second[j])) return ORC_E_INVAL;
  if (g->p.lock_mode == 1) return sequential_update(g, sig, m, winner, second, d1, accepted);
  for (int32_t j = 0; j < m; ++j) {
    if (!accepted[j]) continue;
    const float sx = sig[j], sy = sig[(size_t)m + j], sz = sig[2 * (size_t)m + j];
    const int32_t b = winner[j], s = second[j];
    move_unit(g, b, g->p.eps_b, sx, sy, sz);
    for (int32_t k = 0; k < g->deg[b]; ++k)
      move_unit(g, g->nb[b][k], g->p.eps_n, sx, sy, sz);
    if (edge_pos(g, b, s) < 0) move_unit(g, s, g->p.eps_n, sx, sy, sz);
    g->err[b] = g->err[b] + d1[j];
  }
  for (int32_t i = 0; i < g->n; ++i) g->err[i] = g->err[i] * g->p.err_beta;
  return ORC_OK;
}

/* --------------------------------------------------------------- update edges --- */

int orc_update_edges(orc_net* g, int32_t m, const int32_t* winner, const int32_t* second,
                     const uint8_t* accepted) {
  if (!g || m < 0 || m > g->p.m_max) return ORC_E_INVAL;
  if (m > 0 && (!winner || !second || !accepted)) return ORC_E_INVAL;
  for (int32_t j = 0; j < m; ++j)
    if (accepted[j] && !check_pair(g, winner[j], second[j])) return ORC_E_INVAL;
  if (g->p.lock_mode == 1) return ORC_OK;  /* adapt performed the whole update */
  int32_t* tmp = NULL;
  int32_t tmp_cap = 0;
  for (int32_t j = 0; j < m; ++j) {
    if (!accepted[j]) continue;
    const int32_t b = winner[j], s = second[j];
    /* 1. age every edge at b */
    for (int32_t k = 0; k < g->deg[b]; ++k) {
      int32_t v = g->nb[b][k];
      set_age(g, b, v, g->ag[b][k] + 1);
    }
    /* 2. connect b and s at age 0 */
    if (edge_pos(g, b, s) >= 0) {
      set_age(g, b, s, 0);
    } else {
      int rc = add_edge(g, b, s, 0);
      if (rc) { free(tmp); g->status = rc; return rc; }
    }
    /* 3. remove the edges at b older than max_age */
    if (g->deg[b] > tmp_cap) {
      tmp_cap = g->deg[b];
      int32_t* t = (int32_t*)realloc(tmp, sizeof(int32_t) * (size_t)tmp_cap);
      if (!t) { free(tmp); g->status = ORC_E_CAPACITY; return ORC_E_CAPACITY; }
      tmp = t;
    }
    int32_t nd = 0;
    for (int32_t k = 0; k < g->deg[b]; ++k)
      if (g->ag[b][k] > g->p.max_age) tmp[nd++] = g->nb[b][k];
    for (int32_t k = 0; k < nd; ++k) {
      int32_t v = tmp[k];
      remove_edge(g, b, v);
      if (g->deg[v] == 0) g->orphan[v] = 1;
    }
  }
  free(tmp);
  if (g->n_edges > g->p.e_max) {
    g->status = ORC_E_CAPACITY;
    return ORC_E_CAPACITY;
  }
  return ORC_OK;
}

/* ----------------------------------------------------- greedy resolve (lock_mode 2) --- */

static const orc_net* greedy_net;   /* the comparator's context (the oracle is not reentrant) */
static const float* greedy_d1;

static int by_key_greedy(const void* a, const void* b) {
  const int32_t i = *(const int32_t*)a, j = *(const int32_t*)b;
  const uint64_t ki = signal_key(greedy_net, greedy_d1[i], i);
  const uint64_t kj = signal_key(greedy_net, greedy_d1[j], j);
  return ki < kj ? -1 : (ki > kj ? 1 : 0);
}

/* The signals in ascending key order; each is accepted iff its lock set {b, s} + N(b) (the
 * pre-iteration graph) shares no unit with the lock set of a signal accepted before it. */
static int resolve_greedy(const orc_net* g, int32_t m, const int32_t* winner,
                          const int32_t* second, const float* d1, uint8_t* accepted) {
  int32_t* order = (int32_t*)malloc(sizeof(int32_t) * (size_t)m);
  uint8_t* taken = (uint8_t*)calloc((size_t)(g->n > 0 ? g->n : 1), 1);
  if (!order || !taken) { free(order); free(taken); return ORC_E_CAPACITY; }
  for (int32_t j = 0; j < m; ++j) order[j] = j;
  greedy_net = g;
  greedy_d1 = d1;
  qsort(order, (size_t)m, sizeof(int32_t), by_key_greedy);
  for (int32_t q = 0; q < m; ++q) {
    const int32_t j = order[q], b = winner[j], s = second[j];
    int free_set = !taken[b] && !taken[s];
    for (int32_t k = 0; free_set && k < g->deg[b]; ++k) free_set = !taken[g->nb[b][k]];
    accepted[j] = (uint8_t)free_set;
    if (!free_set) continue;
    taken[b] = 1;
    taken[s] = 1;
    for (int32_t k = 0; k < g->deg[b]; ++k) taken[g->nb[b][k]] = 1;
  }
  free(order);
  free(taken);
  return ORC_OK;
}

/* ------------------------------------------------- sequential update (lock_mode 1) --- */

static const orc_net* sort_net;   /* the comparator's context (the oracle is not reentrant) */
static const float* sort_d1;

static int by_key(const void* a, const void* b) {
  const int32_t i = *(const int32_t*)a, j = *(const int32_t*)b;
  const uint64_t ki = signal_key(sort_net, sort_d1[i], i), kj = signal_key(sort_net, sort_d1[j], j);
  return ki < kj ? -1 : (ki > kj ? 1 : 0);
}

/* The survivors in ascending key order, each with the complete single-signal step of
 * Sec. 2.1 on the current network (see the header); then err *= beta once. */
static int sequential_update(orc_net* g, const float* sig, int32_t m, const int32_t* winner,
                             const int32_t* second, const float* d1, const uint8_t* accepted) {
  int32_t* order = (int32_t*)malloc(sizeof(int32_t) * (size_t)(m > 0 ? m : 1));
  if (!order) return ORC_E_CAPACITY;
  int32_t ns = 0;
  for (int32_t j = 0; j < m; ++j)
    if (accepted[j]) order[ns++] = j;
  sort_net = g;
  sort_d1 = d1;
  qsort(order, (size_t)ns, sizeof(int32_t), by_key);
  int32_t* tmp = NULL;
  int32_t tmp_cap = 0;
  int rc = ORC_OK;
  for (int32_t q = 0; q < ns && rc == ORC_OK; ++q) {
    const int32_t j = order[q];
    const int32_t b = winner[j], s = second[j];
    const float sx = sig[j], sy = sig[(size_t)m + j], sz = sig[2 * (size_t)m + j];
    /* neighbours of b before this step; s moves once, as a neighbour or on its own */
    if (g->deg[b] > tmp_cap) {
      tmp_cap = g->deg[b] + 1;
      int32_t* t = (int32_t*)realloc(tmp, sizeof(int32_t) * (size_t)tmp_cap);
      if (!t) { rc = ORC_E_CAPACITY; break; }
      tmp = t;
    }
    const int32_t nb0 = g->deg[b];
    memcpy(tmp, g->nb[b], sizeof(int32_t) * (size_t)nb0);
    const int s_was_nb = edge_pos(g, b, s) >= 0;
    /* 1. age every edge at b; 2. connect b and s at age 0 */
    for (int32_t k = 0; k < g->deg[b]; ++k) set_age(g, b, g->nb[b][k], g->ag[b][k] + 1);
    if (s_was_nb) {
      set_age(g, b, s, 0);
    } else if ((rc = add_edge(g, b, s, 0)) != ORC_OK) {
      break;
    }
    /* 3. move the winner, its neighbours and the second */
    move_unit(g, b, g->p.eps_b, sx, sy, sz);
    for (int32_t k = 0; k < nb0; ++k) move_unit(g, tmp[k], g->p.eps_n, sx, sy, sz);
    if (!s_was_nb) move_unit(g, s, g->p.eps_n, sx, sy, sz);
    /* 4. remove the edges at b older than max_age */
    int32_t nd = 0;
    for (int32_t k = 0; k < g->deg[b]; ++k)
      if (g->ag[b][k] > g->p.max_age) tmp[nd++] = g->nb[b][k];
    for (int32_t k = 0; k < nd; ++k) {
      remove_edge(g, b, tmp[k]);
      if (g->deg[tmp[k]] == 0) g->orphan[tmp[k]] = 1;
    }
    g->err[b] = g->err[b] + d1[j];
  }
  free(tmp);
  free(order);
  if (rc == ORC_OK && g->n_edges > g->p.e_max) rc = ORC_E_CAPACITY;
  if (rc != ORC_OK) {
    g->status = rc;
    return rc;
  }
  for (int32_t i = 0; i < g->n; ++i) g->err[i] = g->err[i] * g->p.err_beta;
  return ORC_OK;
}

/* ---------------------------------------------------------------------- grow --- */

static int remove_orphans(orc_net* g) {
  int32_t* newid = (int32_t*)malloc(sizeof(int32_t) * (size_t)(g->n > 0 ? g->n : 1));
  if (!newid) return ORC_E_CAPACITY;
  int32_t kept = 0;
  for (int32_t u = 0; u < g->n; ++u) {
    int gone = g->orphan[u] && g->deg[u] == 0;
    newid[u] = gone ? -1 : kept;
    if (!gone) ++kept;
  }
  if (kept == g->n) {
    free(newid);
    memset(g->orphan, 0, (size_t)g->p.n_max);
    return ORC_OK;
  }
  for (int32_t u = 0; u < g->n; ++u) {
    int32_t t = newid[u];
    if (t < 0) {
      free(g->nb[u]); free(g->ag[u]);
      g->nb[u] = NULL; g->ag[u] = NULL; g->cap[u] = 0; g->deg[u] = 0;
      continue;
    }
    /* t <= u: moving downwards never overwrites a unit not yet visited */
    g->x[t] = g->x[u]; g->y[t] = g->y[u]; g->z[t] = g->z[u]; g->err[t] = g->err[u];
    if (t != u) {
      g->nb[t] = g->nb[u]; g->ag[t] = g->ag[u];
      g->deg[t] = g->deg[u]; g->cap[t] = g->cap[u];
      g->nb[u] = NULL; g->ag[u] = NULL; g->deg[u] = 0; g->cap[u] = 0;
    }
    /* remapping is monotone, so rows stay ascending */
    for (int32_t k = 0; k < g->deg[t]; ++k) g->nb[t][k] = newid[g->nb[t][k]];
  }
  for (int32_t u = kept; u < g->n; ++u) {
    g->x[u] = 0.0f; g->y[u] = 0.0f; g->z[u] = 0.0f; g->err[u] = 0.0f;
  }
  g->n = kept;
  memset(g->orphan, 0, (size_t)g->p.n_max);
  free(newid);
  return ORC_OK;
}

static int insert_unit(orc_net* g) {
  if (g->n < 1 || g->n >= g->p.n_max) return ORC_OK;
  int32_t q = 0;
  for (int32_t i = 1; i < g->n; ++i)
    if (g->err[i] > g->err[q]) q = i;
  if (g->deg[q] == 0) return ORC_OK;
  int32_t f = g->nb[q][0];
  for (int32_t k = 1; k < g->deg[q]; ++k) {
    int32_t v = g->nb[q][k];
    if (g->err[v] > g->err[f] || (g->err[v] == g->err[f] && v < f)) f = v;
  }
  if (g->n_edges + 1 > g->p.e_max) {
    g->status = ORC_E_CAPACITY;
    return ORC_E_CAPACITY;
  }
  const int32_t r = g->n;
  g->n += 1;
  g->x[r] = (g->x[q] + g->x[f]) * 0.5f;
  g->y[r] = (g->y[q] + g->y[f]) * 0.5f;
  g->z[r] = (g->z[q] + g->z[f]) * 0.5f;
  remove_edge(g, q, f);
  int rc = add_edge(g, q, r, 0);
  if (!rc) rc = add_edge(g, r, f, 0);
  if (rc) { g->status = rc; return rc; }
  g->err[q] = g->err[q] * g->p.err_alpha;
  g->err[f] = g->err[f] * g->p.err_alpha;
  g->err[r] = g->err[q];
  return ORC_OK;
}

/* Remove orphaned units, then, when iteration % insert_every == 0, insert one unit. */
int orc_grow(orc_net* g, int32_t iteration, int32_t insert_every) {
  if (!g || insert_every < 0) return ORC_E_INVAL;
  int rc = remove_orphans(g);
  if (rc) return rc;
  if (insert_every > 0 && iteration > 0 && iteration % insert_every == 0)
    return insert_unit(g);
  return ORC_OK;
}

/* ------------------------------------------------------------- state transfer --- */

int orc_sizes(const orc_net* g, int32_t* n_units, int64_t* n_edges) {
  if (!g) return ORC_E_INVAL;
  if (n_units) *n_units = g->n;
  if (n_edges) *n_edges = g->n_edges;
  return ORC_OK;
}

int orc_status(const orc_net* g) { return g ? g->status : ORC_E_INVAL; }

/*
 * xyz: SoA [3][n]; err: [n]; edges: SoA [3][n_edges] = (u, v, age) with u < v,
 * ascending by (u, v); orphan: [n].  Any output pointer may be NULL.
 */
int orc_export(const orc_net* g, float* xyz, float* err, int32_t* edges, uint8_t* orphan) {
  if (!g) return ORC_E_INVAL;
  const size_t n = (size_t)g->n, e = (size_t)g->n_edges;
  if (xyz)
    for (size_t i = 0; i < n; ++i) {
      xyz[i] = g->x[i]; xyz[n + i] = g->y[i]; xyz[2 * n + i] = g->z[i];
    }
  if (err) memcpy(err, g->err, sizeof(float) * n);
  if (orphan) memcpy(orphan, g->orphan, n);
  if (edges) {
    size_t t = 0;
    for (int32_t u = 0; u < g->n; ++u)
      for (int32_t k = 0; k < g->deg[u]; ++k) {
        int32_t v = g->nb[u][k];
        if (v > u) {
          edges[t] = u; edges[e + t] = v; edges[2 * e + t] = g->ag[u][k];
          ++t;
        }
      }
  }
  return ORC_OK;
}

/* Replace the whole state.  edges: SoA [3][n_edges] = (u, v, age), any order, u != v. */
int orc_import(orc_net* g, int32_t n, const float* xyz, const float* err, int32_t n_edges,
               const int32_t* edges) {
  if (!g || n < 0 || n > g->p.n_max || n_edges < 0 || n_edges > g->p.e_max) return ORC_E_INVAL;
  if ((n > 0 && !xyz) || (n_edges > 0 && !edges)) return ORC_E_INVAL;
  for (int32_t k = 0; k < n_edges; ++k) {
    int32_t u = edges[k], v = edges[n_edges + k], a = edges[2 * n_edges + k];
    if (u < 0 || v < 0 || u >= n || v >= n || u == v || a < 0) return ORC_E_INVAL;
  }
  for (int32_t u = 0; u < g->p.n_max; ++u) g->deg[u] = 0;
  g->n_edges = 0;
  g->n = n;
  for (int32_t i = 0; i < n; ++i) {
    g->x[i] = xyz[i]; g->y[i] = xyz[(size_t)n + i]; g->z[i] = xyz[2 * (size_t)n + i];
    g->err[i] = err ? err[i] : 0.0f;
  }
  for (int32_t i = n; i < g->p.n_max; ++i) {
    g->x[i] = 0.0f; g->y[i] = 0.0f; g->z[i] = 0.0f; g->err[i] = 0.0f;
  }
  memset(g->orphan, 0, (size_t)g->p.n_max);
  for (int32_t k = 0; k < n_edges; ++k) {
    int32_t u = edges[k], v = edges[n_edges + k], a = edges[2 * n_edges + k];
    if (edge_pos(g, u, v) >= 0) return ORC_E_INVAL;
    int rc = add_edge(g, u, v, a);
    if (rc) return rc;
  }
  g->status = ORC_OK;
  return ORC_OK;
}

int orc_age(const orc_net* g, int32_t u, int32_t v) { return g ? get_age(g, u, v) : -1; }

/* ---------------------------------------------------------------- schedule --- */

typedef struct {
  int32_t m_cap;         /* largest level of parallelism */
  int32_t fixed_m;       /* > 0: this m every iteration instead of the power-of-two rule */
  int64_t insert_every;  /* signals between two insertions; 0 = none */
  int64_t qe_window;     /* signals per stop test */
  int64_t max_signals;   /* stop once this many signals were drawn */
  float qe_threshold;    /* stop when a window's mean is below it */
  uint64_t seed;
} orc_schedule;

typedef struct {
  int64_t iterations, signals, accepted, inserted;
  double qe;             /* the last complete window's mean (the partial one if none) */
  int32_t converged, n_units;
  int64_t n_edges;
} orc_schedule_result;

/* Output number `counter` (1, 2, ...) of SplitMix64 started at `seed`. */
uint64_t orc_splitmix64(uint64_t seed, uint64_t counter) {
  uint64_t z = seed + counter * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

/* The smallest power of two greater than n, capped at m_cap (Sec. 3.1); fixed_m if > 0. */
int32_t orc_schedule_m(int32_t n, int32_t m_cap, int32_t fixed_m) {
  if (fixed_m > 0) return fixed_m;
  int64_t m = 1;
  while (m <= n) m *= 2;
  return m > m_cap ? m_cap : (int32_t)m;
}

static uint64_t qe_units(float d1) {
  if (d1 < 4096.0f) return (uint64_t)(d1 * 4294967296.0f);
  return (uint64_t)1 << 44;  /* also +inf and NaN */
}

int orc_run_schedule(orc_net* g, const float* cloud, int64_t n_points, const orc_schedule* s,
                     orc_schedule_result* r, int threads) {
  if (!g || !cloud || !s || !r) return ORC_E_INVAL;
  if (n_points < 1 || n_points > 0xFFFFFFFFll) return ORC_E_INVAL;
  if (s->m_cap < 1 || s->m_cap > g->p.m_max || s->fixed_m < 0 || s->fixed_m > g->p.m_max)
    return ORC_E_INVAL;
  if (s->insert_every < 0 || s->qe_window < 1 || s->max_signals < 1) return ORC_E_INVAL;
  const int32_t mm = s->fixed_m > 0 ? s->fixed_m : s->m_cap;
  if (s->qe_window + mm > ((int64_t)1 << 19)) return ORC_E_INVAL;
  memset(r, 0, sizeof(*r));
  const size_t cap = (size_t)mm;
  float* sig = (float*)malloc(sizeof(float) * 3 * cap);
  int32_t* w = (int32_t*)malloc(sizeof(int32_t) * cap);
  int32_t* sc = (int32_t*)malloc(sizeof(int32_t) * cap);
  float* d1 = (float*)malloc(sizeof(float) * cap);
  float* d2 = (float*)malloc(sizeof(float) * cap);
  uint8_t* acc = (uint8_t*)malloc(cap);
  int rc = ORC_OK;
  if (!sig || !w || !sc || !d1 || !d2 || !acc) rc = ORC_E_CAPACITY;
  uint64_t wsum = 0;
  int64_t wcount = 0;
  int have_qe = 0;
  while (rc == ORC_OK) {
    if (g->n < 2) { rc = ORC_E_STATE; break; }
    const int32_t m = orc_schedule_m(g->n, s->m_cap, s->fixed_m);
    for (int32_t j = 0; j < m; ++j) {
      const uint64_t z = orc_splitmix64(s->seed, (uint64_t)(r->signals + j + 1));
      const int64_t i = (int64_t)(((z >> 32) * (uint64_t)n_points) >> 32);
      sig[j] = cloud[i];
      sig[m + j] = cloud[n_points + i];
      sig[2 * (size_t)m + j] = cloud[2 * n_points + i];
    }
    if ((rc = orc_find_winners(g, sig, m, w, sc, d1, d2, threads)) != ORC_OK) break;
    if ((rc = orc_resolve_conflicts(g, m, w, sc, d1, acc)) != ORC_OK) break;
    if ((rc = orc_adapt(g, sig, m, w, sc, d1, acc)) != ORC_OK) break;
    if ((rc = orc_update_edges(g, m, w, sc, acc)) != ORC_OK) break;
    for (int32_t j = 0; j < m; ++j) {
      wsum += qe_units(d1[j]);
      r->accepted += acc[j];
    }
    r->signals += m;
    wcount += m;
    r->iterations += 1;
    if ((rc = remove_orphans(g)) != ORC_OK) break;
    const int64_t k = s->insert_every > 0
                          ? r->signals / s->insert_every - (r->signals - m) / s->insert_every
                          : 0;
    for (int64_t i = 0; i < k && rc == ORC_OK; ++i) {
      const int32_t before = g->n;
      rc = insert_unit(g);
      if (g->n == before) break;
      r->inserted += 1;
    }
    if (rc != ORC_OK) break;
    if (wcount >= s->qe_window) {
      r->qe = (double)wsum * 0x1p-32 / (double)wcount;
      have_qe = 1;
      wsum = 0;
      wcount = 0;
      if (r->qe < (double)s->qe_threshold) {
        r->converged = 1;
        break;
      }
    }
    if (r->signals >= s->max_signals) break;
  }
  if (rc == ORC_OK && !have_qe && wcount > 0) r->qe = (double)wsum * 0x1p-32 / (double)wcount;
  r->n_units = g->n;
  r->n_edges = g->n_edges;
  free(sig); free(w); free(sc); free(d1); free(d2); free(acc);
  if (rc != ORC_OK && rc != ORC_E_STATE) g->status = rc;
  return rc;
}

/* ------------------------------------------------------------ indexed search --- */

typedef struct {
  float lo[3];     /* corner of the box */
  float h;         /* side of a cube, > 0 */
  int32_t dims[3]; /* cubes per axis, >= 1 */
} orc_grid;

static int32_t grid_axis(float p, float lo, float inv_h, int32_t dim) {
  const float t = (p - lo) * inv_h;
  if (!(t >= 0.0f)) return 0;          /* below the box (also NaN) */
  if (t >= (float)dim) return dim - 1;  /* beyond it */
  const int32_t c = (int32_t)floorf(t);
  return c < dim ? c : dim - 1;
}

/* Cell coordinates of a point (the reading in the header). */
void orc_grid_cell(const orc_grid* gr, float x, float y, float z, int32_t* c) {
  const float inv_h = 1.0f / gr->h;
  c[0] = grid_axis(x, gr->lo[0], inv_h, gr->dims[0]);
  c[1] = grid_axis(y, gr->lo[1], inv_h, gr->dims[1]);
  c[2] = grid_axis(z, gr->lo[2], inv_h, gr->dims[2]);
}

int orc_find_winners_grid(const orc_net* g, const orc_grid* gr, const float* sig, int32_t m,
                          int32_t* winner, int32_t* second, float* d1, float* d2,
                          int32_t* fell_back, int threads) {
  if (!g || !gr || m < 0 || g->n < 2) return ORC_E_INVAL;
  if (!(gr->h > 0.0f) || gr->dims[0] < 1 || gr->dims[1] < 1 || gr->dims[2] < 1)
    return ORC_E_INVAL;
  if (m > 0 && (!sig || !winner || !second || !d1 || !d2)) return ORC_E_INVAL;
  const int32_t n = g->n;
  int32_t* ucell = (int32_t*)malloc(sizeof(int32_t) * 3 * (size_t)n);
  if (!ucell) return ORC_E_CAPACITY;
  for (int32_t i = 0; i < n; ++i) orc_grid_cell(gr, g->x[i], g->y[i], g->z[i], &ucell[3 * i]);
  int32_t fb = 0;
#ifdef _OPENMP
#pragma omp parallel for schedule(dynamic, 64) num_threads(threads > 0 ? threads : 1) reduction(+ : fb)
#endif
  for (int32_t j = 0; j < m; ++j) {
    const float sx = sig[j], sy = sig[(size_t)m + j], sz = sig[2 * (size_t)m + j];
    int32_t c[3];
    orc_grid_cell(gr, sx, sy, sz, c);
    float bd = 0.0f, sd = 0.0f;
    int32_t bi = -1, si = -1, found = 0;
    for (int32_t i = 0; i < n; ++i) {
      const int32_t* u = &ucell[3 * i];
      if (abs(u[0] - c[0]) > 1 || abs(u[1] - c[1]) > 1 || abs(u[2] - c[2]) > 1) continue;
      ++found;
      const float dx = sx - g->x[i], dy = sy - g->y[i], dz = sz - g->z[i];
      const float d = (dx * dx + dy * dy) + dz * dz;
      if (bi < 0 || key_less(d, i, bd, bi)) {
        si = bi; sd = bd;
        bi = i; bd = d;
      } else if (si < 0 || key_less(d, i, sd, si)) {
        si = i; sd = d;
      }
    }
    if (found < 2) {
      /* the search failed: the exhaustive search */
      ++fb;
      bi = si = -1;
      for (int32_t i = 0; i < n; ++i) {
        const float dx = sx - g->x[i], dy = sy - g->y[i], dz = sz - g->z[i];
        const float d = (dx * dx + dy * dy) + dz * dz;
        if (bi < 0 || key_less(d, i, bd, bi)) {
          si = bi; sd = bd;
          bi = i; bd = d;
        } else if (si < 0 || key_less(d, i, sd, si)) {
          si = i; sd = d;
        }
      }
    }
    winner[j] = bi; second[j] = si; d1[j] = bd; d2[j] = sd;
  }
  free(ucell);
  if (fell_back) *fell_back = fb;
  return ORC_OK;
}
