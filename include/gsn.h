/*
 * gsn.h — C ABI of libgsn, the multi-signal growing self-organizing network iteration
 * on AMD MI355X (gfx950).
 *
 * Method: Parigi, Stramieri, Pau, Piastra, "A Multi-signal Variant for the GPU-based
 * Parallelization of Growing Self-Organizing Networks".  One iteration of the
 * multi-signal variant (Sec. 2.2) is: sample m signals (done by the caller), find the
 * winner and second-nearest unit of every signal against the same snapshot of the
 * network, then update the network for every signal, where signals whose updates would
 * collide are discarded so that one survivor per collision takes effect.
 *
 * Conventions shared by every call
 * --------------------------------
 * Memory.   Every device buffer is allocated and owned by the caller (for example as a
 *           torch tensor) and must outlive the handle.  The network state lives in one
 *           caller-provided device workspace of gsn_workspace_bytes() bytes, aligned to
 *           256 bytes.  The library allocates only the host-side handle (with a few bytes
 *           of pinned host memory in it) and, once gsn_iterate_loop is called, the HIP
 *           runtime objects that call keeps (a stream and its recorded graphs), released by
 *           gsn_destroy.
 * Layout.   Points are structure-of-arrays binary32: a buffer "SoA [3][k]" holds all k x
 *           coordinates, then all y, then all z.  Unit indices are int32 in [0, N).
 * Streams.  `stream` is a hipStream_t passed as void* (NULL = the default stream).  Calls
 *           marked "async" only enqueue work on it and return; their device outputs are
 *           valid once the stream reaches that point.  Calls marked "syncs" wait for the
 *           stream before returning.
 * Order.    Within an iteration the calls are gsn_find_winners -> gsn_resolve_conflicts
 *           -> gsn_adapt -> gsn_update_edges; gsn_grow goes between iterations.  Find and
 *           resolve may be repeated (they do not change the network); any other order
 *           returns GSN_E_STATE and enqueues nothing.
 * Errors.   Argument errors are detected on the host and returned at once, with nothing
 *           enqueued.  Errors only the device can see (a winner index out of range in a
 *           caller-supplied array, an edge or unit capacity overflow) set a sticky device
 *           status that gsn_check() returns; after such an error the network state is
 *           unspecified.  Nothing throws across the ABI and nothing is printed.
 * Results.  Every output is a deterministic function of the inputs and the state: the
 *           same on every run and for every launch configuration (see gsn_tune), and
 *           equal, element by element, to the sequential definition of each step.
 * Threads.  A handle serves one host thread at a time.
 */
#ifndef GSN_H
#define GSN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  GSN_OK = 0,
  GSN_E_INVAL = -1,     /* invalid argument (or, sticky: an invalid index on the device) */
  GSN_E_CAPACITY = -2,  /* n_max, e_max, m_max or the workspace would be exceeded */
  GSN_E_HIP = -3,       /* a HIP runtime call failed */
  GSN_E_STATE = -4      /* call out of the order stated above */
};

typedef struct gsn_net gsn_net;

/* Parameters.  Learning rates and eta follow Eq. (adaptation) of Sec. 2.1; aging follows
 * the footnote on connection aging there; err_alpha / err_beta keep the accumulated error
 * that GNG insertion uses (Sec. 2.1: periodic insertion next to the unit whose accumulated
 * squared error is largest). */
typedef struct gsn_params {
  float eps_b;       /* winner learning rate, in [0, 1] */
  float eps_n;       /* learning rate of the winner's neighbours and second, in [0, 1] */
  int32_t max_age;   /* an edge at an accepted winner whose age exceeds this is removed, >= 0 */
  float err_alpha;   /* error scale applied to q and f when a unit is inserted between them,
                        in [0, 1] */
  float err_beta;    /* error decay applied to every unit once per iteration, in [0, 1] */
  int32_t n_max;     /* unit capacity, >= 2 */
  int32_t e_max;     /* undirected edge capacity, >= 0 */
  int32_t m_max;     /* signals per iteration capacity, >= 1 */
  int32_t lock_mode; /* collision rule: GSN_LOCK_SET (0), GSN_LOCK_WINNER (1) or
                        GSN_LOCK_SET_GREEDY (2), see below */
  int32_t key_mode;  /* survivor priority: GSN_KEY_DIST_INDEX (0) or GSN_KEY_INDEX (1) */
} gsn_params;

/* Collision rules (Sec. 2.2).  The key of signal j orders the signals that collide:
 *   GSN_KEY_DIST_INDEX  key = (bits(d1[j]) << 32) | j: the signal nearest to its winner
 *                       survives, ties to the lower index;
 *   GSN_KEY_INDEX       key = j: the first signal of the batch survives, as with signals
 *                       that arrive in order.
 *   GSN_LOCK_SET        signal j locks L_j = {winner, second} + N(winner); survivors have
 *                       pairwise disjoint lock sets and update in parallel (one pass).
 *   GSN_LOCK_WINNER     the paper's rule: only the winner unit is locked, so the first
 *                       signal (smallest key) of every winner survives and the others are
 *                       discarded; the survivors then take the whole single-signal step of
 *                       Sec. 2.1 (aging, the edge to the second, adaptation, pruning) one
 *                       after another in ascending key order, each on the network its
 *                       predecessors left.  gsn_adapt performs that whole update and
 *                       gsn_update_edges does nothing.
 *   GSN_LOCK_SET_GREEDY the lock sets of GSN_LOCK_SET taken in key order: a signal is
 *                       accepted iff its lock set is disjoint from the lock sets accepted
 *                       before it (a signal whose blockers were all rejected is accepted);
 *                       the accepted sets are pairwise disjoint and the update is that of
 *                       GSN_LOCK_SET.  Resolve runs in rounds (grid-wide, then one
 *                       workgroup) and stays async. */
enum { GSN_LOCK_SET = 0, GSN_LOCK_WINNER = 1, GSN_LOCK_SET_GREEDY = 2 };
enum { GSN_KEY_DIST_INDEX = 0, GSN_KEY_INDEX = 1 };

/* Bytes of device workspace a network with these parameters needs; 0 if the parameters
 * are invalid.  Pure host computation. */
size_t gsn_workspace_bytes(const gsn_params* params);

/* Create a network of n0 units (0 <= n0 <= n_max) at init_xyz (SoA [3][n0] binary32, host
 * or device memory), with no edges and zero accumulated error.  workspace: device memory
 * of at least gsn_workspace_bytes(params) bytes, 256-byte aligned, owned by the caller and
 * used by this handle only.  The handle itself holds a few bytes of pinned host memory
 * (launch feedback of the winner-lock update).  Syncs.  On success *out holds the handle. */
int gsn_create(const gsn_params* params, void* workspace, size_t workspace_bytes, int32_t n0,
               const float* init_xyz, void* stream, gsn_net** out);

/* Find Winners (Sec. 2.1 step 2; Sec. 2.2 step 2).  For every signal j < m (sig: device
 * SoA [3][m] binary32) and every unit i < N, the squared distance
 *     d_ji = (dx*dx + dy*dy) + dz*dz,   dx = sig_x - w_x (likewise y, z),
 * each operation one binary32 rounding to nearest even, no fused multiply-add.  winner[j]
 * is the unit of smallest (d, index) in lexicographic order, second[j] the smallest among
 * the others; d1[j], d2[j] are their distances.  Outputs: device int32[m], int32[m],
 * float[m], float[m].  Requires N >= 2 and 0 <= m <= m_max (m = 0 does nothing).  Async. */
int gsn_find_winners(gsn_net* net, const float* sig, int32_t m, int32_t* winner,
                     int32_t* second, float* d1, float* d2, void* stream);

/* Indexed find winners: the hash index of the paper's "Indexed" implementation (Sec. 3.1)
 * applied to every signal of the batch.  A grid of cubes of side h covers the axis-parallel
 * box with corner lo (the box should hold the input signals); the cube of a point p is
 * c_a = floor((p_a - lo_a) * inv_h), inv_h = 1/h rounded to binary32, each operation in
 * binary32, clamped to [0, dims_a - 1].  For every signal, winner, second, d1 and d2 are
 * those of gsn_find_winners restricted to the units whose cube is within one cube of the
 * signal's on every axis (the signal's cube and its 26 neighbours); when fewer than two
 * units are there, the exhaustive search is used.  Like the paper's index this is
 * approximate: a unit outside the 27 cubes can be nearer than the second found.
 * With exact = 1 the result is instead certified: the two found are kept only when a
 * rigorous lower bound on the distance from the signal to any unit outside its 27 cubes
 * (from the signal's position in its cube, with the rounding of the cell function and of
 * the distances accounted for) exceeds the second's distance; every other signal gets the
 * exhaustive search, so the outputs equal gsn_find_winners' bit for bit.
 * grid_ws: device memory of gsn_grid_workspace_bytes() bytes (256-byte aligned, the
 * caller's, reused across calls; any contents).  Same order rules and outputs as
 * gsn_find_winners; GSN_E_INVAL for an invalid grid, GSN_E_CAPACITY for a small workspace.
 * Async. */
typedef struct gsn_grid {
  float lo[3];       /* box corner, finite */
  float h;           /* side of a cube, finite, > 0 */
  int32_t dims[3];   /* cubes per axis, >= 1, product <= GSN_MAX_GRID_CELLS */
  int32_t exact;     /* 0: the paper's index (approximate); 1: certified, exact */
} gsn_grid;
#define GSN_MAX_GRID_CELLS (1 << 24)
size_t gsn_grid_workspace_bytes(const gsn_grid* grid, int32_t n_max, int32_t m_max);
int gsn_find_winners_grid(gsn_net* net, const gsn_grid* grid, void* grid_ws,
                          size_t grid_ws_bytes, const float* sig, int32_t m, int32_t* winner,
                          int32_t* second, float* d1, float* d2, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): gsn_find_winners_grid with its grid
 * workspace taken from a fixed device array inside the library instead of grid_ws.  The
 * array is GSN_NOALLOC_SCRATCH_BYTES bytes on every GPU the library runs on and is held
 * from the library's load until the process ends; its device address is looked up once
 * per GPU (at gsn_create, else at the first call).  This call allocates nothing (no
 * hipMalloc, no event) and records no timing.  GSN_E_CAPACITY if
 * gsn_grid_workspace_bytes(grid, n_max, m_max) exceeds GSN_NOALLOC_SCRATCH_BYTES, with
 * nothing enqueued; GSN_E_HIP if the array's address cannot be found.  Every call on one
 * GPU, from any handle, uses the same array and leaves its last contents there (each call
 * clears what it needs on the stream): calls that overlap on one GPU (different streams or
 * host threads without ordering between them) race and give undefined results.  Arguments,
 * outputs, order rules and errors otherwise as gsn_find_winners_grid.  Async. */
#define GSN_NOALLOC_SCRATCH_BYTES (32u << 20)
int gsn_find_winners_grid_noalloc(gsn_net* net, const gsn_grid* grid, const float* sig,
                                  int32_t m, int32_t* winner, int32_t* second, float* d1,
                                  float* d2, void* stream);

/* Collision handling (Sec. 2.2: signals whose updates would move the same unit, change
 * the same neighbourhood or add the same edge collide; an implicit lock lets one of them
 * take effect and discards the others).  With GSN_LOCK_SET (and _GREEDY), signal j locks
 * L_j = {winner[j], second[j]} plus the current neighbours of winner[j]; with
 * GSN_LOCK_WINNER, L_j = {winner[j]}.  Keys follow key_mode.  accepted[j] = 1 iff no other
 * signal with a smaller key locks a unit of L_j (with GSN_LOCK_SET_GREEDY: no accepted
 * one), else 0.  With the lock sets, accepted lock sets are pairwise disjoint, so the
 * updates below commute.  Inputs: device arrays of length m as
 * produced by gsn_find_winners (any values with 0 <= winner, second < N and
 * winner != second; others are rejected and flag GSN_E_INVAL on the device).  Output:
 * device uint8[m].  Async. */
int gsn_resolve_conflicts(gsn_net* net, int32_t m, const int32_t* winner,
                          const int32_t* second, const float* d1, uint8_t* accepted,
                          void* stream);

/* Adaptation (Sec. 2.1 step 3, Eq. (adaptation), eta(i, b) = 1 iff i and b are
 * connected).  For every accepted j, with b = winner[j], s = second[j]:
 *     w <- w + eps * (sig_j - w)   per component as t = sig - w; t = eps * t; w = w + t,
 * with eps_b for b and eps_n for every current neighbour of b and for s (once).  The
 * winner's error grows by d1[j]; afterwards every unit's error is multiplied by err_beta.
 * Inputs as for gsn_resolve_conflicts plus sig (SoA [3][m]).  Async with GSN_LOCK_SET.
 * With GSN_LOCK_WINNER it performs, for the accepted signals in ascending key order, the
 * whole single-signal step: every edge at b ages by one, {b, s} is set to age 0 (created if
 * absent), b, its neighbours before that step and s (once) move as above, the edges at b
 * older than max_age are removed (a unit left with no edge is marked for gsn_grow) and
 * err[b] grows by d1[j]; then err *= err_beta.  Any accepted set is valid (signals sharing
 * a winner are applied in key order too); more than e_max edges at the end set
 * GSN_E_CAPACITY on the device.  It runs in rounds (every pending signal whose units
 * {b, s} + N(b) no pending signal of smaller key touches goes in the same round); the
 * first rounds are grid-wide launches (GSN_TUNE_GRID_ROUNDS), the rest run inside one
 * workgroup, so the call stays async. */
int gsn_adapt(gsn_net* net, const float* sig, int32_t m, const int32_t* winner,
              const int32_t* second, const float* d1, const uint8_t* accepted, void* stream);

/* Connection update (Sec. 2.1 step 3 and its footnote on aging); with GSN_LOCK_WINNER
 * gsn_adapt has done it and this call only ends the iteration.  For every accepted j:
 * every edge at b = winner[j] ages by one, the edge {b, second[j]} is set to age 0 (and
 * created if absent), then the edges at b older than max_age are removed; a unit left
 * with no edge by such a removal is marked for removal by gsn_grow.  The adjacency is then
 * rewritten as a compacted CSR with rows in ascending neighbour order.  Exceeding e_max
 * sets GSN_E_CAPACITY on the device.  Async. */
int gsn_update_edges(gsn_net* net, int32_t m, const int32_t* winner, const int32_t* second,
                     const uint8_t* accepted, void* stream);

/* One whole iteration (Sec. 2.2: find winners, resolve, adapt, update edges) in one call:
 * the outputs and the state afterwards are those of the four calls above in order (same
 * order rules: it starts like gsn_find_winners and leaves the handle ready for gsn_grow).
 * With GSN_LOCK_SET the update runs fused: the find's merge makes the claims, resolve's
 * check applies each accepted signal's adaptation and edge marks at once (accepted lock
 * sets are disjoint), and one rewrite of the adjacency applies the error decay: two update
 * launches after the find instead of six.  With GSN_LOCK_WINNER the resolve leaves at most
 * one survivor per winner unit, so each edge changes only in the steps of its two ends'
 * survivors: the update of gsn_adapt is computed per unit in one pass instead of rounds
 * (its moves applied in key order, its edges after the two steps that can change each,
 * its removal mark), in two launches after the resolve, with the same result.
 * With GSN_LOCK_SET_GREEDY the resolve runs its rounds and the fused update of GSN_LOCK_SET
 * applies the accepted signals (disjoint lock sets) without claims or check.  Outputs:
 * device arrays of length m.  Async. */
int gsn_iterate(gsn_net* net, const float* sig, int32_t m, int32_t* winner, int32_t* second,
                float* d1, float* d2, uint8_t* accepted, void* stream);

/* The update of gsn_iterate (resolve, adapt and edges, fused as there) after any find: its
 * outputs and the state afterwards are those of gsn_resolve_conflicts, gsn_adapt and
 * gsn_update_edges called in order on the same arguments, so it serves the hash index
 * (gsn_find_winners_grid) as well as the exhaustive search.  Call it after a find
 * (GSN_E_STATE otherwise); it leaves the handle ready for gsn_grow.  Inputs as for
 * gsn_adapt; output accepted (device uint8[m]).  Async. */
int gsn_update(gsn_net* net, const float* sig, int32_t m, const int32_t* winner,
               const int32_t* second, const float* d1, uint8_t* accepted, void* stream);

/* count whole iterations (Sec. 2.2, the multi-signal loop) in one call: the result, the
 * state afterwards and the outputs (those of the last iteration) are exactly those of count
 * gsn_iterate calls in order over the batches sigs + 3 m k, k = 0 .. count - 1 (each batch
 * laid out as gsn_iterate's sig; device memory, count x 3 x m floats, read by the device
 * when the iterations run).  The launches of the whole loop are recorded once into a HIP
 * graph and replayed: a later call with the same arguments and network state (unit count,
 * tuning, which internal buffer set is current) replays the recorded graph without any
 * per-launch host work, on the caller's stream.  Up to GSN_GRAPH_CACHE graphs are kept per
 * handle (the least recently used one is replaced); GSN_STAT_LOOP_RECORDS counts the calls
 * that recorded one.  A graph reads the batches and writes the outputs at the addresses
 * given, when it runs; it uses no buffer beyond the handle's workspace.  The only
 * difference from the separate calls: the spatial unit order of the staged find is rebuilt
 * at the first iteration when the rebuild would fall inside the loop, never later in it
 * (the order affects speed only).  The event timers (gsn_timing_enable) do not record
 * inside the loop.  count is 1 .. GSN_MAX_LOOP.  Errors as gsn_iterate (checked on the
 * host before anything is recorded).  Async. */
#define GSN_MAX_LOOP 4096
#define GSN_GRAPH_CACHE 4
int gsn_iterate_loop(gsn_net* net, const float* sigs, int32_t m, int32_t count,
                     int32_t* winner, int32_t* second, float* d1, float* d2,
                     uint8_t* accepted, void* stream);

/* Growth (Sec. 2.1: units may be added and removed during the update; GNG inserts next
 * to the unit of largest accumulated error).  First removes, by stable
 * compaction (indices shift down, edges are renumbered), every unit marked by
 * gsn_update_edges that still has no edge.  Then, if insert_every > 0, iteration > 0,
 * iteration % insert_every == 0 and N < n_max: q = argmax error, f = argmax error over the
 * neighbours of q (ties to the lower index; nothing happens if q has none); a unit r = N
 * is added at (w_q + w_f) * 0.5, the edge {q, f} is replaced by {q, r} and {r, f} at age
 * 0, err_q and err_f are multiplied by err_alpha and err_r = err_q.  Syncs. */
int gsn_grow(gsn_net* net, int32_t iteration, int32_t insert_every, void* stream);

/* Growing-network schedule: whole iterations the way the paper's runs drive them (Sec.
 * 3.1: the level of parallelism m of every iteration is the smallest power of two greater
 * than the current N, capped at m_cap, the paper's cap being 8192; Sec. 2.1: GNG insertion
 * at regular intervals, stop on a threshold on the quantization error, the mean squared
 * distance between signals and their winners).  Per iteration, on the device: draw m
 * signals from the cloud, find winners, resolve, adapt, update edges (the handle's collision
 * rule), add the winners' squared distances to the error window, remove orphaned units, and
 * insert k units one after another (GNG rule of gsn_grow), where k is the number of
 * multiples of insert_every passed by the signal count in this iteration.  Then, once the
 * window holds at least qe_window signals, its mean is tested against qe_threshold and the
 * window restarts; the run also stops once max_signals signals were drawn.
 * Signals: the c-th signal of the run (c = 1, 2, ...) is cloud point
 * ((z >> 32) * n_points) >> 32 with z = SplitMix64 output c of `seed` (the mix of
 * seed + c * 0x9E3779B97F4A7C15, Steele, Lea and Flood, 2014).  The error window counts
 * each d1 as the integer floor(d1 * 2^32) (2^44 from d1 >= 4096 on, also for inf and NaN),
 * so its sum is exact in any order; its mean is (double)sum * 2^-32 / (double)count. */
typedef struct gsn_schedule {
  int32_t m_cap;          /* largest m, 1..m_max */
  int32_t fixed_m;        /* 0: the power-of-two rule; > 0 (<= m_max): this m every iteration */
  int64_t insert_every;   /* signals between two insertions, >= 0 (0: no insertion) */
  int64_t qe_window;      /* signals per stop test, >= 1; qe_window + largest m <= 2^19 */
  int64_t max_signals;    /* >= 1 */
  float qe_threshold;     /* stop at the first window whose mean is below it */
  uint64_t seed;
} gsn_schedule;

typedef struct gsn_schedule_result {
  int64_t iterations, signals, accepted, inserted;
  double qe;              /* mean of the last complete window (of the partial one if none) */
  int32_t converged;      /* 1 if the run stopped on the threshold */
  int32_t n_units;
  int64_t n_edges;
} gsn_schedule_result;

/* Runs the schedule from the current network (N >= 2) on cloud (device SoA [3][n_points]
 * binary32, 1 <= n_points < 2^32), continuing the handle's state; the per-iteration buffers
 * are in the workspace.  Must be called between iterations (GSN_E_STATE otherwise, or if N
 * falls below 2).  Syncs (every iteration: growth reads the unit count). */
int gsn_run_schedule(gsn_net* net, const float* cloud, int64_t n_points,
                     const gsn_schedule* schedule, gsn_schedule_result* result, void* stream);

/* Current unit count N and undirected edge count.  Syncs. */
int gsn_sizes(gsn_net* net, int32_t* n_units, int32_t* n_edges, void* stream);

/* Copy the state out (any pointer may be NULL; host or device memory): xyz SoA [3][N],
 * err [N], edges SoA [3][E] = (u, v, age) with u < v in ascending (u, v) order.  Sizes
 * from gsn_sizes.  Syncs. */
int gsn_export(gsn_net* net, float* xyz, float* err, int32_t* edges, void* stream);

/* Replace the state: n units at xyz (SoA [3][n]), errors err (NULL = zeros), and n_edges
 * edges (SoA [3][n_edges] = (u, v, age), any order, u != v, no duplicates, age >= 0).  Host
 * or device memory.  Clears the removal marks and any sticky error.  Syncs. */
int gsn_import(gsn_net* net, int32_t n, const float* xyz, const float* err, int32_t n_edges,
               const int32_t* edges, void* stream);

/* Sticky device status: GSN_OK, or the first GSN_E_INVAL / GSN_E_CAPACITY a kernel
 * raised since creation or the last gsn_import (GSN_E_STATE if the winner-lock update
 * found its lock words not cleared, which only a corrupted workspace causes).  Syncs. */
int gsn_check(gsn_net* net, void* stream);

/* Free the host handle (the workspace stays the caller's).  NULL is ignored. */
void gsn_destroy(gsn_net* net);

/* Launch-configuration knobs, for tests and measurement; results never depend on them.
 *   GSN_TUNE_SPLIT    units are split into this many chunks scanned by separate
 *                     workgroups and merged afterwards (0 = automatic, 1..GSN_MAX_SPLIT)
 *   GSN_TUNE_VARIANT  find-winners kernel: 0 = automatic (4), 1 = direct scan of every
 *                     distance, 2 = screened scan with the screen on the vector unit,
 *                     3 = screened scan with the screen on the matrix cores in binary32,
 *                     4 = the same screen on the matrix cores in split binary16, 5 = variant
 *                     4 with the unit batches dealt out dynamically (every wave takes
 *                     GSN_TUNE_GRAB batches at a time with an atomic counter) (every screen
 *                     carries a rigorous rounding margin; candidates are rechecked in the
 *                     binary32 direct form, so all variants return the same result)
 *   GSN_TUNE_GRAB     batches of 64 units per atomic grab of variant 5: 1..1024, 0 = default
 *   GSN_TUNE_REBUCKET staged find calls (variants 2-5) between rebuilds of the spatial order
 *                     of the units (it is also rebuilt whenever N or the indices change):
 *                     1..4096, 0 = default (64)
 *   GSN_TUNE_GRID_ROUNDS  rounds of the GSN_LOCK_WINNER update of gsn_adapt and of the
 *                     GSN_LOCK_SET_GREEDY resolve launched over the whole device (each
 *                     skipped once fewer than 32 signals are pending) before the remaining
 *                     ones run in a single workgroup: 1..32, or 0 = automatic (winner lock:
 *                     u + u / 4 with u one more than the rounds the previous update could
 *                     have used grid-wide, i.e. the rounds that started with 32 or more
 *                     pending, from a pinned host copy of that count; greedy resolve: 4)
 * Returns GSN_E_INVAL for an unknown key or value. */
enum { GSN_TUNE_SPLIT = 1, GSN_TUNE_VARIANT = 2, GSN_TUNE_GRID_ROUNDS = 3, GSN_TUNE_GRAB = 4,
       GSN_TUNE_REBUCKET = 5 };
#define GSN_MAX_SPLIT 64
int gsn_tune(gsn_net* net, int32_t key, int32_t value);

/* Kernel timing with HIP events recorded on the caller's stream around each step, for
 * measurement.  gsn_timing_enable(net, 1) starts recording; gsn_timing_read returns the
 * summed duration in milliseconds and the number of launches recorded for one step since
 * the last read, and clears them (syncs).  The events are made without the system-scope
 * memory fence (hipEventDisableSystemFence): they time the work, they publish nothing to
 * the host, and recording them does not stall the stream.
 *   GSN_T_FIND_SCAN   the find-winners scan kernel alone.  For the staged scans (variants
 *                     2-5) the pair is bound to the kernel's launch (hipExtLaunchKernel): it
 *                     spans the kernel's own start to end (not the end-of-kernel cache
 *                     flush) and puts no marker on the stream, but costs the host tens of
 *                     microseconds per launch; the unstaged scans (variants 1 and 6, small
 *                     batches, whose steps are bound by launches) take a marker pair
 *   GSN_T_FIND        all of gsn_find_winners
 *   GSN_T_RESOLVE, GSN_T_ADAPT, GSN_T_EDGES   all of the corresponding call
 *   GSN_T_UPDATE      the fused update of gsn_iterate (with GSN_LOCK_SET resolve, adapt
 *                     and edges; with the other rules adapt and edges, the resolve being
 *                     timed as GSN_T_RESOLVE) */
enum { GSN_T_FIND_SCAN = 0, GSN_T_FIND = 1, GSN_T_RESOLVE = 2, GSN_T_ADAPT = 3,
       GSN_T_EDGES = 4, GSN_T_UPDATE = 5, GSN_T_COUNT = 6 };
int gsn_timing_enable(gsn_net* net, int32_t enable);
int gsn_timing_read(gsn_net* net, int32_t which, double* total_ms, int32_t* launches);
/* Restricts the timers that record while timing is enabled to the bits set in mask (bit w
 * for GSN_T_w; all of them after gsn_create), so that a measurement can time one kernel
 * with a single event pair per call.  GSN_E_INVAL for bits beyond GSN_T_COUNT. */
int gsn_timing_select(gsn_net* net, uint32_t mask);

/* Statistics accumulated on the device since creation or the last GSN_STAT_CLEAR, for
 * measurement.  Syncs.
 *   GSN_STAT_ROUNDS      rounds summed over the GSN_LOCK_WINNER updates (a round applies
 *                        every pending survivor whose units no pending survivor of smaller
 *                        key touches)
 *   GSN_STAT_ROUNDS_MAX  the most rounds one such update took
 *   GSN_STAT_UPDATES     gsn_adapt calls that applied the winner-lock update in rounds
 *                        (gsn_iterate takes it in one pass and counts no rounds)
 *   GSN_STAT_CLEAR       sets every statistic to zero (value may be NULL)
 *   GSN_STAT_RESOLVED    signals that went through gsn_resolve_conflicts
 *   GSN_STAT_ACCEPTED    of those, the accepted ones
 *   GSN_STAT_LOOP_RECORDS  gsn_iterate_loop calls that recorded a graph (the others
 *                        replayed one); a host count, the stream is not used */
enum { GSN_STAT_ROUNDS = 0, GSN_STAT_ROUNDS_MAX = 1, GSN_STAT_UPDATES = 2,
       GSN_STAT_CLEAR = 3, GSN_STAT_RESOLVED = 4, GSN_STAT_ACCEPTED = 5,
       GSN_STAT_LOOP_RECORDS = 6 };
int gsn_stat(gsn_net* net, int32_t key, int64_t* value, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* GSN_H */
