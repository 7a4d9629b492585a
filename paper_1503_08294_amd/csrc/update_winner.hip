// The paper's collision rule (Sec. 2.2) on the device: the winner unit alone is locked, the
// first signal of every winner survives, and the survivors take the whole single-signal
// step of Sec. 2.1 one after another in ascending key order.
//
// A survivor j touches the units F_j = {b_j, s_j} + N(b_j) of the network its predecessors
// left: it moves them, and rewrites the rows of b_j, s_j and the neighbours of b_j.  The
// update runs in rounds.  In a round every pending survivor claims F_j with a 64-bit atomic
// minimum of its key; the ones that hold all of F_j apply their step in parallel, on
// disjoint units and rows.  A survivor that goes in a round precedes in key order every
// pending survivor whose F it meets, because those claimed the shared unit with a larger
// key, so the per-unit order of the updates is the key order.  A survivor that goes ahead
// of a smaller-key survivor i it does not meet keeps not meeting it: F_i changes only when
// an edge is inserted at b_i by a survivor that meets F_i, which is also pending and
// precedes i, and such an insertion puts into F_i a winner that the faster survivor would
// have met in the round it went.  The pending survivor of smallest key is always ready,
// so every round makes progress.
//
// The rows are edited in place: before the rounds the CSR is copied with room for every
// insertion the survivors can make (one per survivor at its winner and one at its second),
// and afterwards compacted back, so no round rewrites the adjacency.  The first rounds,
// which hold most of the survivors, are grid-wide launches; the few survivors left then go
// through the remaining rounds inside one workgroup, so that the whole update is enqueued
// without the host waiting to learn how many rounds it takes.
#include "gsn_internal.h"

namespace gsn {
namespace {

inline int blocks(int64_t n) { return static_cast<int>((n + kBlock - 1) / kBlock); }

// Position of v in the ascending slice col[r0, r1), or -1.
__device__ __forceinline__ int32_t slice_find(const int32_t* __restrict__ col, int32_t r0,
                                              int32_t r1, int32_t v) {
  while (r0 < r1) {
    const int32_t mid = (r0 + r1) >> 1;
    const int32_t c = col[mid];
    if (c == v) return mid;
    if (c < v) r0 = mid + 1; else r1 = mid;
  }
  return -1;
}

// Insert v (age a) into the ascending row of u; false if the row has no room left.
__device__ bool row_insert(const int32_t* __restrict__ rp, int32_t* __restrict__ len,
                           int32_t* __restrict__ col, int32_t* __restrict__ age, int32_t u,
                           int32_t v, int32_t a) {
  const int32_t r0 = rp[u], l = len[u];
  if (r0 + l >= rp[u + 1]) return false;
  int32_t k = r0 + l;
  while (k > r0 && col[k - 1] > v) {
    col[k] = col[k - 1];
    age[k] = age[k - 1];
    --k;
  }
  col[k] = v;
  age[k] = a;
  len[u] = l + 1;
  return true;
}

// Position of v in the ascending slice col[r0, r0 + l), or -1: rows of up to 8 entries
// (nearly all of them) are read in one batch of loads rather than by a binary search.
__device__ __forceinline__ int32_t row_find(const int32_t* __restrict__ col, int32_t r0,
                                            int32_t l, int32_t v) {
  if (l > 8) return slice_find(col, r0, r0 + l, v);
  if (l <= 0) return -1;
  // every load in the row (slots past its end repeat the last entry), so none waits on a
  // bounds test
  int32_t c[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) c[k] = col[r0 + min(k, l - 1)];
  int32_t at = -1;
#pragma unroll
  for (int k = 7; k >= 0; --k)
    if (k < l && c[k] == v) at = r0 + k;
  return at;
}

// Remove v from the row of u if present; returns the new length.
__device__ int32_t row_remove(const int32_t* __restrict__ rp, int32_t* __restrict__ len,
                              int32_t* __restrict__ col, int32_t* __restrict__ age, int32_t u,
                              int32_t v) {
  const int32_t r0 = rp[u], l = len[u];
  const int32_t k = row_find(col, r0, l, v);
  if (k < 0) return l;
  for (int32_t q = k; q + 1 < r0 + l; ++q) {
    col[q] = col[q + 1];
    age[q] = age[q + 1];
  }
  len[u] = l - 1;
  return l - 1;
}

// ----------------------------------------------------------------- prologue ----

// Survivors (pend = 1), the insertions each row may receive, the survivor count, and the
// claims of the first round, made on the compact rows (the slack copy holds the same rows).
__global__ void wl_prepare(int32_t m, int32_t n, const int32_t* __restrict__ winner,
                           const int32_t* __restrict__ second, const float* __restrict__ d1,
                           const uint8_t* __restrict__ accepted, int key_mode,
                           const int32_t* __restrict__ rp, const int32_t* __restrict__ col,
                           unsigned long long* __restrict__ lock, uint8_t* __restrict__ pend,
                           int32_t* __restrict__ extra, int32_t* __restrict__ rem,
                           int32_t* __restrict__ status) {
  __shared__ int32_t s_ok;
  if (threadIdx.x == 0) s_ok = 0;
  __syncthreads();
  const int32_t j = blockIdx.x * kBlock + threadIdx.x;
  if (blockIdx.x == 0) spread_clear(rem + rm_round(0), threadIdx.x);
  bool ok = false;
  if (j < m) {
    const bool a = accepted[j] != 0;
    const int32_t b = winner[j], s = second[j];
    ok = a && pair_ok(b, s, n);
    if (a && !ok) raise_error(status, GSN_E_INVAL);
    pend[j] = ok ? 1 : 0;
    if (ok) {
      atomicAdd(&extra[b], 1);
      atomicAdd(&extra[s], 1);
      const unsigned long long key = signal_key(d1[j], j, key_mode);
      atomicMin(&lock[b], key);
      atomicMin(&lock[s], key);
      const int32_t r0 = rp[b];
      claim_row(lock, col, r0, rp[b + 1] - r0, key);
    }
  }
  block_count_spread(ok, rem + kRmSurvivors, &s_ok);
}

// Row sizes for a rewrite: the live length (len, or the CSR row length when len is null)
// plus the room asked in extra (when not null; it is cleared), and per-block sums.  Also
// sets the lock words to all ones when lock is not null (they are all ones after a
// complete update already; this keeps them so after an update that stopped on an error).
__global__ void wl_count(int32_t n, const int32_t* __restrict__ rp,
                         const int32_t* __restrict__ len, int32_t* __restrict__ extra,
                         unsigned long long* __restrict__ lock, int32_t* __restrict__ cnt,
                         int32_t* __restrict__ bsum) {
  __shared__ int32_t red[kBlock];
  const int32_t u = blockIdx.x * kBlock + threadIdx.x;
  int32_t c = 0;
  if (u < n) {
    if (lock) lock[u] = ~0ull;
    c = len ? len[u] : rp[u + 1] - rp[u];
    if (extra) {
      c += extra[u];
      extra[u] = 0;
    }
    cnt[u] = c;
  }
  red[threadIdx.x] = c;
  __syncthreads();
  for (int w = kBlock / 2; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) bsum[blockIdx.x] = red[0];
}

// Copies every row (len[u] entries, or the CSR row when len is null) to the offsets given
// by the block-local scan of cnt plus the block offsets; dst_len (if not null) receives the
// copied length; err (if not null) is multiplied by beta on the way.  Rows stay ascending.
// With fold the block offsets and the capacity check come from the raw block sums
// (fold_offsets, fold_abort); otherwise bsum holds the scanned offsets.
__global__ void wl_write(int32_t n, const int32_t* __restrict__ rp,
                         const int32_t* __restrict__ len, const int32_t* __restrict__ col,
                         const int32_t* __restrict__ age, const int32_t* __restrict__ cnt,
                         const int32_t* __restrict__ bsum, int32_t* __restrict__ dst_rp,
                         int32_t* __restrict__ dst_col, int32_t* __restrict__ dst_age,
                         int32_t* __restrict__ dst_len, float* __restrict__ err, float beta,
                         int32_t* __restrict__ status, int fold, int32_t nb, int64_t cap,
                         int32_t* __restrict__ out_total) {
  __shared__ int32_t sc[kBlock];
  __shared__ int32_t red[2 * kBlock / 64];
  const int32_t u = blockIdx.x * kBlock + threadIdx.x;
  const int32_t c = u < n ? cnt[u] : 0;
  int32_t boff, abort;
  if (fold) {
    int32_t total;
    fold_offsets(bsum, nb, red, &boff, &total);
    abort = fold_abort(total, cap, status, out_total);
  } else {
    boff = bsum[blockIdx.x];
    abort = status[kStAbort];
  }
  sc[threadIdx.x] = c;
  __syncthreads();
  for (int off = 1; off < kBlock; off <<= 1) {
    const int32_t v = threadIdx.x >= off ? sc[threadIdx.x - off] : 0;
    __syncthreads();
    sc[threadIdx.x] += v;
    __syncthreads();
  }
  if (u >= n) return;
  if (err) err[u] = err[u] * beta;
  if (abort) {
    // the rewrite did not fit: leave a valid, empty adjacency (the state is flagged invalid)
    dst_rp[u] = 0;
    if (dst_len) dst_len[u] = 0;
    return;
  }
  const int32_t start = boff + sc[threadIdx.x] - c;
  const int32_t r0 = rp[u];
  const int32_t l = len ? len[u] : rp[u + 1] - r0;
  dst_rp[u] = start;
  if (dst_len) dst_len[u] = l;
  for (int32_t k = 0; k < l; ++k) {
    dst_col[start + k] = col[r0 + k];
    dst_age[start + k] = age[r0 + k];
  }
}

// ------------------------------------------------------------------- rounds ----

constexpr int kRoundBlock = 64;    // threads per workgroup of the grid-wide claims
constexpr int kStepBlock = 256;    // threads per workgroup of the grid-wide steps
constexpr int kTailBlock = 1024;   // threads of the single workgroup of the last rounds

// The lock words are read and released with agent-scope atomics (at L2): the grid-wide
// rounds of several workgroups and the claims (atomic minima) meet there.  The last rounds
// run in one workgroup whose phases are separated by barriers, not by kernel ends; the
// barrier's workgroup-scope ordering covers the rows and flags its waves share.
// Lock words during the rounds.  In the single-workgroup rounds, claims and checks share one
// launch, so the checks read the words atomically (the claims' minima are made at device
// scope).  A grid-wide step reads words that the claims of an earlier launch left (kernel
// boundaries make those visible to plain loads) and writes only releases (all ones), so
// plain loads and stores serve there: a stale or released word reads as some other key or
// all ones, never as the reader's own key unless it held the unit at the end of the
// claims, so a stale read can only make a survivor wait a round.
template <bool kGrid>
__device__ __forceinline__ unsigned long long lock_read(unsigned long long* p) {
  if constexpr (kGrid) return *p;
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <bool kGrid>
__device__ __forceinline__ void lock_release(unsigned long long* p) {
  if constexpr (kGrid) *p = ~0ull;
  else __hip_atomic_store(p, ~0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

struct RoundArgs {
  const float* sig;
  int32_t m;
  const int32_t* winner;
  const int32_t* second;
  const float* d1;
  int key_mode;
  uint8_t* pend;
  const int32_t* rp;
  int32_t* len;
  int32_t* col;
  int32_t* age;
  unsigned long long* lock;
  float *x, *y, *z, *err;
  int32_t* orphan;
  int32_t* status;
  float eps_b, eps_n;
  int32_t max_age;
  int32_t* rem;
  int32_t* list;
  int32_t* feedback;  // pinned host word for the grid rounds used, or null
};

// Claim F_j = {b, s} + N(b) with the key of j.
__device__ void claim(const RoundArgs& a, int32_t j) {
  const int32_t b = a.winner[j], s = a.second[j];
  const unsigned long long key = signal_key(a.d1[j], j, a.key_mode);
  atomicMin(&a.lock[b], key);
  atomicMin(&a.lock[s], key);
  claim_row(a.lock, a.col, a.rp[b], a.len[b], key);
}

__device__ void apply(const RoundArgs& a, int32_t j);

// Applies the step of j if j holds every unit of F_j; returns whether it did.  The winner
// is checked first, and the row of b_j is read only if j holds b_j: a survivor that goes in
// this round edits the rows of its own units only, so the row of a unit that j holds stays
// as claimed.  A survivor that goes releases its units before its step (the others compare
// with their own keys, which differ from the holder's and from all ones in the index half).
// A signal that does not go keeps what it holds: those units stay in its F, because F_j
// loses only winners of survivors that go, which j does not hold, so it claims them again
// with the same key in the next round, and releases them when it goes.
template <bool kGrid>
__device__ bool try_apply(const RoundArgs& a, int32_t j) {
  const int32_t b = a.winner[j], s = a.second[j];
  const unsigned long long key = signal_key(a.d1[j], j, a.key_mode);
  if (lock_read<kGrid>(&a.lock[b]) != key) return false;
  bool ok = lock_read<kGrid>(&a.lock[s]) == key;
  const int32_t r0 = a.rp[b], r1 = r0 + a.len[b];
  for (int32_t k = r0; ok && k < r1; ++k) ok = lock_read<kGrid>(&a.lock[a.col[k]]) == key;
  if (!ok) return false;
  lock_release<kGrid>(&a.lock[b]);
  lock_release<kGrid>(&a.lock[s]);
  for (int32_t k = r0; k < r1; ++k) lock_release<kGrid>(&a.lock[a.col[k]]);
  apply(a, j);
  return true;
}

// The single-signal step of j on the current network.
__device__ void apply(const RoundArgs& a, int32_t j) {
  const int32_t b = a.winner[j], s = a.second[j];
  const int32_t m = a.m;
  const float sx = a.sig[j], sy = a.sig[m + j], sz = a.sig[2 * m + j];
  const int32_t* rp = a.rp;
  int32_t* len = a.len;
  int32_t* col = a.col;
  int32_t* age = a.age;
  const int32_t r0 = rp[b];
  int32_t l = len[b];
  // adaptation: the winner, its neighbours before this step, and the second once
  move_unit(a.x, a.y, a.z, b, a.eps_b, sx, sy, sz);
  bool s_nb = false;
  for (int32_t k = r0; k < r0 + l; ++k) {
    const int32_t v = col[k];
    s_nb |= v == s;
    move_unit(a.x, a.y, a.z, v, a.eps_n, sx, sy, sz);
  }
  if (!s_nb) move_unit(a.x, a.y, a.z, s, a.eps_n, sx, sy, sz);
  // aging of the edges at b, the edge {b, s} at age 0
  for (int32_t k = r0; k < r0 + l; ++k) {
    const int32_t v = col[k];
    const int32_t g = v == s ? 0 : age[k] + 1;
    age[k] = g;
    const int32_t rk = slice_find(col, rp[v], rp[v] + len[v], b);
    if (rk >= 0) age[rk] = g;
  }
  if (!s_nb) {
    if (!row_insert(rp, len, col, age, b, s, 0) || !row_insert(rp, len, col, age, s, b, 0))
      raise_error(a.status, GSN_E_CAPACITY);
  }
  // removal of the edges at b older than max_age
  l = len[b];
  int32_t w = r0;
  for (int32_t k = r0; k < r0 + l; ++k) {
    const int32_t v = col[k];
    const int32_t g = age[k];
    if (g > a.max_age) {
      if (row_remove(rp, len, col, age, v, b) == 0 && !a.orphan[v]) {
        a.orphan[v] = 1;
        atomicAdd(&a.status[kStOrphans], 1);
      }
    } else {
      col[w] = v;
      age[w] = g;
      ++w;
    }
  }
  len[b] = w - r0;
  a.err[b] = a.err[b] + a.d1[j];
}

// Grid-wide round t: rem[t] counts the signals left pending; a round after one that left
// fewer than kTailMin returns at once (the single-workgroup rounds take them), and so do
// the later ones (their counts stay zero).
__global__ void wl_claim(RoundArgs a, int32_t t) {
  if (blockIdx.x == 0) spread_clear(a.rem + rm_round(t), threadIdx.x);
  if (t > 0 && spread_value(a.rem + rm_round(t - 1)) < kTailMin) return;
  const int32_t j = blockIdx.x * kRoundBlock + threadIdx.x;
  if (j < a.m && a.pend[j] == 1) claim(a, j);
}

// The same with a group of kGroup lanes of one wave per signal: lane q takes the q-th
// neighbour of b (ownership, release, its move, the mirror age or its removal), and the
// row of b is rebuilt from ballots over the group.  Rows longer than kGroup go through
// try_apply on the group's first lane, a chain of dependent loads that holds up the whole
// round, so the group is wide enough for nearly every row (16 lanes: the winner rule's
// update took 0.25 instead of 0.32 ms at 16,384 signals with 8).  Every lane of the group
// calls it with the same j; the result is the same on all of them.
constexpr int kGroup = 16;
static_assert(kGroup < 32, "group masks are 32-bit");

__device__ __forceinline__ uint32_t group_bits(unsigned long long wave_mask) {
  const int base = static_cast<int>(threadIdx.x & 63) & ~(kGroup - 1);
  return static_cast<uint32_t>(wave_mask >> base) & ((1u << kGroup) - 1);
}

template <bool kGrid>
__device__ bool group_try_apply(const RoundArgs& a, int32_t j, int q) {
  const int32_t b = a.winner[j], s = a.second[j];
  const float dj = a.d1[j];
  const int32_t m = a.m;
  const float sx = a.sig[j], sy = a.sig[m + j], sz = a.sig[2 * m + j];
  // the loads above are issued together before any of them is waited for
  __builtin_amdgcn_sched_barrier(0);
  const unsigned long long key = signal_key(dj, j, a.key_mode);
  // The row bounds of b are read with its lock word, and what the step reads (positions,
  // error, row bounds of the neighbours) beside the lock words rather than after them:
  // they are used only if j holds F_j, and then nobody else edits those units or rows
  // during the round; otherwise they are dropped.
  const int32_t r0 = a.rp[b], l = a.len[b];
  const unsigned long long lb = lock_read<kGrid>(&a.lock[b]);
  unsigned long long ls = 0;
  int32_t r1b = 0;
  float bx = 0.0f, by = 0.0f, bz = 0.0f, be = 0.0f, tx = 0.0f, ty = 0.0f, tz = 0.0f;
  if (q == 0) {
    ls = lock_read<kGrid>(&a.lock[s]);
    r1b = a.rp[b + 1];
    bx = a.x[b]; by = a.y[b]; bz = a.z[b];
    be = a.err[b];
    tx = a.x[s]; ty = a.y[s]; tz = a.z[s];
  }
  if (lb != key) return false;
  if (l > kGroup) {
    int applied = 0;
    if (q == 0) applied = try_apply<kGrid>(a, j);
    return __shfl(applied, static_cast<int>(threadIdx.x & 63) & ~(kGroup - 1)) != 0;
  }
  const bool has = q < l;
  int32_t v = -1, a_old = 0, vr = 0, vl = 0;
  unsigned long long lv = key;
  float vx = 0.0f, vy = 0.0f, vz = 0.0f;
  if (has) {
    v = a.col[r0 + q];
    a_old = a.age[r0 + q];
    lv = lock_read<kGrid>(&a.lock[v]);
    vx = a.x[v]; vy = a.y[v]; vz = a.z[v];
    vr = a.rp[v];
    vl = a.len[v];
  }
  bool mine = lv == key;
  if (q == 0) mine = mine && ls == key;
  if (group_bits(__ballot(!mine)) != 0) return false;
  // j holds F_j: release it, then the step
  if (has) lock_release<kGrid>(&a.lock[v]);
  if (q == 0) {
    lock_release<kGrid>(&a.lock[b]);
    lock_release<kGrid>(&a.lock[s]);
  }
  // move_unit's expression on positions already loaded
  auto move = [&](int32_t u, float eps, float px, float py, float pz) {
    float t;
    t = sx - px; t = eps * t; a.x[u] = px + t;
    t = sy - py; t = eps * t; a.y[u] = py + t;
    t = sz - pz; t = eps * t; a.z[u] = pz + t;
  };
  const bool is_s = has && v == s;
  const bool new_s = group_bits(__ballot(is_s)) == 0;
  if (q == 0) {
    move(b, a.eps_b, bx, by, bz);
    if (new_s) move(s, a.eps_n, tx, ty, tz);
  }
  if (has) move(v, a.eps_n, vx, vy, vz);
  const int32_t g = is_s ? 0 : a_old + 1;
  const bool keep = has && g <= a.max_age;
  if (keep) {
    const int32_t rk = row_find(a.col, vr, vl, b);
    if (rk >= 0) a.age[rk] = g;
  } else if (has) {
    if (row_remove(a.rp, a.len, a.col, a.age, v, b) == 0 && !a.orphan[v]) {
      a.orphan[v] = 1;
      atomicAdd(&a.status[kStOrphans], 1);
    }
  }
  // the row of b: kept entries in order, with s at its place if the edge is new
  const uint32_t kept_mask = group_bits(__ballot(keep));
  const uint32_t below_s = group_bits(__ballot(keep && v < s));
  const int32_t kept = __popc(kept_mask);
  const int32_t room = __shfl(r1b, static_cast<int>(threadIdx.x & 63) & ~(kGroup - 1)) - r0;
  const bool ins = new_s && kept + 1 <= room;
  if (keep) {
    const int32_t pos = __popc(kept_mask & ((1u << q) - 1)) + (ins && s < v ? 1 : 0);
    a.col[r0 + pos] = v;
    a.age[r0 + pos] = g;
  }
  if (q == 0) {
    if (ins) {
      const int32_t ps = __popc(below_s);
      a.col[r0 + ps] = s;
      a.age[r0 + ps] = 0;
    }
    if (new_s && (!ins || !row_insert(a.rp, a.len, a.col, a.age, s, b, 0)))
      raise_error(a.status, GSN_E_CAPACITY);
    a.len[b] = kept + (ins ? 1 : 0);
    a.err[b] = be + dj;
  }
  return true;
}

__global__ __launch_bounds__(kStepBlock) void wl_step(RoundArgs a, int32_t t) {
  __shared__ int32_t s_left;
  // (the same for every wave: the counter was written by earlier launches)
  if (t > 0 && spread_value(a.rem + rm_round(t - 1)) < kTailMin) return;
  if (threadIdx.x == 0) s_left = 0;
  __syncthreads();
  const int32_t gt = blockIdx.x * kStepBlock + threadIdx.x;
  const int32_t j = gt / kGroup;
  const int q = gt % kGroup;
  bool left = false;
  if (j < a.m && a.pend[j] == 1) {
    if (group_try_apply<true>(a, j, q)) {
      if (q == 0) a.pend[j] = 0;
    } else {
      left = q == 0;
    }
  }
  block_count_spread(left, a.rem + rm_round(t), &s_left);
}

// The remaining rounds in one workgroup: the pending signals are gathered into a list, and
// every round claims, applies where it may and re-gathers them, with a barrier between the
// phases.  Each round applies at least the pending signal of smallest
// key, so the loop ends after at most as many rounds as signals were pending; a round
// without progress ends it with an error.  Also adds this update's round count to the
// statistics and clears the survivor count.
__global__ __launch_bounds__(kTailBlock) void wl_tail(RoundArgs a, int32_t grid_rounds) {
  __shared__ int32_t s_n, s_next, s_rounds, s_ran, s_big;
  __shared__ int32_t s_pend[kMaxGridRounds + 1];  // the counters' values, survivors last
  const int tid = threadIdx.x;
  for (int r = tid >> 6; r <= kMaxGridRounds; r += kTailBlock / 64) {
    const int32_t v = spread_value(a.rem + (r < kMaxGridRounds ? rm_round(r) : kRmSurvivors));
    if ((tid & 63) == 0) s_pend[r] = v;
  }
  __syncthreads();
  if (tid == 0) {
    // grid rounds that ran: the first, then each one after a round that left kTailMin or
    // more; those that applied something: the ones that found survivors pending
    int32_t ran = grid_rounds > 0 ? 1 : 0;
    while (ran < grid_rounds && s_pend[ran - 1] >= kTailMin) ++ran;
    s_rounds = ran > 0 && s_pend[kMaxGridRounds] > 0 ? ran : 0;
    a.rem[kRmGridUsed] = ran;
    s_ran = ran;
    s_big = 0;
    s_n = 0;
    s_next = 0;
  }
  __syncthreads();
  int32_t* cur = a.list;
  int32_t* nxt = a.list + a.m;
  for (int32_t j = tid; j < a.m; j += kTailBlock)
    if (a.pend[j] == 1) cur[atomicAdd(&s_n, 1)] = j;
  __syncthreads();
  for (;;) {
    const int32_t n = s_n;
    if (n == 0) break;
    // a round that starts with kTailMin or more pending would have run grid-wide
    if (tid == 0 && n >= kTailMin) ++s_big;
    for (int32_t i = tid; i < n; i += kTailBlock) claim(a, cur[i]);
    __syncthreads();
    for (int32_t i = tid / kGroup; i < n; i += kTailBlock / kGroup) {
      const int32_t j = cur[i];
      if (group_try_apply<false>(a, j, tid % kGroup) && tid % kGroup == 0) a.pend[j] = 0;
    }
    __syncthreads();
    for (int32_t i = tid; i < n; i += kTailBlock) {
      const int32_t j = cur[i];
      if (a.pend[j] == 1) nxt[atomicAdd(&s_next, 1)] = j;
    }
    __syncthreads();
    if (tid == 0) {
      // no progress means the lock words were not all ones on entry (a corrupted
      // workspace): stop with an error rather than loop
      if (s_next == n) {
        raise_error(a.status, GSN_E_STATE);
        s_next = 0;
      }
      s_n = s_next;
      s_next = 0;
      ++s_rounds;
    }
    __syncthreads();
    int32_t* t = cur;
    cur = nxt;
    nxt = t;
  }
  spread_clear(a.rem + kRmSurvivors, tid);
  if (tid == 0) {
    // the grid-wide rounds this update could have used: those that ran, plus the rounds of
    // this workgroup that started with kTailMin or more pending.  The host reads the count
    // when it enqueues a later update (a stale value only changes how the rounds are split,
    // never a result); a store straight to its pinned word spares the stream a copy.
    if (a.feedback)
      __hip_atomic_store(a.feedback, s_ran + s_big, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    a.rem[kRmRounds] += s_rounds;
    a.rem[kRmRoundsMax] = max(a.rem[kRmRoundsMax], s_rounds);
    a.rem[kRmUpdates] += 1;
  }
}

// ---------------------------------------------------------- one-pass update ----
//
// The same update when no two survivors share a winner, as after the winner-lock resolve.
// Then a unit u is the winner of at most one step E_u (key k_u, second t_u), and the edge
// {u, v} changes only in E_u and E_v: a step ages it by one, or sets it to age 0 (creating
// it) when the step's second is the other end, and then removes it if it is older than
// max_age.  The state of every edge before or after any step therefore follows from its
// state before the update and those two steps alone, and so does all that the sequential
// update does to a unit x:
//   * x moves in E_x (eps_b) and, once with eps_n, in every E_b (b != x) whose second is x
//     or that finds {b, x} alive, which means alive after E_x when k_x < k_b; a move reads
//     and writes the moved unit only, so the moves of x applied to it in ascending key
//     order give its position after the sequential update;
//   * its row afterwards holds its edges alive after the steps of both ends, with their
//     ages;
//   * it is marked for removal when some E_v removes {v, x} and no edge of x is alive right
//     after E_v;
//   * its error grows by d1 in E_x.
// The steps that can involve x are those of x, of its neighbours before the update, of the
// survivors whose second is x (a list per unit, rhead / rnext), and that of the second of
// E_x.  The resolve's check fills the tables (the key and second of each winner's
// survivor, and the list of the survivors by second); then one thread per unit finds the
// steps: two launches and no rounds.  The tables have two
// parities so that the update can clear the other parity while it reads its own: an update
// with parity q finds tables q clean, fills them below n (whi[q] = n), and clears tables
// q ^ 1 below whi[q ^ 1], which the previous update filled.

struct LocalArgs {
  const float* sig;
  int32_t m, n;
  const int32_t* winner;
  const float* d1;
  unsigned long long* wkey;  // tables of this update's parity (records of key and second)
  uint8_t* wflag;            // 1 iff the unit has a record
  int32_t* rhead;
  int32_t* rnext;
  unsigned long long* wkey_o;  // tables of the other parity (cleared by wu_write)
  uint8_t* wflag_o;
  int32_t* rhead_o;
  int32_t* whi;
  int par;
  const int32_t* rp;  // adjacency before the update
  const int32_t* col;
  const int32_t* age;
  int32_t* rp2;  // adjacency after it
  int32_t* col2;
  int32_t* age2;
  float *x, *y, *z, *err;
  int32_t* orphan;
  int32_t* status;
  int32_t* cnt;
  int32_t* bsum;
  float eps_b, eps_n, beta;
  int32_t max_age;
  int64_t cap;
  int32_t nb;
  int fold;
};

struct Surv {
  unsigned long long key;  // all ones: the unit takes no step as a winner
  int32_t sec;             // the step's second (meaningful only with a key)
};

__device__ __forceinline__ Surv surv_of(const LocalArgs& a, int32_t u) {
  const ulonglong2 r = reinterpret_cast<const ulonglong2*>(a.wkey)[u];
  return Surv{r.x, static_cast<int32_t>(static_cast<uint32_t>(r.y))};
}

// The same, reading the unit's flag first and its record only if it has one.
__device__ __forceinline__ Surv surv_flagged(const LocalArgs& a, int32_t u) {
  return a.wflag[u] ? surv_of(a, u) : Surv{~0ull, -1};
}

__device__ __forceinline__ bool has_step(const Surv& s) { return s.key != ~0ull; }

// One step on an edge, taken by one of its ends: age 0 (the edge created if absent) when
// the step's second is the other end, else one year older if alive, then removed if older
// than max_age.  Returns whether this step removed it.
__device__ __forceinline__ bool edge_event(bool& alive, int32_t& ag, bool to_other,
                                           int32_t max_age) {
  if (to_other) {
    alive = true;
    ag = 0;
    return false;
  }
  if (!alive) return false;
  ag += 1;
  if (ag > max_age) {
    alive = false;
    return true;
  }
  return false;
}

struct EdgeState {
  bool alive;
  int32_t age;
  bool removed_by_w;  // the step of w removed it
};

// The edge {x, w} after those steps of x and w whose keys are below limit, from its state
// before the update (alive0, age0).
__device__ __forceinline__ EdgeState edge_state(bool alive0, int32_t age0, int32_t x,
                                                const Surv& sx, int32_t w, const Surv& sw,
                                                int32_t max_age, unsigned long long limit) {
  bool alive = alive0;
  int32_t ag = alive0 ? age0 : 0;
  bool rw = false;
  const bool ex = sx.key < limit, ew = sw.key < limit;
  if (ex && ew && sw.key < sx.key) {
    rw = edge_event(alive, ag, sw.sec == x, max_age);
    edge_event(alive, ag, sx.sec == w, max_age);
  } else {
    if (ex) edge_event(alive, ag, sx.sec == w, max_age);
    if (ew) rw = edge_event(alive, ag, sw.sec == x, max_age);
  }
  return EdgeState{alive, ag, rw};
}

// f(w, alive0, age0, sw) for every unit w that can share an edge with x in this update, each
// once: the neighbours before it (in ascending order), then the winners of the survivors
// whose second is x, then the second of the step of x.
template <typename F>
__device__ __forceinline__ void for_each_incident(const LocalArgs& a, int32_t x, const Surv& sx,
                                                  F&& f) {
  const int32_t r0 = a.rp[x], l = a.rp[x + 1] - r0;
  // the row in batches of eight entries, each batch's entries and then their survivor
  // records loaded together
  for (int32_t k0 = 0; k0 < l; k0 += 8) {
    int32_t w[8], g[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      w[i] = 0;
      g[i] = 0;
      if (k0 + i < l) {
        w[i] = a.col[r0 + k0 + i];
        g[i] = a.age[r0 + k0 + i];
      }
    }
    bool fl[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) fl[i] = k0 + i < l && a.wflag[w[i]] != 0;
    Surv sw[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) sw[i] = fl[i] ? surv_of(a, w[i]) : Surv{~0ull, -1};
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (k0 + i < l) f(w[i], true, g[i], sw[i]);
  }
  // (a list holds distinct signals of this update, so it ends within m links; the bounds
  // only keep a corrupted table from reading out of range)
  int32_t steps = 0;
  for (int32_t j = a.rhead[x]; j >= 0 && j < a.m && steps < a.m; j = a.rnext[j], ++steps) {
    const int32_t b = a.winner[j];
    if (b >= 0 && b < a.n && row_find(a.col, r0, l, b) < 0) f(b, false, 0, surv_of(a, b));
  }
  if (has_step(sx) && sx.sec >= 0 && sx.sec < a.n) {
    const int32_t t = sx.sec;
    const Surv st = surv_flagged(a, t);
    // (a second whose own step has x as its second is in the list above)
    if (row_find(a.col, r0, l, t) < 0 && !(has_step(st) && st.sec == x)) f(t, false, 0, st);
  }
}

constexpr int kMoves = 8;  // moves of a unit gathered per pass

// keys ascending (all ones = empty): keeps the kMoves smallest of keys and k
__device__ __forceinline__ void keep_smallest(unsigned long long (&keys)[kMoves],
                                              unsigned long long k) {
#pragma unroll
  for (int i = 0; i < kMoves; ++i) {
    const bool lt = keys[i] < k;
    const unsigned long long lo = lt ? keys[i] : k;
    k = lt ? k : keys[i];
    keys[i] = lo;
  }
}

// Per unit: its moves in key order, its mark, its error (with the decay), and the length of
// its row after the update (cnt, and per-workgroup sums in bsum).
__global__ __launch_bounds__(kBlock) void wu_apply(LocalArgs a) {
  __shared__ int32_t red[kBlock / 64];
  const int32_t x = blockIdx.x * kBlock + threadIdx.x;
  int32_t c = 0;
  if (x < a.n) {
    const Surv sx = surv_flagged(a, x);
    float px = a.x[x], py = a.y[x], pz = a.z[x];
    bool moved = false;
    // one pass over the incident edges: the row length afterwards, whether a step of the
    // other end removed one of them, and the moves (up to kMoves of them; more take further
    // passes over the keys above those applied)
    unsigned long long keys[kMoves];
    unsigned long long lo = 0;  // keys below lo were applied in earlier passes
    int32_t found = 0;
    auto offer = [&](unsigned long long k) {
      if (k < lo) return;
      ++found;
      keep_smallest(keys, k);
    };
    auto mover = [&](int32_t w, bool alive0, int32_t age0, const Surv& sw) {
      if (has_step(sw) &&
          (sw.sec == x || edge_state(alive0, age0, x, sx, w, sw, a.max_age, sw.key).alive))
        offer(sw.key);
    };
    auto apply_moves = [&]() {
#pragma unroll
      for (int i = 0; i < kMoves; ++i) {
        if (keys[i] == ~0ull) continue;
        const int32_t j = static_cast<int32_t>(static_cast<uint32_t>(keys[i]));
        const float eps = keys[i] == sx.key ? a.eps_b : a.eps_n;
        float t;
        t = a.sig[j] - px; t = eps * t; px = px + t;
        t = a.sig[a.m + j] - py; t = eps * t; py = py + t;
        t = a.sig[2 * a.m + j] - pz; t = eps * t; pz = pz + t;
        moved = true;
      }
    };
#pragma unroll
    for (int i = 0; i < kMoves; ++i) keys[i] = ~0ull;
    if (has_step(sx)) offer(sx.key);
    bool removal = false;
    for_each_incident(a, x, sx, [&](int32_t w, bool alive0, int32_t age0, const Surv& sw) {
      const EdgeState e = edge_state(alive0, age0, x, sx, w, sw, a.max_age, ~0ull);
      c += e.alive ? 1 : 0;
      removal |= e.removed_by_w;
      mover(w, alive0, age0, sw);
    });
    apply_moves();
    while (found > kMoves) {
      lo = keys[kMoves - 1] + 1;
      found = 0;
#pragma unroll
      for (int i = 0; i < kMoves; ++i) keys[i] = ~0ull;
      if (has_step(sx)) offer(sx.key);
      for_each_incident(a, x, sx, mover);
      apply_moves();
    }
    if (moved) {
      a.x[x] = px;
      a.y[x] = py;
      a.z[x] = pz;
    }
    // removal mark: some step of the other end removed an edge of x and left it none
    if (removal) {
      bool lone = false;
      for_each_incident(a, x, sx, [&](int32_t w, bool alive0, int32_t age0, const Surv& sw) {
        if (lone || !edge_state(alive0, age0, x, sx, w, sw, a.max_age, ~0ull).removed_by_w)
          return;
        int32_t d = 0;
        for_each_incident(a, x, sx, [&](int32_t v, bool al0, int32_t ag0, const Surv& sv) {
          if (v != w && edge_state(al0, ag0, x, sx, v, sv, a.max_age, sw.key).alive) ++d;
        });
        lone = d == 0;
      });
      if (lone && !a.orphan[x]) {
        a.orphan[x] = 1;
        atomicAdd(&a.status[kStOrphans], 1);
      }
    }
    float ev = a.err[x];
    if (has_step(sx)) ev = ev + a.d1[static_cast<uint32_t>(sx.key)];
    a.err[x] = ev * a.beta;
    a.cnt[x] = c;
  }
  const int32_t t = block_sum(c, red);
  if (threadIdx.x == 0) a.bsum[blockIdx.x] = t;
}

// Per unit: its row after the update at the offset of the scanned lengths, ascending (the
// neighbours before the update keep their order, each new edge is put in its place); and
// the other parity's tables cleared.  out_total receives the number of half-edges.
__global__ __launch_bounds__(kBlock) void wu_write(LocalArgs a, int32_t* out_total) {
  __shared__ int32_t wt[kBlock / 64];
  __shared__ int32_t red[2 * kBlock / 64];
  const int32_t x = blockIdx.x * kBlock + threadIdx.x;
  const int32_t c = x < a.n ? a.cnt[x] : 0;
  int32_t boff;
  bool abort;
  if (a.fold) {
    int32_t total;
    fold_offsets(a.bsum, a.nb, red, &boff, &total);
    abort = fold_abort(total, a.cap, a.status, out_total);
  } else {
    boff = a.bsum[blockIdx.x];
    abort = a.status[kStAbort] != 0;
  }
  const int32_t inc = block_inclusive_scan(c, wt);
  const int32_t hi_o = a.whi[a.par ^ 1];
  const int32_t stride = static_cast<int32_t>(gridDim.x) * kBlock;
  for (int32_t u = x; u < hi_o; u += stride) {
    a.wkey_o[2 * u] = ~0ull;
    a.wflag_o[u] = 0;
    a.rhead_o[u] = -1;
  }
  if (x >= a.n) return;
  if (abort) {
    // the rewrite did not fit: a valid, empty adjacency (the state is flagged invalid)
    a.rp2[x] = 0;
    return;
  }
  const int32_t start = boff + inc - c;
  a.rp2[x] = start;
  const Surv sx = surv_flagged(a, x);
  int32_t e = start;
  for_each_incident(a, x, sx, [&](int32_t w, bool alive0, int32_t age0, const Surv& sw) {
    const EdgeState st = edge_state(alive0, age0, x, sx, w, sw, a.max_age, ~0ull);
    if (!st.alive) return;
    int32_t k = e;
    if (!alive0)
      for (; k > start && a.col2[k - 1] > w; --k) {
        a.col2[k] = a.col2[k - 1];
        a.age2[k] = a.age2[k - 1];
      }
    a.col2[k] = w;
    a.age2[k] = st.age;
    ++e;
  });
}

}  // namespace

hipError_t launch_winner_update(const DevState& s, int cur, int32_t n, const WinnerStep& w,
                                hipStream_t st) {
  const int nxt = cur ^ 1;
  const int32_t m = w.m;
  const int nb = blocks(n);
  // slack copy of the adjacency
  wl_prepare<<<blocks(m), kBlock, 0, st>>>(m, n, w.winner, w.second, w.d1, w.accepted,
                                           w.key_mode, s.rp[cur], s.col[cur], s.lock, s.pend,
                                           s.extra, s.rem, s.status);
  const int fold = nb <= kFoldBlocks;
  wl_count<<<nb, kBlock, 0, st>>>(n, s.rp[cur], nullptr, s.extra, nullptr, s.cnt, s.bsum);
  hipError_t e = hipSuccess;
  if (!fold) {
    e = launch_scan_blocks(s.bsum, nb, w.slack_cap, s.rp[nxt] + n, s.status, -1, st);
    if (e != hipSuccess) return e;
  }
  wl_write<<<nb, kBlock, 0, st>>>(n, s.rp[cur], nullptr, s.col[cur], s.age[cur], s.cnt, s.bsum,
                                  s.rp[nxt], s.col[nxt], s.age[nxt], s.len, nullptr, 1.0f,
                                  s.status, fold, nb, w.slack_cap, s.rp[nxt] + n);
  // rounds
  RoundArgs a{w.sig,  m,          w.winner,   w.second,  w.d1,    w.key_mode, s.pend,
              s.rp[nxt], s.len,   s.col[nxt], s.age[nxt], s.lock, s.x,        s.y,
              s.z,    s.err,      s.orphan,   s.status,  w.eps_b, w.eps_n,    w.max_age,
              s.rem,  s.list,     w.feedback};
  const int g = static_cast<int>((m + kRoundBlock - 1) / kRoundBlock);
  const int gs = static_cast<int>((static_cast<int64_t>(m) * kGroup + kStepBlock - 1) /
                                  kStepBlock);
  for (int32_t t = 0; t < w.grid_rounds; ++t) {
    // the first round's claims were made with the survivors
    if (t > 0) wl_claim<<<g, kRoundBlock, 0, st>>>(a, t);
    wl_step<<<gs, kStepBlock, 0, st>>>(a, t);
  }
  wl_tail<<<1, kTailBlock, 0, st>>>(a, w.grid_rounds);
  // compact adjacency and error decay
  wl_count<<<nb, kBlock, 0, st>>>(n, s.rp[nxt], s.len, nullptr, s.lock, s.cnt, s.bsum);
  if (!fold) {
    e = launch_scan_blocks(s.bsum, nb, w.half_cap, s.rp[cur] + n, s.status, -1, st);
    if (e != hipSuccess) return e;
  }
  wl_write<<<nb, kBlock, 0, st>>>(n, s.rp[nxt], s.len, s.col[nxt], s.age[nxt], s.cnt, s.bsum,
                                  s.rp[cur], s.col[cur], s.age[cur], nullptr, s.err, w.beta,
                                  s.status, fold, nb, w.half_cap, s.rp[cur] + n);
  return hipGetLastError();
}

}  // namespace gsn

namespace gsn {

WinnerTables winner_tables(const DevState& s, int par, int32_t n_max) {
  const size_t nm = static_cast<size_t>(n_max);
  return WinnerTables{s.wkey + 2 * par * nm, s.wflag + par * nm, s.rhead + par * nm, s.rnext,
                      s.whi, par};
}

hipError_t launch_winner_local(const DevState& s, int cur, int par, int32_t n,
                               const WinnerStep& w, hipStream_t st) {
  const int nxt = cur ^ 1;
  const int po = par ^ 1;
  const size_t nm = static_cast<size_t>(w.n_max);
  const int nb = blocks(n);
  const int fold = nb <= kFoldBlocks;
  LocalArgs a{w.sig, w.m, n, w.winner, w.d1,
              s.wkey + 2 * par * nm, s.wflag + par * nm, s.rhead + par * nm, s.rnext,
              s.wkey + 2 * po * nm, s.wflag + po * nm, s.rhead + po * nm, s.whi, par,
              s.rp[cur], s.col[cur], s.age[cur], s.rp[nxt], s.col[nxt], s.age[nxt],
              s.x, s.y, s.z, s.err, s.orphan, s.status, s.cnt, s.bsum,
              w.eps_b, w.eps_n, w.beta, w.max_age, w.half_cap, nb, fold};
  wu_apply<<<nb, kBlock, 0, st>>>(a);
  if (!fold) {
    const hipError_t e = launch_scan_blocks(s.bsum, nb, w.half_cap, s.rp[nxt] + n, s.status,
                                            -1, st);
    if (e != hipSuccess) return e;
  }
  wu_write<<<nb, kBlock, 0, st>>>(a, s.rp[nxt] + n);
  return hipGetLastError();
}

}  // namespace gsn
