// The update phase of the multi-signal iteration (Sec. 2.1 step 3, Sec. 2.2): conflict
// resolution, adaptation and the connection update, all on the device.
//
// The paper updates sequentially on the host and leaves a parallel update as future work
// because of collisions (Sec. 4).  Here every signal claims its lock set L_j = {b_j, s_j}
// + N(b_j) with a 64-bit atomic minimum of its key, and survives iff it holds every unit
// of L_j.  Surviving lock sets are pairwise disjoint, which makes the adaptation and the
// edge update write-disjoint: no atomics on positions, errors or rows, and the result
// equals any sequential order (a group of eight lanes per signal).  The adjacency is a symmetric CSR (row_ptr, col, age per half-edge),
// rows ascending by neighbour; the edge update modifies ages in place, then rewrites a
// compacted CSR into the other buffer (count -> scan -> scatter).
#include "gsn_internal.h"

namespace gsn {
namespace {

// Rows of up to this many entries (nearly all of them) are read in one batch of loads.
constexpr int kShortRow = 8;

// Position of neighbour v in the ascending row col[lo, hi), or -1.
__device__ __forceinline__ int32_t find_in_span(const int32_t* __restrict__ col, int32_t lo,
                                                int32_t hi, int32_t v) {
  while (lo < hi) {
    const int32_t mid = (lo + hi) >> 1;
    const int32_t c = col[mid];
    if (c == v) return mid;
    if (c < v) lo = mid + 1; else hi = mid;
  }
  return -1;
}

// Position of neighbour v in the row of u, or -1.
__device__ __forceinline__ int32_t find_in_row(const int32_t* __restrict__ rp,
                                               const int32_t* __restrict__ col, int32_t u,
                                               int32_t v) {
  return find_in_span(col, rp[u], rp[u + 1], v);
}

// The same for a row col[r0, r1) of up to 8 entries (nearly all of them), read in one batch
// of loads.
__device__ __forceinline__ int32_t find_in_short_span(const int32_t* __restrict__ col,
                                                      int32_t r0, int32_t r1, int32_t v) {
  const int32_t l = r1 - r0;
  if (l > 8) return find_in_span(col, r0, r1, v);
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

// ------------------------------------------------------------------ resolve ----

// winner_only: L_j = {b}, else L_j = {b, s} + N(b).
__global__ void rs_claim(int32_t m, int32_t n, const int32_t* __restrict__ winner,
                         const int32_t* __restrict__ second, const float* __restrict__ d1,
                         const int32_t* __restrict__ rp, const int32_t* __restrict__ col,
                         unsigned long long* __restrict__ lock, int32_t* __restrict__ status,
                         int winner_only, int key_mode) {
  const int32_t j = blockIdx.x * kBlock + threadIdx.x;
  if (j >= m) return;
  const int32_t b = winner[j], s = second[j];
  if (!pair_ok(b, s, n)) {
    raise_error(status, GSN_E_INVAL);
    return;
  }
  const unsigned long long key = signal_key(d1[j], j, key_mode);
  atomicMin(&lock[b], key);
  if (winner_only) return;
  atomicMin(&lock[s], key);
  const int32_t r0 = rp[b];
  claim_row(lock, col, r0, rp[b + 1] - r0, key);
}

// With the winner alone locked, the survivor also releases its lock (the other claimants
// compare with their own keys, which differ from both values), so the lock array is back
// to all ones afterwards.
// Every claimant visits each unit of its lock set once and releases the units it holds
// (the others compare with their own keys, which differ from the holder's and from all
// ones in the index half), so the lock words are all ones again afterwards and the next
// resolve needs no clearing pass.  Also counts the signals and the accepted ones into the
// 64-bit statistics.
__global__ void rs_check(int32_t m, int32_t n, const int32_t* __restrict__ winner,
                         const int32_t* __restrict__ second, const float* __restrict__ d1,
                         const int32_t* __restrict__ rp, const int32_t* __restrict__ col,
                         unsigned long long* __restrict__ lock,
                         uint8_t* __restrict__ accepted, int winner_only, int key_mode,
                         unsigned long long* __restrict__ acc64, WinnerTables tab) {
  __shared__ int32_t s_acc;
  if (threadIdx.x == 0) s_acc = 0;
  __syncthreads();
  const int32_t j = blockIdx.x * kBlock + threadIdx.x;
  if (tab.wkey && j == 0) tab.whi[tab.par] = n;
  bool ok = false;
  if (j < m) {
    const int32_t b = winner[j], s = second[j];
    if (pair_ok(b, s, n)) {
      const unsigned long long key = signal_key(d1[j], j, key_mode);
      ok = true;
      auto visit = [&](int32_t u) {
        if (lock[u] == key) lock[u] = ~0ull; else ok = false;
      };
      visit(b);
      if (!winner_only) {
        bool s_nb = false;
        for (int32_t k = rp[b]; k < rp[b + 1]; ++k) {
          const int32_t v = col[k];
          s_nb |= v == s;
          visit(v);
        }
        if (!s_nb) visit(s);
      }
      if (ok && tab.wkey) {
        // the survivor tables of the one-pass update (one survivor per winner here)
        reinterpret_cast<ulonglong2*>(tab.wkey)[b] =
            make_ulonglong2(key, static_cast<uint32_t>(s));
        tab.wflag[b] = 1;
        tab.rnext[j] = atomicExch(&tab.rhead[s], j);
      }
    }
    accepted[j] = ok ? 1 : 0;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0)
    atomicAdd(&acc64[kA64Resolved], static_cast<unsigned long long>(m));
  block_count(ok, &acc64[kA64Accepted], &s_acc);
}

// -------------------------------------------------------------------- adapt ----

__global__ void ad_decay(float* __restrict__ err, int32_t n, float beta) {
  const int32_t i = blockIdx.x * kBlock + threadIdx.x;
  if (i < n) err[i] = err[i] * beta;
}

// -------------------------------------------------------------------- edges ----

// The lock-set resolve of rs_check fused with the update of the accepted signals (the
// adaptation of ad_move and the marks of ed_mark): an accepted lock set is held by its
// signal alone, and the other threads of this kernel read only lock words and row layouts,
// which the update leaves alone, so each accepted signal applies its update at once.
struct FusedArgs {
  const float* sig;
  int32_t m, n;
  const int32_t* winner;
  const int32_t* second;
  const float* d1;
  int key_mode;
  const int32_t* rp;
  const int32_t* col;
  unsigned long long* lock;
  uint8_t* accepted;
  unsigned long long* acc64;
  float *x, *y, *z, *err;
  float eps_b, eps_n;
  int32_t* age;
  int32_t* ins;
  int32_t* orphan;
  int32_t* status;
  int32_t max_age;
  int32_t* apart;  // accepted signals of each workgroup (plain stores)
  int32_t* bdelta;  // change of the half-edge count of every block of kBlock units
  const int32_t* order;  // optional: the signals in a spatial order (a permutation of 0..m-1)
  const uint8_t* given;  // optional: the acceptance decided already (the greedy resolve, whose
                         // accepted lock sets are disjoint too): no lock word is read or
                         // written and no statistic counted
};

// The fused kernels give each signal a group of kGroup lanes of one wave: lane q takes the
// neighbours k = q, q + kGroup, ... of the row of b (its claim, its lock word, its move, the
// age of its edge and the mirror half-edge, its removal), lane 0 also the winner and the
// second, and the group agrees on the outcome by ballots.  The neighbours' dependent loads
// (lock word, position, mirror search) then run side by side instead of one after another.
constexpr int kGroup = 8;

__device__ __forceinline__ uint32_t group_bits(unsigned long long wave_mask) {
  const int base = static_cast<int>(threadIdx.x & 63) & ~(kGroup - 1);
  return static_cast<uint32_t>(wave_mask >> base) & ((1u << kGroup) - 1);
}

// The separate adaptation (gsn_adapt) of the accepted signals (Eq. (adaptation)): the winner
// b moves eps_b of the way to the signal, its neighbours and the second (once, when it is no
// neighbour) eps_n, by move_unit, and d1 is added to b's error.  A group of kGroup lanes per
// signal: lane q moves the neighbours k = q, q + kGroup, ... of b, lane 0 the winner and the
// second (whether s is a neighbour comes from a ballot over the group).  Accepted lock sets
// are disjoint, so every unit moves once: the result is that of the signals applied one
// after another.
__global__ void ad_move(const float* __restrict__ sig, int32_t m, int32_t n,
                        const int32_t* __restrict__ winner, const int32_t* __restrict__ second,
                        const float* __restrict__ d1, const uint8_t* __restrict__ accepted,
                        const int32_t* __restrict__ rp, const int32_t* __restrict__ col,
                        float* __restrict__ x, float* __restrict__ y, float* __restrict__ z,
                        float* __restrict__ err, float eps_b, float eps_n) {
  const int64_t gt = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  const int32_t j = static_cast<int32_t>(gt / kGroup);
  const int q = static_cast<int>(gt % kGroup);
  int32_t b = 0, s = 0;
  const bool act = j < m && accepted[j] && pair_ok(b = winner[j], s = second[j], n);
  float sx = 0.0f, sy = 0.0f, sz = 0.0f;
  bool is_s = false;
  if (act) {
    sx = sig[j];
    sy = sig[m + j];
    sz = sig[2 * m + j];
    for (int32_t k = rp[b] + q; k < rp[b + 1]; k += kGroup) {
      const int32_t v = col[k];
      is_s |= v == s;
      move_unit(x, y, z, v, eps_n, sx, sy, sz);
    }
  }
  const bool s_nb = group_bits(__ballot(is_s)) != 0;
  if (act && q == 0) {
    move_unit(x, y, z, b, eps_b, sx, sy, sz);
    if (!s_nb) move_unit(x, y, z, s, eps_n, sx, sy, sz);
    err[b] = err[b] + d1[j];
  }
}

// The separate connection update (gsn_update_edges) of the accepted signals: every edge at b
// is aged by one on both half-edges, the edge {b, s} reset to age 0 (or requested when it is
// missing), the edges at b older than max_age marked dead on both half-edges, and a
// neighbour left without a live or requested edge flagged for removal.  A group of kGroup
// lanes per signal: lane q takes the neighbours k = q, q + kGroup, ... of b (ages, then
// removals), lane 0 the request.  The rows touched belong to L_j only, and the lane of
// neighbour v alone writes the row of v, so the result is that of the signals applied one
// after another.
__global__ void ed_mark(int32_t m, int32_t n, const int32_t* __restrict__ winner,
                        const int32_t* __restrict__ second,
                        const uint8_t* __restrict__ accepted, const int32_t* __restrict__ rp,
                        const int32_t* __restrict__ col, int32_t* __restrict__ age,
                        int32_t* __restrict__ ins, int32_t* __restrict__ orphan,
                        int32_t* __restrict__ status, int32_t max_age,
                        int32_t* __restrict__ bdelta) {
  const int64_t gt = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  const int32_t j = static_cast<int32_t>(gt / kGroup);
  const int q = static_cast<int>(gt % kGroup);
  int32_t b = 0, s = 0;
  const bool act = j < m && accepted[j] && pair_ok(b = winner[j], s = second[j], n);
  int32_t r0 = 0, r1 = 0;
  bool found = false;
  if (act) {
    r0 = rp[b];
    r1 = rp[b + 1];
    for (int32_t k = r0 + q; k < r1; k += kGroup) {
      const int32_t v = col[k];
      int32_t a = age[k] + 1;
      if (v == s) {
        a = 0;
        found = true;
      }
      age[k] = a;
      const int32_t rk = find_in_short_span(col, rp[v], rp[v + 1], b);
      if (rk >= 0) age[rk] = a;
    }
  }
  const bool s_nb = group_bits(__ballot(found)) != 0;
  if (act && q == 0 && !s_nb) {
    ins[b] = s;
    ins[s] = b;
    atomicAdd(&bdelta[b / kBlock], 1);
    atomicAdd(&bdelta[s / kBlock], 1);
  }
  if (!act) return;
  for (int32_t k = r0 + q; k < r1; k += kGroup) {
    if (age[k] <= max_age) continue;
    const int32_t v = col[k];
    age[k] = kDead;
    atomicAdd(&bdelta[b / kBlock], -1);
    const int32_t rk = find_in_row(rp, col, v, b);
    if (rk >= 0) {
      age[rk] = kDead;
      atomicAdd(&bdelta[v / kBlock], -1);
    }
    bool live = ins[v] >= 0;
    for (int32_t kk = rp[v]; !live && kk < rp[v + 1]; ++kk) live = age[kk] != kDead;
    if (!live && !orphan[v]) {
      orphan[v] = 1;
      atomicAdd(&status[kStOrphans], 1);
    }
  }
}

// Claims of the lock sets L_j = {b, s} + N(b), as rs_claim.
__global__ void fu_claim(int32_t m, int32_t n, const int32_t* __restrict__ winner,
                         const int32_t* __restrict__ second, const float* __restrict__ d1,
                         const int32_t* __restrict__ rp, const int32_t* __restrict__ col,
                         unsigned long long* __restrict__ lock, int32_t* __restrict__ status,
                         int key_mode) {
  const int32_t gt = blockIdx.x * kBlock + threadIdx.x;
  const int32_t j = gt / kGroup;
  const int q = gt % kGroup;
  if (j >= m) return;
  const int32_t b = winner[j], s = second[j];
  if (!pair_ok(b, s, n)) {
    if (q == 0) raise_error(status, GSN_E_INVAL);
    return;
  }
  const unsigned long long key = signal_key(d1[j], j, key_mode);
  if (q == 0) {
    atomicMin(&lock[b], key);
    atomicMin(&lock[s], key);
  }
  for (int32_t k = rp[b] + q; k < rp[b + 1]; k += kGroup) atomicMin(&lock[col[k]], key);
}

// The check of rs_check and, for an accepted signal, the adaptation of ad_move and the marks
// of ed_mark, with the same result: each unit of L_j is moved once with the
// same expression, every edge at b is aged (or reset, for {b, s}) and, if older than
// max_age, marked dead on both half-edges, and a neighbour left without a live edge or a
// requested one is flagged.  The lane of neighbour v alone writes the row of v, so its
// orphan test sees that row complete.
// What the update reads (the signal, the positions of b, s and the lane's first neighbour
// v0, b's error, v0's edge age, row bounds and row) is loaded beside the check rather than
// after it: a lock set that passes the check is its signal's alone, so no other thread of
// this launch writes those words, and the check's own reads of lock words taken early
// decide the same (another signal only ever clears a word holding its own key).  The
// dependent loads then form a chain of five rounds instead of about nine.
__global__ void fu_check_apply(FusedArgs a) {
  __shared__ int32_t s_acc;
  if (threadIdx.x == 0) s_acc = 0;
  __syncthreads();
  const int32_t gt = blockIdx.x * kBlock + threadIdx.x;
  // Signal j of the group.  The outcome of every signal does not depend on which group takes
  // it (the claims are all made before this launch and accepted lock sets are disjoint), so
  // with a spatial order the groups of a workgroup take nearby signals, whose lock words,
  // positions and rows share cache lines.
  const int32_t p = gt / kGroup;
  const int q = gt % kGroup;
  const int32_t j = p < a.m && a.order ? a.order[p] : p;
  bool ok = false;
  // (with the acceptance given, a rejected signal's group has nothing to load or do)
  if (p < a.m && j >= 0 && j < a.m && (a.given == nullptr || a.given[j] != 0)) {
    const int32_t b = a.winner[j], s = a.second[j];
    const float dj = a.d1[j];
    const float sx = a.sig[j], sy = a.sig[a.m + j], sz = a.sig[2 * a.m + j];
    // the five loads above are issued together before any of them is waited for
    __builtin_amdgcn_sched_barrier(0);
    if (pair_ok(b, s, a.n)) {
      const unsigned long long key = signal_key(dj, j, a.key_mode);
      const int32_t r0 = a.rp[b], r1 = a.rp[b + 1];
      const bool gv = a.given != nullptr;
      // lane 0: the lock words, positions and error of b and s
      unsigned long long lb = 0, ls = 0;
      float bx = 0.0f, by = 0.0f, bz = 0.0f, be = 0.0f, tx = 0.0f, ty = 0.0f, tz = 0.0f;
      if (q == 0) {
        if (!gv) {
          lb = a.lock[b];
          ls = a.lock[s];
        }
        bx = a.x[b]; by = a.y[b]; bz = a.z[b];
        be = a.err[b];
        tx = a.x[s]; ty = a.y[s]; tz = a.z[s];
      }
      // the lane's first neighbour (a row of up to kGroup entries gives each lane at most one)
      const int32_t k0 = r0 + q;
      const bool has0 = k0 < r1;
      int32_t v0 = -1, g0 = 0, w0 = 0, w1 = 0;
      unsigned long long l0 = 0;
      float vx = 0.0f, vy = 0.0f, vz = 0.0f;
      if (has0) {
        v0 = a.col[k0];
        g0 = a.age[k0];
        if (!gv) l0 = a.lock[v0];
        vx = a.x[v0]; vy = a.y[v0]; vz = a.z[v0];
        w0 = a.rp[v0];
        w1 = a.rp[v0 + 1];
      }
      const int32_t rk0 = has0 ? find_in_short_span(a.col, w0, w1, b) : -1;
      bool mine = true, is_s = false;
      auto visit = [&](int32_t u, unsigned long long word) {
        if (gv) return;
        if (word == key) a.lock[u] = ~0ull; else mine = false;
      };
      if (has0) {
        is_s |= v0 == s;
        visit(v0, l0);
      }
      for (int32_t k = k0 + kGroup; k < r1; k += kGroup) {
        const int32_t v = a.col[k];
        is_s |= v == s;
        if (!gv) visit(v, a.lock[v]);
      }
      const bool s_nb = group_bits(__ballot(is_s)) != 0;
      if (q == 0) {
        visit(b, lb);
        if (!s_nb) visit(s, ls);
      }
      ok = gv ? a.given[j] != 0 : group_bits(__ballot(!mine)) == 0;
      if (ok) {
        // move_unit's expression on positions already loaded
        auto move = [&](int32_t u, float eps, float px, float py, float pz) {
          float t;
          t = sx - px; t = eps * t; a.x[u] = px + t;
          t = sy - py; t = eps * t; a.y[u] = py + t;
          t = sz - pz; t = eps * t; a.z[u] = pz + t;
        };
        if (q == 0) {
          move(b, a.eps_b, bx, by, bz);
          if (!s_nb) {
            move(s, a.eps_n, tx, ty, tz);
            a.ins[b] = s;
            a.ins[s] = b;
            atomicAdd(&a.bdelta[b / kBlock], 1);
            atomicAdd(&a.bdelta[s / kBlock], 1);
          }
          a.err[b] = be + dj;
        }
        for (int32_t k = k0; k < r1; k += kGroup) {
          const bool first = k == k0;
          const int32_t v = first ? v0 : a.col[k];
          if (first) move(v, a.eps_n, vx, vy, vz);
          else move(v, a.eps_n, a.x[v], a.y[v], a.z[v]);
          const int32_t g = v == s ? 0 : (first ? g0 : a.age[k]) + 1;
          const int32_t rk = first ? rk0 : find_in_row(a.rp, a.col, v, b);
          if (g <= a.max_age) {
            a.age[k] = g;
            if (rk >= 0) a.age[rk] = g;
            continue;
          }
          a.age[k] = kDead;
          atomicAdd(&a.bdelta[b / kBlock], -1);
          if (rk >= 0) {
            a.age[rk] = kDead;
            atomicAdd(&a.bdelta[v / kBlock], -1);
          }
          bool live = a.ins[v] >= 0;
          for (int32_t kk = a.rp[v]; !live && kk < a.rp[v + 1]; ++kk) live = a.age[kk] != kDead;
          if (!live && !a.orphan[v]) {
            a.orphan[v] = 1;
            atomicAdd(&a.status[kStOrphans], 1);
          }
        }
      }
    }
    if (q == 0) a.accepted[j] = ok ? 1 : 0;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0 && a.given == nullptr)
    atomicAdd(&a.acc64[kA64Resolved], static_cast<unsigned long long>(a.m));
  // the workgroup's accepted count goes to its own word; the degree count that follows
  // adds them with one atomic (hundreds of same-address atomics at the end of this launch
  // would queue at the cache)
  const unsigned long long acc_mask = __ballot(ok && q == 0);
  if ((threadIdx.x & 63) == 0 && acc_mask != 0)
    atomicAdd(&s_acc, static_cast<int32_t>(__popcll(acc_mask)));
  __syncthreads();
  if (threadIdx.x == 0) a.apart[blockIdx.x] = s_acc;
}

// New degree of every unit (live half-edges + a requested new edge) and per-block sums;
// with err not null also the error decay of the fused iteration, and with apart not null
// workgroup 0 adds the napart per-workgroup counts of the fused check to *acc.
__global__ void ed_count(int32_t n, const int32_t* __restrict__ rp,
                         const int32_t* __restrict__ age, const int32_t* __restrict__ ins,
                         int32_t* __restrict__ cnt, int32_t* __restrict__ bsum,
                         float* __restrict__ err, float beta,
                         const int32_t* __restrict__ apart, int32_t napart,
                         unsigned long long* __restrict__ acc,
                         int32_t* __restrict__ bdelta_next) {
  __shared__ int32_t wt[2][kBlock / 64];
  if (threadIdx.x == 0) bdelta_next[blockIdx.x] = 0;
  if (apart != nullptr && blockIdx.x == 0) {
    int32_t v = 0;
    for (int32_t i = threadIdx.x; i < napart; i += kBlock) v += apart[i];
    v = block_sum(v, wt[0]);
    if (threadIdx.x == 0 && v != 0) atomicAdd(acc, static_cast<unsigned long long>(v));
  }
  const int32_t u = blockIdx.x * kBlock + threadIdx.x;
  int32_t c = 0;
  if (u < n) {
    const float e = err ? err[u] : 0.0f;  // loaded beside the row, stored after it
    const int32_t r0 = rp[u], r1 = rp[u + 1], l = r1 - r0;
    if (l > 0 && l <= kShortRow) {
      // one batch of loads (slots past the row's end repeat its last entry)
      int32_t g[kShortRow];
#pragma unroll
      for (int k = 0; k < kShortRow; ++k) g[k] = age[r0 + min(k, l - 1)];
#pragma unroll
      for (int k = 0; k < kShortRow; ++k) c += k < l && g[k] != kDead;
    } else {
      for (int32_t k = r0; k < r1; ++k) c += age[k] != kDead;
    }
    c += ins[u] >= 0;
    cnt[u] = c;
    if (err) err[u] = e * beta;
  }
  c = block_sum(c, wt[1]);
  if (threadIdx.x == 0) bsum[blockIdx.x] = c;
}

// Exclusive scan of the per-block sums in one workgroup; bsum[nb] receives the total.
// If the total exceeds `cap`, the rewrite is aborted and a capacity error is raised;
// `out_rp_n` (if not null) receives the total, or 0 once aborted, so that the rows written
// afterwards always describe a valid adjacency.
__global__ __launch_bounds__(1024) void scan_blocks(int32_t* __restrict__ bsum, int32_t nb,
                                                    int64_t cap, int32_t* __restrict__ out_rp_n,
                                                    int32_t* __restrict__ status,
                                                    int32_t status_slot_total) {
  __shared__ int32_t part[1024];
  const int32_t t = threadIdx.x;
  const int32_t per = (nb + 1023) / 1024;
  const int32_t a = t * per, e = min(nb, a + per);
  int32_t sum = 0;
  for (int32_t i = a; i < e; ++i) sum += bsum[i];
  part[t] = sum;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    const int32_t v = t >= off ? part[t - off] : 0;
    __syncthreads();
    part[t] += v;
    __syncthreads();
  }
  int32_t run = part[t] - sum;  // exclusive prefix of this thread's slice
  for (int32_t i = a; i < e; ++i) {
    const int32_t v = bsum[i];
    bsum[i] = run;
    run += v;
  }
  if (t == 1023) {
    const int32_t total = part[1023];
    bsum[nb] = total;
    const bool over = static_cast<int64_t>(total) > cap;
    if (over) {
      status[kStAbort] = 1;
      atomicCAS(&status[kStError], 0, GSN_E_CAPACITY);
    }
    if (out_rp_n) *out_rp_n = over || status[kStAbort] ? 0 : total;
    if (status_slot_total >= 0) status[status_slot_total] = total;
  }
}

// Block-local exclusive scan of cnt, plus the block offset, gives each row's start; the
// row is written as the live old entries merged with the requested new neighbour, in
// ascending neighbour order.  Clears the request.  With fold the block offsets and the
// capacity check come from the raw block sums (fold_offsets, fold_abort: cap and out_total
// as for scan_blocks); otherwise bsum holds the scanned offsets.
__global__ void ed_write(int32_t n, const int32_t* __restrict__ rp,
                         const int32_t* __restrict__ col, const int32_t* __restrict__ age,
                         int32_t* __restrict__ ins, const int32_t* __restrict__ cnt,
                         const int32_t* __restrict__ bsum, int32_t* __restrict__ rp_new,
                         int32_t* __restrict__ col_new, int32_t* __restrict__ age_new,
                         int32_t* __restrict__ status, int fold, int32_t nb, int64_t cap,
                         int32_t* __restrict__ out_total, int32_t* __restrict__ taken) {
  __shared__ int32_t wt[kBlock / 64];
  __shared__ int32_t red[2 * kBlock / 64];
  const int32_t u = blockIdx.x * kBlock + threadIdx.x;
  const int32_t c = u < n ? cnt[u] : 0;
  if (taken && u < n) taken[u] = 0;  // the greedy resolve's marks, clear for the next call
  int32_t boff, abort;
  if (fold) {
    int32_t total;
    fold_offsets(bsum, nb, red, &boff, &total);
    abort = fold_abort(total, cap, status, out_total);
  } else {
    boff = bsum[blockIdx.x];
    abort = status[kStAbort];
  }
  const int32_t inc = block_inclusive_scan(c, wt);
  if (u >= n) return;
  const int32_t start = boff + inc - c;
  const int32_t extra = ins[u];
  ins[u] = -1;
  if (abort) {
    // the rewrite did not fit: leave a valid, empty adjacency (state is flagged invalid)
    rp_new[u] = 0;
    return;
  }
  rp_new[u] = start;
  int32_t o = start;
  bool pending = extra >= 0;
  // one live entry (v, g) in ascending order, with the requested neighbour placed before
  // the first larger one
  auto put = [&](int32_t v, int32_t g) {
    if (g == kDead) return;
    if (pending && extra < v) {
      col_new[o] = extra;
      age_new[o] = 0;
      ++o;
      pending = false;
    }
    col_new[o] = v;
    age_new[o] = g;
    ++o;
  };
  const int32_t r0 = rp[u], r1 = rp[u + 1], l = r1 - r0;
  if (l > 0 && l <= kShortRow) {
    // one batch of loads (slots past the row's end repeat its last entry)
    int32_t cv[kShortRow], gv[kShortRow];
#pragma unroll
    for (int k = 0; k < kShortRow; ++k) {
      cv[k] = col[r0 + min(k, l - 1)];
      gv[k] = age[r0 + min(k, l - 1)];
    }
#pragma unroll
    for (int k = 0; k < kShortRow; ++k)
      if (k < l) put(cv[k], gv[k]);
  } else {
    for (int32_t k = r0; k < r1; ++k) put(col[k], age[k]);
  }
  if (pending) {
    col_new[o] = extra;
    age_new[o] = 0;
  }
}

// The rewrite without a separate count (up to kFoldBlocks workgroups): the marking kernels
// added, for every block of kBlock units, the change of its half-edge count (+1 for each
// requested edge, -1 for each half-edge marked dead) to bdelta, so the new start of block
// b is the old start rp[kBlock b] plus the changes of the blocks before it (every workgroup
// sums them itself), and the new total is rp[n] plus all changes.  Each thread counts its
// own row's live entries and request, a block scan places the rows, and the row is written
// as in ed_write.  Also the error decay (err not null), the per-workgroup accepted counts of
// the fused check (apart not null, workgroup 0), and zeroing of the other delta array for
// the next update (every workgroup its own entry).
__global__ void ed_rewrite(int32_t n, const int32_t* __restrict__ rp,
                           const int32_t* __restrict__ col, const int32_t* __restrict__ age,
                           int32_t* __restrict__ ins, const int32_t* __restrict__ bdelta,
                           int32_t* __restrict__ bdelta_next, int32_t* __restrict__ rp_new,
                           int32_t* __restrict__ col_new, int32_t* __restrict__ age_new,
                           int32_t* __restrict__ status, int32_t nb, int64_t cap,
                           float* __restrict__ err, float beta,
                           const int32_t* __restrict__ apart, int32_t napart,
                           unsigned long long* __restrict__ acc, int32_t* __restrict__ taken) {
  __shared__ int32_t wt[kBlock / 64];
  __shared__ int32_t wa[kBlock / 64];
  __shared__ int32_t red[2 * kBlock / 64];
  const int32_t u = blockIdx.x * kBlock + threadIdx.x;
  const bool in = u < n;
  // the row (slots past its end repeat the last entry), the request, the error and the old
  // start of the block, all loaded before any is waited for
  const int32_t r0 = in ? rp[u] : 0, r1 = in ? rp[u + 1] : 0, l = r1 - r0;
  const int32_t extra = in ? ins[u] : -1;
  if (taken && in) taken[u] = 0;  // the greedy resolve's marks, clear for the next call
  const float e = in && err ? err[u] : 0.0f;
  const int32_t base = rp[blockIdx.x * kBlock];
  int32_t cv[kShortRow], gv[kShortRow];
  const bool short_row = l > 0 && l <= kShortRow;
  if (short_row) {
#pragma unroll
    for (int k = 0; k < kShortRow; ++k) {
      cv[k] = col[r0 + min(k, l - 1)];
      gv[k] = age[r0 + min(k, l - 1)];
    }
  }
  int32_t c = extra >= 0 ? 1 : 0;
  if (short_row) {
#pragma unroll
    for (int k = 0; k < kShortRow; ++k) c += k < l && gv[k] != kDead;
  } else {
    // a long row: kShortRow ages per batch of loads (a load per entry, each waited for
    // before the next, would hold up the whole workgroup)
    for (int32_t k0 = r0; k0 < r1; k0 += kShortRow) {
      const int32_t nk = min(kShortRow, r1 - k0);
      int32_t g[kShortRow];
#pragma unroll
      for (int k = 0; k < kShortRow; ++k) g[k] = age[k0 + min(k, nk - 1)];
#pragma unroll
      for (int k = 0; k < kShortRow; ++k) c += k < nk && g[k] != kDead;
    }
  }
  if (apart != nullptr && blockIdx.x == 0) {
    int32_t v = 0;
    for (int32_t i = threadIdx.x; i < napart; i += kBlock) v += apart[i];
    v = block_sum(v, wa);
    if (threadIdx.x == 0 && v != 0) atomicAdd(acc, static_cast<unsigned long long>(v));
  }
  int32_t before, dtotal;
  fold_offsets(bdelta, nb, red, &before, &dtotal);
  const int32_t abort = fold_abort(rp[n] + dtotal, cap, status, rp_new + n);
  const int32_t inc = block_inclusive_scan(c, wt);
  if (threadIdx.x == 0) bdelta_next[blockIdx.x] = 0;
  if (!in) return;
  if (err) err[u] = e * beta;
  ins[u] = -1;
  if (abort) {
    // the rewrite did not fit: leave a valid, empty adjacency (state is flagged invalid)
    rp_new[u] = 0;
    return;
  }
  const int32_t start = base + before + inc - c;
  rp_new[u] = start;
  int32_t o = start;
  bool pending = extra >= 0;
  auto put = [&](int32_t v, int32_t g) {
    if (g == kDead) return;
    if (pending && extra < v) {
      col_new[o] = extra;
      age_new[o] = 0;
      ++o;
      pending = false;
    }
    col_new[o] = v;
    age_new[o] = g;
    ++o;
  };
  if (short_row) {
#pragma unroll
    for (int k = 0; k < kShortRow; ++k)
      if (k < l) put(cv[k], gv[k]);
  } else {
    for (int32_t k0 = r0; k0 < r1; k0 += kShortRow) {
      const int32_t nk = min(kShortRow, r1 - k0);
      int32_t cc[kShortRow], g[kShortRow];
#pragma unroll
      for (int k = 0; k < kShortRow; ++k) {
        cc[k] = col[k0 + min(k, nk - 1)];
        g[k] = age[k0 + min(k, nk - 1)];
      }
#pragma unroll
      for (int k = 0; k < kShortRow; ++k)
        if (k < nk) put(cc[k], g[k]);
    }
  }
  if (pending) {
    col_new[o] = extra;
    age_new[o] = 0;
  }
}

__global__ void init_state(float* __restrict__ err, int32_t* __restrict__ ins,
                           int32_t* __restrict__ orphan, int32_t* __restrict__ rp,
                           unsigned long long* __restrict__ lock, int32_t* __restrict__ extra,
                           int32_t* __restrict__ rem, unsigned long long* __restrict__ acc64,
                           int32_t n_max, int32_t* __restrict__ status,
                           int32_t* __restrict__ bd0, int32_t* __restrict__ bd1,
                           unsigned long long* __restrict__ wkey, uint8_t* __restrict__ wflag,
                           int32_t* __restrict__ rhead, int32_t* __restrict__ whi) {
  const int32_t i = blockIdx.x * kBlock + threadIdx.x;
  if (wkey && i < n_max) {
    wkey[2 * i] = ~0ull;
    wkey[2 * (n_max + i)] = ~0ull;
    wflag[i] = 0;
    wflag[n_max + i] = 0;
    rhead[i] = -1;
    rhead[n_max + i] = -1;
  }
  if (whi && i < 2) whi[i] = 0;
  if (i < n_max / kBlock + 2) {
    bd0[i] = 0;
    bd1[i] = 0;
  }
  if (i < n_max) {
    err[i] = 0.0f;
    ins[i] = -1;
    orphan[i] = 0;
    lock[i] = ~0ull;
    extra[i] = 0;
  }
  if (i <= n_max) rp[i] = 0;
  if (i < kStSlots) status[i] = 0;
  if (i < kRmWords) rem[i] = 0;
  if (i < kA64Slots) acc64[i] = 0;
}

inline int blocks(int64_t n) { return static_cast<int>((n + kBlock - 1) / kBlock); }

}  // namespace

hipError_t launch_init(const DevState& s, int cur, int32_t, int32_t n_max, hipStream_t st) {
  const int64_t cover =
      std::max<int64_t>(static_cast<int64_t>(n_max) + 1, std::max<int>(kStSlots, kRmWords));
  init_state<<<blocks(cover), kBlock, 0, st>>>(s.err, s.ins, s.orphan, s.rp[cur], s.lock,
                                               s.extra, s.rem, s.acc64, n_max, s.status,
                                               s.bdelta[0], s.bdelta[1], s.wkey, s.wflag,
                                               s.rhead,
                                               s.whi);
  return hipGetLastError();
}

hipError_t launch_resolve(const DevState& s, int cur, int32_t n, int32_t m,
                          const int32_t* winner, const int32_t* second, const float* d1,
                          uint8_t* accepted, int lock_mode, int key_mode, hipStream_t st,
                          const WinnerTables* tables, bool claimed) {
  const int wo = lock_mode == 1;
  const WinnerTables tab = tables && wo ? *tables : WinnerTables{};
  // the lock words are all ones between calls (set at creation and import, released by
  // their holders in every check)
  if (!claimed)
    rs_claim<<<blocks(m), kBlock, 0, st>>>(m, n, winner, second, d1, s.rp[cur], s.col[cur],
                                           s.lock, s.status, wo, key_mode);
  rs_check<<<blocks(m), kBlock, 0, st>>>(m, n, winner, second, d1, s.rp[cur], s.col[cur],
                                         s.lock, accepted, wo, key_mode, s.acc64, tab);
  return hipGetLastError();
}

hipError_t launch_adapt(const DevState& s, int cur, int32_t n, const float* sig, int32_t m,
                        const int32_t* winner, const int32_t* second, const float* d1,
                        const uint8_t* accepted, float eps_b, float eps_n, float beta,
                        hipStream_t st) {
  if (m > 0)
    ad_move<<<blocks(static_cast<int64_t>(m) * kGroup), kBlock, 0, st>>>(
        sig, m, n, winner, second, d1, accepted, s.rp[cur], s.col[cur], s.x, s.y, s.z, s.err,
        eps_b, eps_n);
  if (n > 0) ad_decay<<<blocks(n), kBlock, 0, st>>>(s.err, n, beta);
  return hipGetLastError();
}

hipError_t launch_edges(const DevState& s, int cur, int dpar, int32_t n, int32_t m,
                        const int32_t* winner, const int32_t* second,
                        const uint8_t* accepted, int32_t max_age, int64_t half_cap,
                        hipStream_t st, int32_t* taken) {
  const int nxt = cur ^ 1;
  int32_t* bd = s.bdelta[dpar];
  int32_t* bd_next = s.bdelta[dpar ^ 1];
  if (m > 0)
    ed_mark<<<blocks(static_cast<int64_t>(m) * kGroup), kBlock, 0, st>>>(
        m, n, winner, second, accepted, s.rp[cur], s.col[cur], s.age[cur], s.ins, s.orphan,
        s.status, max_age, bd);
  const int nb = blocks(n);
  if (n == 0) return hipGetLastError();
  if (nb <= kFoldBlocks) {
    ed_rewrite<<<nb, kBlock, 0, st>>>(n, s.rp[cur], s.col[cur], s.age[cur], s.ins, bd, bd_next,
                                      s.rp[nxt], s.col[nxt], s.age[nxt], s.status, nb, half_cap,
                                      nullptr, 1.0f, nullptr, 0, nullptr, taken);
    return hipGetLastError();
  }
  ed_count<<<nb, kBlock, 0, st>>>(n, s.rp[cur], s.age[cur], s.ins, s.cnt, s.bsum, nullptr,
                                  1.0f, nullptr, 0, nullptr, bd_next);
  scan_blocks<<<1, 1024, 0, st>>>(s.bsum, nb, half_cap, s.rp[nxt] + n, s.status, -1);
  ed_write<<<nb, kBlock, 0, st>>>(n, s.rp[cur], s.col[cur], s.age[cur], s.ins, s.cnt, s.bsum,
                                  s.rp[nxt], s.col[nxt], s.age[nxt], s.status, 0, nb, half_cap,
                                  s.rp[nxt] + n, taken);
  return hipGetLastError();
}

hipError_t launch_iterate_set(const DevState& s, int cur, int dpar, int32_t n, const float* sig,
                              int32_t m, const int32_t* winner, const int32_t* second,
                              const float* d1, uint8_t* accepted, int key_mode, float eps_b,
                              float eps_n, float beta, int32_t max_age, int64_t half_cap,
                              bool claimed, const int32_t* order, hipStream_t st,
                              const uint8_t* given) {
  const int nxt = cur ^ 1;
  int32_t* bd = s.bdelta[dpar];
  int32_t* bd_next = s.bdelta[dpar ^ 1];
  const int gb = blocks(static_cast<int64_t>(m) * kGroup);
  // the accepted counts go to the statistics unless the resolve that decided them counted
  const int32_t* apart = m > 0 && !given ? s.apart : nullptr;
  // after the greedy resolve its taken marks are cleared for the next call
  int32_t* taken = given ? s.extra : nullptr;
  if (m > 0) {
    if (!claimed && !given)
      fu_claim<<<gb, kBlock, 0, st>>>(m, n, winner, second, d1, s.rp[cur], s.col[cur], s.lock,
                                      s.status, key_mode);
    FusedArgs a{sig,      m,          n,          winner,  second,   d1,     key_mode,
                s.rp[cur], s.col[cur], s.lock,     accepted, s.acc64, s.x,    s.y,
                s.z,      s.err,      eps_b,      eps_n,   s.age[cur], s.ins, s.orphan,
                s.status, max_age, s.apart, bd, order, given};
    fu_check_apply<<<gb, kBlock, 0, st>>>(a);
  }
  // (with no units no signal is accepted, so skipping the rewrite loses nothing)
  if (n == 0) return hipGetLastError();
  const int nb = blocks(n);
  if (nb <= kFoldBlocks) {
    ed_rewrite<<<nb, kBlock, 0, st>>>(n, s.rp[cur], s.col[cur], s.age[cur], s.ins, bd, bd_next,
                                      s.rp[nxt], s.col[nxt], s.age[nxt], s.status, nb, half_cap,
                                      s.err, beta, apart, gb, s.acc64 + kA64Accepted, taken);
    return hipGetLastError();
  }
  ed_count<<<nb, kBlock, 0, st>>>(n, s.rp[cur], s.age[cur], s.ins, s.cnt, s.bsum, s.err, beta,
                                  apart, gb, s.acc64 + kA64Accepted, bd_next);
  scan_blocks<<<1, 1024, 0, st>>>(s.bsum, nb, half_cap, s.rp[nxt] + n, s.status, -1);
  ed_write<<<nb, kBlock, 0, st>>>(n, s.rp[cur], s.col[cur], s.age[cur], s.ins, s.cnt, s.bsum,
                                  s.rp[nxt], s.col[nxt], s.age[nxt], s.status, 0, nb, half_cap,
                                  s.rp[nxt] + n, taken);
  return hipGetLastError();
}

hipError_t launch_scan_blocks(int32_t* bsum, int32_t nb, int64_t cap, int32_t* out_total,
                              int32_t* status, int32_t slot, hipStream_t st) {
  scan_blocks<<<1, 1024, 0, st>>>(bsum, nb, cap, out_total, status, slot);
  return hipGetLastError();
}

}  // namespace gsn
