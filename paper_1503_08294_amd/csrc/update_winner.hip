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
// and afterwards compacted back, so no round rewrites the adjacency.
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

// Remove v from the row of u if present; returns the new length.
__device__ int32_t row_remove(const int32_t* __restrict__ rp, int32_t* __restrict__ len,
                              int32_t* __restrict__ col, int32_t* __restrict__ age, int32_t u,
                              int32_t v) {
  const int32_t r0 = rp[u], l = len[u];
  const int32_t k = slice_find(col, r0, r0 + l, v);
  if (k < 0) return l;
  for (int32_t q = k; q + 1 < r0 + l; ++q) {
    col[q] = col[q + 1];
    age[q] = age[q + 1];
  }
  len[u] = l - 1;
  return l - 1;
}

// Adds the lanes of this wave for which `pred` holds to *ctr with one atomic.
__device__ __forceinline__ void wave_count(bool pred, int32_t* ctr) {
  const unsigned long long mask = __ballot(pred);
  if (mask == 0) return;
  const int lane = static_cast<int>(threadIdx.x & 63);
  if (lane == __ffsll(static_cast<long long>(mask)) - 1)
    atomicAdd(ctr, static_cast<int32_t>(__popcll(mask)));
}

// ----------------------------------------------------------------- prologue ----

// Survivors (pend = 1), the insertions each row may receive, and the survivor count.
__global__ void wl_prepare(int32_t m, int32_t n, const int32_t* __restrict__ winner,
                           const int32_t* __restrict__ second,
                           const uint8_t* __restrict__ accepted, uint8_t* __restrict__ pend,
                           int32_t* __restrict__ extra, int32_t* __restrict__ rem,
                           int32_t* __restrict__ status) {
  const int32_t j = blockIdx.x * kBlock + threadIdx.x;
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
    }
  }
  wave_count(ok, &rem[kRingSurvivors]);
}

// Row sizes for a rewrite: the live length (len, or the CSR row length when len is null)
// plus the room asked in extra (when not null; it is cleared), and per-block sums.
__global__ void wl_count(int32_t n, const int32_t* __restrict__ rp,
                         const int32_t* __restrict__ len, int32_t* __restrict__ extra,
                         int32_t* __restrict__ cnt, int32_t* __restrict__ bsum) {
  __shared__ int32_t red[kBlock];
  const int32_t u = blockIdx.x * kBlock + threadIdx.x;
  int32_t c = 0;
  if (u < n) {
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
__global__ void wl_write(int32_t n, const int32_t* __restrict__ rp,
                         const int32_t* __restrict__ len, const int32_t* __restrict__ col,
                         const int32_t* __restrict__ age, const int32_t* __restrict__ cnt,
                         const int32_t* __restrict__ boff, int32_t* __restrict__ dst_rp,
                         int32_t* __restrict__ dst_col, int32_t* __restrict__ dst_age,
                         int32_t* __restrict__ dst_len, float* __restrict__ err, float beta,
                         const int32_t* __restrict__ status) {
  __shared__ int32_t sc[kBlock];
  const int32_t u = blockIdx.x * kBlock + threadIdx.x;
  const int32_t c = u < n ? cnt[u] : 0;
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
  if (status[kStAbort]) {
    // the rewrite did not fit: leave a valid, empty adjacency (the state is flagged invalid)
    dst_rp[u] = 0;
    if (dst_len) dst_len[u] = 0;
    return;
  }
  const int32_t start = boff[blockIdx.x] + sc[threadIdx.x] - c;
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
// Round t writes slot t % kRing of rem (pending after the round) and reads slot
// (t - 1) % kRing: once a round leaves nothing pending, the later ones return at once.

__global__ void wl_claim(int32_t m, const int32_t* __restrict__ winner,
                         const int32_t* __restrict__ second, const float* __restrict__ d1,
                         int key_mode, const uint8_t* __restrict__ pend,
                         const int32_t* __restrict__ rp, const int32_t* __restrict__ len,
                         const int32_t* __restrict__ col, unsigned long long* __restrict__ lock,
                         int32_t* __restrict__ rem, int32_t slot, int32_t prev, int force) {
  if (blockIdx.x == 0 && threadIdx.x == 0) rem[slot] = 0;
  if (!force && rem[prev] == 0) return;
  const int32_t j = blockIdx.x * kBlock + threadIdx.x;
  if (j >= m || pend[j] != 1) return;
  const int32_t b = winner[j], s = second[j];
  const unsigned long long key = signal_key(d1[j], j, key_mode);
  atomicMin(&lock[b], key);
  atomicMin(&lock[s], key);
  const int32_t r0 = rp[b], r1 = r0 + len[b];
  for (int32_t k = r0; k < r1; ++k) atomicMin(&lock[col[k]], key);
}

// Every claimant visits each unit of F_j once and releases the units it holds; the others
// compare the lock with their own keys, which differ from the holder's key and from all
// ones in the index half, so the release order does not matter and the lock array is all
// ones again afterwards.
__global__ void wl_check(int32_t m, const int32_t* __restrict__ winner,
                         const int32_t* __restrict__ second, const float* __restrict__ d1,
                         int key_mode, uint8_t* __restrict__ pend,
                         const int32_t* __restrict__ rp, const int32_t* __restrict__ len,
                         const int32_t* __restrict__ col, unsigned long long* __restrict__ lock,
                         int32_t* __restrict__ rem, int32_t slot, int32_t prev, int force) {
  if (!force && rem[prev] == 0) return;
  const int32_t j = blockIdx.x * kBlock + threadIdx.x;
  bool left = false;
  if (j < m && pend[j] == 1) {
    const int32_t b = winner[j], s = second[j];
    const unsigned long long key = signal_key(d1[j], j, key_mode);
    bool ok = true;
    if (lock[b] == key) lock[b] = ~0ull; else ok = false;
    bool s_nb = false;
    const int32_t r0 = rp[b], r1 = r0 + len[b];
    for (int32_t k = r0; k < r1; ++k) {
      const int32_t v = col[k];
      s_nb |= v == s;
      if (lock[v] == key) lock[v] = ~0ull; else ok = false;
    }
    if (!s_nb) {
      if (lock[s] == key) lock[s] = ~0ull; else ok = false;
    }
    if (ok) pend[j] = 2;
    left = !ok;
  }
  wave_count(left, &rem[slot]);
}

// The single-signal step of every survivor that holds its units (pend = 2).
__global__ void wl_apply(const float* __restrict__ sig, int32_t m,
                         const int32_t* __restrict__ winner,
                         const int32_t* __restrict__ second, const float* __restrict__ d1,
                         uint8_t* __restrict__ pend, const int32_t* __restrict__ rp,
                         int32_t* __restrict__ len, int32_t* __restrict__ col,
                         int32_t* __restrict__ age, float* __restrict__ x,
                         float* __restrict__ y, float* __restrict__ z,
                         float* __restrict__ err, int32_t* __restrict__ orphan,
                         int32_t* __restrict__ status, float eps_b, float eps_n,
                         int32_t max_age, const int32_t* __restrict__ rem, int32_t prev,
                         int force) {
  if (!force && rem[prev] == 0) return;
  const int32_t j = blockIdx.x * kBlock + threadIdx.x;
  if (j >= m || pend[j] != 2) return;
  pend[j] = 0;
  const int32_t b = winner[j], s = second[j];
  const float sx = sig[j], sy = sig[m + j], sz = sig[2 * m + j];
  const int32_t r0 = rp[b];
  int32_t l = len[b];
  // adaptation: the winner, its neighbours before this step, and the second once
  move_unit(x, y, z, b, eps_b, sx, sy, sz);
  bool s_nb = false;
  for (int32_t k = r0; k < r0 + l; ++k) {
    const int32_t v = col[k];
    s_nb |= v == s;
    move_unit(x, y, z, v, eps_n, sx, sy, sz);
  }
  if (!s_nb) move_unit(x, y, z, s, eps_n, sx, sy, sz);
  // aging of the edges at b, the edge {b, s} at age 0
  for (int32_t k = r0; k < r0 + l; ++k) {
    const int32_t v = col[k];
    const int32_t a = v == s ? 0 : age[k] + 1;
    age[k] = a;
    const int32_t rk = slice_find(col, rp[v], rp[v] + len[v], b);
    if (rk >= 0) age[rk] = a;
  }
  if (!s_nb) {
    if (!row_insert(rp, len, col, age, b, s, 0) || !row_insert(rp, len, col, age, s, b, 0))
      raise_error(status, GSN_E_CAPACITY);
  }
  // removal of the edges at b older than max_age
  l = len[b];
  int32_t w = r0;
  for (int32_t k = r0; k < r0 + l; ++k) {
    const int32_t v = col[k];
    const int32_t a = age[k];
    if (a > max_age) {
      if (row_remove(rp, len, col, age, v, b) == 0 && !orphan[v]) {
        orphan[v] = 1;
        atomicAdd(&status[kStOrphans], 1);
      }
    } else {
      col[w] = v;
      age[w] = a;
      ++w;
    }
  }
  len[b] = w - r0;
  err[b] = err[b] + d1[j];
}

}  // namespace

hipError_t launch_winner_prologue(const DevState& s, int cur, int32_t n, int32_t m,
                                  const int32_t* winner, const int32_t* second,
                                  const uint8_t* accepted, int64_t slack_cap, hipStream_t st) {
  const int nxt = cur ^ 1;
  wl_prepare<<<blocks(m), kBlock, 0, st>>>(m, n, winner, second, accepted, s.pend, s.extra,
                                           s.rem, s.status);
  const int nb = blocks(n);
  wl_count<<<nb, kBlock, 0, st>>>(n, s.rp[cur], nullptr, s.extra, s.cnt, s.bsum);
  hipError_t e = launch_scan_blocks(s.bsum, nb, slack_cap, s.rp[nxt] + n, s.status, -1, st);
  if (e != hipSuccess) return e;
  wl_write<<<nb, kBlock, 0, st>>>(n, s.rp[cur], nullptr, s.col[cur], s.age[cur], s.cnt, s.bsum,
                                  s.rp[nxt], s.col[nxt], s.age[nxt], s.len, nullptr, 1.0f,
                                  s.status);
  return hipGetLastError();
}

hipError_t launch_winner_rounds(const DevState& s, int cur, int32_t n, const float* sig,
                                int32_t m, const int32_t* winner, const int32_t* second,
                                const float* d1, int key_mode, float eps_b, float eps_n,
                                int32_t max_age, int64_t t0, int count, hipStream_t st) {
  (void)n;
  const int nxt = cur ^ 1;
  const int g = blocks(m);
  for (int i = 0; i < count; ++i) {
    const int64_t t = t0 + i;
    const int32_t slot = static_cast<int32_t>(t % kRing);
    const int32_t prev = static_cast<int32_t>((t + kRing - 1) % kRing);
    const int force = t == 0;
    wl_claim<<<g, kBlock, 0, st>>>(m, winner, second, d1, key_mode, s.pend, s.rp[nxt], s.len,
                                   s.col[nxt], s.lock, s.rem, slot, prev, force);
    wl_check<<<g, kBlock, 0, st>>>(m, winner, second, d1, key_mode, s.pend, s.rp[nxt], s.len,
                                   s.col[nxt], s.lock, s.rem, slot, prev, force);
    wl_apply<<<g, kBlock, 0, st>>>(sig, m, winner, second, d1, s.pend, s.rp[nxt], s.len,
                                   s.col[nxt], s.age[nxt], s.x, s.y, s.z, s.err, s.orphan,
                                   s.status, eps_b, eps_n, max_age, s.rem, prev, force);
  }
  return hipGetLastError();
}

hipError_t launch_winner_epilogue(const DevState& s, int cur, int32_t n, float beta,
                                  int64_t half_cap, hipStream_t st) {
  const int nxt = cur ^ 1;
  const int nb = blocks(n);
  wl_count<<<nb, kBlock, 0, st>>>(n, s.rp[nxt], s.len, nullptr, s.cnt, s.bsum);
  hipError_t e = launch_scan_blocks(s.bsum, nb, half_cap, s.rp[cur] + n, s.status, -1, st);
  if (e != hipSuccess) return e;
  wl_write<<<nb, kBlock, 0, st>>>(n, s.rp[nxt], s.len, s.col[nxt], s.age[nxt], s.cnt, s.bsum,
                                  s.rp[cur], s.col[cur], s.age[cur], nullptr, s.err, beta,
                                  s.status);
  return hipGetLastError();
}

}  // namespace gsn
