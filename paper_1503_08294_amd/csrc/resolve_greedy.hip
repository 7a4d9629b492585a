// Greedy lock-set resolve (lock_mode 2): the lock sets L_j = {b_j, s_j} + N(b_j) of the
// lock-set reading of Sec. 2.2, with the signals taken in key order: j is accepted iff L_j
// is disjoint from the lock sets accepted before it.  Computed in rounds: every pending
// signal claims L_j with a 64-bit atomic minimum of its key; a signal that finds a unit of
// L_j taken by an accepted signal is rejected; one that holds all of L_j is accepted and
// marks its units taken; the others stay pending.  A signal is settled once every signal of
// smaller key whose lock set meets L_j is settled, exactly as in the sequential greedy
// order, so the result is that order's; the pending signal of smallest key is always
// settled, so every round makes progress.  The first rounds are grid-wide launches, the
// rest run in one workgroup (as for the winner-lock update).
#include "gsn_internal.h"

namespace gsn {
namespace {

constexpr int kRoundBlock = 256;
constexpr int kTailBlock = 1024;

inline int blocks(int64_t n) { return static_cast<int>((n + kBlock - 1) / kBlock); }

// Lock words in the checks.  The single-workgroup rounds claim and check in one launch, so
// their checks read atomically (the claims' minima are made at device scope); a grid-wide
// check reads words the claims of an earlier launch left (kernel boundaries make them
// visible to plain loads) while the only writes are releases by the holders, so plain
// loads and stores serve there: a stale word reads as its claimed key or as all ones, and
// only the signal that held it at the end of the claims sees its own key.
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

struct GreedyArgs {
  int32_t m, n;
  const int32_t* winner;
  const int32_t* second;
  const float* d1;
  int key_mode;
  const int32_t* rp;
  const int32_t* col;
  unsigned long long* lock;
  int32_t* taken;      // 1: unit of an accepted lock set
  uint8_t* state;      // 0 rejected, 1 pending, 2 accepted
  int32_t* rem;
  int32_t* list;
  int32_t* status;
  unsigned long long* acc64;
};

// Rows of up to this many entries (nearly all of them) are read in one batch of loads
// (indices past the row's end repeat its last entry and are ignored).
constexpr int kShortRow = 8;

__device__ void g_claim(const GreedyArgs& a, int32_t j) {
  const int32_t b = a.winner[j], s = a.second[j];
  const unsigned long long key = signal_key(a.d1[j], j, a.key_mode);
  atomicMin(&a.lock[b], key);
  atomicMin(&a.lock[s], key);
  const int32_t r0 = a.rp[b];
  claim_row(a.lock, a.col, r0, a.rp[b + 1] - r0, key);
}
// Visits b, its neighbours and s (once, when it is no neighbour): a unit taken by an
// accepted signal blocks j for good; j holds the units whose lock word has its key and
// releases them.  For a short row the lock and taken words of all of them are read in one
// round (the units are distinct, another signal only ever clears a word holding its own key,
// and a taken mark seen a round later only delays the same rejection).
template <bool kGrid>
__device__ uint8_t g_check(const GreedyArgs& a, int32_t j) {
  const int32_t b = a.winner[j], s = a.second[j];
  const unsigned long long key = signal_key(a.d1[j], j, a.key_mode);
  bool blocked = false, holds = true;
  auto visit = [&](int32_t u) {
    blocked |= a.taken[u] != 0;
    if (lock_read<kGrid>(&a.lock[u]) == key) lock_release<kGrid>(&a.lock[u]); else holds = false;
  };
  const int32_t r0 = a.rp[b], r1 = a.rp[b + 1], l = r1 - r0;
  if (l > kShortRow || l <= 0) {
    visit(b);
    bool s_nb = false;
    for (int32_t k = r0; k < r1; ++k) {
      const int32_t v = a.col[k];
      s_nb |= v == s;
      visit(v);
    }
    if (!s_nb) visit(s);
  } else {
    int32_t c[kShortRow];
#pragma unroll
    for (int k = 0; k < kShortRow; ++k) c[k] = a.col[r0 + min(k, l - 1)];
    bool s_nb = false;
#pragma unroll
    for (int k = 0; k < kShortRow; ++k) s_nb |= k < l && c[k] == s;
    const bool tb = a.taken[b] != 0, ts = a.taken[s] != 0;
    const unsigned long long lb = lock_read<kGrid>(&a.lock[b]), ls = lock_read<kGrid>(&a.lock[s]);
    bool tk[kShortRow];
    unsigned long long lk[kShortRow];
#pragma unroll
    for (int k = 0; k < kShortRow; ++k) {
      tk[k] = a.taken[c[k]] != 0;
      lk[k] = lock_read<kGrid>(&a.lock[c[k]]);
    }
    auto decide = [&](int32_t u, bool t, unsigned long long w) {
      blocked |= t;
      if (w == key) lock_release<kGrid>(&a.lock[u]); else holds = false;
    };
    decide(b, tb, lb);
#pragma unroll
    for (int k = 0; k < kShortRow; ++k)
      if (k < l) decide(c[k], tk[k], lk[k]);
    if (!s_nb) decide(s, ts, ls);
  }
  if (blocked) return 0;
  if (!holds) return 1;
  a.taken[b] = 1;
  a.taken[s] = 1;
  for (int32_t k = r0; k < r1; ++k) a.taken[a.col[k]] = 1;
  return 2;
}

__global__ void rg_init(GreedyArgs a) {
  const int32_t i = blockIdx.x * kBlock + threadIdx.x;
  if (i < a.n) {
    a.lock[i] = ~0ull;
    a.taken[i] = 0;
  }
  if (i < a.m) {
    const bool ok = pair_ok(a.winner[i], a.second[i], a.n);
    if (!ok) raise_error(a.status, GSN_E_INVAL);
    a.state[i] = ok ? 1 : 0;
  }
}

// Grid-wide round t; the spread counter rm_round(t) counts the signals left pending; rounds
// after one that left fewer than kTailMin return at once.
__global__ void rg_claim(GreedyArgs a, int32_t t) {
  if (blockIdx.x == 0) spread_clear(a.rem + rm_round(t), threadIdx.x);
  if (t > 0 && spread_value(a.rem + rm_round(t - 1)) < kTailMin) return;
  const int32_t j = blockIdx.x * kRoundBlock + threadIdx.x;
  if (j < a.m && a.state[j] == 1) g_claim(a, j);
}

__global__ void rg_check(GreedyArgs a, int32_t t) {
  // (the same for every wave: the counter was written by earlier launches)
  if (t > 0 && spread_value(a.rem + rm_round(t - 1)) < kTailMin) return;
  __shared__ int32_t s_left;
  if (threadIdx.x == 0) s_left = 0;
  __syncthreads();
  const int32_t j = blockIdx.x * kRoundBlock + threadIdx.x;
  bool left = false;
  if (j < a.m && a.state[j] == 1) {
    const uint8_t st = g_check<true>(a, j);
    a.state[j] = st;
    left = st == 1;
  }
  block_count_spread(left, a.rem + rm_round(t), &s_left);
}

// The remaining rounds in one workgroup, then the acceptance flags of all signals (and
// their counts in the statistics).
__global__ __launch_bounds__(kTailBlock) void rg_tail(GreedyArgs a, uint8_t* accepted) {
  __shared__ int32_t s_n, s_next;
  const int tid = threadIdx.x;
  if (tid == 0) {
    s_n = 0;
    s_next = 0;
  }
  __syncthreads();
  int32_t* cur = a.list;
  int32_t* nxt = a.list + a.m;
  for (int32_t j = tid; j < a.m; j += kTailBlock)
    if (a.state[j] == 1) cur[atomicAdd(&s_n, 1)] = j;
  __syncthreads();
  for (;;) {
    const int32_t n = s_n;
    if (n == 0) break;
    for (int32_t i = tid; i < n; i += kTailBlock) g_claim(a, cur[i]);
    __syncthreads();
    for (int32_t i = tid; i < n; i += kTailBlock) a.state[cur[i]] = g_check<false>(a, cur[i]);
    __syncthreads();
    for (int32_t i = tid; i < n; i += kTailBlock)
      if (a.state[cur[i]] == 1) nxt[atomicAdd(&s_next, 1)] = cur[i];
    __syncthreads();
    if (tid == 0) {
      if (s_next == n) {  // no progress: the lock words were not cleared on entry
        raise_error(a.status, GSN_E_STATE);
        s_next = 0;
      }
      s_n = s_next;
      s_next = 0;
    }
    __syncthreads();
    int32_t* t = cur;
    cur = nxt;
    nxt = t;
  }
  // the counts with one atomic each (hundreds of same-address atomics would queue at the
  // cache)
  __shared__ int32_t s_acc;
  if (tid == 0) s_acc = 0;
  __syncthreads();
  int32_t mine = 0;
  for (int32_t j = tid; j < a.m; j += kTailBlock) {
    const bool acc = a.state[j] == 2;
    accepted[j] = acc ? 1 : 0;
    mine += acc;
  }
  for (int o = 32; o > 0; o >>= 1) mine += __shfl_xor(mine, o);
  if ((tid & 63) == 0 && mine != 0) atomicAdd(&s_acc, mine);
  __syncthreads();
  if (tid == 0) {
    atomicAdd(&a.acc64[kA64Resolved], static_cast<unsigned long long>(a.m));
    if (s_acc != 0) atomicAdd(&a.acc64[kA64Accepted], static_cast<unsigned long long>(s_acc));
  }
  // round 0's pending count starts at zero in the next call, whose first claims the find's
  // merge may make (then no launch of this call's kind clears it)
  spread_clear(a.rem + rm_round(0), tid);
}

}  // namespace

hipError_t launch_resolve_greedy(const DevState& s, int cur, int32_t n, int32_t m,
                                 const int32_t* winner, const int32_t* second, const float* d1,
                                 uint8_t* accepted, int key_mode, int grid_rounds,
                                 hipStream_t st, bool claimed) {
  GreedyArgs a{m, n, winner, second, d1, key_mode, s.rp[cur], s.col[cur], s.lock,
               s.extra, s.pend, s.rem, s.list, s.status, s.acc64};
  if (!claimed) rg_init<<<blocks(std::max(n, m)), kBlock, 0, st>>>(a);
  const int g = static_cast<int>((m + kRoundBlock - 1) / kRoundBlock);
  for (int32_t t = 0; t < grid_rounds; ++t) {
    // (round 0's claims may come from the find's merge; the tail of the previous call left
    // round 0's pending count at zero)
    if (t > 0 || !claimed) rg_claim<<<g, kRoundBlock, 0, st>>>(a, t);
    rg_check<<<g, kRoundBlock, 0, st>>>(a, t);
  }
  rg_tail<<<1, kTailBlock, 0, st>>>(a, accepted);
  return hipGetLastError();
}

}  // namespace gsn
