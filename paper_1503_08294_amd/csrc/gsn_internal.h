// Internal declarations shared by the HIP translation units of libgsn.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "../../include/gsn.h"

namespace gsn {

constexpr int kBlock = 256;            // threads per workgroup of the per-unit kernels
constexpr int kMaxSplit = GSN_MAX_SPLIT;
constexpr int kSmallM = 256;           // batches up to this size may take the small-batch scan
constexpr int kSmallRows = 1024;       // its partial rows (workgroups) at most
constexpr int32_t kDead = -1;          // age marking a half-edge removed this iteration

// An event pair bound to one kernel launch: the runtime sets start and stop from the
// kernel's own start and end (hipExtLaunchKernel), which excludes the end-of-kernel cache
// flush and adds no marker to the stream.  Both null: a plain launch.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};

template <typename... KArgs, typename... Args>
inline void launch_with(void (*k)(KArgs...), dim3 grid, dim3 block, hipStream_t st,
                        LaunchEvents ev, Args... args) {
  if (ev.start != nullptr && ev.stop != nullptr)
    hipExtLaunchKernelGGL(k, grid, block, 0, st, ev.start, ev.stop, 0,
                          static_cast<KArgs>(args)...);
  else
    k<<<grid, block, 0, st>>>(static_cast<KArgs>(args)...);
}

// Sticky status word layout (int32 slots in the status area).
enum StatusSlot {
  kStError = 0,       // first error code raised by a kernel (0 = none)
  kStOrphans = 1,     // units marked for removal since the last grow
  kStAbort = 2,       // 1 once the CSR rewrite overflowed (rows are then not written)
  kStInserted = 3,    // grow: 1 if the last insertion added a unit
  kStKept = 4,        // grow: units kept by the last compaction
  kStSlots = 16
};

// Counters of the sequential-survivor update and the greedy resolve (int32 words of
// DevState::rem): round statistics accumulated until the host clears them, then spread
// counters (below) for the signals still pending after each grid-wide round and for the
// survivors of the current call.
constexpr int kMaxGridRounds = 32;
enum RoundSlot {
  kRmRounds,       // rounds summed over the updates since the last clear
  kRmRoundsMax,    // the most rounds one update took
  kRmUpdates,      // updates since the last clear
  kRmGridUsed,     // grid-wide rounds that did work in the last update
  kRmSlots
};
// A spread counter: kSpreadParts words, one per 128-byte line, so that the workgroups of a
// grid-wide launch add to it without queueing at one address (device-scope atomics on one
// word are serialized: ~2,000 workgroups adding to one word cost a round tens of
// microseconds); its value is the sum of the parts.
constexpr int kSpreadParts = 64;
constexpr int kSpreadStride = 32;  // int32 words from one part to the next
constexpr int kSpreadWords = kSpreadParts * kSpreadStride;
constexpr int kRmSpread = 32;      // first word of the spread counters (past the slots)
static_assert(kRmSlots <= kRmSpread, "round slots overlap the spread counters");
// round t's pending count, and the survivors of the current update
__host__ __device__ constexpr int rm_round(int t) { return kRmSpread + t * kSpreadWords; }
constexpr int kRmSurvivors = rm_round(kMaxGridRounds);
constexpr int kRmWords = kRmSurvivors + kSpreadWords;
// A grid-wide round is skipped, and its signals left to the single-workgroup rounds, once
// fewer than this many survivors are pending (a round of the single workgroup, whose claims
// and checks share a launch and so use device-scope atomics, costs about as much as a
// grid-wide round with a few dozen survivors).
constexpr int kTailMin = 32;

// 64-bit accumulators (DevState::acc64).
enum Acc64Slot {
  kA64Window = 0,    // error window of the schedule: sum of floor(d1 * 2^32)
  kA64Resolved = 1,  // signals through resolve since the last statistics clear
  kA64Accepted = 2,  // of those, accepted
  kA64Slots = 4
};

__device__ __forceinline__ void raise_error(int32_t* status, int32_t code) {
  atomicCAS(&status[kStError], 0, code);
}

__device__ __forceinline__ bool pair_ok(int32_t b, int32_t s, int32_t n) {
  return b >= 0 && b < n && s >= 0 && s < n && b != s;
}

// Priority of signal j among the signals that collide (smaller wins): key_mode 0 orders by
// the winner distance, then the index; key_mode 1 by the index alone.
__device__ __forceinline__ unsigned long long signal_key(float d1, int32_t j, int key_mode) {
  const unsigned long long lo = static_cast<uint32_t>(j);
  if (key_mode == 1) return lo;
  return (static_cast<unsigned long long>(__float_as_uint(d1)) << 32) | lo;
}

// Adds the threads of this workgroup for which `pred` holds to *ctr with one atomic per
// workgroup (same-address atomics from thousands of waves queue up at the cache).  Every
// thread of the workgroup calls it (it holds a barrier); `acc` is an LDS word that was
// zeroed before an earlier barrier.
template <typename T>
__device__ __forceinline__ void block_count(bool pred, T* ctr, int32_t* acc) {
  const unsigned long long mask = __ballot(pred);
  if ((threadIdx.x & 63) == 0 && mask != 0)
    atomicAdd(acc, static_cast<int32_t>(__popcll(mask)));
  __syncthreads();
  if (threadIdx.x == 0 && *acc != 0) atomicAdd(ctr, static_cast<T>(*acc));
}

// Claims the units col[r0, r0 + l) with an atomic minimum of key, eight entries per batch of
// loads (slots past the row's end repeat its last entry): the claims of a row wait for one
// round of loads per eight entries rather than one per entry.
__device__ __forceinline__ void claim_row(unsigned long long* lock, const int32_t* col,
                                          int32_t r0, int32_t l, unsigned long long key) {
  for (int32_t k0 = 0; k0 < l; k0 += 8) {
    const int32_t n = min(8, l - k0);
    int32_t c[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) c[k] = col[r0 + k0 + min(k, n - 1)];
#pragma unroll
    for (int k = 0; k < 8; ++k)
      if (k < n) atomicMin(&lock[c[k]], key);
  }
}

// The same into the part blockIdx.x mod kSpreadParts of the spread counter at ctr.
__device__ __forceinline__ void block_count_spread(bool pred, int32_t* ctr, int32_t* acc) {
  block_count(pred, ctr + static_cast<int>(blockIdx.x % kSpreadParts) * kSpreadStride, acc);
}

// The value of the spread counter at ctr, in every lane of the calling wave (lane l reads
// part l).  For a counter written by earlier launches.
__device__ __forceinline__ int32_t spread_value(const int32_t* ctr) {
  static_assert(kSpreadParts == 64, "one part per lane");
  int32_t v = ctr[static_cast<int>(threadIdx.x & 63) * kSpreadStride];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Zeroes the spread counter at ctr: thread tid < kSpreadParts clears part tid.
__device__ __forceinline__ void spread_clear(int32_t* ctr, int tid) {
  if (tid < kSpreadParts) ctr[tid * kSpreadStride] = 0;
}

// Sum of v over a kBlock workgroup, valid in every thread: wave shuffles, then the wave
// totals through LDS (wt holds kBlock / 64 words; one barrier before it may be reused).
__device__ __forceinline__ int32_t block_sum(int32_t v, int32_t* wt) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if ((threadIdx.x & 63) == 0) wt[threadIdx.x >> 6] = v;
  __syncthreads();
  int32_t t = 0;
#pragma unroll
  for (int w = 0; w < kBlock / 64; ++w) t += wt[w];
  return t;
}

// Inclusive prefix sum of v over a kBlock workgroup in thread order: a shuffle scan per
// wave, then the totals of the earlier waves through LDS (one barrier).
__device__ __forceinline__ int32_t block_inclusive_scan(int32_t v, int32_t* wt) {
  const int lane = static_cast<int>(threadIdx.x & 63), w = static_cast<int>(threadIdx.x >> 6);
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int32_t x = __shfl_up(v, o);
    if (lane >= o) v += x;
  }
  if (lane == 63) wt[w] = v;
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kBlock / 64; ++k) v += k < w ? wt[k] : 0;
  return v;
}

// A rewrite of per-row counts into offsets (count -> scan of the per-workgroup sums ->
// write) can skip the single-workgroup scan when it has at most kFoldBlocks workgroups:
// each writing workgroup sums the block sums before its own and all of them itself.
constexpr int kFoldBlocks = 2048;

// The sum of bsum[0, blockIdx.x) and of bsum[0, nb).  Every thread of the workgroup calls
// it (it holds a barrier); red is LDS for 2 ints per wave.
__device__ __forceinline__ void fold_offsets(const int32_t* __restrict__ bsum, int32_t nb,
                                             int32_t* red, int32_t* before, int32_t* total) {
  int32_t a = 0, t = 0;
  const int32_t me = static_cast<int32_t>(blockIdx.x);
  const int32_t bd = static_cast<int32_t>(blockDim.x), tid = static_cast<int32_t>(threadIdx.x);
  if (nb > 0 && nb <= 8 * bd) {
    // up to eight sums per thread in one batch of loads (indices past nb repeat the last)
    int32_t v[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) v[r] = bsum[min(tid + r * bd, nb - 1)];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int32_t i = tid + r * bd;
      const int32_t x = i < nb ? v[r] : 0;
      t += x;
      a += i < me ? x : 0;
    }
  } else {
    for (int32_t i = tid; i < nb; i += bd) {
      const int32_t v = bsum[i];
      t += v;
      a += i < me ? v : 0;
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    a += __shfl_xor(a, o);
    t += __shfl_xor(t, o);
  }
  const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    red[w] = a;
    red[nw + w] = t;
  }
  __syncthreads();
  a = 0;
  t = 0;
  for (int k = 0; k < nw; ++k) {
    a += red[k];
    t += red[nw + k];
  }
  *before = a;
  *total = t;
}

// The capacity decision of a folded rewrite, the same in every workgroup: a total above cap
// (or an abort flagged earlier) aborts it; workgroup 0 records the error and writes the
// total, or 0 once aborted, to *out_total (if not null), as the block-sum scan would.
__device__ __forceinline__ bool fold_abort(int32_t total, int64_t cap, int32_t* status,
                                           int32_t* out_total) {
  const bool over = static_cast<int64_t>(total) > cap;
  const bool abort = over || status[kStAbort] != 0;
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    if (over) {
      status[kStAbort] = 1;
      atomicCAS(&status[kStError], 0, GSN_E_CAPACITY);
    }
    if (out_total) *out_total = abort ? 0 : total;
  }
  return abort;
}

// w <- w + eps (xi - w), one binary32 rounding per operation (no contraction).
__device__ __forceinline__ void move_unit(float* __restrict__ x, float* __restrict__ y,
                                          float* __restrict__ z, int32_t u, float eps,
                                          float sx, float sy, float sz) {
  float t;
  t = sx - x[u]; t = eps * t; x[u] = x[u] + t;
  t = sy - y[u]; t = eps * t; y[u] = y[u] + t;
  t = sz - z[u]; t = eps * t; z[u] = z[u] + t;
}

// Device arrays carved out of the caller's workspace.
struct DevState {
  float *x, *y, *z, *err;          // [n_max]
  int32_t* rp[2];                  // [n_max + 2]   row pointers, ping-pong
  int32_t* col[2];                 // [2 e_max + 2] neighbour ids, ping-pong (2 (e_max +
  int32_t* age[2];                 //  m_max) + 2 with the winner lock); ages, ping-pong
  unsigned long long* lock;        // [n_max]       packed (d1 bits, signal) claims
  int32_t* ins;                    // [n_max]       partner of a new edge, -1 = none
  int32_t* orphan;                 // [n_max]       1 = last edge removed by aging
  int32_t* cnt;                    // [n_max]       per-unit scratch counts / new ids
  int32_t* bsum;                   // [n_max / kBlock + 2] per-block sums / offsets
  int32_t* bdelta[2];              // [n_max / kBlock + 2] each: change of the half-edge count
                                   // of every block of kBlock units in this update (+1 per
                                   // requested edge, -1 per half-edge marked dead); the
                                   // update uses one and zeroes the other for the next
  float* tmp;                      // [4 n_max]     compaction staging
  int32_t* status;                 // [kStSlots]
  unsigned long long* part;        // [kMaxSplit][2][m_max] per-chunk top-2 keys
  unsigned long long* spart;       // [small_part_keys(m_max)] partial keys of the small-batch
                                   // scan: [2 kSmallRows][slots]
  void* scr;                       // staging area of the screened scans (staging.hip)
  // sequential-survivor update (winner lock)
  uint8_t* pend;                   // [m_max]       1 pending survivor, 0 otherwise
  int32_t* len;                    // [n_max]       live length of every row of the slack CSR
  int32_t* extra;                  // [n_max]       insertions a row may receive (kept zero)
  int32_t* rem;                    // [kRmWords]    round counters (RoundSlot, rm_round)
  int32_t* list;                   // [2 m_max]     pending signals of the last rounds
  // one-pass update of the winner-lock survivors (winner lock only; null otherwise): two
  // parities of survivor tables, parity q at offset q n_max, taken by successive updates in
  // turn
  unsigned long long* wkey;        // [2 n_max][2]  per unit: the key of the survivor it is the
                                   //               winner of (all ones for none), and that
                                   //               survivor's second (one 16-byte record)
  uint8_t* wflag;                  // [2 n_max]     1 iff the unit has a survivor record: read
                                   //               first, so that the records of the many
                                   //               units without one are not fetched
  int32_t* rhead;                  // [2 n_max]     a survivor whose second is the unit, -1 none
  int32_t* rnext;                  // [m_max]       the next survivor with the same second
  int32_t* whi;                    // [2]           tables of parity q hold entries below whi[q]
  // growing-network schedule
  float* ssig;                     // [3 m_max]     signals of the iteration, SoA
  int32_t *swin, *ssec;            // [m_max]
  float *sd1, *sd2;                // [m_max]
  uint8_t* sacc;                   // [m_max]
  unsigned long long* acc64;       // [kA64Slots]   64-bit accumulators (Acc64Slot)
  int32_t* apart;                  // [m_max / 32 + 2] accepted signals per workgroup of the
                                   // fused check, added to acc64 by the next degree count
};

struct Layout {
  size_t off[40];
  size_t total;
};

Layout layout_for(const gsn_params& p);
void carve(const gsn_params& p, void* base, DevState* s);

// ---------------------------------------------------------------- launchers ----
// Every launcher enqueues on `stream` and returns the hipGetLastError() of its launches.

struct FindConfig {
  int variant;   // 1 = direct scan, 2 = screened scan (VALU), 3 = screened scan (MFMA),
                 // 4 = screened scan (split binary16 MFMA), 5 = variant 4 with dynamic grabs,
                 // 6 = small-batch unit-parallel scan
  int split;     // unit chunks (variant 5: partial rows, 8 per replica)
};
FindConfig find_config(int32_t n, int32_t m, int cus, int want_split, int want_variant);

hipError_t launch_find_scan(const DevState& s, int32_t n, const float* sig, int32_t m,
                            const FindConfig& cfg, int32_t* winner, int32_t* second,
                            float* d1, float* d2, hipStream_t st, LaunchEvents ev = {});
hipError_t launch_find_merge(const DevState& s, int32_t m, const FindConfig& cfg,
                             int32_t* winner, int32_t* second, float* d1, float* d2,
                             hipStream_t st);

// Small-batch find winners (find_small.hip): unit-parallel, no staging, for
// 1 <= m <= kSmallM (variant 6).  slots = the smallest power of two >= m.
int32_t small_slots(int32_t m);
int32_t small_rows(int32_t n, int32_t m);
size_t small_part_keys(int32_t m_max);
hipError_t launch_find_small_scan(const DevState& s, int32_t n, const float* sig, int32_t m,
                                  hipStream_t st, LaunchEvents ev = {});
struct ClaimArgs;
hipError_t launch_find_small_merge(const DevState& s, int32_t n, int32_t m, int32_t* winner,
                                   int32_t* second, float* d1, float* d2,
                                   const ClaimArgs* claim, hipStream_t st);

// Spatial staging of the screened scans (staging.hip).
constexpr int kBuckets = 32 * 32 * 32;

struct StageBufs {
  float4* pu;       // [ceil64(n_max)] units in bucket order: (x, y, z, |w|^2); slots from n
                    // to the end of the last batch hold stale values
  int32_t* pidx;    // [ceil64(n_max)] original index of every sorted slot (same padding)
  int32_t* ukey;    // [n_max] bucket of every unit at the last bucketing
  int32_t* skey;    // [m_max] bucket of every signal
  int32_t* sperm;   // [m_max] original index of the signal at every sorted position
  float* seed;      // [m_max] seed bound B at every sorted position
  float* ssig;      // [3][m] the signals in sorted order (x, y, z rows of stride m)
  int32_t* stk;     // [m_max] rank of every signal inside its histogram bin (the ticket its
                    // count increment returned)
  int32_t *hist_u, *off_u, *cur_u, *hist_s;  // [kBuckets + 1] each; the signal histogram
                    // uses two sets of kBuckets / 8 in hist_s
  int32_t* acc;     // [16] bounding-box accumulators
  float* bb;        // [8] grid of the last unit bucketing: lo.xyz, cells per length.xyz
  int32_t* mag;     // [4] max |x|, |y|, |z|, |w|^2 of this call (float bits)
  float* bmag;      // [n_max / kBlock + 2][4] per-block magnitude maxima
  float* pm;        // [ceil(n_max / 64) * 256] units in matrix-core operand order
  uint4* pmh;       // [ceil(n_max / 64)][64 lanes][2 groups] scaled units split into binary16
                    // pairs, in the operand order of the 32x32x16 f16 product (16 B each)
  int32_t* wctr;    // [wctr_count(m_max)] grab counters of the dynamic scan, zeroed by the
                    // seed kernel of every call: 8 lists per 64-signal block
};
// 8 counters per 64-signal block, for whole blocks of 256 signals
inline int32_t wctr_count(int32_t m) { return 32 * ((m + 255) / 256); }
size_t stage_bytes(int32_t n_max, int32_t m_max);
StageBufs carve_stage(void* base, int32_t n_max, int32_t m_max);
hipError_t launch_stage_init(const StageBufs& b, hipStream_t st);
// units n0 .. n1 - 1 appended to the spatial order (older indices unchanged)
hipError_t launch_stage_append(const StageBufs& b, int32_t n0, int32_t n1, hipStream_t st);
// parity alternates between calls (two sets of signal histogram and cursors)
hipError_t launch_stage(const DevState& s, const StageBufs& b, int32_t n, const float* sig,
                        int32_t m, bool rebucket, int parity, int variant, hipStream_t st);
// The lock-set claims of the fused iteration, made by the merge once a signal's winner and
// second are known (claim = nullptr: the merge only merges).
struct ClaimArgs {
  int32_t n;
  const int32_t* rp;
  const int32_t* col;
  unsigned long long* lock;
  int32_t* status;
  int key_mode;
  int winner_only;  // the winner-lock rule's claim: the winner alone
  uint8_t* pend;    // greedy rule (round 0 of its resolve): each signal's state, 1 pending,
                    // 0 for an invalid pair (null otherwise)
};
hipError_t launch_stage_merge(const DevState& s, const StageBufs& b, int32_t m, int split,
                              int32_t* winner, int32_t* second, float* d1, float* d2,
                              const ClaimArgs* claim, hipStream_t st);
int screened_split(int32_t n, int32_t m, int cus, int want);
hipError_t launch_scan_screened(const DevState& s, const StageBufs& b, int32_t n,
                                const float* sig, int32_t m, int split, hipStream_t st,
                                LaunchEvents ev = {});
int mfma_split(int32_t n, int32_t m, int cus, int want);
int f16_split(int32_t n, int32_t m, int cus, int want);
hipError_t launch_scan_f16(const DevState& s, const StageBufs& b, int32_t n, const float* sig,
                           int32_t m, int split, hipStream_t st, LaunchEvents ev = {});
// variant 5: split = 8 x replicas (a multiple of 8), grab = list entries per atomic
int f16_dyn_split(int32_t m, int cus, int want);
hipError_t launch_scan_f16_dyn(const DevState& s, const StageBufs& b, int32_t n, int32_t m,
                               int split, int grab, hipStream_t st, LaunchEvents ev = {});
hipError_t launch_scan_mfma(const DevState& s, const StageBufs& b, int32_t n, const float* sig,
                            int32_t m, int split, hipStream_t st, LaunchEvents ev = {});

// The survivor tables of the one-pass winner-lock update (launch_winner_local) of parity par.
struct WinnerTables {
  unsigned long long* wkey;
  uint8_t* wflag;
  int32_t* rhead;
  int32_t* rnext;
  int32_t* whi;
  int par;
};
WinnerTables winner_tables(const DevState& s, int par, int32_t n_max);

// lock_mode: 0 = lock set {b, s} + N(b), 1 = the winner alone; key_mode: 0 = (d1 bits,
// index), 1 = index.  With tables (winner alone only) the check also fills the survivor
// tables of the one-pass update, which then skips that launch.
// claimed: the find's merge made the claims already.
hipError_t launch_resolve(const DevState& s, int cur, int32_t n, int32_t m,
                          const int32_t* winner, const int32_t* second, const float* d1,
                          uint8_t* accepted, int lock_mode, int key_mode, hipStream_t st,
                          const WinnerTables* tables = nullptr, bool claimed = false);
hipError_t launch_adapt(const DevState& s, int cur, int32_t n, const float* sig, int32_t m,
                        const int32_t* winner, const int32_t* second, const float* d1,
                        const uint8_t* accepted, float eps_b, float eps_n, float beta,
                        hipStream_t st);
// taken (greedy rule): the resolve's taken marks, cleared by the rewrite for the next call.
hipError_t launch_edges(const DevState& s, int cur, int dpar, int32_t n, int32_t m,
                        const int32_t* winner, const int32_t* second,
                        const uint8_t* accepted, int32_t max_age, int64_t half_cap,
                        hipStream_t st, int32_t* taken = nullptr);
// Greedy lock-set resolve (resolve_greedy.hip): rounds of claims over L_j = {b, s} + N(b),
// grid_rounds grid-wide, the rest in one workgroup.  Uses lock, extra (as the taken marks),
// pend (signal states), rem and list.
// claimed: the find's merge made the first round's claims and set the signal states (the
// lock words are all ones and the taken marks zero between calls, so there is no set-up
// launch).
hipError_t launch_resolve_greedy(const DevState& s, int cur, int32_t n, int32_t m,
                                 const int32_t* winner, const int32_t* second, const float* d1,
                                 uint8_t* accepted, int key_mode, int grid_rounds,
                                 hipStream_t st, bool claimed = false);

// The sequential-survivor update (update_winner.hip), all enqueued without a host sync:
// the slack copy of the CSR in buffer cur ^ 1, grid_rounds grid-wide rounds, the remaining
// rounds in one workgroup, and the compact CSR back in buffer cur with the error decay.
// half_cap bounds the compact adjacency, slack_cap the slack copy.
struct WinnerStep {
  const float* sig;
  int32_t m;
  const int32_t* winner;
  const int32_t* second;
  const float* d1;
  const uint8_t* accepted;
  int key_mode;
  float eps_b, eps_n, beta;
  int32_t max_age;
  int grid_rounds;   // 0..kMaxGridRounds
  int64_t slack_cap, half_cap;
  int32_t* feedback; // pinned host word (device address) that receives the grid rounds used
  int32_t n_max;     // (the one-pass update: the stride of the table parities)
};
hipError_t launch_winner_update(const DevState& s, int cur, int32_t n, const WinnerStep& w,
                                hipStream_t st);
// The same update in two launches after the winner-lock resolve, whose check (launch_resolve
// with the tables of parity par) leaves one survivor per winner and fills the survivor
// tables: the moves with the new degrees, and the rows, written into buffer cur ^ 1 with the
// error decay (grid_rounds and feedback are not used).  Consecutive calls must alternate
// par.
hipError_t launch_winner_local(const DevState& s, int cur, int par, int32_t n,
                               const WinnerStep& w, hipStream_t st);
// The lock-set resolve, adaptation and edge update of one iteration: the claims (unless the
// find's merge made them, claimed = true); the check fused with the accepted signals'
// updates, taking the signals in the given order when order is not null (a permutation of
// 0..m-1, e.g. the staging's spatial order); the rewrite into buffer cur ^ 1 with the error
// decay (one launch up to kFoldBlocks blocks of units, else degree count, scan and write).
// With given (the acceptance of the greedy resolve, whose accepted lock sets are disjoint
// as well) there are no claims and no check: the accepted signals are applied.
hipError_t launch_iterate_set(const DevState& s, int cur, int dpar, int32_t n, const float* sig,
                              int32_t m, const int32_t* winner, const int32_t* second,
                              const float* d1, uint8_t* accepted, int key_mode, float eps_b,
                              float eps_n, float beta, int32_t max_age, int64_t half_cap,
                              bool claimed, const int32_t* order, hipStream_t st,
                              const uint8_t* given = nullptr);
hipError_t launch_scan_blocks(int32_t* bsum, int32_t nb, int64_t cap, int32_t* out_total,
                              int32_t* status, int32_t slot, hipStream_t st);
hipError_t launch_init(const DevState& s, int cur, int32_t n0, int32_t n_max,
                       hipStream_t st);
hipError_t launch_remove(const DevState& s, int cur, int32_t n, int32_t n_max,
                         hipStream_t st);
// Indexed find winners (find_grid.hip): the grid and the caller's grid workspace.
struct GridSpec {
  float lo[3];
  float inv_h;       // 1 / h rounded to binary32 (the cell function multiplies by it)
  int32_t dims[3];
  int64_t cells;
  int exact;         // certify the 27-cube result, else the exhaustive search
};
struct GridBufs {
  int32_t* cnt;      // [cells + 1] units per cube, then scatter cursors
  int32_t* start;    // [cells + 1] first sorted slot of every cube
  int32_t* bsum;     // [cells / kBlock + 2]
  float4* sorted;    // [n_max] units by cube: (x, y, z, index bits)
  int32_t* ucell;    // [n_max] cube of every unit
  int32_t* fb_list;  // [m_max] signals that fell back to the exhaustive search
  int32_t* nfb;      // their count
};
size_t grid_bytes(int64_t cells, int32_t n_max, int32_t m_max);
GridBufs carve_grid(void* base, int64_t cells, int32_t n_max, int32_t m_max);
hipError_t launch_find_grid(const DevState& s, const GridBufs& gb, const GridSpec& spec,
                            int32_t n, const float* sig, int32_t m, int32_t* winner,
                            int32_t* second, float* d1, float* d2, hipStream_t st);

// Schedule kernels (schedule.hip): draw m signals (signal numbers c0 + 1 .. c0 + m) from
// the cloud, and add the winners' distances of m signals to the error window.
hipError_t launch_draw(const float* cloud, int64_t n_points, uint64_t seed, int64_t c0,
                       int32_t m, float* sig, hipStream_t st);
hipError_t launch_qe(const float* d1, int32_t m, unsigned long long* acc, hipStream_t st);
// Up to `count` GNG insertions one after another; status[kStInserted] receives how many.
hipError_t launch_insert(const DevState& s, int cur, int32_t n, int32_t count, float alpha,
                         int32_t n_max, int64_t half_cap, hipStream_t st);

}  // namespace gsn
