// Find Winners for small batches (m <= kSmallM signals): a unit-parallel exhaustive
// search with no spatial staging, two launches.
//
// With few signals the signal-parallel scans leave most of the device idle (one signal
// block of lanes) and pay the staging (unit gather, signal bucketing, seed bounds) for
// little work.  Here the parallelism comes from the units instead: T = the smallest power
// of two >= m (at most 256) slots per workgroup, thread t takes slot t mod T (signal
// t mod T, idle past m) and sub-lane q = t div T of Q = 256 / T, and every workgroup owns a
// contiguous chunk of units staged through LDS as float4 tiles.  Thread (slot, q) scans
// the tile entries q, q + Q, ... in ascending index order, evaluating the direct-form
// binary32 distance (the definition: signal minus unit per component, squares summed left
// to right, no contraction; this file is compiled with -ffp-contract=off) and keeping the
// lexicographic top-2 of (d, index) as packed keys (bits(d) << 32) | index, whose unsigned
// order is that order for d >= +0.  The threads of one slot then combine their lists with
// wave shuffles and, across waves, through LDS; each workgroup writes one row pair of
// partial keys per signal, and sm_merge (one workgroup per signal) takes the top-2 of the
// rows.  Sub-lanes and workgroups see disjoint units, so every real key is unique and the
// result is the exhaustive one whatever the chunking.
#include "gsn_internal.h"

namespace gsn {
namespace {

constexpr int kSmallTile = 1024;         // units per LDS tile
constexpr int kSmallPerThread = 16;      // units per thread the chunking aims at (one tile
                                         // per workgroup, so one round of global loads)
constexpr unsigned long long kNone = ~0ull;

__device__ __forceinline__ unsigned long long pack(float d, int32_t i) {
  return (static_cast<unsigned long long>(__float_as_uint(d)) << 32) |
         static_cast<uint32_t>(i);
}

// top-2 of two top-2 lists whose real keys are distinct (kNone may repeat)
__device__ __forceinline__ void merge2(unsigned long long& a1, unsigned long long& a2,
                                       unsigned long long b1, unsigned long long b2) {
  const unsigned long long lo = min(a1, b1), hi = max(a1, b1);
  a2 = min(hi, min(a2, b2));
  a1 = lo;
}

// distance of the second key, +inf while the list holds fewer than two units
__device__ __forceinline__ float second_dist(unsigned long long k2) {
  return k2 == kNone ? __builtin_huge_valf() : __uint_as_float(static_cast<uint32_t>(k2 >> 32));
}

// the direct-form distance of the definition, one binary32 rounding per operation
__device__ __forceinline__ float dist(float sx, float sy, float sz, float4 w) {
  const float dx = sx - w.x;
  const float dy = sy - w.y;
  const float dz = sz - w.z;
  return (dx * dx + dy * dy) + dz * dz;
}

// Enters unit i at distance d into the list.  Units arrive in ascending index order: one at
// the second's distance has a larger index and stays out, so the test is strict but for the
// list of fewer than two units (second_dist reports +inf there, and a unit at +inf distance
// must still enter).
__device__ __forceinline__ void consider(float d, int32_t i, unsigned long long& k1,
                                         unsigned long long& k2, float& d2f) {
  if (d < d2f || (d == d2f && k2 == kNone)) {
    const unsigned long long key = pack(d, i);
    const bool lt1 = key < k1;
    k2 = lt1 ? k1 : key;
    k1 = lt1 ? key : k1;
    d2f = second_dist(k2);
  }
}

__global__ __launch_bounds__(kBlock) void sm_scan(const float* __restrict__ ux,
                                                  const float* __restrict__ uy,
                                                  const float* __restrict__ uz, int32_t n,
                                                  int32_t chunk, const float* __restrict__ sig,
                                                  int32_t m, int32_t T,
                                                  unsigned long long* __restrict__ spart) {
  __shared__ float4 tile[kSmallTile];
  __shared__ unsigned long long r1[4][kSmallM], r2[4][kSmallM];
  const int tid = threadIdx.x;
  const int slot = tid & (T - 1);
  const int Q = kBlock / T;
  const int q = tid / T;
  const bool live = slot < m;
  const float sx = live ? sig[slot] : 0.0f;
  const float sy = live ? sig[m + slot] : 0.0f;
  const float sz = live ? sig[2 * m + slot] : 0.0f;
  unsigned long long k1 = kNone, k2 = kNone;
  float d2f = __builtin_huge_valf();
  const int32_t begin = static_cast<int32_t>(blockIdx.x) * chunk;
  const int32_t end = min(n, begin + chunk);
  for (int32_t t0 = begin; t0 < end; t0 += kSmallTile) {
    const int32_t cnt = min(kSmallTile, end - t0);
    __syncthreads();
    for (int32_t k = tid; k < cnt; k += kBlock)
      tile[k] = make_float4(ux[t0 + k], uy[t0 + k], uz[t0 + k], 0.0f);
    __syncthreads();
    // four entries per step (their loads and distances side by side), then the rest
    int32_t k = q;
    for (; k + 3 * Q < cnt; k += 4 * Q) {
      float4 w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) w[i] = tile[k + i * Q];
      float d[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) d[i] = dist(sx, sy, sz, w[i]);
#pragma unroll
      for (int i = 0; i < 4; ++i) consider(d[i], t0 + k + i * Q, k1, k2, d2f);
    }
    for (; k < cnt; k += Q) consider(dist(sx, sy, sz, tile[k]), t0 + k, k1, k2, d2f);
  }
  // the slot's lists: shuffles inside the wave, then LDS across the waves
  const int span = T < 64 ? T : 64;
  for (int off = span; off < 64; off <<= 1) {
    const unsigned long long o1 = __shfl_xor(k1, off);
    const unsigned long long o2 = __shfl_xor(k2, off);
    merge2(k1, k2, o1, o2);
  }
  const int grp = T < 64 ? 64 : T;            // threads per group holding every slot once
  const int groups = kBlock / grp;
  const int g = tid / grp;
  if (tid % grp < T) {
    r1[g][slot] = k1;
    r2[g][slot] = k2;
  }
  __syncthreads();
  if (tid < T && live) {
    unsigned long long a1 = r1[0][tid], a2 = r2[0][tid];
    for (int h = 1; h < groups; ++h) merge2(a1, a2, r1[h][tid], r2[h][tid]);
    spart[(2 * static_cast<size_t>(blockIdx.x)) * T + tid] = a1;
    spart[(2 * static_cast<size_t>(blockIdx.x) + 1) * T + tid] = a2;
  }
}

// One workgroup per signal: top-2 of the 2 * rows partial keys of its slot.  With do_claim
// (the fused lock-set iteration) the workgroup then makes the signal's claims on its lock set
// {b, s} + N(b), each an atomic minimum of the signal's key, as the staged merge does.
__global__ __launch_bounds__(kBlock) void sm_merge(const unsigned long long* __restrict__ spart,
                                                   int32_t rows, int32_t T,
                                                   int32_t* __restrict__ winner,
                                                   int32_t* __restrict__ second,
                                                   float* __restrict__ d1,
                                                   float* __restrict__ d2, ClaimArgs claim,
                                                   int do_claim) {
  __shared__ unsigned long long s1[kBlock / 64], s2[kBlock / 64];
  const int32_t j = static_cast<int32_t>(blockIdx.x);
  const int tid = threadIdx.x;
  unsigned long long a1 = kNone, a2 = kNone;
  for (int32_t r = tid; r < rows; r += kBlock)
    merge2(a1, a2, spart[(2 * static_cast<size_t>(r)) * T + j],
           spart[(2 * static_cast<size_t>(r) + 1) * T + j]);
  for (int off = 32; off > 0; off >>= 1) {
    const unsigned long long o1 = __shfl_xor(a1, off);
    const unsigned long long o2 = __shfl_xor(a2, off);
    merge2(a1, a2, o1, o2);
  }
  if ((tid & 63) == 0) {
    s1[tid >> 6] = a1;
    s2[tid >> 6] = a2;
  }
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < kBlock / 64; ++w) merge2(a1, a2, s1[w], s2[w]);
    winner[j] = static_cast<int32_t>(static_cast<uint32_t>(a1));
    second[j] = static_cast<int32_t>(static_cast<uint32_t>(a2));
    d1[j] = __uint_as_float(static_cast<uint32_t>(a1 >> 32));
    d2[j] = __uint_as_float(static_cast<uint32_t>(a2 >> 32));
    s1[0] = a1;
    s2[0] = a2;
  }
  if (!do_claim) return;
  __syncthreads();
  const unsigned long long ka = s1[0];
  const int32_t bw = static_cast<int32_t>(static_cast<uint32_t>(ka));
  const int32_t sw = static_cast<int32_t>(static_cast<uint32_t>(s2[0]));
  const bool ok = pair_ok(bw, sw, claim.n);
  if (claim.pend && tid == 0) claim.pend[j] = ok ? 1 : 0;
  if (!ok) {
    if (tid == 0) raise_error(claim.status, GSN_E_INVAL);
    return;
  }
  const unsigned long long key =
      signal_key(__uint_as_float(static_cast<uint32_t>(ka >> 32)), j, claim.key_mode);
  if (tid == 0) {
    atomicMin(&claim.lock[bw], key);
    if (!claim.winner_only) atomicMin(&claim.lock[sw], key);
  }
  if (claim.winner_only) return;
  for (int32_t k = claim.rp[bw] + tid; k < claim.rp[bw + 1]; k += kBlock)
    atomicMin(&claim.lock[claim.col[k]], key);
}

}  // namespace

int32_t small_slots(int32_t m) {
  int32_t t = 1;
  while (t < m) t <<= 1;
  return t;
}

size_t small_part_keys(int32_t m_max) {
  return 2 * static_cast<size_t>(kSmallRows) * small_slots(std::min(m_max, kSmallM));
}

// Units per workgroup: about kSmallPerThread per thread within one tile; more (several
// tiles) only when n needs more than kSmallRows workgroups.
int32_t small_chunk(int32_t n, int32_t m) {
  const int64_t want = std::min<int64_t>(kSmallTile, int64_t{kSmallPerThread} * kBlock / small_slots(m));
  const int64_t floor_rows = (n + int64_t{kSmallRows} - 1) / kSmallRows;   // chunk lower bound
  return static_cast<int32_t>(std::max<int64_t>(1, std::max(want, floor_rows)));
}

int32_t small_rows(int32_t n, int32_t m) {
  const int32_t chunk = small_chunk(n, m);
  return (n + chunk - 1) / chunk;
}

hipError_t launch_find_small_scan(const DevState& s, int32_t n, const float* sig, int32_t m,
                                  hipStream_t st, LaunchEvents ev) {
  if (m < 1 || m > kSmallM || n < 2) return hipErrorInvalidValue;
  const int32_t T = small_slots(m);
  const int32_t chunk = small_chunk(n, m);
  const int32_t rows = (n + chunk - 1) / chunk;
  launch_with(sm_scan, dim3(rows), dim3(kBlock), st, ev, s.x, s.y, s.z, n, chunk, sig, m, T,
              s.spart);
  return hipGetLastError();
}

hipError_t launch_find_small_merge(const DevState& s, int32_t n, int32_t m, int32_t* winner,
                                   int32_t* second, float* d1, float* d2,
                                   const ClaimArgs* claim, hipStream_t st) {
  if (m < 1 || m > kSmallM || n < 2) return hipErrorInvalidValue;
  const ClaimArgs none{};
  sm_merge<<<m, kBlock, 0, st>>>(s.spart, small_rows(n, m), small_slots(m), winner, second,
                                 d1, d2, claim ? *claim : none, claim ? 1 : 0);
  return hipGetLastError();
}

}  // namespace gsn
