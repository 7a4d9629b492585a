// Find Winners (Sec. 2.1 step 2, Sec. 2.2 step 2): exhaustive k = 2 search of every
// signal against every unit, signal-parallel as in the paper's Sec. 2.5 kernel (each lane
// owns signals, unit positions are staged through shared memory and read by all lanes of
// the workgroup at once), re-designed for CDNA4:
//   * wave64 lanes each own S signals (register blocking: one LDS broadcast read of a
//     unit feeds S distance evaluations);
//   * the units are split into chunks scanned by separate workgroups so that even a few
//     thousand signals fill the 256 CUs; every chunk keeps an exact top-2 and a second
//     kernel merges the chunk results;
//   * a (distance, index) pair is packed as the 64-bit key (bits(d) << 32) | index.  For
//     d >= +0 the unsigned order of the key is the lexicographic order of the pair, so the
//     merge is a plain unsigned minimum and the result does not depend on the split.
//
// The distance is evaluated exactly as the definition states, every operation rounded to
// binary32 with no contraction (this file is compiled with -ffp-contract=off).
#include "gsn_internal.h"

namespace gsn {
namespace {

constexpr int kTile = 512;    // units per LDS tile
constexpr int kMinChunk = 512;

__device__ __forceinline__ unsigned long long pack(float d, int32_t i) {
  return (static_cast<unsigned long long>(__float_as_uint(d)) << 32) |
         static_cast<uint32_t>(i);
}

// One workgroup: 256 lanes x S signals against the units [u_begin, u_end) of chunk
// blockIdx.y.  Within a chunk each lane sees units in ascending index order, so a strict
// "<" keeps the lower index on equal distances and the running pair is the exact
// lexicographic top-2 of the units seen.
template <int S>
__global__ __launch_bounds__(kBlock) void fw_scan_direct(
    const float* __restrict__ ux, const float* __restrict__ uy, const float* __restrict__ uz,
    int32_t n, int32_t chunk, const float* __restrict__ sig, int32_t m,
    unsigned long long* __restrict__ part) {
  __shared__ float4 tile[kTile];
  const int32_t p = blockIdx.y;
  const int32_t u_begin = p * chunk;
  const int32_t u_end = min(n, u_begin + chunk);

  float sx[S], sy[S], sz[S], d1[S], d2[S];
  int32_t i1[S], i2[S];
  const int32_t j0 = blockIdx.x * (kBlock * S) + threadIdx.x;
#pragma unroll
  for (int s = 0; s < S; ++s) {
    const int32_t j = j0 + s * kBlock;
    const bool live = j < m;
    sx[s] = live ? sig[j] : 0.0f;
    sy[s] = live ? sig[m + j] : 0.0f;
    sz[s] = live ? sig[2 * m + j] : 0.0f;
    d1[s] = __builtin_huge_valf();
    d2[s] = __builtin_huge_valf();
    i1[s] = -1;
    i2[s] = -1;
  }

  for (int32_t t0 = u_begin; t0 < u_end; t0 += kTile) {
    const int32_t cnt = min(kTile, u_end - t0);
    __syncthreads();
    for (int32_t k = threadIdx.x; k < cnt; k += kBlock)
      tile[k] = make_float4(ux[t0 + k], uy[t0 + k], uz[t0 + k], 0.0f);
    __syncthreads();
#pragma unroll 4
    for (int32_t k = 0; k < cnt; ++k) {
      const float4 w = tile[k];
      const int32_t idx = t0 + k;
#pragma unroll
      for (int s = 0; s < S; ++s) {
        const float dx = sx[s] - w.x;
        const float dy = sy[s] - w.y;
        const float dz = sz[s] - w.z;
        const float d = (dx * dx + dy * dy) + dz * dz;
        // an empty slot (index -1) admits any distance, +inf included; units arrive in
        // increasing index order, so the strict test keeps the smaller index on ties
        const bool c1 = d < d1[s] || i1[s] < 0;
        const bool c2 = d < d2[s] || i2[s] < 0;
        d2[s] = c1 ? d1[s] : (c2 ? d : d2[s]);
        i2[s] = c1 ? i1[s] : (c2 ? idx : i2[s]);
        d1[s] = c1 ? d : d1[s];
        i1[s] = c1 ? idx : i1[s];
      }
    }
  }

#pragma unroll
  for (int s = 0; s < S; ++s) {
    const int32_t j = j0 + s * kBlock;
    if (j < m) {
      part[(2 * p) * static_cast<size_t>(m) + j] = pack(d1[s], i1[s]);
      part[(2 * p + 1) * static_cast<size_t>(m) + j] = pack(d2[s], i2[s]);
    }
  }
}

// Top-2 of the union of the chunks' top-2 keys.  Chunk results are exact and disjoint, so
// the two smallest keys of the union are the global winner and second.
__global__ __launch_bounds__(kBlock) void fw_merge(const unsigned long long* __restrict__ part,
                                                   int32_t split, int32_t m,
                                                   int32_t* __restrict__ winner,
                                                   int32_t* __restrict__ second,
                                                   float* __restrict__ d1,
                                                   float* __restrict__ d2) {
  const int32_t j = blockIdx.x * kBlock + threadIdx.x;
  if (j >= m) return;
  unsigned long long a = ~0ull, b = ~0ull;
  for (int32_t q = 0; q < 2 * split; ++q) {
    const unsigned long long k = part[q * static_cast<size_t>(m) + j];
    if (k < a) {
      b = a;
      a = k;
    } else if (k < b) {
      b = k;
    }
  }
  winner[j] = static_cast<int32_t>(static_cast<uint32_t>(a));
  second[j] = static_cast<int32_t>(static_cast<uint32_t>(b));
  d1[j] = __uint_as_float(static_cast<uint32_t>(a >> 32));
  d2[j] = __uint_as_float(static_cast<uint32_t>(b >> 32));
}

int signals_per_lane(int32_t m) { return m >= 8192 ? 4 : (m >= 2048 ? 2 : 1); }

}  // namespace

FindConfig find_config(int32_t n, int32_t m, int cus, int want_split, int want_variant) {
  FindConfig c;
  // small batches take the unit-parallel scan (no staging) unless a variant is asked for;
  // variant 6 is only defined up to kSmallM signals (larger batches take variant 4)
  c.variant = want_variant > 0 ? want_variant : (m <= kSmallM ? 6 : 4);
  if (c.variant == 6 && m > kSmallM) c.variant = 4;
  if (c.variant == 6) {
    c.split = 0;
    return c;
  }
  if (c.variant == 2) {
    c.split = screened_split(n, m, cus, want_split);
    return c;
  }
  if (c.variant == 3) {
    c.split = mfma_split(n, m, cus, want_split);
    return c;
  }
  if (c.variant == 4) {
    c.split = f16_split(n, m, cus, want_split);
    return c;
  }
  if (c.variant == 5) {
    c.split = f16_dyn_split(m, cus, want_split);
    return c;
  }
  const int S = signals_per_lane(m);
  const int64_t sblocks = (m + kBlock * S - 1) / (kBlock * S);
  int split;
  if (want_split > 0) {
    split = want_split;
  } else {
    const int64_t target = 8LL * (cus > 0 ? cus : 256);
    int64_t want = (target + sblocks - 1) / sblocks;
    int64_t by_size = (n + kMinChunk - 1) / kMinChunk;
    split = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(want, by_size)));
  }
  c.split = std::min(std::max(split, 1), kMaxSplit);
  return c;
}

hipError_t launch_find_scan(const DevState& s, int32_t n, const float* sig, int32_t m,
                            const FindConfig& cfg, int32_t*, int32_t*, float*, float*,
                            hipStream_t st, LaunchEvents ev) {
  const int S = signals_per_lane(m);
  const int32_t chunk = (n + cfg.split - 1) / cfg.split;
  dim3 grid((m + kBlock * S - 1) / (kBlock * S), cfg.split);
  switch (S) {
    case 4:
      launch_with(fw_scan_direct<4>, grid, kBlock, st, ev, s.x, s.y, s.z, n, chunk, sig, m,
                  s.part);
      break;
    case 2:
      launch_with(fw_scan_direct<2>, grid, kBlock, st, ev, s.x, s.y, s.z, n, chunk, sig, m,
                  s.part);
      break;
    default:
      launch_with(fw_scan_direct<1>, grid, kBlock, st, ev, s.x, s.y, s.z, n, chunk, sig, m,
                  s.part);
      break;
  }
  return hipGetLastError();
}

hipError_t launch_find_merge(const DevState& s, int32_t m, const FindConfig& cfg,
                             int32_t* winner, int32_t* second, float* d1, float* d2,
                             hipStream_t st) {
  fw_merge<<<(m + kBlock - 1) / kBlock, kBlock, 0, st>>>(s.part, cfg.split, m, winner, second,
                                                        d1, d2);
  return hipGetLastError();
}

}  // namespace gsn
