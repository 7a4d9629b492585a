// Find Winners, screened exhaustive variant.  Same result as the direct scan (the exact
// lexicographic top-2 of the binary32 direct-form distances), with far less arithmetic
// per signal-unit pair.  Units and signals arrive spatially sorted, with a seed bound B
// per signal (staging.hip); then:
//
//  3. Screen.  For every (signal, unit) pair the scan evaluates the expanded form
//        q = fma(-2 sx, wx, fma(-2 sy, wy, fma(-2 sz, wz, |w|^2)))   (= D - |s|^2 exactly)
//     which costs three fused multiply-adds, and keeps the group minimum.  Only a unit with
//     q <= theta(d2) can have a direct-form distance <= d2, where theta adds a rigorous
//     bound on the rounding of both forms (derivation below).  Such candidates are
//     evaluated in the direct form and inserted in the exact (d, index) top-2.  d2 starts
//     at the seed bound B and only decreases, so a unit rejected once stays rejected.
//  4. Merge.  Chunk partial top-2 keys (bits(d) << 32 | index) are merged as in the direct
//     variant and written back at the signals' original positions.
//
// Rounding bound (u = 2^-24, all inputs finite):
//   direct form  D^ = fl(fl(fl(dx^2) + fl(dy^2)) + fl(dz^2)) with dx = fl(sx - wx), etc.:
//     every term is non-negative and passes through at most five roundings, so
//     D (1-u)^5 <= D^ <= D (1+u)^5.
//   norm  n^ = fl(fl(fl(wx^2) + fl(wy^2)) + fl(wz^2)):  |n^ - |w|^2| <= 3.01 u |w|^2.
//   screen  q^ = three fused roundings over T = |2 sx wx| + |2 sy wy| + |2 sz wz| + n^:
//     |q^ - (n^ - 2 s.w)| <= 3.01 u T, so |q^ - q| <= 6.1 u T  with q = |w|^2 - 2 s.w.
//   Bound T <= T_j = 2 (|sx| Xmax + |sy| Ymax + |sz| Zmax) + Nmax with the maxima taken
//   over all units (|x|, |y|, |z|, n^).
//   D^ <= d2  =>  D <= d2 / (1-u)^5  =>  q = D - S <= d2 (1 + 5.01 u) - S
//             =>  q^ <= d2 (1 + 5.01 u) - S^ + 3.01 u S^ + 6.1 u T_j,
//   with S = |s|^2 and S^ its binary32 value.  The kernel uses
//     theta = fl(fl(d2 * (1 + 2^-20)) - S^) + E_j,
//     E_j   = 16 u (T_j + 2 S^ + 2 B_j) + 2^-120,
//   whose slack (16 u against the 6.1 u, 3.01 u and the three roundings of computing theta,
//   each at most u times a quantity bounded by T_j, S^ or B_j >= d2) covers the inequality.
// The screen may admit extra candidates (they are then rejected exactly); it never drops
// a unit of the true top-2.
//
// Range: the bound needs every quantity above to be finite.  A signal whose margin E_j
// exceeds 2^90 (huge or non-finite coordinates of the signal or of some unit) is "open":
// every unit is its candidate, i.e. it is scanned exactly in the direct form.  Below that
// margin T_j, S^ and B_j are at most 2^110, so no product, sum or threshold overflows.
#include "gsn_internal.h"

namespace gsn {
namespace {

constexpr int kTileS = 256;          // units per LDS tile
constexpr int kGroup = 8;            // units per screen group
constexpr int32_t kSentinel = 0x7fffffff;

__device__ __forceinline__ unsigned long long pack(float d, int32_t i) {
  return (static_cast<unsigned long long>(__float_as_uint(d)) << 32) |
         static_cast<uint32_t>(i);
}

__device__ __forceinline__ float norm2(float x, float y, float z) {
  return (x * x + y * y) + z * z;
}

__device__ __forceinline__ bool key_less(float da, int32_t ia, float db, int32_t ib) {
  return da < db || (da == db && ia < ib);
}

template <int S>
__global__ __launch_bounds__(kBlock) void fs_scan(const float4* __restrict__ pu,
                                                  const int32_t* __restrict__ pidx,
                                                  int32_t n, int32_t chunk,
                                                  const float* __restrict__ sig, int32_t m,
                                                  const int32_t* __restrict__ sperm,
                                                  const float* __restrict__ seed,
                                                  const int32_t* __restrict__ mag,
                                                  unsigned long long* __restrict__ part) {
  __shared__ float4 tile[kTileS];
  __shared__ int32_t tid[kTileS];
  const int32_t c = blockIdx.y;
  const int32_t u_begin = c * chunk;
  const int32_t u_end = min(n, u_begin + chunk);
  const float u = 5.9604644775390625e-8f;  // 2^-24
  // unit magnitude bounds of this call (Xmax, Ymax, Zmax, Nmax)
  const float xm = __int_as_float(mag[0]);
  const float ym = __int_as_float(mag[1]);
  const float zm = __int_as_float(mag[2]);
  const float nmx = __int_as_float(mag[3]);

  float ax[S], ay[S], az[S], sx[S], sy[S], sz[S], ss[S], ee[S], th[S];
  bool op[S];  // open: the screen's range does not hold, every unit is a candidate
  float d1[S], d2[S];
  int32_t i1[S], i2[S];
  const int32_t p0 = blockIdx.x * (kBlock * S) + threadIdx.x;
#pragma unroll
  for (int s = 0; s < S; ++s) {
    const int32_t p = p0 + s * kBlock;
    const bool live = p < m;
    const int32_t j = live ? min(max(sperm[p], 0), m - 1) : 0;
    sx[s] = live ? sig[j] : 0.0f;
    sy[s] = live ? sig[m + j] : 0.0f;
    sz[s] = live ? sig[2 * m + j] : 0.0f;
    ax[s] = -2.0f * sx[s];
    ay[s] = -2.0f * sy[s];
    az[s] = -2.0f * sz[s];
    ss[s] = norm2(sx[s], sy[s], sz[s]);
    const float B = live ? seed[p] : 0.0f;
    const float T = 2.0f * (fabsf(sx[s]) * xm + fabsf(sy[s]) * ym + fabsf(sz[s]) * zm) + nmx;
    ee[s] = 16.0f * u * (T + 2.0f * ss[s] + 2.0f * B) + 7.52316384526264e-37f;
    // 2^90 = 0x6c800000; the integer test also catches inf and NaN
    op[s] = (__float_as_uint(ee[s]) & 0x7fffffffu) > 0x6c800000u;
    d1[s] = B;
    d2[s] = B;
    i1[s] = kSentinel;
    i2[s] = kSentinel;
    th[s] = (d2[s] * 1.00000095367431640625f - ss[s]) + ee[s];
  }

  for (int32_t t0 = u_begin; t0 < u_end; t0 += kTileS) {
    const int32_t cnt = min(kTileS, u_end - t0);
    __syncthreads();
    for (int32_t k = threadIdx.x; k < kTileS; k += kBlock) {
      if (k < cnt) {
        tile[k] = pu[t0 + k];
        tid[k] = pidx[t0 + k];
      } else {
        // padding: a far-away unit that never passes the screen (it is never inserted)
        tile[k] = make_float4(0.0f, 0.0f, 0.0f, __builtin_huge_valf());
        tid[k] = kSentinel;
      }
    }
    __syncthreads();
    const int32_t groups = (cnt + kGroup - 1) / kGroup;
    for (int32_t g = 0; g < groups; ++g) {
      float4 w[kGroup];
#pragma unroll
      for (int k = 0; k < kGroup; ++k) w[k] = tile[g * kGroup + k];
      bool hit = false;
      bool hs[S];
#pragma unroll
      for (int s = 0; s < S; ++s) {
        float q[kGroup];
#pragma unroll
        for (int k = 0; k < kGroup; ++k)
          q[k] = __builtin_fmaf(ax[s], w[k].x,
                                __builtin_fmaf(ay[s], w[k].y, __builtin_fmaf(az[s], w[k].z, w[k].w)));
        float mn = q[0];
#pragma unroll
        for (int k = 1; k < kGroup; ++k) mn = fminf(mn, q[k]);
        hs[s] = mn <= th[s] || op[s];
        hit |= hs[s];
      }
      if (hit) {
#pragma unroll
        for (int s = 0; s < S; ++s) {
          if (!hs[s]) continue;
          for (int k = 0; k < kGroup; ++k) {
            const float q = __builtin_fmaf(
                ax[s], w[k].x, __builtin_fmaf(ay[s], w[k].y, __builtin_fmaf(az[s], w[k].z, w[k].w)));
            if (!(q <= th[s]) && !op[s]) continue;
            const int32_t id = tid[g * kGroup + k];
            if (id == kSentinel) continue;
            const float dx = sx[s] - w[k].x;
            const float dy = sy[s] - w[k].y;
            const float dz = sz[s] - w[k].z;
            const float d = (dx * dx + dy * dy) + dz * dz;
            if (key_less(d, id, d1[s], i1[s])) {
              d2[s] = d1[s]; i2[s] = i1[s]; d1[s] = d; i1[s] = id;
            } else if (key_less(d, id, d2[s], i2[s])) {
              d2[s] = d; i2[s] = id;
            } else {
              continue;
            }
            th[s] = (d2[s] * 1.00000095367431640625f - ss[s]) + ee[s];
          }
        }
      }
    }
  }

#pragma unroll
  for (int s = 0; s < S; ++s) {
    const int32_t p = p0 + s * kBlock;
    if (p < m) {
      part[(2 * c) * static_cast<size_t>(m) + p] = pack(d1[s], i1[s]);
      part[(2 * c + 1) * static_cast<size_t>(m) + p] = pack(d2[s], i2[s]);
    }
  }
}

}  // namespace

int screened_signals_per_lane(int32_t m) { return m >= 16384 ? 8 : (m >= 4096 ? 4 : 1); }

int screened_split(int32_t n, int32_t m, int cus, int want) {
  if (want > 0) return std::min(want, kMaxSplit);
  const int S = screened_signals_per_lane(m);
  const int64_t sblocks = (m + kBlock * S - 1) / (kBlock * S);
  const int64_t target = 4LL * (cus > 0 ? cus : 256);
  int64_t sp = (target + sblocks - 1) / sblocks;
  sp = std::min<int64_t>(sp, (n + 1023) / 1024);
  return static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(sp, kMaxSplit)));
}

hipError_t launch_scan_screened(const DevState& s, const StageBufs& b, int32_t n,
                                const float* sig, int32_t m, int split, hipStream_t st,
                                LaunchEvents ev) {
  const int S = screened_signals_per_lane(m);
  const int32_t chunk = (n + split - 1) / split;
  dim3 grid((m + kBlock * S - 1) / (kBlock * S), split);
  switch (S) {
    case 8:
      launch_with(fs_scan<8>, grid, kBlock, st, ev, b.pu, b.pidx, n, chunk, sig, m, b.sperm,
                  b.seed, b.mag, s.part);
      break;
    case 4:
      launch_with(fs_scan<4>, grid, kBlock, st, ev, b.pu, b.pidx, n, chunk, sig, m, b.sperm,
                  b.seed, b.mag, s.part);
      break;
    default:
      launch_with(fs_scan<1>, grid, kBlock, st, ev, b.pu, b.pidx, n, chunk, sig, m, b.sperm,
                  b.seed, b.mag, s.part);
      break;
  }
  return hipGetLastError();
}

}  // namespace gsn
