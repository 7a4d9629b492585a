// Spatial staging shared by the screened find-winners scans (see find_screened.hip for the
// screen and its rounding bound).
//
// Unit order.  Units are counting-sorted by the Morton code of a 32^3 grid cell over their
// bounding box, and every find call gathers the current positions into that order as
// packed (x, y, z, |w|^2) records.  The order only affects speed (every unit is still
// visited for every signal), so it is rebuilt only when the host asks for it: after the
// network changed size or indices, and periodically as units drift.
// Signal order.  Signals are counting-sorted into the same grid on every call, so that a
// wave owns signals that are near each other.
// Seed.  For every signal, the exact direct-form distances to a window of sorted units
// around its cell give B, the second smallest of them: an upper bound on the signal's
// second-winner distance, reached by two real units.
// Merge.  Per-chunk top-2 keys (bits(d) << 32 | index) of the scan are merged per signal
// and written at the signal's original position.
#include "gsn_internal.h"

namespace gsn {
namespace {

constexpr int kGrid = 32;
constexpr int kSignalShift = 3;                        // signals ordered by bucket >> 3
constexpr int kSignalBuckets = kBuckets >> kSignalShift;
constexpr int kSeedWindow = 64;
// operand layouts the gather writes besides the packed records: the binary32 matrix-core
// one (read by the binary32 product scan) and the binary16 one (the split-binary16 scan)
constexpr int kLayoutF32 = 1;
constexpr int kLayoutF16 = 2;
constexpr int kSeedLanes = 16;

__device__ __forceinline__ int32_t ord(float f) {
  const int32_t b = __float_as_int(f);
  return b >= 0 ? b : b ^ 0x7fffffff;
}
__device__ __forceinline__ float unord(int32_t b) {
  return __int_as_float(b >= 0 ? b : b ^ 0x7fffffff);
}

// identities of the bounding-box accumulators: [0..2] ord(min), [3..5] ord(max)
__device__ __forceinline__ int32_t acc_identity(int t) {
  return t < 3 ? ord(__builtin_huge_valf()) : ord(-__builtin_huge_valf());
}

__device__ __forceinline__ uint32_t spread5(uint32_t v) {
  v &= 31u;
  v = (v | (v << 8)) & 0x0300Fu;
  v = (v | (v << 4)) & 0x030C3u;
  v = (v | (v << 2)) & 0x09249u;
  return v;
}

__device__ __forceinline__ uint32_t cell_of(float p, float lo, float inv) {
  const float t = fminf(fmaxf((p - lo) * inv, 0.0f), static_cast<float>(kGrid - 1));
  return static_cast<uint32_t>(t);
}

// bb: lo.x lo.y lo.z inv.x inv.y inv.z
__device__ __forceinline__ int32_t bucket_of(float x, float y, float z, const float* bb) {
  return static_cast<int32_t>(spread5(cell_of(x, bb[0], bb[3])) |
                              (spread5(cell_of(y, bb[1], bb[4])) << 1) |
                              (spread5(cell_of(z, bb[2], bb[5])) << 2));
}

__device__ __forceinline__ float norm2(float x, float y, float z) {
  return (x * x + y * y) + z * z;
}

// Scale of the binary16 operands: sigma = 2^k with sigma M in [16, 32), M the largest
// coordinate magnitude of the bucketing box (so units may grow fourfold before the scan's
// range check, sigma max|w| <= 128, sends the call to the exact path); k in [-60, 60], and
// sigma = 1 for an empty or non-finite box.
__device__ __forceinline__ float scale_of(const int32_t* acc) {
  float mx = 0.0f;
  for (int k = 0; k < 6; ++k) mx = fmaxf(mx, fabsf(unord(acc[k])));
  const uint32_t ex = (__float_as_uint(mx) >> 23) & 0xffu;
  int k = 0;
  if (ex == 0) k = 60;                                    // zero or subnormal
  else if (ex != 0xffu) k = min(60, max(-60, 4 - (static_cast<int>(ex) - 127)));
  return __uint_as_float(static_cast<uint32_t>(k + 127) << 23);
}

typedef _Float16 h8 __attribute__((ext_vector_type(8)));

// v = hi + lo + e with hi, lo binary16 (round to nearest) and |e| <= 2^-22 |v| + 2^-25;
// v - hi is exact in binary32
__device__ __forceinline__ void split16(float v, _Float16& hi, _Float16& lo) {
  hi = static_cast<_Float16>(v);
  lo = static_cast<_Float16>(v - static_cast<float>(hi));
}

// block-wide reduction of up to 4 values with op, result valid in thread 0
template <typename Op>
__device__ void block_reduce4(float v[4], Op op) {
  __shared__ float red[kBlock / 64][4];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1)
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = op(v[k], __shfl_xor(v[k], off));
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0)
#pragma unroll
    for (int k = 0; k < 4; ++k) red[w][k] = v[k];
  __syncthreads();
  if (threadIdx.x == 0)
    for (int ww = 1; ww < kBlock / 64; ++ww)
#pragma unroll
      for (int k = 0; k < 4; ++k) v[k] = op(v[k], red[ww][k]);
}

struct FMin { __device__ float operator()(float a, float b) const { return fminf(a, b); } };
struct FMax { __device__ float operator()(float a, float b) const { return fmaxf(a, b); } };

// every histogram, offset and cursor array cleared; accumulators at their identities
__global__ __launch_bounds__(kBlock) void st_init(StageBufs b) {
  const int32_t i = blockIdx.x * kBlock + threadIdx.x;
  if (i <= kBuckets) {
    b.hist_u[i] = 0;
    b.hist_s[i] = 0;
    b.off_u[i] = 0;
    b.cur_u[i] = 0;
  }
  if (i < 16) b.acc[i] = i < 6 ? acc_identity(i) : 0;
  if (i < 8) b.bb[i] = 0.0f;
}

// ------------------------------------------------------- unit bucketing (rare) ----

__global__ __launch_bounds__(kBlock) void st_bbox(const float* __restrict__ x,
                                                  const float* __restrict__ y,
                                                  const float* __restrict__ z, int32_t n,
                                                  int32_t* __restrict__ acc) {
  float lo[4] = {__builtin_huge_valf(), __builtin_huge_valf(), __builtin_huge_valf(), 0.0f};
  float hi[4] = {-__builtin_huge_valf(), -__builtin_huge_valf(), -__builtin_huge_valf(), 0.0f};
  for (int32_t i = blockIdx.x * kBlock + threadIdx.x; i < n; i += gridDim.x * kBlock) {
    const float p[3] = {x[i], y[i], z[i]};
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      lo[k] = fminf(lo[k], p[k]);
      hi[k] = fmaxf(hi[k], p[k]);
    }
  }
  block_reduce4(lo, FMin());
  __syncthreads();
  block_reduce4(hi, FMax());
  if (threadIdx.x == 0)
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      atomicMin(&acc[k], ord(lo[k]));
      atomicMax(&acc[3 + k], ord(hi[k]));
    }
}

// Grid of this bucketing from the bounding box (written to bb by block 0), bucket of every
// unit, per-bucket counts.
__global__ __launch_bounds__(kBlock) void st_hist_units(const float* __restrict__ x,
                                                        const float* __restrict__ y,
                                                        const float* __restrict__ z, int32_t n,
                                                        const int32_t* __restrict__ acc,
                                                        float* __restrict__ bb,
                                                        int32_t* __restrict__ ukey,
                                                        int32_t* __restrict__ hist_u) {
  __shared__ float sbb[6];
  if (threadIdx.x < 3) {
    const float lo = unord(acc[threadIdx.x]);
    const float hi = unord(acc[3 + threadIdx.x]);
    sbb[threadIdx.x] = lo;
    sbb[3 + threadIdx.x] = hi > lo ? static_cast<float>(kGrid) / (hi - lo) : 0.0f;
    if (blockIdx.x == 0) {
      bb[threadIdx.x] = sbb[threadIdx.x];
      bb[3 + threadIdx.x] = sbb[3 + threadIdx.x];
    }
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) bb[6] = scale_of(acc);
  __syncthreads();
  const int32_t i = blockIdx.x * kBlock + threadIdx.x;
  if (i < n) {
    const int32_t k = bucket_of(x[i], y[i], z[i], sbb);
    ukey[i] = k;
    atomicAdd(&hist_u[k], 1);
  }
}

// Inclusive prefix sum over a 1024-thread workgroup: wave shuffles, then the 16 wave
// totals through LDS (two barriers).
__device__ int32_t block_inclusive_scan(int32_t v, int32_t* total) {
  __shared__ int32_t wsum[16];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int32_t a = __shfl_up(v, o);
    if (lane >= o) v += a;
  }
  if (lane == 63) wsum[w] = v;
  __syncthreads();
  int32_t before = 0, all = 0;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int32_t x = wsum[k];
    before += k < w ? x : 0;
    all += x;
  }
  __syncthreads();
  *total = all;
  return v + before;
}

// One workgroup: exclusive scan of a histogram of B entries into off[] (off[B] = total)
// and cur[], clearing the histogram.  Units (mode 0) also reset the bounding-box
// accumulators.  Signals (mode 1) also reduce the gather's per-block magnitude maxima
// (nmag blocks) into mag[].
template <int B>
__global__ __launch_bounds__(1024) void st_scan_hist(int32_t* __restrict__ hist,
                                                     int32_t* __restrict__ off,
                                                     int32_t* __restrict__ cur,
                                                     int32_t* __restrict__ acc,
                                                     const float* __restrict__ bmag,
                                                     int32_t nmag, int32_t* __restrict__ mag,
                                                     int mode) {
  constexpr int per = B / 1024;
  const int t = threadIdx.x;
  int32_t v[per];
  int32_t sum = 0;
#pragma unroll
  for (int i = 0; i < per; ++i) {
    v[i] = hist[t * per + i];
    sum += v[i];
  }
  int32_t total;
  int32_t run = block_inclusive_scan(sum, &total) - sum;
#pragma unroll
  for (int i = 0; i < per; ++i) {
    off[t * per + i] = run;
    cur[t * per + i] = run;
    hist[t * per + i] = 0;
    run += v[i];
  }
  if (t == 1023) off[B] = total;
  if (mode == 0 && t < 6) acc[t] = acc_identity(t);
  if (mode == 1) {
    float mg[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int32_t b = t; b < nmag; b += 1024)
#pragma unroll
      for (int k = 0; k < 4; ++k) mg[k] = fmaxf(mg[k], bmag[4 * b + k]);
    __shared__ float red[16][4];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
#pragma unroll
      for (int k = 0; k < 4; ++k) mg[k] = fmaxf(mg[k], __shfl_xor(mg[k], o));
    if ((t & 63) == 0)
#pragma unroll
      for (int k = 0; k < 4; ++k) red[t >> 6][k] = mg[k];
    __syncthreads();
    if (t < 4) {
      float r = 0.0f;
      for (int w = 0; w < 16; ++w) r = fmaxf(r, red[w][t]);
      mag[t] = __float_as_int(r);
    }
  }
}

__global__ __launch_bounds__(kBlock) void st_scatter_units(int32_t n,
                                                           const int32_t* __restrict__ ukey,
                                                           int32_t* __restrict__ cur_u,
                                                           int32_t* __restrict__ pidx) {
  const int32_t i = blockIdx.x * kBlock + threadIdx.x;
  if (i >= n) return;
  const int32_t pos = atomicAdd(&cur_u[ukey[i]], 1);
  if (pos >= 0 && pos < n) pidx[pos] = i;  // always true when counts match keys
}

// Units added at the end (indices n0 .. n1 - 1, every older index unchanged) join the
// order at its end: the scan still visits every unit, only their place is not spatial until
// the next bucketing.
__global__ __launch_bounds__(kBlock) void st_append(int32_t n0, int32_t n1,
                                                    int32_t* __restrict__ pidx) {
  const int32_t i = n0 + blockIdx.x * kBlock + threadIdx.x;
  if (i < n1) pidx[i] = i;
}

// ------------------------------------------------------------- every call ----

// Blocks [0, ub): gather the current positions into sorted order and write each block's
// magnitude maxima (max |x|, |y|, |z|, |w|^2) to bmag.  Blocks [ub, ...): bucket of every
// signal in the grid of the last unit bucketing, counted per group of 2^kSignalShift
// buckets (the signal order only needs to be coarsely spatial).
__global__ __launch_bounds__(kBlock) void st_gather(const float* __restrict__ x,
                                                    const float* __restrict__ y,
                                                    const float* __restrict__ z, int32_t n,
                                                    const int32_t* __restrict__ pidx,
                                                    float4* __restrict__ pu,
                                                    float* __restrict__ pm,
                                                    uint4* __restrict__ pmh,
                                                    const float* __restrict__ sig, int32_t m,
                                                    int32_t ub, const float* __restrict__ bb,
                                                    int32_t* __restrict__ skey,
                                                    int32_t* __restrict__ stk,
                                                    int32_t* __restrict__ hist_s,
                                                    int32_t* __restrict__ clear,
                                                    float* __restrict__ bmag, int layouts) {
  if (static_cast<int32_t>(blockIdx.x) < ub) {
    const int32_t pos = blockIdx.x * kBlock + threadIdx.x;
    float mg[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    float cv[4] = {0.0f, 0.0f, 0.0f, __builtin_huge_valf()};  // padding: never a candidate
    if (pos < n) {
      const int32_t i = min(max(pidx[pos], 0), n - 1);
      const float a = x[i], b = y[i], c = z[i];
      const float nn = norm2(a, b, c);
      pu[pos] = make_float4(a, b, c, nn);
      cv[0] = a;
      cv[1] = b;
      cv[2] = c;
      cv[3] = nn;
      mg[0] = fabsf(a);
      mg[1] = fabsf(b);
      mg[2] = fabsf(c);
      mg[3] = nn;
    }
    if (pos < ((n + 63) & ~63)) {
      // matrix-core layout: batch t = pos / 64 holds 4 groups of 16 units; component k of
      // the unit in row i of group e sits at pm[256 t + 4 (16 k + i) + e]
      const int32_t t = pos >> 6, e = (pos >> 4) & 3, i = pos & 15;
      if (layouts & kLayoutF32)
#pragma unroll
        for (int k = 0; k < 4; ++k) pm[256 * t + 4 * (16 * k + i) + e] = cv[k];
      // binary16 layout: batch t holds 2 groups of 32 units; lane h * 32 + r (r the row in
      // the group) reads K slots 8h..8h+7 of its row: h = 0 (x1 x1 x2 x2 y1 y1 y2 y2),
      // h = 1 (z1 z1 z2 z2 n1 n2 0 0) of the scaled unit sigma w and its binary32 norm,
      // at pmh[(64 t + lane) * 2 + group].  Padding carries n1 = +inf: never a candidate.
      if (layouts & kLayoutF16) {
        const int32_t g2 = (pos >> 5) & 1, r = pos & 31;
        const float sg = bb[6];
        h8 o0 = {}, o1 = {};
        if (pos < n) {
          const float sx = sg * cv[0], sy = sg * cv[1], sz = sg * cv[2];
          const float sn = norm2(sx, sy, sz);
          _Float16 a, b;
          split16(sx, a, b);
          o0[0] = a; o0[1] = a; o0[2] = b; o0[3] = b;
          split16(sy, a, b);
          o0[4] = a; o0[5] = a; o0[6] = b; o0[7] = b;
          split16(sz, a, b);
          o1[0] = a; o1[1] = a; o1[2] = b; o1[3] = b;
          split16(sn, a, b);
          o1[4] = a; o1[5] = b;
        } else {
          o1[4] = static_cast<_Float16>(__builtin_huge_valf());
        }
        h8* dst = reinterpret_cast<h8*>(pmh);
        dst[(64 * static_cast<int64_t>(t) + r) * 2 + g2] = o0;
        dst[(64 * static_cast<int64_t>(t) + 32 + r) * 2 + g2] = o1;
      }
    }
    block_reduce4(mg, FMax());
    if (threadIdx.x == 0)
#pragma unroll
      for (int k = 0; k < 4; ++k) bmag[4 * blockIdx.x + k] = mg[k];
  } else {
    const int32_t j = (blockIdx.x - ub) * kBlock + threadIdx.x;
    if (j < m) {
      const int32_t k = bucket_of(sig[j], sig[m + j], sig[2 * m + j], bb);
      skey[j] = k;
      // the count's old value is the signal's rank inside its bin (the order inside a bin
      // is immaterial)
      stk[j] = atomicAdd(&hist_s[k >> kSignalShift], 1);
    }
    // the first signal workgroup zeroes the other parity's histogram, which the next call
    // uses
    if (static_cast<int32_t>(blockIdx.x) == ub)
      for (int32_t i = threadIdx.x; i < kSignalBuckets; i += kBlock) clear[i] = 0;
  }
}


__device__ __forceinline__ unsigned long long pack(float d, int32_t i) {
  return (static_cast<unsigned long long>(__float_as_uint(d)) << 32) |
         static_cast<uint32_t>(i);
}

// top-2 of two top-2 lists of distinct keys
__device__ __forceinline__ void merge2(unsigned long long& a1, unsigned long long& a2,
                                       unsigned long long b1, unsigned long long b2) {
  const unsigned long long lo = min(a1, b1), hi = max(a1, b1);
  a2 = min(hi, min(a2, b2));
  a1 = lo;
}

// Places the signals in bucket order and computes their seed bounds, in one launch.  Every
// workgroup scans the signal histogram (kSignalBuckets bins, zeroed by the previous call) in
// LDS itself, so the bins' offsets need no launch of their own; a signal's sorted position is
// its bin's offset plus its rank inside the bin (stk, from the gather's count).  The signal's index and coordinates are written at that position (sperm,
// ssig), so the scan's prologue reads its signals directly.
// Workgroup 0 also reduces the per-block unit magnitudes of this call.
// kSeedLanes lanes per signal scan a strided part of the kSeedWindow units around the
// signal's unit bucket in the sorted order; the second smallest direct-form distance over
// these distinct units is the seed bound B >= the signal's true second-best distance.  Only
// the distance is kept, so the window slot (distinct per unit) stands in for the unit's
// index in the keys and the indices are not read.
__global__ __launch_bounds__(kBlock) void st_place_seed(
    const int32_t* __restrict__ hist_s, const int32_t* __restrict__ stk,
    const int32_t* __restrict__ skey, const float* __restrict__ sig, int32_t m,
    const float4* __restrict__ pu, int32_t n, const int32_t* __restrict__ off_u, int32_t* __restrict__ sperm, float* __restrict__ seed,
    float* __restrict__ ssig, const float* __restrict__ bmag,
    int32_t nmag, int32_t* __restrict__ mag, int32_t* __restrict__ wctr, int32_t nctr) {
  static_assert(kBlock == 256 && kSignalBuckets % kBlock == 0, "four waves, whole bins");
  constexpr int per = kSignalBuckets / kBlock;
  __shared__ int32_t soff[kSignalBuckets];
  __shared__ int32_t wsum[kBlock / 64];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int32_t t = blockIdx.x * kBlock + tid;
  const int32_t j = t / kSeedLanes;
  const int q = t % kSeedLanes;

  // The seed first: its chain of loads (key, bucket bounds, window units) does not depend on
  // the placement, so it runs beside the histogram scan below instead of after it.
  unsigned long long k1 = ~0ull, k2 = ~0ull;
  float sx = 0.0f, sy = 0.0f, sz = 0.0f;
  int32_t key = 0, rank = 0;
  if (j < m) {
    if (q == 0) rank = stk[j];
    sx = sig[j];
    sy = sig[m + j];
    sz = sig[2 * m + j];
    key = skey[j];
    const int32_t b0 = off_u[key], b1 = off_u[key + 1];
    int32_t lo = (b0 + b1) / 2 - kSeedWindow / 2;
    lo = max(0, min(lo, n - kSeedWindow));
    const int32_t hi = min(n, lo + kSeedWindow);
    // the lane's kSeedWindow / kSeedLanes units in one batch of loads (indices past hi
    // repeat the last unit and enter as the all-ones key, which changes nothing)
    constexpr int kPer = kSeedWindow / kSeedLanes;
    if (hi > lo) {
      float4 wu[kPer];
#pragma unroll
      for (int i = 0; i < kPer; ++i) wu[i] = pu[min(lo + q + i * kSeedLanes, hi - 1)];
#pragma unroll
      for (int i = 0; i < kPer; ++i) {
        const int32_t r = lo + q + i * kSeedLanes;
        const float dx = sx - wu[i].x, dy = sy - wu[i].y, dz = sz - wu[i].z;
        const unsigned long long kk =
            r < hi ? pack((dx * dx + dy * dy) + dz * dz, r) : ~0ull;
        merge2(k1, k2, kk, ~0ull);
      }
    }
  }
#pragma unroll
  for (int off = 1; off < kSeedLanes; off <<= 1) {
    const unsigned long long o1 = __shfl_xor(k1, off);
    const unsigned long long o2 = __shfl_xor(k2, off);
    merge2(k1, k2, o1, o2);
  }

  {
    int32_t v[per], sum = 0;
#pragma unroll
    for (int i = 0; i < per; ++i) {
      v[i] = hist_s[tid * per + i];
      sum += v[i];
    }
    int32_t inc = sum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int32_t a = __shfl_up(inc, o);
      if (lane >= o) inc += a;
    }
    if (lane == 63) wsum[w] = inc;
    __syncthreads();
    int32_t run = inc - sum;
    for (int k = 0; k < w; ++k) run += wsum[k];
#pragma unroll
    for (int i = 0; i < per; ++i) {
      soff[tid * per + i] = run;
      run += v[i];
    }
  }
  if (blockIdx.x == 0) {
    float mg[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int32_t b = tid; b < nmag; b += kBlock)
#pragma unroll
      for (int k = 0; k < 4; ++k) mg[k] = fmaxf(mg[k], bmag[4 * b + k]);
    __shared__ float red[kBlock / 64][4];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
#pragma unroll
      for (int k = 0; k < 4; ++k) mg[k] = fmaxf(mg[k], __shfl_xor(mg[k], o));
    if (lane == 0)
#pragma unroll
      for (int k = 0; k < 4; ++k) red[w][k] = mg[k];
    __syncthreads();
    if (tid < 4) {
      float r = 0.0f;
      for (int q = 0; q < kBlock / 64; ++q) r = fmaxf(r, red[q][tid]);
      mag[tid] = __float_as_int(r);
    }
  }
  __syncthreads();

  if (t < nctr) wctr[t] = 0;  // grab counters of the dynamic scan (variant 5)
  if (j < m && q == 0) {
    const int32_t bin = key >> kSignalShift;
    const int32_t pos = soff[bin] + rank;
    if (pos >= 0 && pos < m) {  // always true when counts match keys
      sperm[pos] = j;
      ssig[pos] = sx;
      ssig[m + pos] = sy;
      ssig[2 * m + pos] = sz;
      seed[pos] = k2 != ~0ull ? __uint_as_float(static_cast<uint32_t>(k2 >> 32))
                              : __builtin_huge_valf();
    }
  }
}

// 32 signals per workgroup, 8 groups of lanes split the partial rows, merged in LDS.
// With claim set (the fused iteration), the merge then makes the claims of each signal's
// lock set {b, s} + N(b): its eight threads (one per group) take the neighbours k = g,
// g + 8, ... of b's row, the first also b and s, each an atomic minimum of the key (with
// winner_only, the winner-lock rule's claim of b alone).
__global__ __launch_bounds__(kBlock) void st_merge(const unsigned long long* __restrict__ part,
                                                   int32_t rows, int32_t m,
                                                   const int32_t* __restrict__ sperm,
                                                   int32_t* __restrict__ winner,
                                                   int32_t* __restrict__ second,
                                                   float* __restrict__ d1,
                                                   float* __restrict__ d2, ClaimArgs claim,
                                                   int do_claim) {
  __shared__ unsigned long long sa[8][32], sb[8][32];
  __shared__ int32_t sj[32];
  const int c = threadIdx.x & 31, g = threadIdx.x >> 5;
  const int32_t p = blockIdx.x * 32 + c;
  unsigned long long a = ~0ull, b = ~0ull;
  // Rows may repeat a sentinel key (a chunk with fewer than two units under the seed bound
  // reports (B, sentinel)); real keys are unique.  insert() keeps the two smallest
  // distinct keys.
  // (branch-free: a wave's lanes see different rows)
  auto insert = [&](unsigned long long k) {
    const bool lt1 = k < a;
    const bool lt2 = k < b && k != a;
    b = lt1 ? a : (lt2 ? k : b);
    a = lt1 ? k : a;
  };
  // the output position first, then eight rows per step, all loaded before any is
  // inserted, so the loads overlap (64 rows, the usual count, take one step; rows beyond
  // the last read the all-ones key, which changes nothing)
  const int32_t jp = g == 0 && p < m ? sperm[p] : 0;
  if (p < m)
    for (int32_t q = g; q < rows; q += 64) {
      unsigned long long k[8];
#pragma unroll
      for (int i = 0; i < 8; ++i)
        k[i] = q + 8 * i < rows ? part[(q + 8 * i) * static_cast<size_t>(m) + p] : ~0ull;
#pragma unroll
      for (int i = 0; i < 8; ++i) insert(k[i]);
    }
  sa[g][c] = a;
  sb[g][c] = b;
  __syncthreads();
  if (g == 0 && p < m) {
    for (int h = 1; h < 8; ++h) {
      insert(sa[h][c]);
      insert(sb[h][c]);
    }
    const int32_t j = min(max(jp, 0), m - 1);
    winner[j] = static_cast<int32_t>(static_cast<uint32_t>(a));
    second[j] = static_cast<int32_t>(static_cast<uint32_t>(b));
    d1[j] = __uint_as_float(static_cast<uint32_t>(a >> 32));
    d2[j] = __uint_as_float(static_cast<uint32_t>(b >> 32));
    sa[0][c] = a;
    sb[0][c] = b;
    sj[c] = j;
  }
  if (!do_claim) return;
  __syncthreads();
  if (p >= m) return;
  const unsigned long long ka = sa[0][c];
  const int32_t bw = static_cast<int32_t>(static_cast<uint32_t>(ka));
  const int32_t sw = static_cast<int32_t>(static_cast<uint32_t>(sb[0][c]));
  const bool ok = pair_ok(bw, sw, claim.n);
  if (claim.pend && g == 0) claim.pend[sj[c]] = ok ? 1 : 0;
  if (!ok) {
    if (g == 0) raise_error(claim.status, GSN_E_INVAL);
    return;
  }
  const unsigned long long key =
      signal_key(__uint_as_float(static_cast<uint32_t>(ka >> 32)), sj[c], claim.key_mode);
  if (g == 0) {
    atomicMin(&claim.lock[bw], key);
    if (!claim.winner_only) atomicMin(&claim.lock[sw], key);
  }
  if (claim.winner_only) return;
  for (int32_t k = claim.rp[bw] + g; k < claim.rp[bw + 1]; k += 8)
    atomicMin(&claim.lock[claim.col[k]], key);
}

inline int blocks(int64_t n) { return static_cast<int>((n + kBlock - 1) / kBlock); }

}  // namespace

size_t stage_bytes(int32_t n_max, int32_t m_max) {
  size_t b = 0;
  auto add = [&](size_t x) { b += (x + 255) & ~static_cast<size_t>(255); };
  const size_t nm = static_cast<size_t>(n_max), mm = static_cast<size_t>(m_max);
  const size_t hb = 4 * static_cast<size_t>(kBuckets + 1);
  const size_t nb64 = (nm + 63) / 64 * 64;  // pu and pidx cover whole batches of 64 units
  add(16 * nb64);  // pu
  add(4 * nb64);   // pidx
  add(4 * nm);   // ukey
  add(4 * mm);   // skey
  add(4 * mm);   // stk
  add(4 * mm);   // sperm
  add(4 * mm);   // seed
  add(12 * mm);  // ssig
  for (int i = 0; i < 4; ++i) add(hb);  // hist/off/cur for units, hist for signals
  add(4 * 16);   // acc
  add(4 * 8);    // bb
  add(4 * 4);    // mag
  add(16 * (nm / kBlock + 2));  // bmag
  add(16 * ((nm + 63) / 64 * 64));  // pm
  add(32 * ((nm + 63) / 64 * 64));  // pmh
  add(4 * wctr_count(m_max));        // wctr
  return b;
}

StageBufs carve_stage(void* base, int32_t n_max, int32_t m_max) {
  StageBufs s;
  char* b = static_cast<char*>(base);
  size_t o = 0;
  auto take = [&](size_t x) {
    char* r = b + o;
    o += (x + 255) & ~static_cast<size_t>(255);
    return r;
  };
  const size_t nm = static_cast<size_t>(n_max), mm = static_cast<size_t>(m_max);
  const size_t hb = 4 * static_cast<size_t>(kBuckets + 1);
  const size_t nb64 = (nm + 63) / 64 * 64;
  s.pu = reinterpret_cast<float4*>(take(16 * nb64));
  s.pidx = reinterpret_cast<int32_t*>(take(4 * nb64));
  s.ukey = reinterpret_cast<int32_t*>(take(4 * nm));
  s.skey = reinterpret_cast<int32_t*>(take(4 * mm));
  s.stk = reinterpret_cast<int32_t*>(take(4 * mm));
  s.sperm = reinterpret_cast<int32_t*>(take(4 * mm));
  s.seed = reinterpret_cast<float*>(take(4 * mm));
  s.ssig = reinterpret_cast<float*>(take(12 * mm));
  s.hist_u = reinterpret_cast<int32_t*>(take(hb));
  s.off_u = reinterpret_cast<int32_t*>(take(hb));
  s.cur_u = reinterpret_cast<int32_t*>(take(hb));
  s.hist_s = reinterpret_cast<int32_t*>(take(hb));
  s.acc = reinterpret_cast<int32_t*>(take(4 * 16));
  s.bb = reinterpret_cast<float*>(take(4 * 8));
  s.mag = reinterpret_cast<int32_t*>(take(4 * 4));
  s.bmag = reinterpret_cast<float*>(take(16 * (nm / kBlock + 2)));
  s.pm = reinterpret_cast<float*>(take(16 * ((nm + 63) / 64 * 64)));
  s.pmh = reinterpret_cast<uint4*>(take(32 * ((nm + 63) / 64 * 64)));
  s.wctr = reinterpret_cast<int32_t*>(take(4 * wctr_count(m_max)));
  return s;
}

hipError_t launch_stage_append(const StageBufs& b, int32_t n0, int32_t n1, hipStream_t st) {
  if (n1 <= n0) return hipSuccess;
  st_append<<<blocks(n1 - n0), kBlock, 0, st>>>(n0, n1, b.pidx);
  return hipGetLastError();
}

hipError_t launch_stage_init(const StageBufs& b, hipStream_t st) {
  st_init<<<blocks(kBuckets + 1), kBlock, 0, st>>>(b);
  return hipGetLastError();
}

hipError_t launch_stage(const DevState& s, const StageBufs& b, int32_t n, const float* sig,
                        int32_t m, bool rebucket, int parity, int variant, hipStream_t st) {
  const int layouts = variant == 3 ? kLayoutF32 : variant >= 4 ? kLayoutF16 : 0;
  const int nb_u = blocks(n);
  if (rebucket) {
    st_bbox<<<std::min(nb_u, 64), kBlock, 0, st>>>(s.x, s.y, s.z, n, b.acc);
    st_hist_units<<<nb_u, kBlock, 0, st>>>(s.x, s.y, s.z, n, b.acc, b.bb, b.ukey, b.hist_u);
    st_scan_hist<kBuckets><<<1, 1024, 0, st>>>(b.hist_u, b.off_u, b.cur_u, b.acc, nullptr, 0,
                                              b.mag, 0);
    st_scatter_units<<<nb_u, kBlock, 0, st>>>(n, b.ukey, b.cur_u, b.pidx);
  }
  const int nb_g = blocks((static_cast<int64_t>(n) + 63) & ~static_cast<int64_t>(63));
  // the signal histogram alternates between two sets by call parity; each call's gather
  // zeroes the other set for the next call
  int32_t* hist = b.hist_s + parity * kSignalBuckets;
  int32_t* hist_next = b.hist_s + (parity ^ 1) * kSignalBuckets;
  st_gather<<<nb_g + blocks(m), kBlock, 0, st>>>(s.x, s.y, s.z, n, b.pidx, b.pu, b.pm, b.pmh, sig,
                                                 m, nb_g, b.bb, b.skey, b.stk, hist, hist_next,
                                                 b.bmag, layouts);
  st_place_seed<<<blocks(static_cast<int64_t>(m) * kSeedLanes), kBlock, 0, st>>>(
      hist, b.stk, b.skey, sig, m, b.pu, n, b.off_u, b.sperm, b.seed, b.ssig,
      b.bmag, nb_g, b.mag, b.wctr, wctr_count(m));
  return hipGetLastError();
}

hipError_t launch_stage_merge(const DevState& s, const StageBufs& b, int32_t m, int split,
                              int32_t* winner, int32_t* second, float* d1, float* d2,
                              const ClaimArgs* claim, hipStream_t st) {
  const ClaimArgs none{};
  st_merge<<<(m + 31) / 32, kBlock, 0, st>>>(s.part, 2 * split, m, b.sperm, winner, second, d1,
                                             d2, claim ? *claim : none, claim ? 1 : 0);
  return hipGetLastError();
}

}  // namespace gsn
