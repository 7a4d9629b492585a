// Device parts of the growing-network schedule: drawing the signals of an iteration from the
// point cloud, and the quantization-error window (Sec. 2.1: the convergence criterion is a
// threshold on the mean squared distance between signals and their winners).
#include "gsn_internal.h"

namespace gsn {
namespace {

// SplitMix64 (Steele, Lea and Flood, 2014): output number c of the sequence started at seed.
__device__ __forceinline__ unsigned long long splitmix64(unsigned long long seed,
                                                         unsigned long long c) {
  unsigned long long z = seed + c * 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Signal j of the iteration is the run's signal c0 + j + 1; it takes cloud point
// ((z >> 32) * P) >> 32.
__global__ void sc_draw(const float* __restrict__ cloud, int64_t n_points,
                        unsigned long long seed, int64_t c0, int32_t m,
                        float* __restrict__ sig) {
  const int32_t j = blockIdx.x * kBlock + threadIdx.x;
  if (j >= m) return;
  const unsigned long long z =
      splitmix64(seed, static_cast<unsigned long long>(c0 + j + 1));
  const int64_t i = static_cast<int64_t>(
      ((z >> 32) * static_cast<unsigned long long>(n_points)) >> 32);
  sig[j] = cloud[i];
  sig[m + j] = cloud[n_points + i];
  sig[2 * static_cast<int64_t>(m) + j] = cloud[2 * n_points + i];
}

// floor(d1 * 2^32) as an integer (exact: the scaling by a power of two is exact), 2^44 from
// 4096 on and for inf and NaN; the window sum of these is exact in any order.
__device__ __forceinline__ unsigned long long qe_units(float d1) {
  if (d1 < 4096.0f) return static_cast<unsigned long long>(d1 * 4294967296.0f);
  return 1ull << 44;
}

__global__ void sc_qe(const float* __restrict__ d1, int32_t m,
                      unsigned long long* __restrict__ acc) {
  const int32_t j = blockIdx.x * kBlock + threadIdx.x;
  unsigned long long v = j < m ? qe_units(d1[j]) : 0ull;
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  if ((threadIdx.x & 63) == 0 && v != 0) atomicAdd(acc, v);
}

inline int blocks(int64_t n) { return static_cast<int>((n + kBlock - 1) / kBlock); }

}  // namespace

hipError_t launch_draw(const float* cloud, int64_t n_points, uint64_t seed, int64_t c0,
                       int32_t m, float* sig, hipStream_t st) {
  if (m <= 0) return hipSuccess;
  sc_draw<<<blocks(m), kBlock, 0, st>>>(cloud, n_points, seed, c0, m, sig);
  return hipGetLastError();
}

hipError_t launch_qe(const float* d1, int32_t m, unsigned long long* acc, hipStream_t st) {
  if (m <= 0) return hipSuccess;
  sc_qe<<<blocks(m), kBlock, 0, st>>>(d1, m, acc);
  return hipGetLastError();
}

}  // namespace gsn
