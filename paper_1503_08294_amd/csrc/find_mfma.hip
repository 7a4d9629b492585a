// Find Winners, screened exhaustive variant on the matrix cores.  Same result as the
// direct scan (the exact lexicographic top-2 of the binary32 direct-form distances); the
// screen of find_screened.hip is evaluated as a dense K = 4 contraction with
// v_mfma_f32_16x16x4f32, and the vector unit only tests the products.
//
// Per 16-unit group and 16-signal block one MFMA computes
//     D[i][j] = x_i (-2 sx_j) + y_i (-2 sy_j) + z_i (-2 sz_j) + n_i * 1  +  C[i][j]
// with n_i = |w_i|^2 (binary32) and C[i][j] = -theta_j, i.e. D = q - theta.  A unit is a
// candidate for signal j iff D <= 0, which for every non-NaN binary32 value is the signed
// integer test bits(D) <= 0; the 16 results a lane holds per group are reduced with integer
// min3 (no NaN canonicalization) and one compare.  Candidates are evaluated in the direct
// form and inserted in the exact (d, index) top-2.
//
// Lane layout (wave64, 16x16x4 f32): lane l = 16 g + j supplies A[j][g] (component g of unit
// j of the group), B[g][j] (component g of signal j: -2 sx, -2 sy, -2 sz, 1) and receives
// D[4 g + r][j], r = 0..3.  So lane l owns signal j of every block and sees units 4g..4g+3 of
// every group.  It keeps its own top-2 per owned signal over the units it sees; such a
// partial second-best is an upper bound on the signal's true second-best, so its threshold
// is valid, and the four partial states of a signal are merged at the end.
//
// Rounding bound (u = 2^-24): as in find_screened.hip, with the MFMA's own rounding of the
// five-term sum (products and C): measured at most 3.2 u (sum of |terms|) on the target, and
// at most 5 u for any sequence of binary32 roundings of exact or rounded products; the margin
// below allows 8 u.  With T_j = 2(|sx| Xmax + |sy| Ymax + |sz| Zmax) + Nmax and theta =
// fl(fl(d2 (1 + 2^-20)) - S^) + E_j, a unit whose direct-form distance is <= d2 has
//     D^ <= d2 (1 + 5.01u) - S^ + 3.01u S^ + 3.01u n + 8u (T + |theta|) - theta <= 0
// whenever E_j (1 - u) >= 11.01u T_j + 13.01u S^ + 8.01u B_j + 8u E_j; the kernel uses
//     E_j = 32u (T_j + 2 S^ + 2 B_j) + 2^-120,
// which satisfies it with room to spare.  (B_j >= d2 >= 0 is the seed bound.)
#include "gsn_internal.h"

namespace gsn {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kBlocksPerWave = 4;     // 16-signal blocks per wave: 64 signals per wave
constexpr int kSignalsPerWG = 4 * 16 * kBlocksPerWave;  // 4 waves
constexpr int32_t kSentinel = 0x7fffffff;

__device__ __forceinline__ unsigned long long pack(float d, int32_t i) {
  return (static_cast<unsigned long long>(__float_as_uint(d)) << 32) |
         static_cast<uint32_t>(i);
}

__device__ __forceinline__ float norm2(float x, float y, float z) {
  return (x * x + y * y) + z * z;
}

// insert a key into a top-2 of distinct keys (branch-free, so the per-block key arrays stay
// in registers)
__device__ __forceinline__ bool insert2(unsigned long long& k1, unsigned long long& k2,
                                        unsigned long long key) {
  const bool lt1 = key < k1;
  const bool lt2 = key < k2 && key != k1;
  const unsigned long long n2 = lt1 ? k1 : (lt2 ? key : k2);
  k1 = lt1 ? key : k1;
  k2 = n2;
  return lt1 || lt2;
}

__device__ __forceinline__ float theta_of(unsigned long long k2, float ss, float ee) {
  const float d2 = __uint_as_float(static_cast<uint32_t>(k2 >> 32));
  return (d2 * 1.00000095367431640625f - ss) + ee;
}

__device__ __forceinline__ int32_t imin3(int32_t a, int32_t b, int32_t c) {
  return min(a, min(b, c));
}

__device__ __forceinline__ int32_t bits(float f) { return __float_as_int(f); }

template <int NB>
__device__ __forceinline__ void mfma_group(float a, const float (&bop)[NB], const v4f (&cc)[NB],
                                           v4f (&d)[NB]) {
#pragma unroll
  for (int b = 0; b < NB; ++b) d[b] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, bop[b], cc[b], 0, 0, 0);
}

// the 4 groups of a batch: results for 4 groups x NB blocks x 4 rows stay in registers
template <int NB>
__device__ __forceinline__ void mfma_batch(const float4& a, const float (&bop)[NB],
                                           const v4f (&cc)[NB], v4f (&d)[4][NB]) {
  mfma_group<NB>(a.x, bop, cc, d[0]);
  mfma_group<NB>(a.y, bop, cc, d[1]);
  mfma_group<NB>(a.z, bop, cc, d[2]);
  mfma_group<NB>(a.w, bop, cc, d[3]);
}

// minimum of the 16 NB result bit patterns with three-input integer minima
template <int NB>
__device__ __forceinline__ int32_t batch_min(const v4f (&d)[4][NB]) {
  int32_t acc[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    int32_t m = imin3(bits(d[e][0][0]), bits(d[e][0][1]), bits(d[e][0][2]));
    int32_t x = bits(d[e][0][3]);
#pragma unroll
    for (int b = 1; b < NB; ++b) {
      m = imin3(m, bits(d[e][b][0]), bits(d[e][b][1]));
      x = imin3(x, bits(d[e][b][2]), bits(d[e][b][3]));
    }
    acc[e] = min(m, x);
  }
  return imin3(acc[0], acc[1], min(acc[2], acc[3]));
}

// Candidates of a batch as one 16-bit mask per block: bit 4 e + r is set when the unit of
// group e, row 4 g + r passes the screen for the lane's signal of block b.
template <int NB>
__device__ __forceinline__ void batch_masks(const v4f (&d)[4][NB], uint32_t (&mk)[NB]) {
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    uint32_t x = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e)
#pragma unroll
      for (int r = 0; r < 4; ++r) x |= (bits(d[e][b][r]) <= 0 ? 1u : 0u) << (4 * e + r);
    mk[b] = x;
  }
}

// Exact recheck of the lane's candidates in batch t: the unit of group e, row i = 4 g + r
// is 64 t + 16 e + i; its component k is slot[4 (16 k + i) + e] of the wave's LDS copy of
// the batch.  The unit's index is read from pidx only when the distance can enter the
// top-2.  Returns true if a top-2 improved.
template <int NB>
__device__ __forceinline__ bool batch_recheck(const uint32_t (&mk)[NB], int32_t t, int g,
                                              int32_t n, const float* __restrict__ slot,
                                              const int32_t* __restrict__ pidx,
                                              const float (&sx)[NB], const float (&sy)[NB],
                                              const float (&sz)[NB],
                                              unsigned long long (&k1)[NB],
                                              unsigned long long (&k2)[NB]) {
  bool improved = false;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    uint32_t x = mk[b];
    while (x) {
      const int s = __builtin_ctz(x);
      x &= x - 1;
      const int e = s >> 2, i = 4 * g + (s & 3);
      const int32_t uu = 64 * t + 16 * e + i;
      if (uu >= n) continue;  // padding
      const float dx = sx[b] - slot[4 * i + e];
      const float dy = sy[b] - slot[4 * (16 + i) + e];
      const float dz = sz[b] - slot[4 * (32 + i) + e];
      const float dd = (dx * dx + dy * dy) + dz * dz;
      // keys order by distance first: only a distance <= the current second can enter
      if (__float_as_uint(dd) > static_cast<uint32_t>(k2[b] >> 32)) continue;
      improved |= insert2(k1[b], k2[b], pack(dd, pidx[uu]));
    }
  }
  return improved;
}

// Units arrive in batches of 64 (four groups of 16) in matrix-core operand order: lane
// (j, g) finds component g of the unit in row j of groups 0..3 of batch t as the float4 at
// pm[256 t + 4 (16 g + j)], so a wave's operands for a batch are one contiguous 1 KB load.
// Waves are independent (no barriers); each operand load is issued a batch ahead of its
// use.  Thresholds are
// refreshed from the lanes' top-2 states after every pair of batches (a stale, larger
// threshold only admits extra candidates), so the C operands stay fixed inside the body.
__global__ __launch_bounds__(256) void fm_scan(const float4* __restrict__ pu,
                                               const float* __restrict__ pm,
                                               const int32_t* __restrict__ pidx, int32_t n,
                                               int32_t chunk_batches,
                                               const float* __restrict__ sig, int32_t m,
                                               const int32_t* __restrict__ sperm,
                                               const float* __restrict__ seed,
                                               const int32_t* __restrict__ mag,
                                               unsigned long long* __restrict__ part) {
  constexpr int NB = kBlocksPerWave;
  __shared__ __attribute__((aligned(16))) float lds[4][256];   // one batch per wave
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j = lane & 15, g = lane >> 4;
  float* slot = lds[wave];
  const int32_t c = blockIdx.y;
  const int32_t n_batches = (n + 63) >> 6;
  const int32_t t_begin = c * chunk_batches;
  const int32_t t_end = min(n_batches, t_begin + chunk_batches);
  const float u = 5.9604644775390625e-8f;
  const float xm = __int_as_float(mag[0]), ym = __int_as_float(mag[1]);
  const float zm = __int_as_float(mag[2]), nmx = __int_as_float(mag[3]);

  // the lane's signal in block b: sorted position p = base + 16 b + j
  const int32_t base = blockIdx.x * kSignalsPerWG + wave * 16 * NB;
  float sx[NB], sy[NB], sz[NB], ss[NB], ee[NB], bop[NB];
  unsigned long long k1[NB], k2[NB];
  v4f cc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int32_t p = base + 16 * b + j;
    const bool live = p < m;
    const int32_t jj = live ? min(max(sperm[p], 0), m - 1) : 0;
    sx[b] = live ? sig[jj] : 0.0f;
    sy[b] = live ? sig[m + jj] : 0.0f;
    sz[b] = live ? sig[2 * m + jj] : 0.0f;
    ss[b] = norm2(sx[b], sy[b], sz[b]);
    // signals past m get B = -inf: their threshold is -inf and nothing is a candidate
    const float B = live ? seed[p] : -__builtin_huge_valf();
    const float T = 2.0f * (fabsf(sx[b]) * xm + fabsf(sy[b]) * ym + fabsf(sz[b]) * zm) + nmx;
    ee[b] = live ? 32.0f * u * (T + 2.0f * ss[b] + 2.0f * B) + 7.52316384526264e-37f : 0.0f;
    k1[b] = pack(B, kSentinel);
    k2[b] = k1[b];
    const float th = live ? theta_of(k2[b], ss[b], ee[b]) : -__builtin_huge_valf();
    cc[b] = (v4f){-th, -th, -th, -th};
    bop[b] = g == 0 ? -2.0f * sx[b] : (g == 1 ? -2.0f * sy[b] : (g == 2 ? -2.0f * sz[b] : 1.0f));
  }

  const float4* opnd = reinterpret_cast<const float4*>(pm) + 16 * g + j;
  float4 a0 = t_begin < t_end ? opnd[64 * t_begin] : make_float4(0.f, 0.f, 0.f, 0.f);
  float4 a1 = t_begin + 1 < t_end ? opnd[64 * (t_begin + 1)] : make_float4(0.f, 0.f, 0.f, 0.f);
  // the wave's copy of a batch in LDS serves the candidates' exact rechecks
  float4* my = reinterpret_cast<float4*>(slot) + 16 * g + j;
  for (int32_t t = t_begin; t < t_end; t += 2) {
    bool improved = false;
    v4f d[4][NB];
    // every lane writes its part of the batch (uniform control flow): a lane's recheck
    // reads rows that other lanes loaded
    *my = a0;
    mfma_batch<NB>(a0, bop, cc, d);
    if (batch_min<NB>(d) <= 0) {
      uint32_t mk[NB];
      batch_masks<NB>(d, mk);
      improved |= batch_recheck<NB>(mk, t, g, n, slot, pidx, sx, sy, sz, k1, k2);
    }
    if (t + 2 < t_end) a0 = opnd[64 * (t + 2)];
    if (t + 1 < t_end) {
      *my = a1;
      mfma_batch<NB>(a1, bop, cc, d);
      if (batch_min<NB>(d) <= 0) {
        uint32_t mk[NB];
        batch_masks<NB>(d, mk);
        improved |= batch_recheck<NB>(mk, t + 1, g, n, slot, pidx, sx, sy, sz, k1, k2);
      }
      if (t + 3 < t_end) a1 = opnd[64 * (t + 3)];
    }
    if (improved) {
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const float th = theta_of(k2[b], ss[b], ee[b]);
        cc[b] = (v4f){-th, -th, -th, -th};
      }
    }
  }

  // merge the partial states of the four lanes that share each signal (lanes j + 16 g)
#pragma unroll
  for (int b = 0; b < NB; ++b) {
#pragma unroll
    for (int off = 16; off <= 32; off <<= 1) {
      const unsigned long long o1 = __shfl_xor(k1[b], off);
      const unsigned long long o2 = __shfl_xor(k2[b], off);
      insert2(k1[b], k2[b], o1);
      insert2(k1[b], k2[b], o2);
    }
  }
  // lane (j, g) writes block g's signal j (one predicated store per block, so the
  // per-block arrays are never indexed by a lane-dependent value)
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int32_t p = base + 16 * b + j;
    if (g == b && p < m) {
      part[(2 * c) * static_cast<size_t>(m) + p] = k1[b];
      part[(2 * c + 1) * static_cast<size_t>(m) + p] = k2[b];
    }
  }
}

}  // namespace

int mfma_split(int32_t n, int32_t m, int cus, int want) {
  if (want > 0) return std::min(want, kMaxSplit);
  const int64_t sblocks = (m + kSignalsPerWG - 1) / kSignalsPerWG;
  const int64_t target = 4LL * (cus > 0 ? cus : 256);   // ~4 waves per SIMD in one round
  int64_t sp = (target + sblocks - 1) / sblocks;
  sp = std::min<int64_t>(sp, (n + 2047) / 2048);
  return static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(sp, kMaxSplit)));
}

hipError_t launch_scan_mfma(const DevState& s, const StageBufs& b, int32_t n, const float* sig,
                            int32_t m, int split, hipStream_t st) {
  const int32_t n_batches = (n + 63) / 64;
  const int32_t chunk_batches = (n_batches + split - 1) / split;
  dim3 grid((m + kSignalsPerWG - 1) / kSignalsPerWG, split);
  fm_scan<<<grid, 256, 0, st>>>(b.pu, b.pm, b.pidx, n, chunk_batches, sig, m, b.sperm, b.seed,
                                b.mag, s.part);
  return hipGetLastError();
}

}  // namespace gsn
