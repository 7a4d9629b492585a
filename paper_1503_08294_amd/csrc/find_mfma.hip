// Find Winners, screened exhaustive variant on the matrix cores.  Same result as the
// direct scan (the exact lexicographic top-2 of the binary32 direct-form distances); the
// screen of find_screened.hip is evaluated as a dense K = 4 contraction with
// v_mfma_f32_16x16x4f32, and the vector unit only tests the products.
//
// Per 16-unit group and 16-signal block one MFMA computes
//     Q[i][j] = x_i (-2 sx_j) + y_i (-2 sy_j) + z_i (-2 sz_j) + n_i * 1
// with n_i = |w_i|^2 (binary32): the expanded form q of |s - w|^2 - |s|^2.  A unit is a
// candidate for signal j iff Q <= theta_j.  The 16 results a lane holds per block are reduced
// with the NaN-propagating binary32 minimum (v_minimum3_f32: it needs no canonicalization of
// the inputs, and binary32 vector instructions issue at twice the rate of 32-bit integer
// ones), and the block's minimum is tested with one subtraction (fl(a - b) <= 0 iff a <= b).
// Candidates are evaluated in the direct form and inserted in the exact (d, index) top-2.
//
// Range: the screen is applied to a signal only when its margin E_j (below) is at most 2^90.
// That bounds T_j, S^ and B_j by 2^113, so no product, sum or threshold of the screen
// overflows and Q is never NaN.  A signal outside that range (huge or non-finite
// coordinates) is "open": every unit is its candidate, i.e. it is scanned exactly in the
// direct form.
//
// Lane layout (wave64, 16x16x4 f32): lane l = 16 g + j supplies A[j][g] (component g of unit
// j of the group), B[g][j] (component g of signal j: -2 sx, -2 sy, -2 sz, 1) and receives
// Q[4 g + r][j], r = 0..3.  So lane l owns signal j of every block and sees units 4g..4g+3 of
// every group.  It keeps its own top-2 per owned signal over the units it sees; such a
// partial second-best is an upper bound on the signal's true second-best, so its threshold
// is valid, and the four partial states of a signal are merged at the end.
//
// Rounding bound (u = 2^-24).  The matrix core sums the four products (exact, since -2 s is
// exact) with an error measured at most 3.2 u of the sum of |terms| on the target; the bound
// below allows 8 u, which also covers truncating rather than rounding additions.  The sum
// of |terms| is at most T_j = 2(|sx| Xmax + |sy| Ymax + |sz| Zmax) + Nmax.  The computed norms
// n^ and S^ are within 3.01 u of |w|^2 and |s|^2, and the direct-form distance d^ within
// 5.01 u of |s - w|^2.  So a unit with d^ <= d2 has
//     Q^ <= d2 (1 + 5.01u) - S^ + 3.01u S^ + 11.02u T_j,
// while theta = fl(fl(fl(d2 (1 + 2^-20)) - S^) + E_j) is at least
//     d2 (1 + 14.99u) - S^ + E_j (1 - u) - (2 + u) u (B_j (1 + 17u) + S^),
// so Q^ <= theta whenever E_j (1 - u) >= 11.02u T_j + 5.02u S^ + 2.01u B_j.  The kernel uses
//     E_j = 12u T_j + 6u S^ + 3u B_j + 2^-120,
// evaluated in binary32 (at most four roundings, relative error below 4.01u, which the slack
// 0.97u T_j + 0.97u S^ + 0.98u B_j absorbs).  B_j >= d2 >= 0 is the seed bound; the last
// term covers underflow.
#include "gsn_internal.h"

namespace gsn {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kBlocksPerWave = 4;     // 16-signal blocks per wave: 64 signals per wave
constexpr int kSignalsPerWG = 4 * 16 * kBlocksPerWave;  // 4 waves
constexpr int32_t kSentinel = 0x7fffffff;
constexpr int kDepth = 4;             // operand ring: loads run kDepth - 1 batches ahead
static_assert(kDepth % 2 == 0, "the result sets alternate by batch parity");

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

// binary32 minimum of three (NaN-propagating; inputs here are never NaN)
__device__ __forceinline__ float fmin3(float a, float b, float c) {
  return __builtin_elementwise_minimum(__builtin_elementwise_minimum(a, b), c);
}


// The products of group e of a batch for the NB blocks: r[b][e] = Q of block b, group e.
template <int NB>
__device__ __forceinline__ void mfma_group(float a, const float (&bop)[NB], v4f (&r)[NB][4],
                                           int e) {
  const v4f z = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int b = 0; b < NB; ++b) r[b][e] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, bop[b], z, 0, 0, 0);
}

// Minimum of the 16 results of a block.
__device__ __forceinline__ float block_min(const v4f (&r)[4]) {
  const float m0 = fmin3(r[0][0], r[0][1], r[0][2]);
  const float m1 = fmin3(r[0][3], r[1][0], r[1][1]);
  const float m2 = fmin3(r[1][2], r[1][3], r[2][0]);
  const float m3 = fmin3(r[2][1], r[2][2], r[2][3]);
  const float m4 = fmin3(r[3][0], r[3][1], r[3][2]);
  return __builtin_elementwise_minimum(fmin3(m0, m1, m2), fmin3(m3, m4, r[3][3]));
}

// The rare path of block b in a batch where some lane of the wave has a candidate.  It runs
// under a wave-uniform condition and reads the block's results r, still held from the
// common path.  Bit 15 - (4 e + k) of the lane's mask is set when the unit of group e,
// row i = 4 g + k passes the screen Q <= th; that unit is 64 t + 16 e + i, its component c is
// slot[4 (16 c + i) + e] and its index is idx[16 e + i] (the wave's LDS copies of the batch).
// The exact direct-form distance of a candidate is inserted into the top-2.  Returns true if
// the lane's top-2 of block b improved.
__device__ __forceinline__ bool block_recheck(const v4f (&r)[4], float th, bool open, int32_t t,
                                              int g, int32_t n, const float* __restrict__ slot,
                                              const int32_t* __restrict__ idx, float sx,
                                              float sy, float sz, unsigned long long& k1,
                                              unsigned long long& k2) {
  uint32_t x = 0;
#pragma unroll
  for (int e = 0; e < 4; ++e)
#pragma unroll
    for (int k = 0; k < 4; ++k) x = (x << 1) | (r[e][k] <= th ? 1u : 0u);
  if (open) x = 0xffffu;
  bool improved = false;
  while (x) {
    const int s = 15 - __builtin_ctz(x);
    x &= x - 1;
    const int e = s >> 2, i = 4 * g + (s & 3);
    const int32_t uu = 64 * t + 16 * e + i;
    if (uu >= n) continue;  // padding
    const float dx = sx - slot[4 * i + e];
    const float dy = sy - slot[4 * (16 + i) + e];
    const float dz = sz - slot[4 * (32 + i) + e];
    const float dd = (dx * dx + dy * dy) + dz * dz;
    // keys order by distance first: only a distance <= the current second can enter
    if (__float_as_uint(dd) > static_cast<uint32_t>(k2 >> 32)) continue;
    improved |= insert2(k1, k2, pack(dd, idx[16 * e + i]));
  }
  return improved;
}

// Per-lane signal data that only the rare path reads, kept in LDS to spare registers:
// sd[(b * 5 + k) * 64 + lane], k = sx, sy, sz, S^, E.
constexpr int kSigFields = 5;

// Completes batch t once the minima mn[b] of its blocks are known: the rare path is entered
// only under wave-uniform conditions (valid is uniform; it is false for the placeholder batch
// before a chunk's first).  Bit b of open is set when the lane's signal of block b is open;
// wave_open is nonzero when any lane of the wave has an open signal.  res holds the batch's
// products; slot and idx address the wave's LDS copies of its operands and unit indices.  A lane whose top-2 improved refreshes its thresholds, which
// the products screened afterwards use (a stale, larger threshold only admits extra
// candidates).
template <int NB>
__device__ __forceinline__ void finish_batch(const v4f (&res)[NB][4], const float (&mn)[NB],
                                             bool valid, int32_t t, int g, int lane, int32_t n,
                                             const float* __restrict__ slot,
                                             const int32_t* __restrict__ idx, const float* sd,
                                             float (&th)[NB], unsigned long long (&k1)[NB],
                                             unsigned long long (&k2)[NB], uint32_t open,
                                             unsigned long long wave_open) {
  float lo = mn[0] - th[0];
#pragma unroll
  for (int b = 1; b < NB; ++b) lo = __builtin_elementwise_minimum(lo, mn[b] - th[b]);
  // the ballot is taken unconditionally, so the minima are computed where the caller placed
  // them (between the products) instead of being sunk into the branch
  const unsigned long long hit = __ballot(lo <= 0.0f) | wave_open;
  if (valid && hit != 0) {
    bool improved = false;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const bool ob = (open >> b) & 1u;
      if (__ballot(mn[b] <= th[b] || ob) != 0) {
        const float* f = sd + b * kSigFields * 64 + lane;
        improved |= block_recheck(res[b], th[b], ob, t, g, n, slot, idx, f[0], f[64], f[128],
                                  k1[b], k2[b]);
      }
    }
    if (improved) {
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        const float* f = sd + b * kSigFields * 64 + lane;
        th[b] = theta_of(k2[b], f[192], f[256]);
      }
    }
  }
}

// Units arrive in batches of 64 (four groups of 16) in matrix-core operand order: lane
// (j, g) finds component g of the unit in row j of groups 0..3 of batch t as the float4 at
// pm[256 t + 4 (16 g + j)], so a wave's operands for a batch are one contiguous 1 KB load.
// Waves are independent (no barriers).
//
// Software pipeline: the products of batch t go to one of two result sets (by the parity of
// t) while the minima of batch t - 1 are taken from the other, block by block, and batch
// t - 1 is completed after that.  A vector instruction that reads a matrix-core result soon
// after the product was issued stalls the SIMD; reading it a whole batch (16 products) later
// does not, which is worth about a quarter of the scan's time.  The wave's LDS copy of a
// batch is double-buffered by the same parity, so batch t - 1's rows stay in place for its
// rare path.
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void fm_scan(const float4* __restrict__ pu,
                                               const float* __restrict__ pm,
                                               const int32_t* __restrict__ pidx, int32_t n,
                                               int32_t chunk_batches,
                                               const float* __restrict__ sig, int32_t m,
                                               const int32_t* __restrict__ sperm,
                                               const int32_t* __restrict__ skey,
                                               const int32_t* __restrict__ off_u,
                                               const float* __restrict__ seed,
                                               const int32_t* __restrict__ mag,
                                               unsigned long long* __restrict__ part) {
  constexpr int NB = kBlocksPerWave;
  __shared__ __attribute__((aligned(16))) float lds[4][2][256];   // two batches per wave
  __shared__ int32_t lds_idx[4][2][64];                             // their unit indices
  __shared__ float sdata[4][kBlocksPerWave * kSigFields * 64];     // rare-path signal data
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j = lane & 15, g = lane >> 4;
  const int32_t n_batches = (n + 63) >> 6;
  // Chunk order: the signal block's candidates (and so its rare-path work) concentrate in the
  // chunk holding the units of the same grid cells, its home chunk, found from the bucket of
  // the block's middle signal.  Row y of the grid takes chunk home + 0, +1, -1, +2, -2, ...
  // (mod split, a bijection), so the work-groups with the most rare-path work start first
  // instead of forming the tail.
  int32_t c;
  {
    const int32_t split = static_cast<int32_t>(gridDim.y);
    const int32_t pm_ = min(blockIdx.x * kSignalsPerWG + kSignalsPerWG / 2, m - 1);
    const int32_t key = min(max(skey[min(max(sperm[pm_], 0), m - 1)], 0), kBuckets - 1);
    const int32_t pos = min(max(off_u[key], 0), n);
    const int32_t home = min(pos / (64 * chunk_batches), split - 1);
    const int32_t y = static_cast<int32_t>(blockIdx.y);
    const int32_t d = (y & 1) ? (y + 1) / 2 : -(y / 2);
    c = ((home + d) % split + split) % split;
  }
  const int32_t t_begin = c * chunk_batches;
  const int32_t t_end = min(n_batches, t_begin + chunk_batches);
  const float u = 5.9604644775390625e-8f;
  const float xm = __int_as_float(mag[0]), ym = __int_as_float(mag[1]);
  const float zm = __int_as_float(mag[2]), nmx = __int_as_float(mag[3]);

  // the lane's signal in block b: sorted position p = base + 16 b + j
  const int32_t base = blockIdx.x * kSignalsPerWG + wave * 16 * NB;
  float* sd = sdata[wave];
  float bop[NB], th[NB];
  unsigned long long k1[NB], k2[NB];
  uint32_t open = 0;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int32_t p = base + 16 * b + j;
    const bool live = p < m;
    const int32_t jj = live ? min(max(sperm[p], 0), m - 1) : 0;
    const float sx = live ? sig[jj] : 0.0f;
    const float sy = live ? sig[m + jj] : 0.0f;
    const float sz = live ? sig[2 * m + jj] : 0.0f;
    const float ss = norm2(sx, sy, sz);
    // signals past m get B = -inf: their threshold is -inf and nothing is a candidate
    const float B = live ? seed[p] : -__builtin_huge_valf();
    const float T = 2.0f * (fabsf(sx) * xm + fabsf(sy) * ym + fabsf(sz) * zm) + nmx;
    const float ee = live ? (12.0f * u * T + 6.0f * u * ss) + 3.0f * u * B + 7.52316384526264e-37f
                          : 0.0f;
    // 2^90 = 0x6c800000; the integer test also catches inf and NaN
    if ((__float_as_uint(ee) & 0x7fffffffu) > 0x6c800000u) open |= 1u << b;
    k1[b] = pack(B, kSentinel);
    k2[b] = k1[b];
    th[b] = live ? theta_of(k2[b], ss, ee) : -__builtin_huge_valf();
    bop[b] = g == 0 ? -2.0f * sx : (g == 1 ? -2.0f * sy : (g == 2 ? -2.0f * sz : 1.0f));
    float* f = sd + b * kSigFields * 64 + lane;  // read back only by this lane
    f[0] = sx;
    f[64] = sy;
    f[128] = sz;
    f[192] = ss;
    f[256] = ee;
  }

  const unsigned long long wave_open = __ballot(open != 0);

  // Batches are taken kDepth at a time (t .. t + kDepth - 1) with clamped indices, from a
  // ring of kDepth operand registers, so every operand load is unconditional and issued
  // kDepth - 1 batches ahead of its use: batches past the chunk's end rescan its last batch,
  // which leaves the top-2 unchanged (insert2 ignores a key already held).  The first loads
  // are unconditional too (a conditional load makes the compiler wait for every load at the
  // loop's head): for an empty chunk (t_begin >= n_batches) the index is the last batch,
  // still in bounds since the caller guarantees n >= 2, and no iteration runs.
  const float4* opnd = reinterpret_cast<const float4*>(pm) + 16 * g + j;
  float4 ring[kDepth];
  int32_t ridx[kDepth];  // unit index of slot `lane` of the batch (clamped: pidx holds n)
#pragma unroll
  for (int q = 0; q < kDepth; ++q) {
    ring[q] = opnd[64 * min(t_begin + q, t_end - 1)];
    ridx[q] = pidx[min(64 * min(t_begin + q, t_end - 1) + lane, n - 1)];
    asm volatile("" ::: "memory");  // issue in ring order, so the loop waits for one load
  }
  // the wave's copies of batches in LDS serve the candidates' exact rechecks
  const float* slot[2] = {lds[wave][0], lds[wave][1]};
  float4* my[2] = {reinterpret_cast<float4*>(lds[wave][0]) + 16 * g + j,
                   reinterpret_cast<float4*>(lds[wave][1]) + 16 * g + j};
  const int32_t* idx[2] = {lds_idx[wave][0], lds_idx[wave][1]};
  // result sets of even and odd batches; the odd set starts as a placeholder batch with no
  // candidates, completed with valid = false
  v4f res[2][NB][4];
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float inf = __builtin_huge_valf();
      res[1][b][e] = (v4f){inf, inf, inf, inf};
    }
  for (int32_t t = t_begin; t < t_end; t += kDepth) {
#pragma unroll
    for (int q = 0; q < kDepth; ++q) {
      const int cur = q & 1, prv = cur ^ 1;
      // every lane writes its part of the batch (uniform control flow): a lane's recheck
      // reads rows that other lanes loaded
      *my[cur] = ring[q];
      lds_idx[wave][cur][lane] = ridx[q];
      // Products in group-major order: four consecutive MFMAs share their A operand (one
      // component of the group's units) and differ only in B.  Fewer operand bits switch
      // between consecutive products, which the matrix cores turn into throughput under this
      // load (7-10% in a probe of this loop).  Between the groups, the minimum of one block of
      // the previous batch.
      static_assert(NB == 4, "one block minimum per group");
      const float av[4] = {ring[q].x, ring[q].y, ring[q].z, ring[q].w};
      float mn[NB];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        mfma_group(av[e], bop, res[cur], e);
        __builtin_amdgcn_sched_barrier(0);
        mn[e] = block_min(res[prv][e]);
        __builtin_amdgcn_sched_barrier(0);
      }
      ring[q] = opnd[64 * min(t + kDepth + q, t_end - 1)];
      ridx[q] = pidx[min(64 * min(t + kDepth + q, t_end - 1) + lane, n - 1)];
      // keep the load here: without the barrier the compiler sinks all ring loads to the
      // loop's end, which removes the prefetch distance
      asm volatile("" ::: "memory");
      finish_batch<NB>(res[prv], mn, q > 0 || t > t_begin, min(t + q - 1, t_end - 1), g, lane,
                       n, slot[prv], idx[prv], sd, th, k1, k2, open, wave_open);
    }
  }
  // the chunk's last batch, t_end - 1, sits in the odd set (kDepth is even)
  if (t_begin < t_end) {
    float mn[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) mn[b] = block_min(res[1][b]);
    finish_batch<NB>(res[1], mn, true, t_end - 1, g, lane, n, slot[1], idx[1], sd, th, k1, k2,
                     open, wave_open);
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
                            int32_t m, int split, hipStream_t st, LaunchEvents ev) {
  const int32_t n_batches = (n + 63) / 64;
  const int32_t chunk_batches = (n_batches + split - 1) / split;
  dim3 grid((m + kSignalsPerWG - 1) / kSignalsPerWG, split);
  launch_with(fm_scan, grid, dim3(256), st, ev, b.pu, b.pm, b.pidx, n, chunk_batches, sig, m,
              b.sperm, b.skey, b.off_u, b.seed, b.mag, s.part);
  return hipGetLastError();
}

}  // namespace gsn
