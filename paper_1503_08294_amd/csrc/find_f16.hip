// Find Winners, screened exhaustive variant on the matrix cores in split binary16.  Same
// result as the direct scan (the exact lexicographic top-2 of the binary32 direct-form
// distances); the screen of find_mfma.hip is evaluated with v_mfma_f32_32x32x16_f16, which
// produces four times as many pairs per instruction as the binary32 16x16x4 product at
// 1.6 times its issue cost.
//
// Scaling and split.  Units and signals are scaled by sigma = 2^k (staging: sigma times
// the largest coordinate of the bucketing box lies in [16, 32)), which is exact, and every
// scaled coordinate v is split as v = v1 + v2 + e with v1, v2 binary16.  One product per
// 32-unit group and 32-signal block computes, for unit i and signal j,
//     Q[i][j] = sum over axes a of (w1 + w2)_a (b1 + b2)_a + n1 + n2,   b = -2 sigma s,
// where n1 + n2 splits the binary32 norm of the scaled unit: K = 14 of the 16 slots (lane
// half h = 0 carries x and y, h = 1 carries z and the norm).  Every product of two binary16
// numbers is exact in binary32.  A unit is a candidate for signal j iff Q <= theta_j (scaled).
//
// Lane layout (wave64, 32x32x16 f16, measured): lane l = 32 h + j supplies A[j][8h..8h+7]
// (unit j of the group) and B[8h..8h+7][j] (signal j of the block) and receives
// D[8q + 4h + r][j] as item 4q + r.  So lane l owns signal j of every block and sees the 16
// units 8q + 4h + r of every group; the two partial top-2 states of a signal are merged at
// the end.
//
// Rounding bound (u = 2^-24; everything scaled by sigma, sigma^2 for squares, exactly).
//   split: |e| <= 2^-22 |v| + 2^-25, so the products of the pieces miss at most
//     sum_a (2^-21 |w_a| |b_a| + 2^-25 (|w_a| + |b_a|)) + 2^-22 n + 2^-25;
//   the matrix core sums the 14 exact products with an error measured at most 3.0 u of the
//   sum of |terms|; the bound allows 32 u (15 additions, truncating);
//   the sum of |terms| is at most (1 + 2^-9) T_j, T_j = 2(|sx| Xmax + |sy| Ymax + |sz| Zmax)
//   + Nmax (scaled maxima over all units); the binary32 norms are within 3.01 u.
//   So |Q^ - q| <= 43.1u T_j + 2^-25 (2 (|sx| + |sy| + |sz|) + 385) with q the exact
//   |w|^2 - 2 s.w, and as in find_mfma.hip a unit with direct-form distance <= d2 has
//   Q^ <= theta = fl(fl(fl(d2 (1 + 2^-20)) - S^) + E_j) whenever
//   E_j (1 - u) >= 43.1u T_j + 5.02u S^ + 2.01u B_j + 2^-25 (2 (|sx| + |sy| + |sz|) + 385).
//   The kernel uses E_j = 46u T_j + 6u S^ + 3u B_j + 2^-24 (2 (|sx| + |sy| + |sz|) + 400)
//   + 2^-120, whose slack covers the five roundings of computing it.
//
// Range: the bound needs the binary16 pieces finite and the norm split meaningful: the call
// is screened only if sigma max|w| <= 128 over the units of this call (so n <= 49152 <
// 65504), and a signal only if its scaled coordinates are at most 2^14 in magnitude and its
// margin at most 2^90.  Otherwise the call, or the signal, is "open": every unit is a
// candidate, scanned exactly in the direct form from the binary32 copy.
#include "gsn_internal.h"

namespace gsn {
namespace {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef float f4 __attribute__((ext_vector_type(4)));   // a native vector: stays in registers

constexpr int kBlocks = 2;                        // 32-signal blocks per wave
constexpr int kSignalsPerWG = 4 * 32 * kBlocks;   // 4 waves
constexpr int32_t kSentinel = 0x7fffffff;
constexpr int kDepth = 2;             // operand ring: loads run kDepth - 1 batches ahead
constexpr int kSigFields = 5;         // rare-path signal data: sx, sy, sz, S^, E (scaled S, E)

__device__ __forceinline__ unsigned long long pack(float d, int32_t i) {
  return (static_cast<unsigned long long>(__float_as_uint(d)) << 32) |
         static_cast<uint32_t>(i);
}

__device__ __forceinline__ float norm2(float x, float y, float z) {
  return (x * x + y * y) + z * z;
}

// insert a key into a top-2 of distinct keys (branch-free)
__device__ __forceinline__ bool insert2(unsigned long long& k1, unsigned long long& k2,
                                        unsigned long long key) {
  const bool lt1 = key < k1;
  const bool lt2 = key < k2 && key != k1;
  const unsigned long long n2 = lt1 ? k1 : (lt2 ? key : k2);
  k1 = lt1 ? key : k1;
  k2 = n2;
  return lt1 || lt2;
}

// scaled threshold from the lane's second key (unscaled distance) and the scale squared
__device__ __forceinline__ float theta_of(unsigned long long k2, float sig2, float ss,
                                          float ee) {
  const float d2 = __uint_as_float(static_cast<uint32_t>(k2 >> 32)) * sig2;
  return (d2 * 1.00000095367431640625f - ss) + ee;
}

__device__ __forceinline__ float fmin3(float a, float b, float c) {
  return __builtin_elementwise_minimum(__builtin_elementwise_minimum(a, b), c);
}

// Minimum of the 32 results of a block (two groups): fifteen three-input minima leave two
// values, one two-input minimum joins them (31 reductions in 16 instructions).
__device__ __forceinline__ float block_min(const v16f (&r)[2]) {
  float x[10];
#pragma unroll
  for (int e = 0; e < 2; ++e)
#pragma unroll
    for (int i = 0; i < 5; ++i) x[5 * e + i] = fmin3(r[e][3 * i], r[e][3 * i + 1], r[e][3 * i + 2]);
  const float y0 = fmin3(x[0], x[1], x[2]);
  const float y1 = fmin3(x[3], x[4], r[0][15]);
  const float y2 = fmin3(x[5], x[6], x[7]);
  const float y3 = fmin3(x[8], x[9], r[1][15]);
  return __builtin_elementwise_minimum(fmin3(y0, y1, y2), y3);
}

// The rare path of block b of batch t, under a wave-uniform condition: bit 16 e + 4 q + r of
// the lane's mask is set when its unit of group e, row 8 q + 4 h + r passes the screen
// (r[e][4q + r] <= th, or the signal is open); that unit is 64 t + 32 e + 8 q + 4 h + r, its
// binary32 coordinates are lu[32 e + 8 q + 4 h + r] and its index li[...] (the wave's LDS
// copies of the batch).  The exact direct-form distance of a candidate is inserted into the
// top-2 when it can enter it.  Returns true if the lane's top-2 improved.
__device__ __forceinline__ bool block_recheck(const v16f (&r)[2], float th, bool open,
                                              int32_t t, int h, int32_t n,
                                              const f4* __restrict__ lu,
                                              const int32_t* __restrict__ li, float sx,
                                              float sy, float sz, unsigned long long& k1,
                                              unsigned long long& k2) {
  uint32_t x = 0;
#pragma unroll
  for (int e = 1; e >= 0; --e)
#pragma unroll
    for (int k = 15; k >= 0; --k) x = (x << 1) | (r[e][k] <= th ? 1u : 0u);
  if (open) x = 0xffffffffu;
  bool improved = false;
  while (x) {
    const int s = __builtin_ctz(x);
    x &= x - 1;
    const int e = s >> 4, q = (s >> 2) & 3, rr = s & 3;
    const int uu = 32 * e + 8 * q + 4 * h + rr;
    if (64 * t + uu >= n) continue;  // padding
    const f4 w = lu[uu];
    const float dx = sx - w[0];
    const float dy = sy - w[1];
    const float dz = sz - w[2];
    const float dd = (dx * dx + dy * dy) + dz * dz;
    // keys order by distance first: only a distance <= the current second can enter
    if (__float_as_uint(dd) > static_cast<uint32_t>(k2 >> 32)) continue;
    improved |= insert2(k1, k2, pack(dd, li[uu]));
  }
  return improved;
}

// Completes batch t (tq batches past the work-group's first) once the minima mn[b] of its
// blocks are known (see find_mfma.hip): the ballot is unconditional; valid is uniform (false
// skips the batch).
__device__ __forceinline__ void finish_batch(const v16f (&res)[kBlocks][2],
                                             const float (&mn)[kBlocks], bool valid, int32_t t,
                                             int h, int lane, int32_t n,
                                             __amdgpu_buffer_rsrc_t ru_,
                                             __amdgpu_buffer_rsrc_t ri_, int32_t tq,
                                             f4* __restrict__ lu, int32_t* __restrict__ li,
                                             const float* sd, float sig2, float (&th)[kBlocks],
                                             unsigned long long (&k1)[kBlocks],
                                             unsigned long long (&k2)[kBlocks], uint32_t open,
                                             unsigned long long wave_open) {
  // one ballot per block: each compare then writes its lane mask directly
  unsigned long long hit = wave_open;
#pragma unroll
  for (int b = 0; b < kBlocks; ++b) hit |= __ballot(mn[b] <= th[b]);
  if (valid && hit != 0) {
    // the batch's binary32 units and indices, for the candidates' exact distances: each
    // lane fetches one unit into the wave's LDS copy (the slots past n get stale values,
    // which the recheck skips)
    lu[lane] = __builtin_bit_cast(
        f4, __builtin_amdgcn_raw_buffer_load_b128(ru_, 16 * lane, 1024 * tq, 0));
    li[lane] = static_cast<int32_t>(
        __builtin_amdgcn_raw_buffer_load_b32(ri_, 4 * lane, 256 * tq, 0));
    bool improved = false;
#pragma unroll
    for (int b = 0; b < kBlocks; ++b) {
      const bool ob = (open >> b) & 1u;
      if (__ballot(mn[b] <= th[b] || ob) != 0) {
        const float* f = sd + b * kSigFields * 64 + lane;
        improved |= block_recheck(res[b], th[b], ob, t, h, n, lu, li, f[0], f[64], f[128],
                                  k1[b], k2[b]);
      }
    }
    if (improved) {
#pragma unroll
      for (int b = 0; b < kBlocks; ++b) {
        const float* f = sd + b * kSigFields * 64 + lane;
        th[b] = theta_of(k2[b], sig2, f[192], f[256]);
      }
    }
  }
}

// Units arrive in batches of 64 (two groups of 32): lane l reads its two 16-byte operands of
// batch t at pmh[(64 t + l) * 2 + group] (2 KB contiguous per wave).  The binary32 units and
// their indices are read only for a batch in which some lane has a candidate: lane l then
// fetches unit 64 t + l (pu) and its index (pidx) into the wave's LDS copy (finish_batch).
// One result set: the minima of a batch follow its own products, and the other waves of the
// SIMD cover their latency (122 VGPRs, four waves per SIMD; measured faster than the
// two-set pipeline of find_mfma.hip at two waves per SIMD, whose 200 VGPRs allow no more).
// Products in group-major order.
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void fh_scan(
    const float4* __restrict__ pu, const uint4* __restrict__ pmh,
    const int32_t* __restrict__ pidx, int32_t n, const float* __restrict__ ssig, int32_t m,
    const float* __restrict__ seed, const int32_t* __restrict__ mag,
    const float* __restrict__ bb, unsigned long long* __restrict__ part) {
  constexpr int NB = kBlocks;
  __shared__ f4 lds_u[4][64];                      // binary32 units of a batch, per wave
  __shared__ int32_t lds_i[4][64];                 // their indices
  __shared__ float sdata[4][NB * kSigFields * 64];  // rare-path signal data
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j = lane & 31, h = lane >> 5;
  const int32_t n_batches = (n + 63) >> 6;
  // Work-group -> (signal block sb, chunk c).  Chunk c holds the batches t = c (mod split),
  // so every chunk samples the whole spatial order evenly: the few batches near a block's
  // signals, where its candidates and so its rare-path work lie, spread over all of its
  // work-groups instead of weighing on one.  Work-groups go to the 8 XCDs round-robin by
  // linear id; when the split is a multiple of 8, XCD r gets the chunks c = r (mod 8) only,
  // so its L2 holds an eighth of the operand array (the batches t = r (mod 8)).
  const int32_t split = static_cast<int32_t>(gridDim.y);
  int32_t c, sb;
  if (split % 8 == 0) {
    const int32_t sblocks = static_cast<int32_t>(gridDim.x);
    const int32_t id = static_cast<int32_t>(blockIdx.x) + static_cast<int32_t>(blockIdx.y) * sblocks;
    const int32_t k = id / 8;
    sb = k % sblocks;
    c = id % 8 + 8 * (k / sblocks);
  } else {
    sb = static_cast<int32_t>(blockIdx.x);
    c = static_cast<int32_t>(blockIdx.y);
  }
  // batches c + split i, i < cnt, of the chunk (none when c >= n_batches)
  const int32_t cnt = c < n_batches ? (n_batches - 1 - c) / split + 1 : 0;
  const int32_t last = max(cnt - 1, 0);
  const float u = 5.9604644775390625e-8f;
  const float sgm = bb[6], sig2 = sgm * sgm;
  const float xm = sgm * __int_as_float(mag[0]), ym = sgm * __int_as_float(mag[1]);
  const float zm = sgm * __int_as_float(mag[2]), nmx = sig2 * __int_as_float(mag[3]);
  // the call's units fit the binary16 operands (false for NaN as well)
  const bool range_ok = fmaxf(xm, fmaxf(ym, zm)) <= 128.0f;

  // the lane's signal in block b: sorted position p = base + 32 b + j
  const int32_t base = sb * kSignalsPerWG + wave * 32 * NB;
  float* sd = sdata[wave];
  h8 bop[NB];
  float th[NB];
  unsigned long long k1[NB], k2[NB];
  uint32_t open = 0;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int32_t p = base + 32 * b + j;
    const bool live = p < m;
    const float sx = live ? ssig[p] : 0.0f;
    const float sy = live ? ssig[m + p] : 0.0f;
    const float sz = live ? ssig[2 * m + p] : 0.0f;
    const float tx = sgm * sx, ty = sgm * sy, tz = sgm * sz;  // exact
    const float ss = norm2(tx, ty, tz);
    // signals past m get B = -inf: their threshold is -inf and nothing is a candidate
    const float B = live ? seed[p] : -__builtin_huge_valf();
    const float T = 2.0f * (fabsf(tx) * xm + fabsf(ty) * ym + fabsf(tz) * zm) + nmx;
    const float A = 2.0f * ((fabsf(tx) + fabsf(ty)) + fabsf(tz)) + 400.0f;
    const float ee = live ? (((46.0f * u * T + 6.0f * u * ss) + 3.0f * u * (B * sig2)) +
                             u * A) + 7.52316384526264e-37f
                          : 0.0f;
    // 2^90 = 0x6c800000; the integer test also catches inf and NaN
    const bool big = !(fmaxf(fabsf(tx), fmaxf(fabsf(ty), fabsf(tz))) <= 16384.0f);
    if (!range_ok || big || (__float_as_uint(ee) & 0x7fffffffu) > 0x6c800000u) open |= 1u << b;
    k1[b] = pack(B, kSentinel);
    k2[b] = k1[b];
    th[b] = live ? theta_of(k2[b], sig2, ss, ee) : -__builtin_huge_valf();
    // B operand: K slots 8h..8h+7 of signal j, b = -2 sigma s split in binary16 pairs
    const float bx = -2.0f * tx, by = -2.0f * ty, bz = -2.0f * tz;
    auto split = [](float v, _Float16& hi, _Float16& lo) {
      hi = static_cast<_Float16>(v);
      lo = static_cast<_Float16>(v - static_cast<float>(hi));
    };
    _Float16 a1, a2, c1, c2;
    h8 o;
    if (h == 0) {
      split(bx, a1, a2);
      split(by, c1, c2);
      o = (h8){a1, a2, a1, a2, c1, c2, c1, c2};
    } else {
      split(bz, a1, a2);
      const _Float16 one = static_cast<_Float16>(1.0f), zero = static_cast<_Float16>(0.0f);
      o = (h8){a1, a2, a1, a2, one, one, zero, zero};
    }
    bop[b] = o;
    float* f = sd + b * kSigFields * 64 + lane;  // read back only by this lane
    f[0] = sx;
    f[64] = sy;
    f[128] = sz;
    f[192] = ss;
    f[256] = ee;
  }
  const unsigned long long wave_open = __ballot(open != 0);

  // Operand ring with clamped, unconditional loads issued in ring order (find_mfma.hip).  Each
  // load is a uniform batch base plus a per-lane offset that never changes, so no vector
  // instruction computes addresses; pu and pidx cover whole batches (the slots past n hold
  // stale values that the rare path skips).
  // The loads are raw buffer loads from a per-workgroup base at batch tb0 (the chunk's first,
  // or the last batch for an empty chunk): the lane's offset sits in the vector offset and
  // the batch's in the scalar offset.  Every access is in bounds by construction (batches
  // are clamped to the chunk, the host keeps chunk offsets below 2^31).
  const int32_t tb0 = min(c, n_batches - 1);
  const int32_t stride = 2048 * split;  // operand bytes from one batch of the chunk to the next
  const __amdgpu_buffer_rsrc_t rh = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint4*>(pmh) + 128 * static_cast<int64_t>(tb0), 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t ru_ = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float4*>(pu) + 64 * static_cast<int64_t>(tb0), 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t ri_ = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<int32_t*>(pidx) + 64 * static_cast<int64_t>(tb0), 0, 0x7fffffff, 0x00020000);
  const int32_t vh = 32 * lane;
  h8 ra[kDepth][2];
#pragma unroll
  for (int q = 0; q < kDepth; ++q) {
    const int32_t iq = min(q, last);
    ra[q][0] = __builtin_bit_cast(h8, __builtin_amdgcn_raw_buffer_load_b128(rh, vh, stride * iq, 0));
    ra[q][1] = __builtin_bit_cast(h8, __builtin_amdgcn_raw_buffer_load_b128(rh, vh + 16, stride * iq, 0));
    asm volatile("" ::: "memory");
  }
  v16f res[NB][2];
  const v16f zero16 = {};
  // Issue priority by progress: a wave starts at the highest priority and steps down at a
  // quarter, a half and three quarters of its chunk, so that the SIMD favours the waves that
  // are furthest behind (the hardware otherwise favours the oldest wave, and the youngest
  // waves of a SIMD finish last); priority only orders the issue of ready waves.
  __builtin_amdgcn_s_setprio(3);
  const int32_t p1 = cnt / 4, p2 = cnt / 2, p3 = (3 * cnt) / 4;
  for (int32_t i = 0; i < cnt; i += kDepth) {
    if (i >= p1 && i < p1 + kDepth) __builtin_amdgcn_s_setprio(2);
    if (i >= p2 && i < p2 + kDepth) __builtin_amdgcn_s_setprio(1);
    if (i >= p3 && i < p3 + kDepth) __builtin_amdgcn_s_setprio(0);
#pragma unroll
    for (int q = 0; q < kDepth; ++q) {
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const h8 a = ra[q][e];
#pragma unroll
        for (int b = 0; b < NB; ++b)
          res[b][e] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, bop[b], zero16, 0, 0, 0);
      }
      const int32_t in = min(i + kDepth + q, last);
      ra[q][0] = __builtin_bit_cast(h8, __builtin_amdgcn_raw_buffer_load_b128(rh, vh, stride * in, 0));
      ra[q][1] = __builtin_bit_cast(h8, __builtin_amdgcn_raw_buffer_load_b128(rh, vh + 16, stride * in, 0));
      asm volatile("" ::: "memory");
      float mn[NB];
#pragma unroll
      for (int b = 0; b < NB; ++b) mn[b] = block_min(res[b]);
      const int32_t ic = min(i + q, last);
      finish_batch(res, mn, true, c + split * ic, h, lane, n, ru_, ri_, split * ic,
                   lds_u[wave], lds_i[wave], sd, sig2, th, k1, k2, open, wave_open);
    }
  }

  // merge the two partial states of each signal (lanes j and j + 32); lane (j, h) writes
  // block h's signal j
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const unsigned long long o1 = __shfl_xor(k1[b], 32);
    const unsigned long long o2 = __shfl_xor(k2[b], 32);
    insert2(k1[b], k2[b], o1);
    insert2(k1[b], k2[b], o2);
  }
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int32_t p = base + 32 * b + j;
    if (h == b && p < m) {
      part[(2 * c) * static_cast<size_t>(m) + p] = k1[b];
      part[(2 * c + 1) * static_cast<size_t>(m) + p] = k2[b];
    }
  }
}

// Variant 5: the same scan with dynamic work distribution.  The batches are dealt out as
// eight lists, list x holding the batches t = x + 8 i (so list x is the eighth of the
// operand array that the XCD with the same number keeps in its L2); for every wave-level
// signal block (64 signals) each list has a counter in wctr, zeroed by the staging before
// the call.  Work-group id = 8 k + x runs on XCD x (work-groups reach the XCDs round-robin)
// and its four waves take the signal blocks of work-group k mod sblocks; a wave repeatedly
// takes `grab` consecutive list entries with one atomic addition (the next grab's atomic is
// issued before the current grab's work), drains its own list first and then the other
// seven, so all waves of a signal block finish within about one grab of each other, and
// keeps its top-2 in registers across grabs: it writes one partial row pair, row
// 8 (k div sblocks) + x, at the end.  Every batch is scanned by exactly one wave of each
// signal block, so the merged result is the exhaustive one, independent of which wave took
// which batch.
__device__ __forceinline__ int32_t take(int32_t* ctr, int32_t grab, int lane) {
  int32_t v = 0;
  if (lane == 0) v = atomicAdd(ctr, grab);
  return __builtin_amdgcn_readfirstlane(v);
}

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void fh_scan_dyn(
    const float4* __restrict__ pu, const uint4* __restrict__ pmh,
    const int32_t* __restrict__ pidx, int32_t n, const float* __restrict__ ssig, int32_t m,
    const float* __restrict__ seed, const int32_t* __restrict__ mag,
    const float* __restrict__ bb, unsigned long long* __restrict__ part,
    int32_t* __restrict__ wctr, int32_t sblocks, int32_t grab) {
  constexpr int NB = kBlocks;
  __shared__ f4 lds_u[4][64];
  __shared__ int32_t lds_i[4][64];
  __shared__ float sdata[4][NB * kSigFields * 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j = lane & 31, h = lane >> 5;
  const int32_t n_batches = (n + 63) >> 6;
  const int32_t id = static_cast<int32_t>(blockIdx.x);
  const int32_t xcd = id & 7, k = id >> 3;
  const int32_t sb = k % sblocks, rep = k / sblocks;
  const int32_t row = 8 * rep + xcd;
  int32_t* ctr = wctr + 8 * (4 * sb + wave);
  const float u = 5.9604644775390625e-8f;
  const float sgm = bb[6], sig2 = sgm * sgm;
  const float xm = sgm * __int_as_float(mag[0]), ym = sgm * __int_as_float(mag[1]);
  const float zm = sgm * __int_as_float(mag[2]), nmx = sig2 * __int_as_float(mag[3]);
  const bool range_ok = fmaxf(xm, fmaxf(ym, zm)) <= 128.0f;

  // the wave's first grab goes out before the signal set-up
  int32_t x = xcd;
  int32_t i0 = take(ctr + x, grab, lane);

  const int32_t base = sb * kSignalsPerWG + wave * 32 * NB;
  float* sd = sdata[wave];
  h8 bop[NB];
  float th[NB];
  unsigned long long k1[NB], k2[NB];
  uint32_t open = 0;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int32_t p = base + 32 * b + j;
    const bool live = p < m;
    const float sx = live ? ssig[p] : 0.0f;
    const float sy = live ? ssig[m + p] : 0.0f;
    const float sz = live ? ssig[2 * m + p] : 0.0f;
    const float tx = sgm * sx, ty = sgm * sy, tz = sgm * sz;
    const float ss = norm2(tx, ty, tz);
    const float B = live ? seed[p] : -__builtin_huge_valf();
    const float T = 2.0f * (fabsf(tx) * xm + fabsf(ty) * ym + fabsf(tz) * zm) + nmx;
    const float A = 2.0f * ((fabsf(tx) + fabsf(ty)) + fabsf(tz)) + 400.0f;
    const float ee = live ? (((46.0f * u * T + 6.0f * u * ss) + 3.0f * u * (B * sig2)) +
                             u * A) + 7.52316384526264e-37f
                          : 0.0f;
    const bool big = !(fmaxf(fabsf(tx), fmaxf(fabsf(ty), fabsf(tz))) <= 16384.0f);
    if (!range_ok || big || (__float_as_uint(ee) & 0x7fffffffu) > 0x6c800000u) open |= 1u << b;
    k1[b] = pack(B, kSentinel);
    k2[b] = k1[b];
    th[b] = live ? theta_of(k2[b], sig2, ss, ee) : -__builtin_huge_valf();
    const float bx = -2.0f * tx, by = -2.0f * ty, bz = -2.0f * tz;
    auto split = [](float v, _Float16& hi, _Float16& lo) {
      hi = static_cast<_Float16>(v);
      lo = static_cast<_Float16>(v - static_cast<float>(hi));
    };
    _Float16 a1, a2, c1, c2;
    h8 o;
    if (h == 0) {
      split(bx, a1, a2);
      split(by, c1, c2);
      o = (h8){a1, a2, a1, a2, c1, c2, c1, c2};
    } else {
      split(bz, a1, a2);
      const _Float16 one = static_cast<_Float16>(1.0f), zero = static_cast<_Float16>(0.0f);
      o = (h8){a1, a2, a1, a2, one, one, zero, zero};
    }
    bop[b] = o;
    float* f = sd + b * kSigFields * 64 + lane;
    f[0] = sx;
    f[64] = sy;
    f[128] = sz;
    f[192] = ss;
    f[256] = ee;
  }
  const unsigned long long wave_open = __ballot(open != 0);

  // buffer resources at batch 0: batch t's operands sit 2048 t bytes further (the host
  // keeps 2048 n_batches below 2^31), its units 1024 t and its indices 256 t
  const __amdgpu_buffer_rsrc_t rh = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint4*>(pmh), 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t ru_ = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float4*>(pu), 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t ri_ = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<int32_t*>(pidx), 0, 0x7fffffff, 0x00020000);
  const int32_t vh = 32 * lane;
  const v16f zero16 = {};
  int32_t tried = 1;   // lists whose counter this wave has read (its own so far)
  while (true) {
    // list x holds the batches x, x + 8, ...: len entries
    int32_t len = x < n_batches ? (n_batches - 1 - x) / 8 + 1 : 0;
    while (i0 >= len && tried < 8) {
      x = (x + 1) & 7;
      ++tried;
      i0 = take(ctr + x, grab, lane);
      len = x < n_batches ? (n_batches - 1 - x) / 8 + 1 : 0;
    }
    if (i0 >= len) break;
    const int32_t cnt = min(grab, len - i0);
    const int32_t last = cnt - 1;
    const int32_t nxt = take(ctr + x, grab, lane);  // the next grab of the same list
    // batch of entry e of this grab: t = x + 8 (i0 + e)
    const int32_t t0 = x + 8 * i0;
    h8 ra[kDepth][2];
#pragma unroll
    for (int q = 0; q < kDepth; ++q) {
      const int32_t tq = t0 + 8 * min(q, last);
      ra[q][0] = __builtin_bit_cast(h8, __builtin_amdgcn_raw_buffer_load_b128(rh, vh, 2048 * tq, 0));
      ra[q][1] = __builtin_bit_cast(h8, __builtin_amdgcn_raw_buffer_load_b128(rh, vh + 16, 2048 * tq, 0));
      asm volatile("" ::: "memory");
    }
    v16f res[NB][2];
    for (int32_t i = 0; i < cnt; i += kDepth) {
#pragma unroll
      for (int q = 0; q < kDepth; ++q) {
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const h8 a = ra[q][e];
#pragma unroll
          for (int b = 0; b < NB; ++b)
            res[b][e] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, bop[b], zero16, 0, 0, 0);
        }
        const int32_t tn = t0 + 8 * min(i + kDepth + q, last);
        ra[q][0] = __builtin_bit_cast(h8, __builtin_amdgcn_raw_buffer_load_b128(rh, vh, 2048 * tn, 0));
        ra[q][1] = __builtin_bit_cast(h8, __builtin_amdgcn_raw_buffer_load_b128(rh, vh + 16, 2048 * tn, 0));
        asm volatile("" ::: "memory");
        float mn[NB];
#pragma unroll
        for (int b = 0; b < NB; ++b) mn[b] = block_min(res[b]);
        const int32_t tc = t0 + 8 * min(i + q, last);
        finish_batch(res, mn, true, tc, h, lane, n, ru_, ri_, tc, lds_u[wave], lds_i[wave],
                     sd, sig2, th, k1, k2, open, wave_open);
      }
    }
    i0 = nxt;
  }

#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const unsigned long long o1 = __shfl_xor(k1[b], 32);
    const unsigned long long o2 = __shfl_xor(k2[b], 32);
    insert2(k1[b], k2[b], o1);
    insert2(k1[b], k2[b], o2);
  }
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int32_t p = base + 32 * b + j;
    if (h == b && p < m) {
      part[(2 * row) * static_cast<size_t>(m) + p] = k1[b];
      part[(2 * row + 1) * static_cast<size_t>(m) + p] = k2[b];
    }
  }
}

}  // namespace

int f16_dyn_split(int32_t m, int cus, int want) {
  // 8 rep rows per signal (one per XCD list per replica); replicas fill the resident slots
  // (four work-groups of four waves per CU), at most kMaxSplit / 8
  if (want > 0) return std::max(1, std::min(want / 8, kMaxSplit / 8)) * 8;
  const int64_t sblocks = (m + kSignalsPerWG - 1) / kSignalsPerWG;
  const int64_t slots = 4LL * (cus > 0 ? cus : 256);
  const int64_t reps = std::max<int64_t>(1, std::min<int64_t>(slots / (8 * sblocks), kMaxSplit / 8));
  return static_cast<int>(8 * reps);
}

hipError_t launch_scan_f16_dyn(const DevState& s, const StageBufs& b, int32_t n, int32_t m,
                               int split, int grab, hipStream_t st, LaunchEvents ev) {
  const int32_t n_batches = (n + 63) / 64;
  if (static_cast<int64_t>(n_batches) * 2048 >= (1LL << 31)) return hipErrorInvalidValue;
  if (split < 8 || split % 8 != 0 || split > kMaxSplit || grab < 1) return hipErrorInvalidValue;
  const int32_t sblocks = (m + kSignalsPerWG - 1) / kSignalsPerWG;
  launch_with(fh_scan_dyn, dim3(8 * sblocks * (split / 8)), dim3(256), st, ev, b.pu, b.pmh,
              b.pidx, n, b.ssig, m, b.seed, b.mag, b.bb, s.part, b.wctr, sblocks, grab);
  return hipGetLastError();
}

int f16_split(int32_t n, int32_t m, int cus, int want) {
  if (want > 0) return std::min(want, kMaxSplit);
  const int64_t sblocks = (m + kSignalsPerWG - 1) / kSignalsPerWG;
  // one round of work-groups: four per CU (four waves per SIMD), all resident from the
  // start; with the scan's progress-ordered priority they then finish close together
  // (measured better than two rounds at 8,192 and 16,384 signals, equal at 65,536)
  const int64_t target = 4LL * (cus > 0 ? cus : 256);
  int64_t sp = (target + sblocks - 1) / sblocks;
  sp = std::min<int64_t>(sp, (n + 2047) / 2048);
  return static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(sp, kMaxSplit)));
}

hipError_t launch_scan_f16(const DevState& s, const StageBufs& b, int32_t n, const float* sig,
                           int32_t m, int split, hipStream_t st, LaunchEvents ev) {
  const int32_t n_batches = (n + 63) / 64;
  // buffer offsets from a chunk's first batch are 32-bit: 2 KB per batch
  if (static_cast<int64_t>(n_batches) * 2048 >= (1LL << 31)) return hipErrorInvalidValue;
  dim3 grid((m + kSignalsPerWG - 1) / kSignalsPerWG, split);
  launch_with(fh_scan, grid, dim3(256), st, ev, b.pu, b.pmh, b.pidx, n, b.ssig, m, b.seed, b.mag,
              b.bb, s.part);
  return hipGetLastError();
}

}  // namespace gsn
