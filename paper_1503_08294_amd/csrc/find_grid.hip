// Indexed find winners: the hash index of the paper's "Indexed" implementation (Sec. 3.1)
// applied to every signal of the batch.  A grid of cubes of side h over an axis-parallel
// box holds the units, counting-sorted by cube every call (units move every iteration); the
// winner and the second of a signal are searched among the units of its cube and the 26
// neighbours, one lane per cube (a group of 32 lanes per signal, the lanes' top-2 keys
// merged by shuffles), and signals whose 27 cubes hold fewer than two units get the
// exhaustive search.  Results equal the oracle's indexed search bit for bit: the same cell
// function, the same direct-form distance, the same (d, index) order.  In exact mode the
// 27-cube result is kept only where it is certified to be the exhaustive one.
#include "gsn_internal.h"

namespace gsn {
namespace {

constexpr int kGroupLanes = 32;            // lanes per signal (27 cubes, 5 idle)
constexpr int kQueryBlock = 256;           // 8 signals per workgroup
constexpr int kFallbackBlocks = 256;
constexpr unsigned long long kNoKey = ~0ull;

inline int blocks(int64_t n) { return static_cast<int>((n + kBlock - 1) / kBlock); }

__device__ __forceinline__ int32_t grid_axis(float p, float lo, float inv_h, int32_t dim) {
  const float t = (p - lo) * inv_h;
  if (!(t >= 0.0f)) return 0;                              // below the box (and NaN)
  if (t >= static_cast<float>(dim)) return dim - 1;        // beyond it
  const int32_t c = static_cast<int32_t>(floorf(t));
  return c < dim ? c : dim - 1;
}

struct GridArgs {
  float lo0, lo1, lo2, inv_h;
  int32_t d0, d1, d2;
  int exact;
};

__device__ __forceinline__ void cell_of(const GridArgs& g, float x, float y, float z,
                                        int32_t* c) {
  c[0] = grid_axis(x, g.lo0, g.inv_h, g.d0);
  c[1] = grid_axis(y, g.lo1, g.inv_h, g.d1);
  c[2] = grid_axis(z, g.lo2, g.inv_h, g.d2);
}

// (d, index) key: the unsigned order of the key is the lexicographic order (d >= +0).
__device__ __forceinline__ unsigned long long dkey(float d, int32_t i) {
  return (static_cast<unsigned long long>(__float_as_uint(d)) << 32) | static_cast<uint32_t>(i);
}

__device__ __forceinline__ float direct_d(float sx, float sy, float sz, float wx, float wy,
                                          float wz) {
  const float dx = sx - wx, dy = sy - wy, dz = sz - wz;
  return (dx * dx + dy * dy) + dz * dz;
}

// Certification of a signal's 27-cube result (exact mode).  With t = fl(fl(p - lo) inv_h)
// and x = (p - lo) inv_h exactly, t = x (1 + eta), |eta| <= 2u + u^2.  A unit in a cube two
// or more above the signal's on axis a has t_w >= c + 2, so x_w >= (c + 2) / (1 + |eta|);
// the signal has t_s < c + 1 (or t_s < 0), so x_s <= max(t_s, 0) / (1 - |eta|); below
// likewise with x_w < (c - 1) / (1 - |eta|) and x_s >= t_s / (1 + |eta|).  Every unit outside
// the 27 cubes is outside on some axis, so its true distance is at least r = the least of
// these gaps divided by inv_h (gaps computed in binary64 with a relative margin of 3e-7 >
// 2.01 u per factor and an absolute one for subnormal differences).  Its computed binary32
// distance is at least (1 - 5u) times the true one, so if d2 < r^2 (1 - 4e-7) every outside
// unit's computed distance exceeds d2 and the 27-cube top-2 is the exhaustive one.
__device__ bool certified(const GridArgs& g, float sx, float sy, float sz, const int32_t* c,
                          float d2) {
  const double up = 1.0 + 3e-7, dn = 1.0 - 3e-7;
  const float p[3] = {sx, sy, sz};
  const float lo[3] = {g.lo0, g.lo1, g.lo2};
  const int32_t dims[3] = {g.d0, g.d1, g.d2};
  double gap = __builtin_huge_val();  // in cells
  for (int a = 0; a < 3; ++a) {
    const double t = static_cast<double>((p[a] - lo[a]) * g.inv_h);
    if (c[a] + 2 <= dims[a] - 1) gap = fmin(gap, (c[a] + 2) * dn - fmax(t, 0.0) * up);
    if (c[a] - 2 >= 0) gap = fmin(gap, t * dn - (c[a] - 1) * up);
  }
  if (gap == __builtin_huge_val()) return d2 < __builtin_huge_valf();  // the cubes hold all
  gap -= 1e-30;
  if (!(gap > 0.0)) return false;
  const double r = gap / static_cast<double>(g.inv_h) * (1.0 - 1e-12);
  return static_cast<double>(d2) < r * r * (1.0 - 4e-7);
}

__device__ __forceinline__ void top2_insert(unsigned long long k, unsigned long long& k1,
                                            unsigned long long& k2) {
  if (k < k1) {
    k2 = k1;
    k1 = k;
  } else if (k < k2) {
    k2 = k;
  }
}

__global__ void gx_clear(int32_t* __restrict__ cnt, int32_t cells, int32_t* __restrict__ nfb) {
  const int32_t stride = gridDim.x * kBlock;
  for (int32_t c = blockIdx.x * kBlock + threadIdx.x; c < cells; c += stride) cnt[c] = 0;
  if (blockIdx.x == 0 && threadIdx.x == 0) *nfb = 0;
}

__global__ void gx_count(int32_t n, const float* __restrict__ x, const float* __restrict__ y,
                         const float* __restrict__ z, GridArgs g, int32_t* __restrict__ ucell,
                         int32_t* __restrict__ cnt) {
  const int32_t u = blockIdx.x * kBlock + threadIdx.x;
  if (u >= n) return;
  int32_t c[3];
  cell_of(g, x[u], y[u], z[u], c);
  const int32_t lin = (c[2] * g.d1 + c[1]) * g.d0 + c[0];
  ucell[u] = lin;
  atomicAdd(&cnt[lin], 1);
}

__global__ void gx_bsum(int32_t cells, const int32_t* __restrict__ cnt,
                        int32_t* __restrict__ bsum) {
  __shared__ int32_t red[kBlock];
  const int32_t c = blockIdx.x * kBlock + threadIdx.x;
  red[threadIdx.x] = c < cells ? cnt[c] : 0;
  __syncthreads();
  for (int w = kBlock / 2; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) bsum[blockIdx.x] = red[0];
}

// start[c] = units in the cubes before c; cnt[c] becomes the scatter cursor start[c].
__global__ void gx_start(int32_t cells, int32_t n, int32_t* __restrict__ cnt,
                         const int32_t* __restrict__ boff, int32_t* __restrict__ start) {
  __shared__ int32_t sc[kBlock];
  const int32_t c = blockIdx.x * kBlock + threadIdx.x;
  const int32_t v = c < cells ? cnt[c] : 0;
  sc[threadIdx.x] = v;
  __syncthreads();
  for (int off = 1; off < kBlock; off <<= 1) {
    const int32_t t = threadIdx.x >= off ? sc[threadIdx.x - off] : 0;
    __syncthreads();
    sc[threadIdx.x] += t;
    __syncthreads();
  }
  if (c < cells) {
    const int32_t s = boff[blockIdx.x] + sc[threadIdx.x] - v;
    start[c] = s;
    cnt[c] = s;
  }
  if (c == 0) start[cells] = n;
}

__global__ void gx_scatter(int32_t n, const float* __restrict__ x, const float* __restrict__ y,
                           const float* __restrict__ z, const int32_t* __restrict__ ucell,
                           int32_t* __restrict__ cursor, float4* __restrict__ sorted) {
  const int32_t u = blockIdx.x * kBlock + threadIdx.x;
  if (u >= n) return;
  const int32_t pos = atomicAdd(&cursor[ucell[u]], 1);
  sorted[pos] = make_float4(x[u], y[u], z[u], __int_as_float(u));
}

// 32 lanes per signal: lane q < 27 scans cube (cx + q % 3 - 1, cy + (q / 3) % 3 - 1,
// cz + q / 9 - 1).  The lanes' top-2 keys and candidate counts are merged by shuffles
// within the 32 lanes; fewer than two candidates (or, in exact mode, a result that cannot
// be certified) sends the signal to the fallback list.
__global__ void gx_query(const float* __restrict__ sig, int32_t m, GridArgs g,
                         const int32_t* __restrict__ start, const float4* __restrict__ sorted,
                         int32_t* __restrict__ winner, int32_t* __restrict__ second,
                         float* __restrict__ d1, float* __restrict__ d2,
                         int32_t* __restrict__ fb_list, int32_t* __restrict__ nfb) {
  const int32_t gt = blockIdx.x * kQueryBlock + threadIdx.x;
  const int32_t j = gt / kGroupLanes;
  const int q = gt % kGroupLanes;
  if (j >= m) return;  // whole groups: m groups fill the grid exactly up to the last block
  const float sx = sig[j], sy = sig[m + j], sz = sig[2 * m + j];
  int32_t c[3];
  cell_of(g, sx, sy, sz, c);
  unsigned long long k1 = kNoKey, k2 = kNoKey;
  int32_t found = 0;
  if (q < 27) {
    const int32_t cx = c[0] + q % 3 - 1, cy = c[1] + (q / 3) % 3 - 1, cz = c[2] + q / 9 - 1;
    if (cx >= 0 && cx < g.d0 && cy >= 0 && cy < g.d1 && cz >= 0 && cz < g.d2) {
      const int32_t lin = (cz * g.d1 + cy) * g.d0 + cx;
      const int32_t a = start[lin], b = start[lin + 1];
      found = b - a;
      for (int32_t k = a; k < b; ++k) {
        const float4 w = sorted[k];
        top2_insert(dkey(direct_d(sx, sy, sz, w.x, w.y, w.z), __float_as_int(w.w)), k1, k2);
      }
    }
  }
  for (int off = kGroupLanes / 2; off > 0; off >>= 1) {
    const unsigned long long o1 = __shfl_xor(k1, off, kGroupLanes);
    const unsigned long long o2 = __shfl_xor(k2, off, kGroupLanes);
    found += __shfl_xor(found, off, kGroupLanes);
    // top two of {k1, k2, o1, o2} (each pair ascending, all keys distinct or none)
    const unsigned long long lo = k1 < o1 ? k1 : o1, hi = k1 < o1 ? o1 : k1;
    const unsigned long long rest = k2 < o2 ? k2 : o2;
    k1 = lo;
    k2 = hi < rest ? hi : rest;
  }
  if (q != 0) return;
  if (found < 2 ||
      (g.exact && !certified(g, sx, sy, sz, c, __uint_as_float(static_cast<uint32_t>(k2 >> 32))))) {
    fb_list[atomicAdd(nfb, 1)] = j;
    return;
  }
  winner[j] = static_cast<int32_t>(k1 & 0xFFFFFFFFu);
  second[j] = static_cast<int32_t>(k2 & 0xFFFFFFFFu);
  d1[j] = __uint_as_float(static_cast<uint32_t>(k1 >> 32));
  d2[j] = __uint_as_float(static_cast<uint32_t>(k2 >> 32));
}

// The exhaustive search for the signals on the fallback list: one workgroup per signal at a
// time (a fixed grid looping over the list), the threads' top-2 keys merged in LDS.
__global__ void gx_fallback(const float* __restrict__ sig, int32_t m, int32_t n,
                            const float* __restrict__ x, const float* __restrict__ y,
                            const float* __restrict__ z, const int32_t* __restrict__ fb_list,
                            const int32_t* __restrict__ nfb, int32_t* __restrict__ winner,
                            int32_t* __restrict__ second, float* __restrict__ d1,
                            float* __restrict__ d2) {
  __shared__ unsigned long long s1[kBlock], s2[kBlock];
  const int32_t count = *nfb;
  for (int32_t e = blockIdx.x; e < count; e += gridDim.x) {
    const int32_t j = fb_list[e];
    const float sx = sig[j], sy = sig[m + j], sz = sig[2 * m + j];
    unsigned long long k1 = kNoKey, k2 = kNoKey;
    for (int32_t i = threadIdx.x; i < n; i += kBlock)
      top2_insert(dkey(direct_d(sx, sy, sz, x[i], y[i], z[i]), i), k1, k2);
    s1[threadIdx.x] = k1;
    s2[threadIdx.x] = k2;
    __syncthreads();
    for (int w = kBlock / 2; w > 0; w >>= 1) {
      if (threadIdx.x < w) {
        const unsigned long long a1 = s1[threadIdx.x], a2 = s2[threadIdx.x];
        const unsigned long long b1 = s1[threadIdx.x + w], b2 = s2[threadIdx.x + w];
        const unsigned long long lo = a1 < b1 ? a1 : b1, hi = a1 < b1 ? b1 : a1;
        const unsigned long long rest = a2 < b2 ? a2 : b2;
        s1[threadIdx.x] = lo;
        s2[threadIdx.x] = hi < rest ? hi : rest;
      }
      __syncthreads();
    }
    if (threadIdx.x == 0) {
      winner[j] = static_cast<int32_t>(s1[0] & 0xFFFFFFFFu);
      second[j] = static_cast<int32_t>(s2[0] & 0xFFFFFFFFu);
      d1[j] = __uint_as_float(static_cast<uint32_t>(s1[0] >> 32));
      d2[j] = __uint_as_float(static_cast<uint32_t>(s2[0] >> 32));
    }
    __syncthreads();
  }
}

}  // namespace

// Regions of the caller's grid workspace (offsets from its 256-aligned base).
static void grid_layout(int64_t cells, int32_t n_max, int32_t m_max, size_t* off) {
  size_t o = 0;
  const size_t sz[7] = {4 * static_cast<size_t>(cells + 1), 4 * static_cast<size_t>(cells + 1),
                        4 * static_cast<size_t>(cells / kBlock + 2),
                        16 * static_cast<size_t>(n_max), 4 * static_cast<size_t>(n_max),
                        4 * static_cast<size_t>(m_max), 256};
  for (int i = 0; i < 7; ++i) {
    off[i] = o;
    o = (o + sz[i] + 255) & ~static_cast<size_t>(255);
  }
  off[7] = o;
}

size_t grid_bytes(int64_t cells, int32_t n_max, int32_t m_max) {
  size_t off[8];
  grid_layout(cells, n_max, m_max, off);
  return off[7];
}

GridBufs carve_grid(void* base, int64_t cells, int32_t n_max, int32_t m_max) {
  size_t off[8];
  grid_layout(cells, n_max, m_max, off);
  char* b = static_cast<char*>(base);
  GridBufs g;
  g.cnt = reinterpret_cast<int32_t*>(b + off[0]);
  g.start = reinterpret_cast<int32_t*>(b + off[1]);
  g.bsum = reinterpret_cast<int32_t*>(b + off[2]);
  g.sorted = reinterpret_cast<float4*>(b + off[3]);
  g.ucell = reinterpret_cast<int32_t*>(b + off[4]);
  g.fb_list = reinterpret_cast<int32_t*>(b + off[5]);
  g.nfb = reinterpret_cast<int32_t*>(b + off[6]);
  return g;
}

hipError_t launch_find_grid(const DevState& s, const GridBufs& gb, const GridSpec& spec,
                            int32_t n, const float* sig, int32_t m, int32_t* winner,
                            int32_t* second, float* d1, float* d2, hipStream_t st) {
  const int32_t cells = static_cast<int32_t>(spec.cells);
  const GridArgs g{spec.lo[0], spec.lo[1], spec.lo[2], spec.inv_h,
                   spec.dims[0], spec.dims[1], spec.dims[2], spec.exact};
  gx_clear<<<std::min(blocks(cells), 1024), kBlock, 0, st>>>(gb.cnt, cells, gb.nfb);
  gx_count<<<blocks(n), kBlock, 0, st>>>(n, s.x, s.y, s.z, g, gb.ucell, gb.cnt);
  const int nb = blocks(cells);
  gx_bsum<<<nb, kBlock, 0, st>>>(cells, gb.cnt, gb.bsum);
  hipError_t e = launch_scan_blocks(gb.bsum, nb, INT64_MAX, nullptr, s.status, -1, st);
  if (e != hipSuccess) return e;
  gx_start<<<nb, kBlock, 0, st>>>(cells, n, gb.cnt, gb.bsum, gb.start);
  gx_scatter<<<blocks(n), kBlock, 0, st>>>(n, s.x, s.y, s.z, gb.ucell, gb.cnt, gb.sorted);
  const int64_t lanes = static_cast<int64_t>(m) * kGroupLanes;
  gx_query<<<static_cast<int>((lanes + kQueryBlock - 1) / kQueryBlock), kQueryBlock, 0, st>>>(
      sig, m, g, gb.start, gb.sorted, winner, second, d1, d2, gb.fb_list, gb.nfb);
  gx_fallback<<<kFallbackBlocks, kBlock, 0, st>>>(sig, m, n, s.x, s.y, s.z, gb.fb_list, gb.nfb,
                                                  winner, second, d1, d2);
  return hipGetLastError();
}

}  // namespace gsn
