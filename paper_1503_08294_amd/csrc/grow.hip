// Growth of the network (Sec. 2.1: units are added and removed during the update; GNG
// inserts periodically next to the unit of largest accumulated error).
//
// Removal is a stable compaction: units marked by the edge update that still have no edge
// are dropped, the others keep their relative order, and every neighbour id is renumbered.
// Removed rows are empty, so the half-edge arrays keep their positions; only the row
// pointers are compacted and the column ids remapped.
//
// Insertion is a single small edit done by one workgroup: an argmax reduction over the
// errors, then one lane rewrites the rows of q and f in place and appends the row of the
// new unit r = N (its index is the largest, so appending keeps every row ascending).
#include "gsn_internal.h"

namespace gsn {
namespace {

inline int blocks(int64_t n) { return static_cast<int>((n + kBlock - 1) / kBlock); }

__global__ void gr_keep(int32_t n, const int32_t* __restrict__ rp,
                        const int32_t* __restrict__ orphan, int32_t* __restrict__ keep,
                        int32_t* __restrict__ bsum) {
  __shared__ int32_t red[kBlock];
  const int32_t u = blockIdx.x * kBlock + threadIdx.x;
  int32_t k = 0;
  if (u < n) {
    k = !(orphan[u] && rp[u + 1] == rp[u]);
    keep[u] = k;
  }
  red[threadIdx.x] = k;
  __syncthreads();
  for (int w = kBlock / 2; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) bsum[blockIdx.x] = red[0];
}

// New id of every unit (or -1), staged positions/errors at the new ids, compacted row
// pointers.  Overwrites keep[] with the new ids.
__global__ void gr_compact(int32_t n, int32_t n_max, int32_t* __restrict__ keep,
                           const int32_t* __restrict__ boff, const int32_t* __restrict__ rp,
                           int32_t* __restrict__ rp_new, const float* __restrict__ x,
                           const float* __restrict__ y, const float* __restrict__ z,
                           const float* __restrict__ err, float* __restrict__ tmp,
                           int32_t* __restrict__ orphan, const int32_t* __restrict__ status) {
  __shared__ int32_t sc[kBlock];
  const int32_t u = blockIdx.x * kBlock + threadIdx.x;
  const int32_t k = u < n ? keep[u] : 0;
  sc[threadIdx.x] = k;
  __syncthreads();
  for (int off = 1; off < kBlock; off <<= 1) {
    const int32_t v = threadIdx.x >= off ? sc[threadIdx.x - off] : 0;
    __syncthreads();
    sc[threadIdx.x] += v;
    __syncthreads();
  }
  if (u >= n) return;
  const int32_t id = k ? boff[blockIdx.x] + sc[threadIdx.x] - 1 : -1;
  keep[u] = id;
  orphan[u] = 0;
  if (id >= 0) {
    tmp[id] = x[u];
    tmp[n_max + id] = y[u];
    tmp[2 * n_max + id] = z[u];
    tmp[3 * n_max + id] = err[u];
    rp_new[id] = rp[u];
  }
  if (u == n - 1) rp_new[status[kStKept]] = rp[n];
}

// Renumber the neighbour ids of every kept row (positions unchanged).
__global__ void gr_remap(int32_t n, const int32_t* __restrict__ newid,
                         const int32_t* __restrict__ rp, const int32_t* __restrict__ col,
                         const int32_t* __restrict__ age, int32_t* __restrict__ col_new,
                         int32_t* __restrict__ age_new) {
  const int32_t u = blockIdx.x * kBlock + threadIdx.x;
  if (u >= n) return;
  for (int32_t k = rp[u]; k < rp[u + 1]; ++k) {
    col_new[k] = newid[col[k]];
    age_new[k] = age[k];
  }
}

__global__ void gr_copyback(int32_t n, int32_t n_max, const float* __restrict__ tmp,
                            float* __restrict__ x, float* __restrict__ y,
                            float* __restrict__ z, float* __restrict__ err,
                            int32_t* __restrict__ status) {
  const int32_t i = blockIdx.x * kBlock + threadIdx.x;
  const int32_t kept = status[kStKept];
  if (i == 0) status[kStOrphans] = 0;
  if (i >= n) return;
  if (i < kept) {
    x[i] = tmp[i];
    y[i] = tmp[n_max + i];
    z[i] = tmp[2 * n_max + i];
    err[i] = tmp[3 * n_max + i];
  } else {
    x[i] = 0.0f;
    y[i] = 0.0f;
    z[i] = 0.0f;
    err[i] = 0.0f;
  }
}

// Remove neighbour `gone` from the ascending row of u and append `added` (larger than
// every id in the row) at age 0.  The row keeps its length.
__device__ void replace_in_row(const int32_t* __restrict__ rp, int32_t* __restrict__ col,
                               int32_t* __restrict__ age, int32_t u, int32_t gone,
                               int32_t added) {
  const int32_t r0 = rp[u], r1 = rp[u + 1];
  int32_t k = r0;
  while (k < r1 && col[k] != gone) ++k;
  for (; k + 1 < r1; ++k) {
    col[k] = col[k + 1];
    age[k] = age[k + 1];
  }
  col[r1 - 1] = added;
  age[r1 - 1] = 0;
}

// One GNG insertion at unit index n (thread 0 only): q = argmax err (given), f = argmax err
// over the neighbours of q, r = n at the midpoint, {q, f} replaced by {q, r} and {r, f}.
// Returns 1 if a unit was added.
__device__ int insert_one(int32_t n, int32_t q, float alpha, int64_t half_cap,
                          int32_t* __restrict__ rp, int32_t* __restrict__ col,
                          int32_t* __restrict__ age, float* __restrict__ x,
                          float* __restrict__ y, float* __restrict__ z,
                          float* __restrict__ err, int32_t* __restrict__ status) {
  if (q < 0 || rp[q + 1] == rp[q]) return 0;
  int32_t f = col[rp[q]];
  for (int32_t k = rp[q] + 1; k < rp[q + 1]; ++k) {
    const int32_t v = col[k];
    if (err[v] > err[f]) f = v;  // ascending row: ties keep the lower index
  }
  const int32_t e2 = rp[n];
  if (static_cast<int64_t>(e2) + 2 > half_cap) {
    atomicCAS(&status[kStError], 0, GSN_E_CAPACITY);
    return 0;
  }
  const int32_t r = n;
  x[r] = (x[q] + x[f]) * 0.5f;
  y[r] = (y[q] + y[f]) * 0.5f;
  z[r] = (z[q] + z[f]) * 0.5f;
  replace_in_row(rp, col, age, q, f, r);
  replace_in_row(rp, col, age, f, q, r);
  col[e2] = min(q, f);
  col[e2 + 1] = max(q, f);
  age[e2] = 0;
  age[e2 + 1] = 0;
  rp[r + 1] = e2 + 2;
  err[q] = err[q] * alpha;
  err[f] = err[f] * alpha;
  err[r] = err[q];
  return 1;
}

// Up to `count` insertions one after another (each sees the errors and edges the previous
// one left), while N < n_max and the unit of largest error has a neighbour.  One workgroup:
// the argmax is a block reduction, the edge surgery runs on thread 0, and a device-scope
// fence and a barrier separate the insertions.
__global__ __launch_bounds__(1024) void gr_insert(int32_t n0, int32_t count, int32_t n_max,
                                                  float alpha, int64_t half_cap,
                                                  int32_t* __restrict__ rp,
                                                  int32_t* __restrict__ col,
                                                  int32_t* __restrict__ age,
                                                  float* __restrict__ x, float* __restrict__ y,
                                                  float* __restrict__ z,
                                                  float* __restrict__ err,
                                                  int32_t* __restrict__ status) {
  __shared__ float be[1024];
  __shared__ int32_t bi[1024];
  __shared__ int32_t added;
  const int32_t t = threadIdx.x;
  int32_t n = n0;
  int32_t done = 0;
  for (int32_t it = 0; it < count && n < n_max; ++it) {
    float e = -__builtin_huge_valf();
    int32_t idx = -1;
    for (int32_t i = t; i < n; i += 1024) {
      const float v = err[i];
      if (idx < 0 || v > e) {  // ascending i per lane: strict > keeps the lower index
        e = v;
        idx = i;
      }
    }
    be[t] = e;
    bi[t] = idx;
    __syncthreads();
    for (int w = 512; w > 0; w >>= 1) {
      if (t < w) {
        const float oe = be[t + w];
        const int32_t oi = bi[t + w];
        if (oi >= 0 && (bi[t] < 0 || oe > be[t] || (oe == be[t] && oi < bi[t]))) {
          be[t] = oe;
          bi[t] = oi;
        }
      }
      __syncthreads();
    }
    if (t == 0) added = insert_one(n, bi[0], alpha, half_cap, rp, col, age, x, y, z, err, status);
    __threadfence();
    __syncthreads();
    if (!added) break;
    ++n;
    ++done;
  }
  if (t == 0) status[kStInserted] = done;
}

}  // namespace

hipError_t launch_remove(const DevState& s, int cur, int32_t n, int32_t n_max,
                         hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int nxt = cur ^ 1;
  const int nb = blocks(n);
  gr_keep<<<nb, kBlock, 0, st>>>(n, s.rp[cur], s.orphan, s.cnt, s.bsum);
  hipError_t e = launch_scan_blocks(s.bsum, nb, INT64_MAX, nullptr, s.status, kStKept, st);
  if (e != hipSuccess) return e;
  gr_compact<<<nb, kBlock, 0, st>>>(n, n_max, s.cnt, s.bsum, s.rp[cur], s.rp[nxt], s.x, s.y,
                                    s.z, s.err, s.tmp, s.orphan, s.status);
  gr_remap<<<nb, kBlock, 0, st>>>(n, s.cnt, s.rp[cur], s.col[cur], s.age[cur], s.col[nxt],
                                  s.age[nxt]);
  gr_copyback<<<nb, kBlock, 0, st>>>(n, n_max, s.tmp, s.x, s.y, s.z, s.err, s.status);
  return hipGetLastError();
}

hipError_t launch_insert(const DevState& s, int cur, int32_t n, int32_t count, float alpha,
                         int32_t n_max, int64_t half_cap, hipStream_t st) {
  gr_insert<<<1, 1024, 0, st>>>(n, count, n_max, alpha, half_cap, s.rp[cur], s.col[cur],
                                s.age[cur], s.x, s.y, s.z, s.err, s.status);
  return hipGetLastError();
}

}  // namespace gsn
