// Growth of the network (Sec. 2.1: units are added and removed during the update; GNG
// inserts periodically next to the unit of largest accumulated error).
//
// Removal is a stable compaction: units marked by the edge update that still have no edge
// are dropped, the others keep their relative order, and every neighbour id is renumbered.
// Removed rows are empty, so the half-edge arrays keep their positions; only the row
// pointers are compacted and the column ids remapped.
//
// Insertion runs in one workgroup, one unit after another: the argmax over per-segment
// maxima of the errors held in LDS, the rows of q and f rewritten in place and the row of
// the new unit r = N appended (its index is the largest, so every row stays ascending);
// only the segments of q, f and r are rescanned after an insertion.
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

// ------------------------------------------------------------------ insertion ----
// GNG insertion (Sec. 2.1): q = the unit of largest error, f = the neighbour of q of
// largest error (ties to the lower index for both), a unit r = N at their midpoint, the edge
// {q, f} replaced by {q, r} and {r, f} at age 0, err_q and err_f scaled by alpha, and
// err_r = err_q.  Several insertions run one after another in one workgroup; the argmax
// over all units goes over per-segment maxima held in LDS, and after every insertion only
// the segments of q, f and r are rescanned.

constexpr int kMaxSeg = 4096;  // segments held in LDS

// Order key for the argmax: larger error first, then the lower index (errors are >= +0, so
// their bits order like their values).  0 means "no unit".
__device__ __forceinline__ unsigned long long err_key(float e, int32_t i) {
  return (static_cast<unsigned long long>(__float_as_uint(e)) << 32) |
         (0xFFFFFFFFu - static_cast<uint32_t>(i));
}
__device__ __forceinline__ int32_t key_index(unsigned long long k) {
  return static_cast<int32_t>(0xFFFFFFFFu - static_cast<uint32_t>(k));
}

__device__ __forceinline__ unsigned long long wave_max(unsigned long long v) {
  for (int off = 32; off > 0; off >>= 1) {
    const unsigned long long o = __shfl_xor(v, off);
    v = o > v ? o : v;
  }
  return v;
}

// Key of the best unit of segment sg (units [sg len, sg len + len) below n), by one wave.
__device__ unsigned long long segment_key(const float* __restrict__ err, int32_t n, int32_t sg,
                                          int32_t len) {
  const int lane = static_cast<int>(threadIdx.x & 63);
  unsigned long long best = 0;
  const int32_t end = min(n, (sg + 1) * len);
  for (int32_t i = sg * len + lane; i < end; i += 64) {
    const unsigned long long k = err_key(err[i], i);
    best = k > best ? k : best;
  }
  return wave_max(best);
}

__global__ void gr_segmax(int32_t n, int32_t len, int32_t nseg, const float* __restrict__ err,
                          unsigned long long* __restrict__ seg) {
  const int32_t sg = (blockIdx.x * kBlock + threadIdx.x) >> 6;
  if (sg >= nseg) return;  // whole waves
  const unsigned long long k = segment_key(err, n, sg, len);
  if ((threadIdx.x & 63) == 0) seg[sg] = k;
}

// Remove `gone` from the ascending row of u and append `added` (larger than every id in the
// row) at age 0, by one wave: lanes hold the entries, the ones after `gone` move down.
__device__ void wave_replace(const int32_t* __restrict__ rp, int32_t* __restrict__ col,
                             int32_t* __restrict__ age, int32_t u, int32_t gone,
                             int32_t added) {
  const int lane = static_cast<int>(threadIdx.x & 63);
  const int32_t r0 = rp[u], r1 = rp[u + 1], l = r1 - r0;
  if (l > 64) {
    if (lane == 0) {
      int32_t k = r0;
      while (k < r1 && col[k] != gone) ++k;
      for (; k + 1 < r1; ++k) {
        col[k] = col[k + 1];
        age[k] = age[k + 1];
      }
      col[r1 - 1] = added;
      age[r1 - 1] = 0;
    }
    return;
  }
  int32_t c = -1, a = 0;
  if (lane < l) {
    c = col[r0 + lane];
    a = age[r0 + lane];
  }
  const unsigned long long at = __ballot(lane < l && c == gone);
  const int pos = at ? __ffsll(static_cast<long long>(at)) - 1 : l;
  if (lane < l && lane > pos) {
    col[r0 + lane - 1] = c;
    age[r0 + lane - 1] = a;
  }
  if (lane == 0) {
    col[r1 - 1] = added;
    age[r1 - 1] = 0;
  }
}

// One insertion at r = n with q given, by one wave; returns 1 if a unit was added and the
// chosen f in *f_out.
__device__ int wave_insert(int32_t n, int32_t q, float alpha, int64_t half_cap,
                           int32_t* __restrict__ rp, int32_t* __restrict__ col,
                           int32_t* __restrict__ age, float* __restrict__ x,
                           float* __restrict__ y, float* __restrict__ z,
                           float* __restrict__ err, int32_t* __restrict__ status,
                           int32_t* f_out) {
  const int lane = static_cast<int>(threadIdx.x & 63);
  if (q < 0) return 0;
  const int32_t r0 = rp[q], r1 = rp[q + 1];
  if (r1 == r0) return 0;
  unsigned long long best = 0;
  for (int32_t k = r0 + lane; k < r1; k += 64) {
    const int32_t v = col[k];
    const unsigned long long kk = err_key(err[v], v);
    best = kk > best ? kk : best;
  }
  const int32_t f = key_index(wave_max(best));
  const int32_t e2 = rp[n];
  if (static_cast<int64_t>(e2) + 2 > half_cap) {
    if (lane == 0) atomicCAS(&status[kStError], 0, GSN_E_CAPACITY);
    return 0;
  }
  const int32_t r = n;
  wave_replace(rp, col, age, q, f, r);
  wave_replace(rp, col, age, f, q, r);
  if (lane == 0) {
    x[r] = (x[q] + x[f]) * 0.5f;
    y[r] = (y[q] + y[f]) * 0.5f;
    z[r] = (z[q] + z[f]) * 0.5f;
    col[e2] = min(q, f);
    col[e2 + 1] = max(q, f);
    age[e2] = 0;
    age[e2 + 1] = 0;
    rp[r + 1] = e2 + 2;
    err[q] = err[q] * alpha;
    err[f] = err[f] * alpha;
    err[r] = err[q];
  }
  *f_out = f;
  return 1;
}

// Up to `count` insertions one after another (each sees the errors and edges the previous
// one left), while N < n_max and the unit of largest error has a neighbour.  seg holds the
// segment keys of the n0 units on entry (gr_segmax).  A barrier separates the phases of an
// insertion (one workgroup: its ordering covers what the waves share).  Per insertion, wave
// 0 takes q (the best segment key), then in three dependent rounds of loads q's row bounds,
// position and error; q's row; every neighbour's error, row bounds and position, so that
// f's come with the choice of f.  It writes the three new errors, and while waves 1-3
// rescan the segments of q, f and r, it rewrites the rows of q and f (one more round of
// loads, f's row) and adds r.  Rows longer than 64 entries take the one-lane path.
__global__ __launch_bounds__(1024) void gr_insert(int32_t n0, int32_t count, int32_t n_max,
                                                  int32_t len, float alpha, int64_t half_cap,
                                                  const unsigned long long* __restrict__ seg,
                                                  int32_t* __restrict__ rp,
                                                  int32_t* __restrict__ col,
                                                  int32_t* __restrict__ age,
                                                  float* __restrict__ x, float* __restrict__ y,
                                                  float* __restrict__ z,
                                                  float* __restrict__ err,
                                                  int32_t* __restrict__ status) {
  __shared__ unsigned long long sk[kMaxSeg];
  __shared__ unsigned long long red[16];
  __shared__ int32_t s_q, s_f, s_added, s_long;
  const int t = threadIdx.x, w = t >> 6, lane = t & 63;
  int32_t nseg = (n0 + len - 1) / len;
  for (int32_t i = t; i < nseg; i += 1024) sk[i] = seg[i];
  __syncthreads();
  int32_t n = n0;
  int32_t done = 0;
  for (int32_t it = 0; it < count && n < n_max; ++it) {
    // q: the best segment key
    unsigned long long best = 0;
    for (int32_t i = t; i < nseg; i += 1024) best = sk[i] > best ? sk[i] : best;
    best = wave_max(best);
    if (lane == 0) red[w] = best;
    __syncthreads();
    if (w == 0) {
      unsigned long long b = lane < 16 ? red[lane] : 0;
      b = wave_max(b);
      if (lane == 0) s_q = b ? key_index(b) : -1;
    }
    __syncthreads();
    const int32_t q = s_q, r = n;
    // wave 0: choose f, write the new errors (registers keep q's row for the surgery)
    int32_t r0 = 0, r1 = 0, e2 = 0, l = 0, v = -1, av = 0, kf = 0, f = -1, f0 = 0, f1 = 0;
    float xq = 0.0f, yq = 0.0f, zq = 0.0f, xf = 0.0f, yf = 0.0f, zf = 0.0f;
    if (w == 0) {
      int added = 0, longrow = 0;
      if (q >= 0) {
        r0 = rp[q];
        r1 = rp[q + 1];
        e2 = rp[n];
        xq = x[q];
        yq = y[q];
        zq = z[q];
        const float eq = err[q];
        l = r1 - r0;
        if (l > 64) {
          longrow = 1;
        } else if (l > 0) {
          if (static_cast<int64_t>(e2) + 2 > half_cap) {
            if (lane == 0) atomicCAS(&status[kStError], 0, GSN_E_CAPACITY);
          } else {
            float ev = 0.0f, xv = 0.0f, yv = 0.0f, zv = 0.0f;
            int32_t rv0 = 0, rv1 = 0;
            unsigned long long kv = 0;
            if (lane < l) {
              v = col[r0 + lane];
              av = age[r0 + lane];
            }
            if (lane < l) {
              ev = err[v];
              rv0 = rp[v];
              rv1 = rp[v + 1];
              xv = x[v];
              yv = y[v];
              zv = z[v];
              kv = err_key(ev, v);
            }
            f = key_index(wave_max(kv));
            kf = __ffsll(static_cast<long long>(__ballot(lane < l && v == f))) - 1;
            f0 = __shfl(rv0, kf);
            f1 = __shfl(rv1, kf);
            xf = __shfl(xv, kf);
            yf = __shfl(yv, kf);
            zf = __shfl(zv, kf);
            const float ef = __shfl(ev, kf);
            if (lane == 0) {
              err[q] = eq * alpha;
              err[f] = ef * alpha;
              err[r] = eq * alpha;
            }
            added = 1;
          }
        }
      }
      if (lane == 0) {
        s_added = added;
        s_long = longrow;
        s_f = f;
      }
    }
    __syncthreads();
    if (s_long) {
      // a row longer than 64 entries: the whole insertion on one wave as before
      if (w == 0) {
        int32_t ff = -1;
        const int a = wave_insert(n, q, alpha, half_cap, rp, col, age, x, y, z, err, status,
                                  &ff);
        if (lane == 0) {
          s_added = a;
          s_f = ff;
        }
      }
      __syncthreads();
    }
    if (!s_added) break;
    ++n;
    ++done;
    if (w >= 1 && w <= 3) {
      // rescan the segments of q, f and r (equal segments give equal keys)
      const int32_t u = w == 1 ? q : (w == 2 ? s_f : r);
      const unsigned long long k = segment_key(err, n, u / len, len);
      if (lane == 0) sk[u / len] = k;
    } else if (w == 0 && !s_long) {
      // rows of q (f -> r) and f (q -> r), and the new unit r
      if (lane < l && lane > kf) {
        col[r0 + lane - 1] = v;
        age[r0 + lane - 1] = av;
      }
      if (lane == 0) {
        col[r1 - 1] = r;
        age[r1 - 1] = 0;
      }
      const int32_t lf = f1 - f0;
      if (lf > 64) {
        if (lane == 0) {
          int32_t k = f0;
          while (k < f1 && col[k] != q) ++k;
          for (; k + 1 < f1; ++k) {
            col[k] = col[k + 1];
            age[k] = age[k + 1];
          }
          col[f1 - 1] = r;
          age[f1 - 1] = 0;
        }
      } else {
        int32_t c = -1, a = 0;
        if (lane < lf) {
          c = col[f0 + lane];
          a = age[f0 + lane];
        }
        const unsigned long long at = __ballot(lane < lf && c == q);
        const int pos = at ? __ffsll(static_cast<long long>(at)) - 1 : lf;
        if (lane < lf && lane > pos) {
          col[f0 + lane - 1] = c;
          age[f0 + lane - 1] = a;
        }
        if (lane == 0) {
          col[f1 - 1] = r;
          age[f1 - 1] = 0;
        }
      }
      if (lane == 0) {
        x[r] = (xq + xf) * 0.5f;
        y[r] = (yq + yf) * 0.5f;
        z[r] = (zq + zf) * 0.5f;
        col[e2] = min(q, f);
        col[e2 + 1] = max(q, f);
        age[e2] = 0;
        age[e2 + 1] = 0;
        rp[r + 1] = e2 + 2;
      }
    }
    nseg = (n + len - 1) / len;
    __syncthreads();
  }
  if (t == 0) status[kStInserted] = done;
}

// --------------------------------------------------- speculative insertion rounds ----
// Many insertions per call are taken in rounds that each apply, at once, a prefix of the
// sequential order that is known to be exact.  A round selects the pool: the units whose key
// exceeds T, T being the (K + 1)-th largest segment key (every unit above T lies in one of
// the K segments above it), sorted by key.  It guesses that step i takes q_i = the i-th
// pool unit and f_i = the best neighbour in q_i's row as it is now, and accepts the
// longest prefix in which (a) every lowered key of the earlier steps (alpha e_q for q_j and
// r_j, alpha e_f for f_j) stays below the key of q_i, and (b) neither q_i nor any neighbour
// of q_i is a q_j or f_j of an earlier step.  Then q_i is the largest key after the earlier
// steps (the pool holds every larger original key, all of them earlier q's), q_i's row and
// its neighbours' keys are untouched, so f_i is the sequential f, and f_i's row too; the
// q's and f's of the prefix are pairwise distinct and the prefix applies in one parallel
// pass.  Step 0 always qualifies, unless q_0's row is longer than 64 entries (it then takes
// the one-wave insertion) or empty (insertion stops, as in the sequential order).
constexpr int kSpecSeg = 64;      // segments above T at most (halved while the pool overflows)
constexpr int kSpecPool = 512;    // pool units
constexpr int kSpecRows = 4096;   // row entries of the pool units
constexpr int kSpecHash = 2048;   // unit -> first step that touches it (power of two)
constexpr int kSpecMin = 8;       // fewer insertions: the sequential kernel

__device__ __forceinline__ float key_err(unsigned long long k) {
  return __uint_as_float(static_cast<uint32_t>(k >> 32));
}

// The k-th largest (1-based, k <= nk) of nk distinct keys, by an 8-bit radix select from
// the top byte down; every thread of the workgroup calls it (it holds barriers).
__device__ unsigned long long kth_largest(const unsigned long long* keys, int32_t nk,
                                          int32_t k, int32_t* hist, int32_t* s_bin,
                                          int32_t* s_k) {
  const int t = threadIdx.x, lane = t & 63;
  unsigned long long prefix = 0, mask = 0;
  int32_t kk = k;
  for (int shift = 56; shift >= 0; shift -= 8) {
    for (int32_t i = t; i < 256; i += blockDim.x) hist[i] = 0;
    __syncthreads();
    for (int32_t i = t; i < nk; i += blockDim.x) {
      const unsigned long long v = keys[i];
      if ((v & mask) == prefix) atomicAdd(&hist[(v >> shift) & 255], 1);
    }
    __syncthreads();
    if (t < 64) {
      // lane l holds bins 255 - 4l ... 252 - 4l; counts accumulate from the top bin down
      int32_t c[4], sum = 0;
      for (int a = 0; a < 4; ++a) {
        c[a] = hist[255 - 4 * lane - a];
        sum += c[a];
      }
      int32_t incl = sum;
      for (int o = 1; o < 64; o <<= 1) {
        const int32_t v = __shfl_up(incl, o);
        if (lane >= o) incl += v;
      }
      const int32_t excl = incl - sum;
      if (excl < kk && kk <= incl) {
        int32_t run = excl;
        for (int a = 0; a < 4; ++a) {
          if (run + c[a] >= kk) {
            *s_bin = 255 - 4 * lane - a;
            *s_k = kk - run;
            break;
          }
          run += c[a];
        }
      }
    }
    __syncthreads();
    prefix |= static_cast<unsigned long long>(*s_bin) << shift;
    mask |= 255ull << shift;
    kk = *s_k;
    __syncthreads();
  }
  return prefix;
}

__device__ __forceinline__ uint32_t spec_hash(int32_t u) {
  return (static_cast<uint32_t>(u) * 2654435761u) & (kSpecHash - 1);
}

// first step touching u, or INT32_MAX
__device__ int32_t touch_find(const int32_t* hk, const int32_t* hv, int32_t u) {
  uint32_t h = spec_hash(u);
  for (int probe = 0; probe < kSpecHash; ++probe) {
    const int32_t v = hk[h];
    if (v == u) return hv[h];
    if (v < 0) return INT32_MAX;
    h = (h + 1) & (kSpecHash - 1);
  }
  return INT32_MAX;
}

// records that step i touches u (at most 2 kSpecPool < kSpecHash units per round)
__device__ void touch_put(int32_t* hk, int32_t* hv, int32_t u, int32_t i) {
  uint32_t h = spec_hash(u);
  for (int probe = 0; probe < kSpecHash; ++probe) {
    const int32_t prev = atomicCAS(&hk[h], -1, u);
    if (prev == -1 || prev == u) {
      atomicMin(&hv[h], i);
      return;
    }
    h = (h + 1) & (kSpecHash - 1);
  }
}

// key of segment sg by a group of 16 consecutive lanes (sub = lane within the group); every
// lane of the wave calls it (sg < 0: a group with nothing to scan)
__device__ unsigned long long segment_key16(const float* __restrict__ err, int32_t n,
                                            int32_t sg, int32_t len, int sub) {
  unsigned long long best = 0;
  if (sg >= 0) {
    const int32_t end = min(n, (sg + 1) * len);
    for (int32_t i = sg * len + sub; i < end; i += 16) {
      const unsigned long long k = err_key(err[i], i);
      best = k > best ? k : best;
    }
  }
  for (int off = 8; off > 0; off >>= 1) {
    const unsigned long long o = __shfl_xor(best, off, 16);
    best = o > best ? o : best;
  }
  return best;
}

__global__ __launch_bounds__(1024) void gr_insert_spec(
    int32_t n0, int32_t count, int32_t n_max, int32_t len, float alpha, int64_t half_cap,
    const unsigned long long* __restrict__ seg, int32_t* __restrict__ rp,
    int32_t* __restrict__ col, int32_t* __restrict__ age, float* __restrict__ x,
    float* __restrict__ y, float* __restrict__ z, float* __restrict__ err,
    int32_t* __restrict__ status) {
  __shared__ unsigned long long sk[kMaxSeg];
  __shared__ int32_t hist[256];
  __shared__ unsigned long long pkey[kSpecPool], skey[kSpecPool];
  __shared__ unsigned long long st_best[kSpecPool], st_mod[kSpecPool];
  __shared__ int32_t st_r0[kSpecPool], st_deg[kSpecPool], st_off[kSpecPool], st_f[kSpecPool];
  __shared__ int32_t row_nb[kSpecRows], row_age[kSpecRows];
  __shared__ int32_t hk[kSpecHash], hv[kSpecHash];
  __shared__ uint32_t mark[kMaxSeg / 32];
  __shared__ int32_t list[3 * kSpecPool];
  __shared__ int32_t s_bin, s_k, s_cnt, s_lbad, s_lzero, s_total, s_e2, s_ok;
  const int t = threadIdx.x, w = t >> 6, lane = t & 63;
  int32_t nseg = (n0 + len - 1) / len;
  for (int32_t i = t; i < nseg; i += 1024) sk[i] = seg[i];
  __syncthreads();
  int32_t n = n0, done = 0, kseg = kSpecSeg;
  bool stop = false;
  while (!stop && done < count && n < n_max) {
    // ---- T and the pool (the units above T, at most kSpecPool of them)
    const unsigned long long T = nseg > kseg ? kth_largest(sk, nseg, kseg + 1, hist, &s_bin, &s_k)
                                             : 0ull;
    if (t == 0) s_cnt = 0;
    __syncthreads();
    for (int32_t i = t; i < nseg; i += 1024)
      if (sk[i] > T) {
        const int32_t k = atomicAdd(&s_cnt, 1);
        if (k < 3 * kSpecPool) list[k] = i;
      }
    __syncthreads();
    const int32_t nl = min(s_cnt, 3 * kSpecPool);
    __syncthreads();
    if (t == 0) s_cnt = 0;
    __syncthreads();
    for (int32_t e = t; e < nl * len; e += 1024) {
      const int32_t u = list[e / len] * len + e % len;
      if (u < n) {
        const unsigned long long k = err_key(err[u], u);
        if (k > T) {
          const int32_t at = atomicAdd(&s_cnt, 1);
          if (at < kSpecPool) pkey[at] = k;
        }
      }
    }
    __syncthreads();
    const int32_t C = s_cnt;
    __syncthreads();
    bool slow = false;
    if (C > kSpecPool) {
      if (kseg > 1) {
        kseg >>= 1;
        continue;
      }
      slow = true;  // one segment holds more pool units than fit: one sequential insertion
    }
    int32_t L = 0;
    if (!slow) {
      // ---- the pool in descending key order (ranks of distinct keys)
      if (t < C) {
        const unsigned long long k = pkey[t];
        int32_t r = 0;
        for (int32_t j = 0; j < C; ++j) r += pkey[j] > k;
        skey[r] = k;
      }
      for (int32_t i = t; i < kSpecHash; i += 1024) {
        hk[i] = -1;
        hv[i] = INT32_MAX;
      }
      if (t == 0) {
        s_e2 = rp[n];
        s_lbad = INT32_MAX;
        s_lzero = INT32_MAX;
      }
      __syncthreads();
      // ---- the rows of the guessed q's (rows over 64 entries, or past kSpecRows, stay out)
      if (t < C) {
        const int32_t q = key_index(skey[t]);
        const int32_t r0 = rp[q];
        st_r0[t] = r0;
        st_deg[t] = rp[q + 1] - r0;
        st_best[t] = 0;
      }
      __syncthreads();
      if (w == 0) {
        int32_t run = 0;
        for (int32_t b = 0; b < C; b += 64) {
          const int32_t i = b + lane;
          const int32_t l = i < C && st_deg[i] <= 64 ? st_deg[i] : 0;
          int32_t inc = l;
          for (int o = 1; o < 64; o <<= 1) {
            const int32_t v = __shfl_up(inc, o);
            if (lane >= o) inc += v;
          }
          if (i < C) st_off[i] = run + inc - l <= kSpecRows - l ? run + inc - l : -1;
          run += __shfl(inc, 63);
        }
        if (lane == 0) s_total = min(run, kSpecRows);
      }
      __syncthreads();
      const int32_t total = s_total;
      for (int32_t e = t; e < total; e += 1024) {
        int32_t lo = 0, hi = C - 1;  // the last step whose offset is <= e
        while (lo < hi) {
          const int32_t mid = (lo + hi + 1) >> 1;
          if (st_off[mid] >= 0 && st_off[mid] <= e) lo = mid; else hi = mid - 1;
        }
        const int32_t k = e - st_off[lo];
        if (st_off[lo] >= 0 && st_deg[lo] <= 64 && k >= 0 && k < st_deg[lo]) {
          const int32_t v = col[st_r0[lo] + k];
          row_nb[e] = v;
          row_age[e] = age[st_r0[lo] + k];
          atomicMax(&st_best[lo], err_key(err[v], v));
        }
      }
      __syncthreads();
      // ---- f, the lowered keys, and the first step touching each unit
      if (t < C) {
        const int32_t q = key_index(skey[t]);
        const bool fetched = st_off[t] >= 0 && st_deg[t] <= 64;
        if (fetched && st_deg[t] > 0) {
          const int32_t f = key_index(st_best[t]);
          st_f[t] = f;
          const unsigned long long kq = err_key(key_err(skey[t]) * alpha, q);
          const unsigned long long kf = err_key(key_err(st_best[t]) * alpha, f);
          st_mod[t] = kq > kf ? kq : kf;
          touch_put(hk, hv, f, t);
        } else {
          st_f[t] = -1;
          st_mod[t] = 0;
          if (!fetched) atomicMin(&s_lbad, t);
          else atomicMin(&s_lzero, t);
        }
        touch_put(hk, hv, q, t);
      }
      __syncthreads();
      // ---- (a): the key of q_i above every lowered key of the earlier steps (the exclusive
      // prefix maximum of st_mod replaces it), (b): q_i and its row untouched before i
      if (w == 0) {
        unsigned long long run = 0;
        for (int32_t b = 0; b < C; b += 64) {
          const int32_t i = b + lane;
          const unsigned long long v = i < C ? st_mod[i] : 0ull;
          unsigned long long inc = v;
          for (int o = 1; o < 64; o <<= 1) {
            const unsigned long long u = __shfl_up(inc, o);
            if (lane >= o) inc = u > inc ? u : inc;
          }
          const unsigned long long excl0 = __shfl_up(inc, 1);
          const unsigned long long excl = lane == 0 ? run : (excl0 > run ? excl0 : run);
          if (i < C) st_mod[i] = excl;
          const unsigned long long top = __shfl(inc, 63);
          run = top > run ? top : run;
        }
      }
      __syncthreads();
      if (t < C) {
        const int32_t q = key_index(skey[t]);
        if (touch_find(hk, hv, q) < t || (t > 0 && !(skey[t] > st_mod[t])))
          atomicMin(&s_lbad, t);
      }
      for (int32_t e = t; e < total; e += 1024) {
        int32_t lo = 0, hi = C - 1;
        while (lo < hi) {
          const int32_t mid = (lo + hi + 1) >> 1;
          if (st_off[mid] >= 0 && st_off[mid] <= e) lo = mid; else hi = mid - 1;
        }
        const int32_t k = e - st_off[lo];
        if (st_off[lo] >= 0 && st_deg[lo] <= 64 && k >= 0 && k < st_deg[lo] &&
            touch_find(hk, hv, row_nb[e]) < lo)
          atomicMin(&s_lbad, lo);
      }
      __syncthreads();
      // ---- the prefix: up to the first failed guess, the first empty row, the counts
      // The sequential order at step L (when the counts allow one more): a q without a
      // neighbour stops the call; a q with one but no room for its edge is a capacity error;
      // a first guess whose row is too long takes the one-wave path; any other failed guess
      // (or an exhausted pool) starts another round.
      const int32_t e2 = s_e2;
      const int64_t room64 = max((half_cap - static_cast<int64_t>(e2)) / 2, int64_t{0});
      const int32_t room = static_cast<int32_t>(min(room64, static_cast<int64_t>(INT32_MAX)));
      const int32_t lbad = s_lbad, lzero = s_lzero;
      const int32_t j = min(min(lbad, lzero), C);
      const int32_t lim = min(count - done, n_max - n);
      L = min(j, min(room, lim));
      if (L < lim) {
        if (L == lzero) {
          stop = true;
        } else if (L == room && L < j) {
          if (t == 0) atomicCAS(&status[kStError], 0, GSN_E_CAPACITY);
          stop = true;
        } else if (L == 0 && lbad == 0) {
          slow = true;
        }
      }
      // ---- apply steps 0 .. L-1 (their q's and f's are pairwise distinct)
      if (t < L) {
        const int32_t q = key_index(skey[t]), f = st_f[t], r = n + t;
        const float eq = key_err(skey[t]) * alpha;
        const float ef = key_err(st_best[t]) * alpha;
        err[q] = eq;
        err[f] = ef;
        err[r] = eq;
        // q's row: f out, r appended
        const int32_t r0 = st_r0[t], d = st_deg[t], o = st_off[t];
        int32_t wpos = 0;
        for (int32_t k = 0; k < d; ++k) {
          const int32_t v = row_nb[o + k];
          if (v == f) continue;
          col[r0 + wpos] = v;
          age[r0 + wpos] = row_age[o + k];
          ++wpos;
        }
        col[r0 + d - 1] = r;
        age[r0 + d - 1] = 0;
        // f's row: q out, r appended
        const int32_t f0 = rp[f], f1 = rp[f + 1];
        int32_t k = f0;
        while (k < f1 && col[k] != q) ++k;
        for (; k + 1 < f1; ++k) {
          col[k] = col[k + 1];
          age[k] = age[k + 1];
        }
        col[f1 - 1] = r;
        age[f1 - 1] = 0;
        // r's row and position
        col[e2 + 2 * t] = min(q, f);
        col[e2 + 2 * t + 1] = max(q, f);
        age[e2 + 2 * t] = 0;
        age[e2 + 2 * t + 1] = 0;
        rp[r + 1] = e2 + 2 * (t + 1);
        x[r] = (x[q] + x[f]) * 0.5f;
        y[r] = (y[q] + y[f]) * 0.5f;
        z[r] = (z[q] + z[f]) * 0.5f;
      }
    }
    // ---- the segments of every unit touched
    for (int32_t i = t; i < kMaxSeg / 32; i += 1024) mark[i] = 0;
    if (t == 0) s_cnt = 0;
    __syncthreads();
    const int32_t n1 = n + L;
    for (int32_t i = t; i < 3 * L; i += 1024) {
      const int32_t s3 = i / 3, which = i % 3;
      const int32_t u = which == 0 ? key_index(skey[s3]) : (which == 1 ? st_f[s3] : n + s3);
      const int32_t sg = u / len;
      if ((atomicOr(&mark[sg >> 5], 1u << (sg & 31)) & (1u << (sg & 31))) == 0)
        list[atomicAdd(&s_cnt, 1)] = sg;
    }
    __syncthreads();
    const int32_t nmark = s_cnt;
    for (int32_t b = 0; b < nmark; b += 64) {
      const int32_t my = b + (t >> 4);
      const int32_t sg = my < nmark ? list[my] : -1;
      const unsigned long long k = segment_key16(err, n1, sg, len, t & 15);
      if ((t & 15) == 0 && sg >= 0) sk[sg] = k;
    }
    n = n1;
    done += L;
    nseg = (n + len - 1) / len;
    if (L > 0 && kseg < kSpecSeg) kseg <<= 1;
    __syncthreads();
    if (!slow || stop || done >= count || n >= n_max) continue;
    // ---- one insertion by the one-wave path: q = the largest segment key
    unsigned long long best = 0;
    for (int32_t i = t; i < nseg; i += 1024) best = sk[i] > best ? sk[i] : best;
    best = wave_max(best);
    if (lane == 0) pkey[w] = best;
    __syncthreads();
    if (w == 0) {
      unsigned long long b2 = lane < 16 ? pkey[lane] : 0ull;
      b2 = wave_max(b2);
      const int32_t q = b2 ? key_index(b2) : -1;
      int32_t ff = -1;
      const int a = wave_insert(n, q, alpha, half_cap, rp, col, age, x, y, z, err, status, &ff);
      if (lane == 0) {
        s_ok = a;
        st_f[0] = ff;
        st_r0[0] = q;
      }
    }
    __syncthreads();
    if (!s_ok) {
      stop = true;
      continue;
    }
    const int32_t qs = st_r0[0], fs = st_f[0];
    ++n;
    ++done;
    nseg = (n + len - 1) / len;
    if (w < 3) {
      const int32_t u = w == 0 ? qs : (w == 1 ? fs : n - 1);
      const unsigned long long k = segment_key(err, n, u / len, len);
      if (lane == 0) sk[u / len] = k;
    }
    __syncthreads();
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
  // segment length: whole waves, at most kMaxSeg segments over n_max units
  const int32_t waves = (n_max + 63) / 64;
  const int32_t len = 64 * ((waves + kMaxSeg - 1) / kMaxSeg);
  const int32_t nseg = (n + len - 1) / len;
  // the per-unit count array is free between iterations; it holds the segment keys
  unsigned long long* seg = reinterpret_cast<unsigned long long*>(s.cnt);
  if (nseg > 0)
    gr_segmax<<<(nseg * 64 + kBlock - 1) / kBlock, kBlock, 0, st>>>(n, len, nseg, s.err, seg);
  if (count >= kSpecMin)
    gr_insert_spec<<<1, 1024, 0, st>>>(n, count, n_max, len, alpha, half_cap, seg, s.rp[cur],
                                       s.col[cur], s.age[cur], s.x, s.y, s.z, s.err, s.status);
  else
    gr_insert<<<1, 1024, 0, st>>>(n, count, n_max, len, alpha, half_cap, seg, s.rp[cur],
                                  s.col[cur], s.age[cur], s.x, s.y, s.z, s.err, s.status);
  return hipGetLastError();
}

}  // namespace gsn
