// Host side of the C ABI declared in include/gsn.h: argument validation, workspace
// carving, launch configuration, call ordering and event timing.  All device memory is the
// caller's; this file allocates only the handle (and short-lived host vectors in the
// synchronous export/import calls).
#include <stdlib.h>
#include <string.h>

#include <cmath>
#include <cstddef>
#include <mutex>
#include <new>
#include <vector>

#include "gsn_internal.h"

// The grid workspace of gsn_find_winners_grid_noalloc, for callers that cannot allocate:
// one fixed array per GPU, held from the library's load until the process ends.  In host
// code the name only stands for the symbol; its device address on each GPU comes from
// hipGetSymbolAddress (noalloc_scratch below), and only that address is used.
static __device__ __align__(256) unsigned char scratch[GSN_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

// Device address of `scratch` on the current device, looked up once per device with that
// device current; nullptr if the lookup fails.
void* noalloc_scratch() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    g_scratch_dev[dev] = ptr;
  }
  return g_scratch_dev[dev];
}

}  // namespace

namespace gsn {

Layout layout_for(const gsn_params& p) {
  Layout L{};
  size_t o = 0;
  int i = 0;
  auto add = [&](size_t bytes) {
    o = (o + 255) & ~static_cast<size_t>(255);
    L.off[i++] = o;
    o += bytes;
  };
  const size_t nm = static_cast<size_t>(p.n_max);
  const size_t mm = static_cast<size_t>(p.m_max);
  // the winner-lock update works on a copy of the adjacency with room for one insertion
  // per survivor at its winner and one at its second
  const size_t hc = 2 * (static_cast<size_t>(p.e_max) + (p.lock_mode == 1 ? mm : 0)) + 2;
  add(4 * nm);                 // 0 x
  add(4 * nm);                 // 1 y
  add(4 * nm);                 // 2 z
  add(4 * nm);                 // 3 err
  add(4 * (nm + 2));           // 4 rp0
  add(4 * (nm + 2));           // 5 rp1
  add(4 * hc);                 // 6 col0
  add(4 * hc);                 // 7 col1
  add(4 * hc);                 // 8 age0
  add(4 * hc);                 // 9 age1
  add(8 * nm);                 // 10 lock
  add(4 * nm);                 // 11 ins
  add(4 * nm);                 // 12 orphan
  add(4 * nm);                 // 13 cnt
  add(4 * (nm / kBlock + 2));  // 14 bsum
  add(16 * nm);                // 15 tmp
  add(4 * kStSlots);           // 16 status
  add(8 * static_cast<size_t>(kMaxSplit) * 2 * mm);  // 17 part
  add(stage_bytes(p.n_max, p.m_max));                 // 18 screened staging
  add(mm);                     // 19 pend
  add(4 * nm);                 // 20 len
  add(4 * nm);                 // 21 extra
  add(4 * kRmWords);           // 22 rem
  add(8 * mm);                 // 23 list
  add(12 * mm);                // 24 schedule signals
  add(4 * mm);                 // 25 schedule winners
  add(4 * mm);                 // 26 schedule seconds
  add(4 * mm);                 // 27 schedule d1
  add(4 * mm);                 // 28 schedule d2
  add(mm);                     // 29 schedule acceptance
  add(8 * kA64Slots);          // 30 64-bit accumulators
  add(4 * (mm / 32 + 2));      // 31 accepted signals per workgroup of the fused check
  add(8 * small_part_keys(p.m_max));  // 32 partial keys of the small-batch scan
  add(4 * (nm / kBlock + 2));  // 33 per-block half-edge changes, set 0
  add(4 * (nm / kBlock + 2));  // 34 per-block half-edge changes, set 1
  const bool wl = p.lock_mode == 1;
  add(wl ? 32 * nm : 0);       // 35 survivor records (key, second), two parities
  add(wl ? 2 * nm : 0);        // 36 survivor flags, two parities
  add(wl ? 8 * nm : 0);        // 37 heads of the second lists, two parities
  add(wl ? 4 * mm : 0);        // 38 links of the second lists
  add(wl ? 8 : 0);             // 39 table bounds
  L.total = (o + 255) & ~static_cast<size_t>(255);
  return L;
}

void carve(const gsn_params& p, void* base, DevState* s) {
  const Layout L = layout_for(p);
  char* b = static_cast<char*>(base);
  s->x = reinterpret_cast<float*>(b + L.off[0]);
  s->y = reinterpret_cast<float*>(b + L.off[1]);
  s->z = reinterpret_cast<float*>(b + L.off[2]);
  s->err = reinterpret_cast<float*>(b + L.off[3]);
  s->rp[0] = reinterpret_cast<int32_t*>(b + L.off[4]);
  s->rp[1] = reinterpret_cast<int32_t*>(b + L.off[5]);
  s->col[0] = reinterpret_cast<int32_t*>(b + L.off[6]);
  s->col[1] = reinterpret_cast<int32_t*>(b + L.off[7]);
  s->age[0] = reinterpret_cast<int32_t*>(b + L.off[8]);
  s->age[1] = reinterpret_cast<int32_t*>(b + L.off[9]);
  s->lock = reinterpret_cast<unsigned long long*>(b + L.off[10]);
  s->ins = reinterpret_cast<int32_t*>(b + L.off[11]);
  s->orphan = reinterpret_cast<int32_t*>(b + L.off[12]);
  s->cnt = reinterpret_cast<int32_t*>(b + L.off[13]);
  s->bsum = reinterpret_cast<int32_t*>(b + L.off[14]);
  s->tmp = reinterpret_cast<float*>(b + L.off[15]);
  s->status = reinterpret_cast<int32_t*>(b + L.off[16]);
  s->part = reinterpret_cast<unsigned long long*>(b + L.off[17]);
  s->scr = b + L.off[18];
  s->pend = reinterpret_cast<uint8_t*>(b + L.off[19]);
  s->len = reinterpret_cast<int32_t*>(b + L.off[20]);
  s->extra = reinterpret_cast<int32_t*>(b + L.off[21]);
  s->rem = reinterpret_cast<int32_t*>(b + L.off[22]);
  s->list = reinterpret_cast<int32_t*>(b + L.off[23]);
  s->ssig = reinterpret_cast<float*>(b + L.off[24]);
  s->swin = reinterpret_cast<int32_t*>(b + L.off[25]);
  s->ssec = reinterpret_cast<int32_t*>(b + L.off[26]);
  s->sd1 = reinterpret_cast<float*>(b + L.off[27]);
  s->sd2 = reinterpret_cast<float*>(b + L.off[28]);
  s->sacc = reinterpret_cast<uint8_t*>(b + L.off[29]);
  s->acc64 = reinterpret_cast<unsigned long long*>(b + L.off[30]);
  s->apart = reinterpret_cast<int32_t*>(b + L.off[31]);
  s->spart = reinterpret_cast<unsigned long long*>(b + L.off[32]);
  s->bdelta[0] = reinterpret_cast<int32_t*>(b + L.off[33]);
  s->bdelta[1] = reinterpret_cast<int32_t*>(b + L.off[34]);
  const bool wl = p.lock_mode == 1;
  s->wkey = wl ? reinterpret_cast<unsigned long long*>(b + L.off[35]) : nullptr;
  s->wflag = wl ? reinterpret_cast<uint8_t*>(b + L.off[36]) : nullptr;
  s->rhead = wl ? reinterpret_cast<int32_t*>(b + L.off[37]) : nullptr;
  s->rnext = wl ? reinterpret_cast<int32_t*>(b + L.off[38]) : nullptr;
  s->whi = wl ? reinterpret_cast<int32_t*>(b + L.off[39]) : nullptr;
}

}  // namespace gsn

using gsn::DevState;

enum Phase { kReady = 0, kFound = 1, kResolved = 2, kAdapted = 3 };
constexpr int kRebucketEvery = 64;     // default calls between rebuilds of the unit order
constexpr int kDefaultGrab = 4;        // batches per grab of the dynamic scan
constexpr int kDefaultGridRounds = 6;  // before any update has reported back
constexpr int kGreedyGridRounds = 4;   // grid-wide rounds of the greedy lock-set resolve

struct gsn_net {
  gsn_params p;
  DevState s;
  int32_t n;        // live units (host copy, changed only by grow/import)
  int cur;          // current CSR buffer
  int dpar;         // which per-block delta array the next lock-set edge update uses
  int wpar;         // which survivor tables the next one-pass winner-lock update uses
  int phase;
  int cus;          // compute units of the device
  int tune_split;
  int tune_variant;
  int tune_grab;    // list entries per atomic of the dynamic scan
  int tune_rebucket;  // staged find calls between rebuilds of the spatial unit order
  int stage_parity;  // which set of signal histogram and cursors the next call uses
  bool timing;
  uint32_t timing_mask;  // timers that record while timing is on (bit GSN_T_*)
  int32_t bucket_n;            // unit count at the last spatial bucketing (-1: none yet)
  int32_t finds_since_bucket;
  int grid_rounds;             // grid-wide rounds of the winner-lock update (0: automatic)
  int32_t* feedback;           // pinned host word: the last update's grid rounds used
  int32_t* feedback_dev;       // its device address, stored by the update's last kernel
  void* scratch_dev;           // device address of the no-allocation grid workspace
  std::vector<hipEvent_t> pool;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> rec[GSN_T_COUNT];
  // gsn_iterate_loop: recorded loops, the stream they are recorded on, and the recording
  // state (event timers off; the unit-order rule of the first staged find overridden)
  struct LoopGraph {
    // what the recorded launches depend on
    const float* sigs;
    int32_t m, count;
    int32_t *winner, *second;
    float *d1, *d2;
    uint8_t* accepted;
    int32_t n;
    int cur, dpar, wpar, stage_parity;
    bool rebuild_first;
    int tune_split, tune_variant, tune_grab, tune_rebucket, grid_rounds;
    // the host state the loop leaves
    bool rebuilt;   // the first find rebuilt the unit order (else finds_delta counts finds)
    int cur_after, dpar_after, wpar_after, stage_parity_after;
    int32_t finds_after, finds_delta, bucket_n_after;
    hipGraphExec_t exec;
    uint64_t used;
  };
  std::vector<LoopGraph> graphs;
  uint64_t graph_clock;
  int64_t loop_records;   // loop calls that recorded a graph
  hipStream_t cap_stream;
  bool capturing;
  int loop_rebuild;   // -1, or the unit-order decision (0/1) of the next staged find
};

namespace {

bool params_ok(const gsn_params* p) {
  if (!p) return false;
  if (!(p->eps_b >= 0.0f && p->eps_b <= 1.0f)) return false;
  if (!(p->eps_n >= 0.0f && p->eps_n <= 1.0f)) return false;
  // errors stay >= +0 and only shrink under the two factors (the argmax keys rely on it)
  if (!(p->err_alpha >= 0.0f && p->err_alpha <= 1.0f)) return false;
  if (!(p->err_beta >= 0.0f && p->err_beta <= 1.0f)) return false;
  if (p->max_age < 0) return false;
  if (p->n_max < 2 || p->e_max < 0 || p->m_max < 1) return false;
  if (p->lock_mode < 0 || p->lock_mode > 2 || p->key_mode < 0 || p->key_mode > 1) return false;
  // keep every derived index inside int32
  const int64_t slack = p->lock_mode == 1 ? p->m_max : 0;
  if ((static_cast<int64_t>(p->e_max) + slack) * 2 + 2 > INT32_MAX) return false;
  if (static_cast<int64_t>(p->n_max) + 2 > INT32_MAX / 4) return false;
  if (static_cast<int64_t>(p->m_max) * 2 * gsn::kMaxSplit > INT32_MAX) return false;
  return true;
}

inline hipStream_t as_stream(void* st) { return static_cast<hipStream_t>(st); }

bool grid_ok(const gsn_grid* g, int64_t* cells) {
  if (!g) return false;
  if (!(g->h > 0.0f) || !std::isfinite(g->h)) return false;
  if (!std::isfinite(1.0f / g->h)) return false;
  int64_t c = 1;
  for (int a = 0; a < 3; ++a) {
    if (!std::isfinite(g->lo[a]) || g->dims[a] < 1) return false;
    c *= g->dims[a];
    if (c > GSN_MAX_GRID_CELLS) return false;
  }
  if (g->exact != 0 && g->exact != 1) return false;
  *cells = c;
  return true;
}

inline int hip_ok(hipError_t e) { return e == hipSuccess ? GSN_OK : GSN_E_HIP; }

hipEvent_t take_event(gsn_net* net) {
  if (!net->pool.empty()) {
    hipEvent_t e = net->pool.back();
    net->pool.pop_back();
    return e;
  }
  // timing only: no system-scope fence at the record (the default one writes back and
  // invalidates the caches, which stalls the stream for several microseconds per record)
  hipEvent_t e = nullptr;
  if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
  return e;
}

// Records an event pair around the launches made between begin() and end().
struct TimedRegion {
  gsn_net* net;
  int which;
  hipStream_t st;
  hipEvent_t a = nullptr;
  TimedRegion(gsn_net* n, int w, hipStream_t s) : net(n), which(w), st(s) {
    if (net->timing && !net->capturing && ((net->timing_mask >> w) & 1u)) {
      a = take_event(net);
      if (a && hipEventRecord(a, st) != hipSuccess) {
        net->pool.push_back(a);
        a = nullptr;
      }
    }
  }
  void end() {
    if (!a) return;
    hipEvent_t b = take_event(net);
    if (!b) {
      net->pool.push_back(a);
      a = nullptr;
      return;
    }
    if (hipEventRecord(b, st) == hipSuccess) {
      net->rec[which].emplace_back(a, b);
    } else {
      net->pool.push_back(a);
      net->pool.push_back(b);
    }
    a = nullptr;
  }
};

// A timer whose event pair is bound to one kernel launch (gsn::LaunchEvents): the pair is
// taken from the pool when the timer records, and end() keeps it only if the launch was made.
struct LaunchTimer {
  gsn_net* net;
  int which;
  gsn::LaunchEvents ev;
  LaunchTimer(gsn_net* n, int w) : net(n), which(w) {
    if (net->timing && !net->capturing && ((net->timing_mask >> w) & 1u)) {
      ev.start = take_event(net);
      ev.stop = ev.start ? take_event(net) : nullptr;
      if (ev.start && !ev.stop) {
        net->pool.push_back(ev.start);
        ev.start = nullptr;
      }
    }
  }
  void end(bool launched) {
    if (!ev.start) return;
    if (launched) {
      net->rec[which].emplace_back(ev.start, ev.stop);
    } else {
      net->pool.push_back(ev.start);
      net->pool.push_back(ev.stop);
    }
    ev = {};
  }
};

int read_status_slot(gsn_net* net, int slot, int32_t* out, hipStream_t st) {
  if (hipMemcpyAsync(out, net->s.status + slot, sizeof(int32_t), hipMemcpyDeviceToHost, st) !=
      hipSuccess)
    return GSN_E_HIP;
  return hip_ok(hipStreamSynchronize(st));
}

int read_acc64(gsn_net* net, int slot, int64_t* out, hipStream_t st) {
  unsigned long long v = 0;
  if (hipMemcpyAsync(&v, net->s.acc64 + slot, sizeof(v), hipMemcpyDeviceToHost, st) !=
      hipSuccess)
    return GSN_E_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return GSN_E_HIP;
  *out = static_cast<int64_t>(v);
  return GSN_OK;
}

// Between iterations: remove the units orphaned since the last call, then up to `count` GNG
// insertions one after another (while N < n_max).  Syncs to learn the new unit count.
int grow_step(gsn_net* net, int32_t count, int32_t* inserted_out, hipStream_t st) {
  int32_t orphans = 0;
  int rc = read_status_slot(net, gsn::kStOrphans, &orphans, st);
  if (rc) return rc;
  if (orphans > 0) {
    if (gsn::launch_remove(net->s, net->cur, net->n, net->p.n_max, st) != hipSuccess)
      return GSN_E_HIP;
    net->cur ^= 1;
    int32_t kept = 0;
    rc = read_status_slot(net, gsn::kStKept, &kept, st);
    if (rc) return rc;
    net->n = kept;
    net->bucket_n = -1;  // indices changed
  }
  int32_t inserted = 0;
  if (count > 0 && net->n >= 1 && net->n < net->p.n_max) {
    if (gsn::launch_insert(net->s, net->cur, net->n, count, net->p.err_alpha, net->p.n_max,
                           2 * static_cast<int64_t>(net->p.e_max), st) != hipSuccess)
      return GSN_E_HIP;
    rc = read_status_slot(net, gsn::kStInserted, &inserted, st);
    if (rc) return rc;
    const int32_t n_before = net->n;
    net->n += inserted;
    if (inserted) {
      // new units take the next indices: they join the spatial order at its end (the
      // periodic rebucketing restores locality); after a removal the order is rebuilt
      if (net->bucket_n == n_before) {
        const gsn::StageBufs sb = gsn::carve_stage(net->s.scr, net->p.n_max, net->p.m_max);
        if (gsn::launch_stage_append(sb, n_before, net->n, st) != hipSuccess) return GSN_E_HIP;
        net->bucket_n = net->n;
      } else {
        net->bucket_n = -1;
      }
    }
  }
  if (inserted_out) *inserted_out = inserted;
  return GSN_OK;
}

}  // namespace

extern "C" {

size_t gsn_workspace_bytes(const gsn_params* params) {
  if (!params_ok(params)) return 0;
  return gsn::layout_for(*params).total;
}

int gsn_create(const gsn_params* params, void* workspace, size_t workspace_bytes, int32_t n0,
               const float* init_xyz, void* stream, gsn_net** out) {
  if (!out) return GSN_E_INVAL;
  *out = nullptr;
  if (!params_ok(params) || !workspace || n0 < 0 || n0 > params->n_max) return GSN_E_INVAL;
  if (n0 > 0 && !init_xyz) return GSN_E_INVAL;
  if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0) return GSN_E_INVAL;
  if (workspace_bytes < gsn::layout_for(*params).total) return GSN_E_CAPACITY;
  gsn_net* net = new (std::nothrow) gsn_net();
  if (!net) return GSN_E_CAPACITY;
  net->p = *params;
  gsn::carve(*params, workspace, &net->s);
  net->n = n0;
  net->cur = 0;
  net->dpar = 0;
  net->wpar = 0;
  net->phase = kReady;
  net->tune_split = 0;
  net->tune_variant = 0;
  net->tune_grab = kDefaultGrab;
  net->tune_rebucket = kRebucketEvery;
  net->stage_parity = 0;
  net->timing = false;
  net->timing_mask = (1u << GSN_T_COUNT) - 1;
  net->bucket_n = -1;
  net->finds_since_bucket = 0;
  net->grid_rounds = 0;
  net->graph_clock = 0;
  net->loop_records = 0;
  net->cap_stream = nullptr;
  net->capturing = false;
  net->loop_rebuild = -1;
  net->feedback = nullptr;
  if (hipHostMalloc(reinterpret_cast<void**>(&net->feedback), sizeof(int32_t)) != hipSuccess) {
    delete net;
    return GSN_E_HIP;
  }
  *net->feedback = kDefaultGridRounds - 1;
  net->feedback_dev = nullptr;
  // set-up of the no-allocation entry point on this device (null if the lookup failed;
  // that entry point then tries once more and reports GSN_E_HIP)
  net->scratch_dev = noalloc_scratch();
  if (hipHostGetDevicePointer(reinterpret_cast<void**>(&net->feedback_dev), net->feedback, 0) !=
      hipSuccess) {
    gsn_destroy(net);
    return GSN_E_HIP;
  }
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) == hipSuccess &&
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess)
    net->cus = cus;
  else
    net->cus = 256;
  hipStream_t st = as_stream(stream);
  hipError_t e = gsn::launch_init(net->s, 0, n0, params->n_max, st);
  if (e == hipSuccess)
    e = gsn::launch_stage_init(gsn::carve_stage(net->s.scr, params->n_max, params->m_max), st);
  const size_t bytes = sizeof(float) * static_cast<size_t>(n0);
  if (e == hipSuccess && n0 > 0) {
    e = hipMemcpyAsync(net->s.x, init_xyz, bytes, hipMemcpyDefault, st);
    if (e == hipSuccess)
      e = hipMemcpyAsync(net->s.y, init_xyz + n0, bytes, hipMemcpyDefault, st);
    if (e == hipSuccess)
      e = hipMemcpyAsync(net->s.z, init_xyz + 2 * static_cast<size_t>(n0), bytes,
                         hipMemcpyDefault, st);
  }
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) {
    gsn_destroy(net);  // frees the pinned feedback word with the handle
    return GSN_E_HIP;
  }
  *out = net;
  return GSN_OK;
}

}  // extern "C"

namespace {

// gsn_find_winners; with claim not null the merge of the staged scans also makes the
// lock-set claims of every signal, and *claimed says whether it did (the direct scan's
// merge does not).
int find_impl(gsn_net* net, const float* sig, int32_t m, int32_t* winner, int32_t* second,
              float* d1, float* d2, void* stream, const gsn::ClaimArgs* claim,
              bool* claimed, const int32_t** order = nullptr) {
  if (claimed) *claimed = false;
  if (order) *order = nullptr;
  if (!net || m < 0 || m > net->p.m_max) return GSN_E_INVAL;
  if (net->phase != kReady && net->phase != kFound) return GSN_E_STATE;
  if (net->n < 2) return GSN_E_INVAL;
  if (m > 0 && (!sig || !winner || !second || !d1 || !d2)) return GSN_E_INVAL;
  net->phase = kFound;
  if (m == 0) return GSN_OK;
  hipStream_t st = as_stream(stream);
  const gsn::FindConfig cfg =
      gsn::find_config(net->n, m, net->cus, net->tune_split, net->tune_variant);
  TimedRegion all(net, GSN_T_FIND, st);
  hipError_t e;
  if (cfg.variant == 6) {
    // a marker pair here: binding a pair to a launch costs the host tens of microseconds,
    // which a launch-bound small batch would show in its step time
    TimedRegion scan(net, GSN_T_FIND_SCAN, st);
    e = gsn::launch_find_small_scan(net->s, net->n, sig, m, st);
    scan.end();
    if (e == hipSuccess) {
      e = gsn::launch_find_small_merge(net->s, net->n, m, winner, second, d1, d2, claim, st);
      if (claimed) *claimed = claim != nullptr;
    }
  } else if (cfg.variant >= 2) {
    const gsn::StageBufs sb = gsn::carve_stage(net->s.scr, net->p.n_max, net->p.m_max);
    // the unit order is rebuilt when the network changed and every kRebucketEvery calls
    bool rebucket = net->bucket_n != net->n || net->finds_since_bucket >= net->tune_rebucket;
    if (net->loop_rebuild >= 0) {  // the first staged find of a recorded loop
      rebucket = net->loop_rebuild == 1;
      net->loop_rebuild = -1;
    }
    e = gsn::launch_stage(net->s, sb, net->n, sig, m, rebucket, net->stage_parity,
                          cfg.variant, st);
    net->stage_parity ^= 1;
    if (rebucket) {
      net->bucket_n = net->n;
      net->finds_since_bucket = 0;
    }
    ++net->finds_since_bucket;
    if (e == hipSuccess) {
      LaunchTimer scan(net, GSN_T_FIND_SCAN);
      e = cfg.variant == 5   ? gsn::launch_scan_f16_dyn(net->s, sb, net->n, m, cfg.split,
                                                    net->tune_grab, st, scan.ev)
          : cfg.variant == 4 ? gsn::launch_scan_f16(net->s, sb, net->n, sig, m, cfg.split, st,
                                                    scan.ev)
          : cfg.variant == 3 ? gsn::launch_scan_mfma(net->s, sb, net->n, sig, m, cfg.split, st,
                                                     scan.ev)
                             : gsn::launch_scan_screened(net->s, sb, net->n, sig, m, cfg.split,
                                                         st, scan.ev);
      scan.end(e == hipSuccess);
    }
    if (e == hipSuccess) {
      e = gsn::launch_stage_merge(net->s, sb, m, cfg.split, winner, second, d1, d2, claim, st);
      if (claimed) *claimed = claim != nullptr;
      if (order) *order = sb.sperm;  // the signals' spatial order of this call
    }
  } else {
    TimedRegion scan(net, GSN_T_FIND_SCAN, st);
    e = gsn::launch_find_scan(net->s, net->n, sig, m, cfg, winner, second, d1, d2, st);
    scan.end();
    if (e == hipSuccess) e = gsn::launch_find_merge(net->s, m, cfg, winner, second, d1, d2, st);
  }
  all.end();
  return hip_ok(e);
}

// Resolve, adapt and edges after a find, fused where the rule allows (the outputs and state
// of gsn_resolve_conflicts, gsn_adapt and gsn_update_edges in order).  claimed: the find's
// merge made the lock-set claims; order: the signals in the staging's spatial order, or null.
int update_impl(gsn_net* net, const float* sig, int32_t m, const int32_t* winner,
                const int32_t* second, const float* d1, uint8_t* accepted, void* stream,
                bool claimed, const int32_t* order) {
  hipStream_t st = as_stream(stream);
  const int64_t half_cap = 2 * static_cast<int64_t>(net->p.e_max);
  if (net->p.lock_mode == 1) {
    if (m == 0) {
      int rc = gsn_resolve_conflicts(net, m, winner, second, d1, accepted, stream);
      if (!rc) rc = gsn_adapt(net, sig, m, winner, second, d1, accepted, stream);
      if (!rc) rc = gsn_update_edges(net, m, winner, second, accepted, stream);
      return rc;
    }
    // the resolve leaves one survivor per winner: the update in one pass, no rounds (the
    // resolve's check fills the survivor tables)
    const gsn::WinnerTables tab = gsn::winner_tables(net->s, net->wpar, net->p.n_max);
    {
      TimedRegion tr(net, GSN_T_RESOLVE, st);
      const hipError_t e = gsn::launch_resolve(net->s, net->cur, net->n, m, winner, second, d1,
                                               accepted, 1, net->p.key_mode, st, &tab,
                                               claimed);
      tr.end();
      if (e != hipSuccess) return GSN_E_HIP;
    }
    TimedRegion t(net, GSN_T_UPDATE, st);
    const gsn::WinnerStep w{sig, m, winner, second, d1, accepted, net->p.key_mode,
                            net->p.eps_b, net->p.eps_n, net->p.err_beta, net->p.max_age, 0, 0,
                            half_cap, nullptr, net->p.n_max};
    const hipError_t e = gsn::launch_winner_local(net->s, net->cur, net->wpar, net->n, w, st);
    t.end();
    if (e != hipSuccess) return GSN_E_HIP;
    net->cur ^= 1;
    net->wpar ^= 1;
    net->phase = kReady;
    return GSN_OK;
  }
  // the lock sets: the fused check and update; greedy: the resolve's rounds decide, and the
  // same update applies the accepted signals (disjoint lock sets) without claims or check
  const bool greedy = net->p.lock_mode == 2;
  if (greedy && m > 0) {
    // (with claimed the find's merge made the first round's claims and the signal states)
    TimedRegion tr(net, GSN_T_RESOLVE, st);
    const hipError_t e = gsn::launch_resolve_greedy(
        net->s, net->cur, net->n, m, winner, second, d1, accepted, net->p.key_mode,
        net->grid_rounds ? net->grid_rounds : kGreedyGridRounds, st, claimed);
    tr.end();
    if (e != hipSuccess) return GSN_E_HIP;
  }
  TimedRegion t(net, GSN_T_UPDATE, st);
  const hipError_t e = gsn::launch_iterate_set(
      net->s, net->cur, net->dpar, net->n, sig, m, winner, second, d1, accepted,
      net->p.key_mode, net->p.eps_b, net->p.eps_n, net->p.err_beta, net->p.max_age, half_cap,
      greedy || claimed, order, st, greedy ? accepted : nullptr);
  t.end();
  if (e != hipSuccess) return GSN_E_HIP;
  net->cur ^= 1;
  net->dpar ^= 1;
  net->phase = kReady;
  return GSN_OK;
}

}  // namespace

extern "C" {

int gsn_find_winners(gsn_net* net, const float* sig, int32_t m, int32_t* winner,
                     int32_t* second, float* d1, float* d2, void* stream) {
  return find_impl(net, sig, m, winner, second, d1, d2, stream, nullptr, nullptr);
}

size_t gsn_grid_workspace_bytes(const gsn_grid* grid, int32_t n_max, int32_t m_max) {
  int64_t cells = 0;
  if (!grid_ok(grid, &cells) || n_max < 2 || m_max < 1) return 0;
  return gsn::grid_bytes(cells, n_max, m_max);
}

}  // extern "C"

namespace {

int find_grid_impl(gsn_net* net, const gsn_grid* grid, void* grid_ws, size_t grid_ws_bytes,
                   const float* sig, int32_t m, int32_t* winner, int32_t* second, float* d1,
                   float* d2, void* stream, bool timed) {
  if (!net || m < 0 || m > net->p.m_max) return GSN_E_INVAL;
  if (net->phase != kReady && net->phase != kFound) return GSN_E_STATE;
  int64_t cells = 0;
  if (!grid_ok(grid, &cells) || !grid_ws) return GSN_E_INVAL;
  if (reinterpret_cast<uintptr_t>(grid_ws) % 256 != 0) return GSN_E_INVAL;
  if (grid_ws_bytes < gsn::grid_bytes(cells, net->p.n_max, net->p.m_max)) return GSN_E_CAPACITY;
  if (net->n < 2) return GSN_E_INVAL;
  if (m > 0 && (!sig || !winner || !second || !d1 || !d2)) return GSN_E_INVAL;
  net->phase = kFound;
  if (m == 0) return GSN_OK;
  hipStream_t st = as_stream(stream);
  gsn::GridSpec spec{};
  for (int a = 0; a < 3; ++a) {
    spec.lo[a] = grid->lo[a];
    spec.dims[a] = grid->dims[a];
  }
  spec.inv_h = 1.0f / grid->h;
  spec.cells = cells;
  spec.exact = grid->exact;
  const gsn::GridBufs gb = gsn::carve_grid(grid_ws, cells, net->p.n_max, net->p.m_max);
  hipError_t e;
  if (timed) {
    TimedRegion t(net, GSN_T_FIND, st);
    e = gsn::launch_find_grid(net->s, gb, spec, net->n, sig, m, winner, second, d1, d2, st);
    t.end();
  } else {
    e = gsn::launch_find_grid(net->s, gb, spec, net->n, sig, m, winner, second, d1, d2, st);
  }
  return hip_ok(e);
}

}  // namespace

extern "C" {

int gsn_find_winners_grid(gsn_net* net, const gsn_grid* grid, void* grid_ws,
                          size_t grid_ws_bytes, const float* sig, int32_t m, int32_t* winner,
                          int32_t* second, float* d1, float* d2, void* stream) {
  return find_grid_impl(net, grid, grid_ws, grid_ws_bytes, sig, m, winner, second, d1, d2,
                        stream, true);
}

int gsn_find_winners_grid_noalloc(gsn_net* net, const gsn_grid* grid, const float* sig,
                                  int32_t m, int32_t* winner, int32_t* second, float* d1,
                                  float* d2, void* stream) {
  if (!net) return GSN_E_INVAL;
  int64_t cells = 0;
  if (!grid_ok(grid, &cells)) return GSN_E_INVAL;
  if (gsn::grid_bytes(cells, net->p.n_max, net->p.m_max) > GSN_NOALLOC_SCRATCH_BYTES)
    return GSN_E_CAPACITY;
  if (!net->scratch_dev) net->scratch_dev = noalloc_scratch();
  if (!net->scratch_dev) return GSN_E_HIP;
  // no event timing here: a first event record would create (allocate) an event
  return find_grid_impl(net, grid, net->scratch_dev, GSN_NOALLOC_SCRATCH_BYTES, sig, m, winner,
                        second, d1, d2, stream, false);
}

int gsn_resolve_conflicts(gsn_net* net, int32_t m, const int32_t* winner,
                          const int32_t* second, const float* d1, uint8_t* accepted,
                          void* stream) {
  if (!net || m < 0 || m > net->p.m_max) return GSN_E_INVAL;
  if (net->phase != kFound && net->phase != kResolved) return GSN_E_STATE;
  if (m > 0 && (!winner || !second || !d1 || !accepted)) return GSN_E_INVAL;
  net->phase = kResolved;
  if (m == 0) return GSN_OK;
  hipStream_t st = as_stream(stream);
  TimedRegion t(net, GSN_T_RESOLVE, st);
  hipError_t e =
      net->p.lock_mode == 2
          ? gsn::launch_resolve_greedy(net->s, net->cur, net->n, m, winner, second, d1,
                                       accepted, net->p.key_mode,
                                       net->grid_rounds ? net->grid_rounds : kGreedyGridRounds,
                                       st)
          : gsn::launch_resolve(net->s, net->cur, net->n, m, winner, second, d1, accepted,
                                net->p.lock_mode, net->p.key_mode, st);
  t.end();
  return hip_ok(e);
}

int gsn_adapt(gsn_net* net, const float* sig, int32_t m, const int32_t* winner,
              const int32_t* second, const float* d1, const uint8_t* accepted, void* stream) {
  if (!net || m < 0 || m > net->p.m_max) return GSN_E_INVAL;
  if (net->phase != kResolved) return GSN_E_STATE;
  if (m > 0 && (!sig || !winner || !second || !d1 || !accepted)) return GSN_E_INVAL;
  net->phase = kAdapted;
  hipStream_t st = as_stream(stream);
  TimedRegion t(net, GSN_T_ADAPT, st);
  hipError_t e;
  if (net->p.lock_mode == 1 && m > 0 && net->n > 0) {
    // automatic: from the grid rounds the last update could use (read from the pinned copy
    // of its count; a stale value only changes the split, never the result)
    int g = net->grid_rounds;
    if (g == 0) {
      // a quarter more than the last update could use grid-wide: the single-workgroup tail
      // is the slow part, and a recorded loop keeps this count for all its iterations while
      // the network (and the rounds its updates need) grows
      const int used = *static_cast<volatile int32_t*>(net->feedback) + 1;
      g = std::clamp(used + used / 4, 1, gsn::kMaxGridRounds);
    }
    gsn::WinnerStep w{sig, m, winner, second, d1, accepted, net->p.key_mode, net->p.eps_b,
                      net->p.eps_n, net->p.err_beta, net->p.max_age, g,
                      2 * (static_cast<int64_t>(net->p.e_max) + net->p.m_max),
                      2 * static_cast<int64_t>(net->p.e_max), net->feedback_dev};
    e = gsn::launch_winner_update(net->s, net->cur, net->n, w, st);
  } else {
    e = gsn::launch_adapt(net->s, net->cur, net->n, sig, m, winner, second, d1, accepted,
                          net->p.eps_b, net->p.eps_n, net->p.err_beta, st);
  }
  t.end();
  return hip_ok(e);
}

int gsn_update_edges(gsn_net* net, int32_t m, const int32_t* winner, const int32_t* second,
                     const uint8_t* accepted, void* stream) {
  if (!net || m < 0 || m > net->p.m_max) return GSN_E_INVAL;
  if (net->phase != kAdapted) return GSN_E_STATE;
  if (m > 0 && (!winner || !second || !accepted)) return GSN_E_INVAL;
  hipStream_t st = as_stream(stream);
  if (net->p.lock_mode == 1) {  // gsn_adapt has updated the edges
    net->phase = kReady;
    return GSN_OK;
  }
  TimedRegion t(net, GSN_T_EDGES, st);
  hipError_t e = gsn::launch_edges(net->s, net->cur, net->dpar, net->n, m, winner, second,
                                   accepted,
                                   net->p.max_age, 2 * static_cast<int64_t>(net->p.e_max), st,
                                   net->p.lock_mode == 2 ? net->s.extra : nullptr);
  t.end();
  if (e != hipSuccess) return GSN_E_HIP;
  net->cur ^= 1;
  net->dpar ^= 1;
  net->phase = kReady;
  return GSN_OK;
}

int gsn_iterate(gsn_net* net, const float* sig, int32_t m, int32_t* winner, int32_t* second,
                float* d1, float* d2, uint8_t* accepted, void* stream) {
  if (!net || m < 0 || m > net->p.m_max) return GSN_E_INVAL;
  if (net->phase != kReady && net->phase != kFound) return GSN_E_STATE;
  if (m > 0 && !accepted) return GSN_E_INVAL;
  // with the lock-set and winner-lock rules the find's merge makes the claims where it can
  const gsn::ClaimArgs claim{net->n, net->s.rp[net->cur], net->s.col[net->cur], net->s.lock,
                             net->s.status, net->p.key_mode, net->p.lock_mode == 1 ? 1 : 0,
                             net->p.lock_mode == 2 ? net->s.pend : nullptr};
  bool claimed = false;
  const int32_t* order = nullptr;
  const int rc = find_impl(net, sig, m, winner, second, d1, d2, stream, &claim, &claimed,
                           &order);
  if (rc) return rc;
  return update_impl(net, sig, m, winner, second, d1, accepted, stream, claimed, order);
}

int gsn_update(gsn_net* net, const float* sig, int32_t m, const int32_t* winner,
               const int32_t* second, const float* d1, uint8_t* accepted, void* stream) {
  if (!net || m < 0 || m > net->p.m_max) return GSN_E_INVAL;
  if (net->phase != kFound && net->phase != kResolved) return GSN_E_STATE;
  if (m > 0 && (!sig || !winner || !second || !d1 || !accepted)) return GSN_E_INVAL;
  return update_impl(net, sig, m, winner, second, d1, accepted, stream, false, nullptr);
}

int gsn_iterate_loop(gsn_net* net, const float* sigs, int32_t m, int32_t count,
                     int32_t* winner, int32_t* second, float* d1, float* d2,
                     uint8_t* accepted, void* stream) {
  if (!net || count < 1 || count > GSN_MAX_LOOP || m < 0 || m > net->p.m_max)
    return GSN_E_INVAL;
  if (net->phase != kReady && net->phase != kFound) return GSN_E_STATE;
  if (net->n < 2) return GSN_E_INVAL;
  if (m > 0 && (!sigs || !winner || !second || !d1 || !d2 || !accepted)) return GSN_E_INVAL;
  hipStream_t st = as_stream(stream);
  // the unit order is rebuilt at the first iteration if the usual rule would rebuild it
  // anywhere inside the loop (after that the usual rule applies, from a fresh count)
  const bool rebuild_first =
      net->bucket_n != net->n || net->finds_since_bucket + count > net->tune_rebucket;
  using LoopGraph = gsn_net::LoopGraph;
  auto same = [&](const LoopGraph& g) {
    return g.sigs == sigs && g.m == m && g.count == count && g.winner == winner &&
           g.second == second && g.d1 == d1 && g.d2 == d2 && g.accepted == accepted &&
           g.n == net->n && g.cur == net->cur && g.dpar == net->dpar && g.wpar == net->wpar &&
           g.stage_parity == net->stage_parity && g.rebuild_first == rebuild_first &&
           g.tune_split == net->tune_split && g.tune_variant == net->tune_variant &&
           g.tune_grab == net->tune_grab && g.tune_rebucket == net->tune_rebucket &&
           g.grid_rounds == net->grid_rounds;
  };
  LoopGraph* hit = nullptr;
  for (auto& g : net->graphs)
    if (same(g)) hit = &g;
  if (!hit) {
    if (!net->cap_stream &&
        hipStreamCreateWithFlags(&net->cap_stream, hipStreamNonBlocking) != hipSuccess) {
      net->cap_stream = nullptr;
      return GSN_E_HIP;
    }
    LoopGraph g{};
    g.sigs = sigs; g.m = m; g.count = count;
    g.winner = winner; g.second = second; g.d1 = d1; g.d2 = d2; g.accepted = accepted;
    g.n = net->n; g.cur = net->cur; g.dpar = net->dpar; g.wpar = net->wpar;
    g.stage_parity = net->stage_parity;
    g.rebuild_first = rebuild_first;
    g.tune_split = net->tune_split; g.tune_variant = net->tune_variant;
    g.tune_grab = net->tune_grab; g.tune_rebucket = net->tune_rebucket;
    g.grid_rounds = net->grid_rounds;
    // record the loop: the calls run on the host as usual (argument checks, state), their
    // launches go into the graph
    const int cur0 = net->cur, dpar0 = net->dpar, wpar0 = net->wpar, sp0 = net->stage_parity;
    const int phase0 = net->phase;
    const int32_t bn0 = net->bucket_n, f0 = net->finds_since_bucket;
    (void)hipGetLastError();
    if (hipStreamBeginCapture(net->cap_stream, hipStreamCaptureModeThreadLocal) != hipSuccess)
      return GSN_E_HIP;
    net->capturing = true;
    net->loop_rebuild = rebuild_first ? 1 : 0;
    int rc = GSN_OK;
    for (int32_t k = 0; k < count && rc == GSN_OK; ++k)
      rc = gsn_iterate(net, sigs ? sigs + 3 * static_cast<size_t>(m) * k : nullptr, m, winner,
                       second, d1, d2, accepted, net->cap_stream);
    net->capturing = false;
    // a staged find consumed the unit-order decision; other finds leave the order alone
    const bool rebuilt = rebuild_first && net->loop_rebuild == -1;
    net->loop_rebuild = -1;
    hipGraph_t graph = nullptr;
    const hipError_t ec = hipStreamEndCapture(net->cap_stream, &graph);
    hipGraphExec_t exec = nullptr;
    if (rc == GSN_OK && ec == hipSuccess && graph &&
        hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0) != hipSuccess) {
      exec = nullptr;
    }
    if (graph) (void)hipGraphDestroy(graph);
    if (rc != GSN_OK || !exec) {
      // nothing ran: the handle is as before the call
      net->cur = cur0; net->dpar = dpar0; net->wpar = wpar0; net->stage_parity = sp0;
      net->phase = phase0;
      net->bucket_n = bn0; net->finds_since_bucket = f0;
      (void)hipGetLastError();
      return rc != GSN_OK ? rc : GSN_E_HIP;
    }
    g.exec = exec;
    g.rebuilt = rebuilt;
    g.cur_after = net->cur; g.dpar_after = net->dpar; g.wpar_after = net->wpar;
    g.stage_parity_after = net->stage_parity;
    g.finds_after = net->finds_since_bucket;
    g.finds_delta = net->finds_since_bucket - f0;
    g.bucket_n_after = net->bucket_n;
    // the host state is back at the start until the graph is launched below
    net->cur = cur0; net->dpar = dpar0; net->wpar = wpar0; net->stage_parity = sp0;
    net->bucket_n = bn0; net->finds_since_bucket = f0;
    if (net->graphs.size() >= GSN_GRAPH_CACHE) {
      size_t old = 0;
      for (size_t i = 1; i < net->graphs.size(); ++i)
        if (net->graphs[i].used < net->graphs[old].used) old = i;
      (void)hipGraphExecDestroy(net->graphs[old].exec);
      net->graphs.erase(net->graphs.begin() + static_cast<std::ptrdiff_t>(old));
    }
    net->graphs.push_back(g);
    hit = &net->graphs.back();
    ++net->loop_records;
  }
  hit->used = ++net->graph_clock;
  if (hipGraphLaunch(hit->exec, st) != hipSuccess) return GSN_E_HIP;
  net->cur = hit->cur_after;
  net->dpar = hit->dpar_after;
  net->wpar = hit->wpar_after;
  net->stage_parity = hit->stage_parity_after;
  if (hit->rebuilt) {
    net->finds_since_bucket = hit->finds_after;
    net->bucket_n = hit->bucket_n_after;
  } else {
    net->finds_since_bucket += hit->finds_delta;
  }
  net->phase = kReady;
  return GSN_OK;
}

int gsn_grow(gsn_net* net, int32_t iteration, int32_t insert_every, void* stream) {
  if (!net || insert_every < 0) return GSN_E_INVAL;
  if (net->phase != kReady) return GSN_E_STATE;
  const bool insert = insert_every > 0 && iteration > 0 && iteration % insert_every == 0;
  return grow_step(net, insert ? 1 : 0, nullptr, as_stream(stream));
}

int gsn_run_schedule(gsn_net* net, const float* cloud, int64_t n_points,
                     const gsn_schedule* sc, gsn_schedule_result* res, void* stream) {
  if (!net || !cloud || !sc || !res) return GSN_E_INVAL;
  if (n_points < 1 || n_points > static_cast<int64_t>(UINT32_MAX)) return GSN_E_INVAL;
  if (sc->m_cap < 1 || sc->m_cap > net->p.m_max || sc->fixed_m < 0 ||
      sc->fixed_m > net->p.m_max)
    return GSN_E_INVAL;
  if (sc->insert_every < 0 || sc->qe_window < 1 || sc->max_signals < 1) return GSN_E_INVAL;
  const int32_t m_big = sc->fixed_m > 0 ? sc->fixed_m : sc->m_cap;
  if (sc->qe_window + m_big > (int64_t{1} << 19)) return GSN_E_INVAL;
  if (net->phase != kReady || net->n < 2) return GSN_E_STATE;
  hipStream_t st = as_stream(stream);
  const gsn::DevState& s = net->s;
  *res = gsn_schedule_result{};
  int64_t accepted0 = 0, accepted1 = 0;
  int rc = read_acc64(net, gsn::kA64Accepted, &accepted0, st);
  if (rc) return rc;
  if (hipMemsetAsync(s.acc64 + gsn::kA64Window, 0, 8, st) != hipSuccess) return GSN_E_HIP;
  int64_t wcount = 0;
  bool have_qe = false;
  for (;;) {
    if (net->n < 2) return GSN_E_STATE;
    int32_t m = sc->fixed_m;
    if (m == 0) {
      int64_t p2 = 1;
      while (p2 <= net->n) p2 *= 2;  // the smallest power of two greater than N
      m = static_cast<int32_t>(std::min<int64_t>(p2, sc->m_cap));
    }
    if (gsn::launch_draw(cloud, n_points, sc->seed, res->signals, m, s.ssig, st) != hipSuccess)
      return GSN_E_HIP;
    if ((rc = gsn_iterate(net, s.ssig, m, s.swin, s.ssec, s.sd1, s.sd2, s.sacc, stream)))
      return rc;
    if (gsn::launch_qe(s.sd1, m, s.acc64 + gsn::kA64Window, st) != hipSuccess) return GSN_E_HIP;
    res->signals += m;
    res->iterations += 1;
    wcount += m;
    const int64_t k = sc->insert_every > 0 ? res->signals / sc->insert_every -
                                                 (res->signals - m) / sc->insert_every
                                           : 0;
    int32_t inserted = 0;
    if ((rc = grow_step(net, static_cast<int32_t>(std::min<int64_t>(k, INT32_MAX)), &inserted,
                        st)))
      return rc;
    res->inserted += inserted;
    if (wcount >= sc->qe_window) {
      int64_t sum = 0;
      if ((rc = read_acc64(net, gsn::kA64Window, &sum, st))) return rc;
      if (hipMemsetAsync(s.acc64 + gsn::kA64Window, 0, 8, st) != hipSuccess) return GSN_E_HIP;
      res->qe = static_cast<double>(static_cast<uint64_t>(sum)) * 0x1p-32 /
                static_cast<double>(wcount);
      have_qe = true;
      wcount = 0;
      if (res->qe < static_cast<double>(sc->qe_threshold)) {
        res->converged = 1;
        break;
      }
    }
    if (res->signals >= sc->max_signals) break;
  }
  if (!have_qe && wcount > 0) {
    int64_t sum = 0;
    if ((rc = read_acc64(net, gsn::kA64Window, &sum, st))) return rc;
    res->qe = static_cast<double>(static_cast<uint64_t>(sum)) * 0x1p-32 /
              static_cast<double>(wcount);
  }
  if ((rc = read_acc64(net, gsn::kA64Accepted, &accepted1, st))) return rc;
  res->accepted = accepted1 - accepted0;
  int32_t nu = 0, ne = 0;
  if ((rc = gsn_sizes(net, &nu, &ne, stream))) return rc;
  res->n_units = nu;
  res->n_edges = ne;
  return GSN_OK;
}

int gsn_sizes(gsn_net* net, int32_t* n_units, int32_t* n_edges, void* stream) {
  if (!net) return GSN_E_INVAL;
  hipStream_t st = as_stream(stream);
  int32_t half = 0;
  if (hipMemcpyAsync(&half, net->s.rp[net->cur] + net->n, sizeof(int32_t),
                     hipMemcpyDeviceToHost, st) != hipSuccess)
    return GSN_E_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return GSN_E_HIP;
  if (n_units) *n_units = net->n;
  if (n_edges) *n_edges = half / 2;
  return GSN_OK;
}

int gsn_export(gsn_net* net, float* xyz, float* err, int32_t* edges, void* stream) {
  if (!net) return GSN_E_INVAL;
  hipStream_t st = as_stream(stream);
  const size_t n = static_cast<size_t>(net->n);
  // every copy is ordered on the caller's stream, each group followed by its sync
  auto copy = [&](void* dst, const void* src, size_t bytes) {
    return hipMemcpyAsync(dst, src, bytes, hipMemcpyDefault, st) == hipSuccess;
  };
  auto sync = [&]() { return hipStreamSynchronize(st) == hipSuccess; };
  try {
    bool ok = true;
    if (xyz && n > 0)
      ok = copy(xyz, net->s.x, 4 * n) && copy(xyz + n, net->s.y, 4 * n) &&
           copy(xyz + 2 * n, net->s.z, 4 * n);
    if (ok && err && n > 0) ok = copy(err, net->s.err, 4 * n);
    if (!ok || !sync()) return GSN_E_HIP;
    if (edges) {
      std::vector<int32_t> rp(n + 1);
      if (!copy(rp.data(), net->s.rp[net->cur], 4 * (n + 1)) || !sync()) return GSN_E_HIP;
      const size_t half = static_cast<size_t>(rp[n]);
      std::vector<int32_t> col(half), age(half);
      if (half > 0 && (!copy(col.data(), net->s.col[net->cur], 4 * half) ||
                       !copy(age.data(), net->s.age[net->cur], 4 * half) || !sync()))
        return GSN_E_HIP;
      const size_t e = half / 2;
      std::vector<int32_t> out(3 * e);
      size_t t = 0;
      for (size_t u = 0; u < n; ++u)
        for (int32_t k = rp[u]; k < rp[u + 1]; ++k)
          if (static_cast<size_t>(col[k]) > u && t < e) {
            out[t] = static_cast<int32_t>(u);
            out[e + t] = col[k];
            out[2 * e + t] = age[k];
            ++t;
          }
      if (e > 0 && (!copy(edges, out.data(), 4 * 3 * e) || !sync())) return GSN_E_HIP;
    }
  } catch (const std::bad_alloc&) {
    return GSN_E_CAPACITY;
  }
  return GSN_OK;
}

int gsn_import(gsn_net* net, int32_t n, const float* xyz, const float* err, int32_t n_edges,
               const int32_t* edges, void* stream) {
  if (!net || n < 0 || n > net->p.n_max || n_edges < 0) return GSN_E_INVAL;
  if (n_edges > net->p.e_max) return GSN_E_CAPACITY;
  if ((n > 0 && !xyz) || (n_edges > 0 && !edges)) return GSN_E_INVAL;
  hipStream_t st = as_stream(stream);
  try {
    if (hipStreamSynchronize(st) != hipSuccess) return GSN_E_HIP;
    const size_t nn = static_cast<size_t>(n), ne = static_cast<size_t>(n_edges);
    std::vector<int32_t> ed(3 * ne);
    if (ne > 0 && (hipMemcpyAsync(ed.data(), edges, 4 * 3 * ne, hipMemcpyDefault, st) !=
                       hipSuccess ||
                   hipStreamSynchronize(st) != hipSuccess))
      return GSN_E_HIP;
    std::vector<int32_t> deg(nn + 1, 0);
    for (size_t k = 0; k < ne; ++k) {
      const int32_t u = ed[k], v = ed[ne + k], a = ed[2 * ne + k];
      if (u < 0 || v < 0 || u >= n || v >= n || u == v || a < 0) return GSN_E_INVAL;
      ++deg[u];
      ++deg[v];
    }
    std::vector<int32_t> rp(nn + 1, 0);
    for (size_t u = 0; u < nn; ++u) rp[u + 1] = rp[u] + deg[u];
    std::vector<int32_t> fill(rp.begin(), rp.end() - 1);
    std::vector<std::pair<int32_t, int32_t>> half(2 * ne);
    for (size_t k = 0; k < ne; ++k) {
      const int32_t u = ed[k], v = ed[ne + k], a = ed[2 * ne + k];
      half[fill[u]++] = {v, a};
      half[fill[v]++] = {u, a};
    }
    std::vector<int32_t> col(2 * ne), age(2 * ne);
    for (size_t u = 0; u < nn; ++u) {
      std::sort(half.begin() + rp[u], half.begin() + rp[u + 1]);
      for (int32_t k = rp[u]; k < rp[u + 1]; ++k) {
        if (k > rp[u] && half[k].first == half[k - 1].first) return GSN_E_INVAL;
        col[k] = half[k].first;
        age[k] = half[k].second;
      }
    }
    // everything below is ordered on the caller's stream; the host vectors stay alive
    // until the stream synchronization at the end
    net->cur = 0;
    const DevState& s = net->s;
    bool ok = true;
    auto copy = [&](void* dst, const void* src, size_t bytes) {
      ok = ok && hipMemcpyAsync(dst, src, bytes, hipMemcpyDefault, st) == hipSuccess;
    };
    auto fill_bytes = [&](void* dst, int value, size_t bytes) {
      ok = ok && hipMemsetAsync(dst, value, bytes, st) == hipSuccess;
    };
    if (n > 0) {
      copy(s.x, xyz, 4 * nn);
      copy(s.y, xyz + nn, 4 * nn);
      copy(s.z, xyz + 2 * nn, 4 * nn);
      if (err)
        copy(s.err, err, 4 * nn);
      else
        fill_bytes(s.err, 0, 4 * nn);
    }
    copy(s.rp[0], rp.data(), 4 * (nn + 1));
    if (ne > 0) {
      copy(s.col[0], col.data(), 8 * ne);
      copy(s.age[0], age.data(), 8 * ne);
    }
    const size_t nm = static_cast<size_t>(net->p.n_max);
    fill_bytes(s.ins, 0xff, 4 * nm);
    fill_bytes(s.orphan, 0, 4 * nm);
    fill_bytes(s.lock, 0xff, 8 * nm);
    fill_bytes(s.extra, 0, 4 * nm);
    fill_bytes(s.rem, 0, 4 * gsn::kRmWords);
    fill_bytes(s.status, 0, 4 * gsn::kStSlots);
    fill_bytes(s.bdelta[0], 0, 4 * (nm / gsn::kBlock + 2));
    fill_bytes(s.bdelta[1], 0, 4 * (nm / gsn::kBlock + 2));
    if (s.wkey) {
      fill_bytes(s.wkey, 0xff, 32 * nm);
      fill_bytes(s.wflag, 0, 2 * nm);
      fill_bytes(s.rhead, 0xff, 8 * nm);
      fill_bytes(s.whi, 0, 8);
    }
    ok = ok && gsn::launch_stage_init(gsn::carve_stage(s.scr, net->p.n_max, net->p.m_max),
                                      st) == hipSuccess;
    ok = hipStreamSynchronize(st) == hipSuccess && ok;
    if (!ok) return GSN_E_HIP;
    net->n = n;
    net->dpar = 0;
    net->wpar = 0;
    net->stage_parity = 0;   // both histogram sets were cleared above
    net->phase = kReady;
    net->bucket_n = -1;
  } catch (const std::bad_alloc&) {
    return GSN_E_CAPACITY;
  }
  return GSN_OK;
}

int gsn_check(gsn_net* net, void* stream) {
  if (!net) return GSN_E_INVAL;
  int32_t code = 0;
  int rc = read_status_slot(net, gsn::kStError, &code, as_stream(stream));
  if (rc) return rc;
  return code;
}

void gsn_destroy(gsn_net* net) {
  if (!net) return;
  for (auto& g : net->graphs) (void)hipGraphExecDestroy(g.exec);
  if (net->cap_stream) (void)hipStreamDestroy(net->cap_stream);
  for (auto& v : net->rec)
    for (auto& pr : v) {
      (void)hipEventDestroy(pr.first);
      (void)hipEventDestroy(pr.second);
    }
  for (hipEvent_t e : net->pool) (void)hipEventDestroy(e);
  if (net->feedback) (void)hipHostFree(net->feedback);
  delete net;
}

int gsn_tune(gsn_net* net, int32_t key, int32_t value) {
  if (!net) return GSN_E_INVAL;
  switch (key) {
    case GSN_TUNE_SPLIT:
      if (value < 0 || value > GSN_MAX_SPLIT) return GSN_E_INVAL;
      net->tune_split = value;
      return GSN_OK;
    case GSN_TUNE_VARIANT:
      if (value < 0 || value > 6) return GSN_E_INVAL;
      net->tune_variant = value;
      return GSN_OK;
    case GSN_TUNE_GRAB:
      if (value < 0 || value > 1024) return GSN_E_INVAL;
      net->tune_grab = value ? value : kDefaultGrab;
      return GSN_OK;
    case GSN_TUNE_REBUCKET:
      if (value < 0 || value > 4096) return GSN_E_INVAL;
      net->tune_rebucket = value ? value : kRebucketEvery;
      return GSN_OK;
    case GSN_TUNE_GRID_ROUNDS:
      if (value < 0 || value > gsn::kMaxGridRounds) return GSN_E_INVAL;  // 0: automatic
      net->grid_rounds = value;
      return GSN_OK;
    default:
      return GSN_E_INVAL;
  }
}

int gsn_stat(gsn_net* net, int32_t key, int64_t* value, void* stream) {
  if (!net || key < 0 || key > GSN_STAT_LOOP_RECORDS) return GSN_E_INVAL;
  if (key != GSN_STAT_CLEAR && !value) return GSN_E_INVAL;
  if (key == GSN_STAT_LOOP_RECORDS) {
    *value = net->loop_records;
    return GSN_OK;
  }
  hipStream_t st = as_stream(stream);
  int32_t* slots = net->s.rem + gsn::kRmRounds;
  if (key == GSN_STAT_CLEAR) {
    net->loop_records = 0;
    const int32_t zero[3] = {0, 0, 0};
    const unsigned long long zero64[2] = {0, 0};
    if (hipMemcpyAsync(slots, zero, sizeof(zero), hipMemcpyHostToDevice, st) != hipSuccess ||
        hipMemcpyAsync(net->s.acc64 + gsn::kA64Resolved, zero64, sizeof(zero64),
                       hipMemcpyHostToDevice, st) != hipSuccess)
      return GSN_E_HIP;
    return hip_ok(hipStreamSynchronize(st));
  }
  if (key == GSN_STAT_RESOLVED)
    return read_acc64(net, gsn::kA64Resolved, value, st);
  if (key == GSN_STAT_ACCEPTED)
    return read_acc64(net, gsn::kA64Accepted, value, st);
  int32_t h[3];
  if (hipMemcpyAsync(h, slots, sizeof(h), hipMemcpyDeviceToHost, st) != hipSuccess)
    return GSN_E_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return GSN_E_HIP;
  *value = key == GSN_STAT_ROUNDS ? h[0] : key == GSN_STAT_ROUNDS_MAX ? h[1] : h[2];
  return GSN_OK;
}

int gsn_timing_enable(gsn_net* net, int32_t enable) {
  if (!net) return GSN_E_INVAL;
  net->timing = enable != 0;
  return GSN_OK;
}

int gsn_timing_select(gsn_net* net, uint32_t mask) {
  if (!net || (mask >> GSN_T_COUNT) != 0) return GSN_E_INVAL;
  net->timing_mask = mask;
  return GSN_OK;
}

int gsn_timing_read(gsn_net* net, int32_t which, double* total_ms, int32_t* launches) {
  if (!net || which < 0 || which >= GSN_T_COUNT) return GSN_E_INVAL;
  double sum = 0.0;
  int32_t cnt = 0;
  int rc = GSN_OK;
  for (auto& pr : net->rec[which]) {
    float ms = 0.0f;
    if (hipEventSynchronize(pr.second) != hipSuccess ||
        hipEventElapsedTime(&ms, pr.first, pr.second) != hipSuccess)
      rc = GSN_E_HIP;
    sum += ms;
    ++cnt;
    net->pool.push_back(pr.first);
    net->pool.push_back(pr.second);
  }
  net->rec[which].clear();
  if (total_ms) *total_ms = sum;
  if (launches) *launches = cnt;
  return rc;
}

}  // extern "C"
