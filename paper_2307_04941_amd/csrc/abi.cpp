// The C ABI (include/mg3m.h): validation, planning and dispatch.
//
// Validation is synchronous and finishes before anything is launched, so a
// rejected call writes nothing.  No exception crosses the interface.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <exception>
#include <functional>
#include <mutex>
#include <string>
#include <unordered_map>
#include <utility>
#include <vector>

#include "mg3m.h"
#include "mg3m_internal.h"

namespace {

thread_local std::string g_last_error;
// one-shot kernel timing events (mg3m_time_next_kernel)
thread_local hipEvent_t g_ev_start = nullptr, g_ev_stop = nullptr;

int fail(int status, const std::string& msg) {
  g_last_error = msg;
  return status;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  uintptr_t pa = reinterpret_cast<uintptr_t>(a), pb = reinterpret_cast<uintptr_t>(b);
  return pa < pb + nb && pb < pa + na;
}

using Geom = mg3m::ConvGeom;

Geom geom(int N, int C, int H, int W, int K, int R, int S, int sh, int sw, int ph, int pw, int layout,
          bool acc64 = false) {
  return Geom{N, C, H, W, K, R, S, sh, sw, ph, pw, layout, acc64};
}

// Plans already made, by everything a plan depends on: the selector scores
// about 170 candidates (several microseconds of host time), which for the
// small layers of a network is as long as the kernel.  Bounded; cleared when
// full.  Guarded by a mutex: calls may come from several host threads.
struct PlanKey {
  int v[16];
  std::string override_text;
  bool operator==(const PlanKey& o) const {
    return std::memcmp(v, o.v, sizeof v) == 0 && override_text == o.override_text;
  }
};
struct PlanKeyHash {
  size_t operator()(const PlanKey& k) const {
    size_t h = std::hash<std::string>()(k.override_text);
    for (int x : k.v) h = h * 1000003u ^ std::hash<int>()(x);
    return h;
  }
};
struct PlanCache {
  std::mutex mu;
  std::unordered_map<PlanKey, std::pair<mg3m::ConvShape, mg3m::Plan>, PlanKeyHash> map;
};
PlanCache& plan_cache() {
  static PlanCache* c = new PlanCache();   // never destroyed: usable from exit-time destructors
  return *c;
}
constexpr size_t kPlanCacheMax = 4096;

// MG3M_FORCE_PLAN stands in for a missing override; MG3M_LOG=1 reports each
// new plan on stderr.
const char* forced_plan() {
  const char* e = std::getenv("MG3M_FORCE_PLAN");
  return (e != nullptr && *e != 0) ? e : nullptr;
}
bool log_plans() {
  const char* e = std::getenv("MG3M_LOG");
  return e != nullptr && *e != 0 && std::strcmp(e, "0") != 0;
}

int shape_and_plan(const Geom& g, const char* plan, bool x16, bool w16, bool y16,
                   mg3m::ConvShape* s, mg3m::Plan* p) {
  const char* forced = plan == nullptr ? forced_plan() : nullptr;
  if (forced != nullptr) plan = forced;
  PlanKey key{{g.N, g.C, g.H, g.W, g.K, g.R, g.S, g.sh, g.sw, g.ph, g.pw, g.layout,
               (g.acc64 ? 1 : 0), (x16 ? 4 : 0) | (w16 ? 2 : 0) | (y16 ? 1 : 0),
               (int)(uint32_t)((uint64_t)g.ws_cap >> 32), (int)(uint32_t)g.ws_cap},
              plan ? std::string(plan) : std::string("\x01")};
  PlanCache& cache = plan_cache();
  {
    std::lock_guard<std::mutex> lock(cache.mu);
    auto it = cache.map.find(key);
    if (it != cache.map.end()) {
      *s = it->second.first;
      *p = it->second.second;
      return MG3M_OK;
    }
  }
  std::string err;
  int rc = mg3m::make_shape(g.N, g.C, g.H, g.W, g.K, g.R, g.S, g.sh, g.sw, g.ph, g.pw, g.layout, s, &err);
  if (rc) return fail(rc, err);
  rc = mg3m::make_plan(*s, plan, g.acc64, x16, w16, y16, p, &err, g.ws_cap);
  if (rc) return fail(rc, forced != nullptr ? err + " (plan forced by MG3M_FORCE_PLAN)" : err);
  if (log_plans())
    std::fprintf(stderr, "mg3m plan: N=%d C=%d H=%d W=%d K=%d R=%d S=%d stride=%dx%d pad=%dx%d %s%s%s: %s\n",
                 g.N, g.C, g.H, g.W, g.K, g.R, g.S, g.sh, g.sw, g.ph, g.pw,
                 g.layout == mg3m::kHWCN ? "HWCN" : "NCHW", g.acc64 ? " acc64" : "",
                 forced != nullptr ? " (MG3M_FORCE_PLAN)" : "", mg3m::plan_to_string(*s, *p).c_str());
  std::lock_guard<std::mutex> lock(cache.mu);
  if (cache.map.size() >= kPlanCacheMax) cache.map.clear();
  cache.map.emplace(std::move(key), std::make_pair(*s, *p));
  return MG3M_OK;
}

// The plain entry points take their partials from one stream-ordered pool per
// device, made on first use.  Its release threshold is the maximum, so a freed
// block stays mapped in the pool and the next call on that device reuses it.
// With the default pool (threshold 0) every call mapped its 20-100 MB of
// partials afresh, which cost 5-16 us per call on the VGG-16 layers.  A pool
// holds the most that calls on its device had live at once, until the process
// ends or mg3m_trim_workspace_pool() gives back what no call is using.
struct WsPools {
  std::mutex mu;
  std::unordered_map<int, hipMemPool_t> pools;
};
WsPools& ws_pools() {
  static WsPools* p = new WsPools();   // never destroyed, like the plan cache
  return *p;
}

int workspace_pool(void* stream, hipMemPool_t* pool, std::string* err) {
  int dev = 0;
  hipError_t e = stream != nullptr ? hipStreamGetDevice(static_cast<hipStream_t>(stream), &dev)
                                   : hipGetDevice(&dev);
  if (e != hipSuccess) {
    *err = std::string("device of the stream: ") + hipGetErrorString(e);
    return MG3M_ERR_HIP;
  }
  WsPools& wp = ws_pools();
  std::lock_guard<std::mutex> lock(wp.mu);
  auto it = wp.pools.find(dev);
  if (it != wp.pools.end()) {
    *pool = it->second;
    return MG3M_OK;
  }
  hipMemPoolProps props{};
  props.allocType = hipMemAllocationTypePinned;
  props.handleTypes = hipMemHandleTypeNone;
  props.location.type = hipMemLocationTypeDevice;
  props.location.id = dev;
  hipMemPool_t p = nullptr;
  e = hipMemPoolCreate(&p, &props);
  if (e != hipSuccess) {
    *err = std::string("hipMemPoolCreate: ") + hipGetErrorString(e);
    return MG3M_ERR_HIP;
  }
  uint64_t keep = UINT64_MAX;
  e = hipMemPoolSetAttribute(p, hipMemPoolAttrReleaseThreshold, &keep);
  if (e != hipSuccess) {
    (void)hipMemPoolDestroy(p);
    *err = std::string("hipMemPoolSetAttribute: ") + hipGetErrorString(e);
    return MG3M_ERR_HIP;
  }
  wp.pools.emplace(dev, p);
  *pool = p;
  return MG3M_OK;
}

// Above the pool sits one grow-only workspace per (device, stream handle) for
// streams that are not being captured: each call on a stream reuses the
// buffer the last call there left, so the steady state neither allocates nor
// frees.  (Taking and giving back a pool block per call made
// hipMallocFromPoolAsync wait for the stream's queued work whenever the last
// block was freed by a call not yet run, which kept the host from running
// ahead: 300-600 us per call on the ResNet-50 layers.)  Each buffer carries
// the event recorded after the last call that used it, and a call first makes
// its stream wait for that event: on the same stream this orders nothing new,
// and if a destroyed stream's handle comes back for a new stream, the new
// stream's calls still start after the old ones.  A larger plan frees the old
// buffer on the stream (after that wait) and takes a larger one.  The lock is
// held from the lookup until the call's launches and its event are queued.
// At most kWsStreamsPerDevice streams per device get a buffer, later ones
// use the pool per call; captured calls use the pool too, whose blocks the
// graph then owns.
constexpr int kWsStreamsPerDevice = 32;
struct WsCache {
  struct Entry {
    int dev;
    void* stream;
    void* ptr;
    size_t bytes;
    hipEvent_t last;      // recorded after the last call that used ptr
  };
  std::mutex mu;
  std::vector<Entry> entries;
};
WsCache& ws_cache() {
  static WsCache* c = new WsCache();   // never destroyed, like the pools
  return *c;
}

// The workspace of one call.  Either the stream's cached buffer: *lock then
// holds the cache and *done is the event the caller records on the stream
// after its last launch; or (the stream is being captured, or the device
// already has kWsStreamsPerDevice cached streams) a pool block that the
// caller gives back with hipFreeAsync (*done = nullptr).
int own_workspace_for(void* stream, size_t bytes, float** ws, hipEvent_t* done,
                      std::unique_lock<std::mutex>* lock, std::string* err) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  *done = nullptr;
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  hipError_t e = hipStreamIsCapturing(st, &cap);
  if (e != hipSuccess) {
    *err = std::string("hipStreamIsCapturing: ") + hipGetErrorString(e);
    return MG3M_ERR_HIP;
  }
  int dev = 0;
  e = st != nullptr ? hipStreamGetDevice(st, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess) {
    *err = std::string("device of the stream: ") + hipGetErrorString(e);
    return MG3M_ERR_HIP;
  }
  hipMemPool_t pool = nullptr;
  if (int rc = workspace_pool(stream, &pool, err)) return rc;
  if (cap == hipStreamCaptureStatusNone) {
    WsCache& c = ws_cache();
    std::unique_lock<std::mutex> lk(c.mu);
    WsCache::Entry* hit = nullptr;
    int on_dev = 0;
    for (auto& en : c.entries) {
      if (en.dev == dev && en.stream == stream) hit = &en;
      on_dev += en.dev == dev;
    }
    if (hit == nullptr && on_dev < kWsStreamsPerDevice) {
      // the event belongs to the stream's device, whichever device is current
      hipEvent_t ev = nullptr;
      int cur = dev;
      e = hipGetDevice(&cur);
      if (e == hipSuccess && cur != dev) e = hipSetDevice(dev);
      if (e == hipSuccess) e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
      if (cur != dev) {
        const hipError_t e2 = hipSetDevice(cur);
        if (e == hipSuccess) e = e2;
      }
      if (e != hipSuccess) {
        *err = std::string("hipEventCreateWithFlags: ") + hipGetErrorString(e);
        return MG3M_ERR_HIP;
      }
      c.entries.push_back({dev, stream, nullptr, 0, ev});
      hit = &c.entries.back();
    } else if (hit != nullptr) {
      e = hipStreamWaitEvent(st, hit->last, 0);
      if (e != hipSuccess) {
        *err = std::string("hipStreamWaitEvent: ") + hipGetErrorString(e);
        return MG3M_ERR_HIP;
      }
    }
    if (hit != nullptr) {
      if (hit->bytes < bytes) {
        if (hit->ptr != nullptr) {
          e = hipFreeAsync(hit->ptr, st);      // after every call that used it
          if (e != hipSuccess) {
            *err = std::string("hipFreeAsync: ") + hipGetErrorString(e);
            return MG3M_ERR_HIP;
          }
          hit->ptr = nullptr;
          hit->bytes = 0;
        }
        e = hipMallocFromPoolAsync(&hit->ptr, bytes, pool, st);
        if (e != hipSuccess) {
          hit->ptr = nullptr;
          *err = std::string("hipMallocFromPoolAsync: ") + hipGetErrorString(e);
          return MG3M_ERR_HIP;
        }
        hit->bytes = bytes;
      }
      *ws = static_cast<float*>(hit->ptr);
      *done = hit->last;
      *lock = std::move(lk);
      return MG3M_OK;
    }
  }
  e = hipMallocFromPoolAsync(reinterpret_cast<void**>(ws), bytes, pool, st);
  if (e != hipSuccess) {
    *err = std::string("hipMallocFromPoolAsync: ") + hipGetErrorString(e);
    return MG3M_ERR_HIP;
  }
  return MG3M_OK;
}

int run(const float* x, const float* w, float* y, const Geom& g, void* workspace,
        size_t workspace_bytes, bool own_workspace, const char* plan, void* stream,
        const float* add = nullptr, int relu = 0) {
  g_last_error.clear();
  if (x == nullptr || w == nullptr || y == nullptr) return fail(MG3M_ERR_NULL, "x, w and y must be non-NULL");
  if (!aligned(x, 4) || !aligned(w, 4) || !aligned(y, 4) || !aligned(add, 4))
    return fail(MG3M_ERR_ALIGN, "x, w, y and add must be 4-byte aligned");
  if (relu != 0 && relu != 1) return fail(MG3M_ERR_ARG, "relu must be 0 or 1");
  mg3m::ConvShape s;
  mg3m::Plan p;
  int rc = shape_and_plan(g, plan, aligned(x, 16), aligned(w, 16), aligned(y, 16), &s, &p);
  if (rc) return rc;
  const int N = g.N, C = g.C, H = g.H, W = g.W, K = g.K, R = g.R, S = g.S;
  const size_t xb = 4ull * N * C * H * W, wb = 4ull * K * C * R * S;
  const size_t yb = 4ull * (size_t)s.Mg * (size_t)s.Ng;
  if (overlap(y, yb, x, xb) || overlap(y, yb, w, wb))
    return fail(MG3M_ERR_ALIAS, "y overlaps x or w");
  // add may be y itself (each output reads its own add element first), or disjoint from it
  if (add != nullptr && add != y && overlap(add, yb, y, yb))
    return fail(MG3M_ERR_ALIAS, "add partly overlaps y");

  float* ws = nullptr;
  bool pooled = false;                       // ws is a pool block to give back after the launches
  hipEvent_t ws_done = nullptr;              // else, with own_workspace: recorded after the launches
  std::unique_lock<std::mutex> ws_lock;      // holds the per-stream workspace until then
  if (p.ws_bytes > 0) {
    if (own_workspace) {
      std::string perr;
      if (int prc = own_workspace_for(stream, p.ws_bytes, &ws, &ws_done, &ws_lock, &perr)) return fail(prc, perr);
      pooled = ws_done == nullptr;
    } else {
      if (workspace == nullptr || workspace_bytes < p.ws_bytes)
        return fail(MG3M_ERR_WORKSPACE, "plan needs " + std::to_string(p.ws_bytes) + " workspace bytes");
      if (!aligned(workspace, 16)) return fail(MG3M_ERR_WORKSPACE, "workspace must be 16-byte aligned");
      if (overlap(workspace, p.ws_bytes, x, xb) || overlap(workspace, p.ws_bytes, w, wb) ||
          overlap(workspace, p.ws_bytes, y, yb))
        return fail(MG3M_ERR_ALIAS, "workspace overlaps x, w or y");
      ws = static_cast<float*>(workspace);
    }
  }

  // workspace: [R][S][C][K] filter copy (tap-major NCHW plans) or the HWCN
  // copies of x, w and y (NCHW calls run as HWCN), then the partials
  const bool via = p.via_hwcn != 0;
  auto at_byte = [&](size_t off) { return reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + off); };
  const size_t xr = (xb + 255) / 256 * 256, wr = (wb + 255) / 256 * 256;
  float* const wt = p.wt_bytes > 0 ? ws : nullptr;
  float* const xh = via ? at_byte(0) : nullptr;
  float* const wh = via ? at_byte(xr) : nullptr;
  float* const yh = via ? at_byte(xr + wr) : nullptr;
  float* const part = ws != nullptr ? at_byte(p.wt_bytes + p.via_bytes) : nullptr;
  float* const yk = via ? yh : y;                  // the output the kernels write
  mg3m::KArgs a{};
  a.x = via ? xh : x; a.w = via ? wh : (wt != nullptr ? wt : w); a.y = yk; a.ws = part;
  a.x_bytes = (unsigned)xb; a.w_bytes = (unsigned)wb; a.y_bytes = (unsigned)yb;
  a.N = s.N; a.C = s.C; a.H = s.H; a.W = s.W; a.K = s.K; a.R = s.R; a.S = s.S;
  a.sh = s.sh; a.sw = s.sw; a.ph = s.ph; a.pw = s.pw; a.Ho = s.Ho; a.Wo = s.Wo;
  a.Mg = (int)s.Mg; a.Ng = (int)s.Ng; a.Kg = (int)s.Kg;
  a.tiles_m = p.tiles_m; a.k_tiles = p.k_tiles;
  a.dp_tiles = p.dp_tiles; a.tail_tiles = p.tail_tiles; a.sk_q = p.sk_q; a.sk_r = p.sk_r; a.sk_s = p.sk_s;
  a.e_mode = p.e_mode;
  const int klayout = via ? mg3m::kHWCN : s.layout;   // the layout the kernels run in
  a.mstride = klayout == mg3m::kHWCN ? s.N : s.Ho * s.Wo;
  // an NCHW call run as HWCN applies its output stage on the way back to NCHW
  a.add = via ? nullptr : add;
  a.relu = via ? 0 : relu;

  std::string err;
  if (wt != nullptr) rc = mg3m::launch_filter_to_rsck(w, wt, s.K, s.C, s.R, s.S, stream, &err);
  if (via) {
    // one launch: [N][C][H][W] -> [H][W][C][N] and [K][C][R][S] -> [R][S][C][K]
    mg3m::SwapJob jobs[2] = {};
    jobs[0].in = x; jobs[0].out = xh; jobs[0].A = s.N; jobs[0].Cm = s.C; jobs[0].B = s.H * s.W;
    jobs[1].in = w; jobs[1].out = wh; jobs[1].A = s.K; jobs[1].Cm = s.C; jobs[1].B = s.R * s.S;
    unsigned tiles = 0;
    rc = mg3m::prepare_swap_batch(jobs, 2, &tiles, &err);
    if (rc == MG3M_OK) rc = mg3m::launch_swap_outer_inner_pair(jobs, tiles, stream, &err);
  }
  hipEvent_t ev0 = g_ev_start, ev1 = g_ev_stop;
  g_ev_start = g_ev_stop = nullptr;
  if (rc == MG3M_OK) rc = mg3m::launch_conv(p, a, stream, &err, ev0, ev1);
  if (rc == MG3M_OK && p.tail_tiles > 0) {
    mg3m::RArgs r{};
    r.ws = part; r.y = yk; r.mt = p.t.mt; r.nt = p.t.nt;
    r.tiles_m = p.tiles_m; r.dp_tiles = p.dp_tiles; r.tail_tiles = p.tail_tiles;
    r.k_tiles = p.k_tiles; r.sk_q = p.sk_q; r.sk_r = p.sk_r; r.sk_s = p.sk_s;
    r.layout = klayout; r.N = s.N; r.K = s.K; r.HoWo = s.Ho * s.Wo;
    r.Mg = (int)s.Mg; r.Ng = (int)s.Ng;
    const bool contiguous4 = klayout == mg3m::kHWCN ? s.N % 4 == 0 : (s.Ho * s.Wo) % 4 == 0;
    r.vec4 = contiguous4 && aligned(yk, 16);
    r.f64 = p.acc64;
    r.add = a.add;
    r.relu = a.relu;
    rc = mg3m::launch_tail_reduce(r, stream, &err);
  }
  // [Ho][Wo][K][N] -> [N][K][Ho][Wo], with the output stage
  if (rc == MG3M_OK && via) rc = mg3m::launch_swap_outer_inner(yh, y, s.Ho * s.Wo, s.K, s.N, stream, &err, add, relu);
  if (ws_done != nullptr) {
    // recorded even after a failed launch: a later call waits for what was queued
    hipError_t e = hipEventRecord(ws_done, static_cast<hipStream_t>(stream));
    if (rc == MG3M_OK && e != hipSuccess) {
      rc = MG3M_ERR_HIP;
      err = std::string("hipEventRecord: ") + hipGetErrorString(e);
    }
  }
  if (pooled) {
    hipError_t e = hipFreeAsync(ws, static_cast<hipStream_t>(stream));
    if (rc == MG3M_OK && e != hipSuccess) {
      rc = MG3M_ERR_HIP;
      err = std::string("hipFreeAsync: ") + hipGetErrorString(e);
    }
  }
  if (rc) return fail(rc, err);
  return MG3M_OK;
}

}  // namespace

namespace mg3m {

int set_error(int status, const std::string& msg) { return fail(status, msg); }
void clear_error() { g_last_error.clear(); }

int conv_run(const float* x, const float* w, float* y, const ConvGeom& g, void* workspace,
             size_t workspace_bytes, bool own_workspace, const char* plan, const float* add, int relu,
             void* stream) {
  try {
    return run(x, w, y, g, workspace, workspace_bytes, own_workspace, plan, stream, add, relu);
  } catch (const std::exception& e) {
    return fail(MG3M_ERR_HIP, e.what());
  } catch (...) {
    return fail(MG3M_ERR_HIP, "unknown exception");
  }
}

int conv_plan(const ConvGeom& g, const char* plan, ConvShape* s, Plan* p) {
  return shape_and_plan(g, plan, true, true, true, s, p);
}

int maxpool_dims(int H, int W, int R, int S, int sh, int sw, int ph, int pw, int* Ho, int* Wo,
                 std::string* err) {
  if (H < 1 || W < 1 || R < 1 || S < 1 || sh < 1 || sw < 1 || ph < 0 || pw < 0) {
    *err = "pooling: sizes and strides must be >= 1, pads >= 0";
    return MG3M_ERR_SHAPE;
  }
  if (2 * ph > R || 2 * pw > S) {
    *err = "pooling: padding must be at most half the window";
    return MG3M_ERR_SHAPE;
  }
  ConvShape s;
  int rc = make_shape(1, 1, H, W, 1, R, S, sh, sw, ph, pw, kHWCN, &s, err);
  if (rc) return rc;
  *Ho = s.Ho;
  *Wo = s.Wo;
  return MG3M_OK;
}

int maxpool_run(const float* x, float* y, int N, int C, int H, int W, int R, int S, int sh, int sw,
                int ph, int pw, int layout, void* stream) {
  try {
    g_last_error.clear();
    if (x == nullptr || y == nullptr) return fail(MG3M_ERR_NULL, "x and y must be non-NULL");
    if (!aligned(x, 4) || !aligned(y, 4)) return fail(MG3M_ERR_ALIGN, "x and y must be 4-byte aligned");
    if (layout != kHWCN && layout != kNCHW) return fail(MG3M_ERR_LAYOUT, "unknown layout");
    if (N < 1 || C < 1) return fail(MG3M_ERR_SHAPE, "N and C must be >= 1");
    std::string err;
    int Ho = 0, Wo = 0;
    int rc = maxpool_dims(H, W, R, S, sh, sw, ph, pw, &Ho, &Wo, &err);
    if (rc) return fail(rc, err);
    const long long xe = (long long)N * C * H * W, ye = (long long)N * C * Ho * Wo;
    if (xe > kMaxTensorBytes / 4 || ye > kMaxTensorBytes / 4)
      return fail(MG3M_ERR_TOO_LARGE, "a tensor is larger than 4 GiB - 64 bytes");
    if (overlap(y, 4 * (size_t)ye, x, 4 * (size_t)xe)) return fail(MG3M_ERR_ALIAS, "y overlaps x");
    PArgs p{};
    p.x = x; p.y = y;
    p.N = N; p.C = C; p.H = H; p.W = W; p.R = R; p.S = S;
    p.sh = sh; p.sw = sw; p.ph = ph; p.pw = pw; p.Ho = Ho; p.Wo = Wo;
    p.layout = layout;
    p.aligned16 = aligned(x, 16) && aligned(y, 16);
    rc = launch_maxpool(p, stream, &err);
    if (rc) return fail(rc, err);
    return MG3M_OK;
  } catch (...) {
    return fail(MG3M_ERR_HIP, "unknown exception");
  }
}

}  // namespace mg3m

extern "C" {

int conv2d_fwd_f32_fused(const float* x, const float* w, float* y, const float* add, int relu, int N,
                         int C, int H, int W, int K, int R, int S, int stride_h, int stride_w,
                         int pad_h, int pad_w, int layout, void* workspace, size_t workspace_bytes,
                         const char* plan, void* stream) {
  return mg3m::conv_run(x, w, y, geom(N, C, H, W, K, R, S, stride_h, stride_w, pad_h, pad_w, layout),
                        workspace, workspace_bytes, false, plan, add, relu, stream);
}

int maxpool2d_f32(const float* x, float* y, int N, int C, int H, int W, int R, int S, int stride_h,
                  int stride_w, int pad_h, int pad_w, int layout, void* stream) {
  return mg3m::maxpool_run(x, y, N, C, H, W, R, S, stride_h, stride_w, pad_h, pad_w, layout, stream);
}

int maxpool2d_out_dims(int H, int W, int R, int S, int stride_h, int stride_w, int pad_h, int pad_w,
                       int* Ho, int* Wo) {
  g_last_error.clear();
  if (Ho == nullptr || Wo == nullptr) return fail(MG3M_ERR_NULL, "Ho and Wo must be non-NULL");
  std::string err;
  int rc = mg3m::maxpool_dims(H, W, R, S, stride_h, stride_w, pad_h, pad_w, Ho, Wo, &err);
  return rc ? fail(rc, err) : MG3M_OK;
}

int conv2d_out_dims_hw(int H, int W, int R, int S, int stride_h, int stride_w, int pad_h, int pad_w,
                       int* Ho, int* Wo) {
  g_last_error.clear();
  if (Ho == nullptr || Wo == nullptr) return fail(MG3M_ERR_NULL, "Ho and Wo must be non-NULL");
  mg3m::ConvShape s;
  std::string err;
  int rc = mg3m::make_shape(1, 1, H, W, 1, R, S, stride_h, stride_w, pad_h, pad_w, MG3M_LAYOUT_HWCN,
                            &s, &err);
  if (rc) return fail(rc, err);
  *Ho = s.Ho;
  *Wo = s.Wo;
  return MG3M_OK;
}

int conv2d_out_dims(int H, int W, int R, int S, int stride, int pad, int* Ho, int* Wo) {
  return conv2d_out_dims_hw(H, W, R, S, stride, stride, pad, pad, Ho, Wo);
}

int conv2d_fwd_f32(const float* x, const float* w, float* y, int N, int C, int H, int W, int K,
                   int R, int S, int stride, int pad, int layout, void* stream) {
  try {
    return run(x, w, y, geom(N, C, H, W, K, R, S, stride, stride, pad, pad, layout), nullptr, 0,
               true, nullptr, stream);
  } catch (const std::exception& e) {
    return fail(MG3M_ERR_HIP, e.what());
  } catch (...) {
    return fail(MG3M_ERR_HIP, "unknown exception");
  }
}

int conv2d_fwd_f32_ex(const float* x, const float* w, float* y, int N, int C, int H, int W, int K,
                      int R, int S, int stride, int pad, int layout, void* workspace,
                      size_t workspace_bytes, const char* plan, void* stream) {
  try {
    return run(x, w, y, geom(N, C, H, W, K, R, S, stride, stride, pad, pad, layout), workspace,
               workspace_bytes, false, plan, stream);
  } catch (const std::exception& e) {
    return fail(MG3M_ERR_HIP, e.what());
  } catch (...) {
    return fail(MG3M_ERR_HIP, "unknown exception");
  }
}

int conv2d_fwd_f32_hw(const float* x, const float* w, float* y, int N, int C, int H, int W, int K,
                      int R, int S, int stride_h, int stride_w, int pad_h, int pad_w, int layout,
                      void* workspace, size_t workspace_bytes, const char* plan, void* stream) {
  try {
    return run(x, w, y, geom(N, C, H, W, K, R, S, stride_h, stride_w, pad_h, pad_w, layout),
               workspace, workspace_bytes, false, plan, stream);
  } catch (const std::exception& e) {
    return fail(MG3M_ERR_HIP, e.what());
  } catch (...) {
    return fail(MG3M_ERR_HIP, "unknown exception");
  }
}

static int workspace_bytes(const Geom& g, const char* plan, size_t* bytes) {
  try {
    g_last_error.clear();
    if (bytes == nullptr) return fail(MG3M_ERR_NULL, "bytes must be non-NULL");
    mg3m::ConvShape s;
    mg3m::Plan p;
    int rc = shape_and_plan(g, plan, true, true, true, &s, &p);
    if (rc) return rc;
    *bytes = p.ws_bytes;
    return MG3M_OK;
  } catch (...) {
    return fail(MG3M_ERR_HIP, "unknown exception");
  }
}

int conv2d_fwd_f32_workspace_bytes(int N, int C, int H, int W, int K, int R, int S, int stride,
                                   int pad, int layout, const char* plan, size_t* bytes) {
  return workspace_bytes(geom(N, C, H, W, K, R, S, stride, stride, pad, pad, layout), plan, bytes);
}

int conv2d_fwd_f32_hw_workspace_bytes(int N, int C, int H, int W, int K, int R, int S, int stride_h,
                                      int stride_w, int pad_h, int pad_w, int layout, const char* plan,
                                      size_t* bytes) {
  return workspace_bytes(geom(N, C, H, W, K, R, S, stride_h, stride_w, pad_h, pad_w, layout), plan,
                         bytes);
}

static int plan_string(const Geom& g, const char* plan, char* buf, size_t len) {
  try {
    g_last_error.clear();
    if (buf == nullptr) return fail(MG3M_ERR_NULL, "buf must be non-NULL");
    mg3m::ConvShape s;
    mg3m::Plan p;
    int rc = shape_and_plan(g, plan, true, true, true, &s, &p);
    if (rc) return rc;
    std::string text = mg3m::plan_to_string(s, p);
    if (len < text.size() + 1) return fail(MG3M_ERR_ARG, "buffer too short for the plan string");
    std::memcpy(buf, text.c_str(), text.size() + 1);
    return MG3M_OK;
  } catch (...) {
    return fail(MG3M_ERR_HIP, "unknown exception");
  }
}

int conv2d_fwd_f32_plan_string(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                               int layout, const char* plan, char* buf, size_t len) {
  return plan_string(geom(N, C, H, W, K, R, S, stride, stride, pad, pad, layout), plan, buf, len);
}

int conv2d_fwd_f32_acc64(const float* x, const float* w, float* y, int N, int C, int H, int W,
                         int K, int R, int S, int stride_h, int stride_w, int pad_h, int pad_w,
                         int layout, const char* plan, void* stream) {
  try {
    return run(x, w, y, geom(N, C, H, W, K, R, S, stride_h, stride_w, pad_h, pad_w, layout, true),
               nullptr, 0, true, plan, stream);
  } catch (const std::exception& e) {
    return fail(MG3M_ERR_HIP, e.what());
  } catch (...) {
    return fail(MG3M_ERR_HIP, "unknown exception");
  }
}

int conv2d_fwd_f32_acc64_plan_string(int N, int C, int H, int W, int K, int R, int S, int stride_h,
                                     int stride_w, int pad_h, int pad_w, int layout, const char* plan,
                                     char* buf, size_t len) {
  return plan_string(geom(N, C, H, W, K, R, S, stride_h, stride_w, pad_h, pad_w, layout, true), plan,
                     buf, len);
}

int conv2d_fwd_f32_plan_info(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                             int layout, const char* plan, mg3m_plan_info* info) {
  try {
    g_last_error.clear();
    if (info == nullptr) return fail(MG3M_ERR_NULL, "info must be non-NULL");
    mg3m::ConvShape s;
    mg3m::Plan p;
    int rc = shape_and_plan(geom(N, C, H, W, K, R, S, stride, stride, pad, pad, layout), plan, true,
                            true, true, &s, &p);
    if (rc) return rc;
    info->mt = p.t.mt; info->nt = p.t.nt; info->kt = p.t.kt;
    info->waves_m = p.t.wm; info->waves_n = p.t.wn;
    info->split = p.split; info->k_tiles = p.k_tiles;
    info->k_tiles_per_wg = p.tail_wgs > 0 ? p.sk_q + (p.sk_r > 0 ? 1 : 0) : p.k_tiles;
    info->dp_tiles = p.dp_tiles; info->tail_tiles = p.tail_tiles; info->tail_wgs = p.tail_wgs;
    info->tiles_m = p.tiles_m; info->tiles_n = p.tiles_n; info->grid = p.grid;
    info->Mg = s.Mg; info->Ng = s.Ng; info->Kg = s.Kg;
    info->workspace_bytes = p.ws_bytes; info->lds_bytes = p.lds_bytes;
    info->pad_efficiency = p.pad_eff; info->est_us = p.est_us;
    info->layout = p.layout; info->a_mode = p.a_mode; info->b_mode = p.b_mode;
    info->e_mode = p.e_mode;
    info->persistent = p.persist;
    info->via_hwcn = p.via_hwcn;
    return MG3M_OK;
  } catch (...) {
    return fail(MG3M_ERR_HIP, "unknown exception");
  }
}

int mg3m_time_next_kernel(void* start, void* stop) {
  g_last_error.clear();
  if ((start == nullptr) != (stop == nullptr)) return fail(MG3M_ERR_ARG, "give both events or neither");
  g_ev_start = static_cast<hipEvent_t>(start);
  g_ev_stop = static_cast<hipEvent_t>(stop);
  return MG3M_OK;
}

int mg3m_padding_overhead(int M, int N, int C, int mt, int nt, double* flop_overhead,
                          double* data_overhead) {
  g_last_error.clear();
  if (flop_overhead == nullptr || data_overhead == nullptr)
    return fail(MG3M_ERR_NULL, "out-parameters must be non-NULL");
  if (M < 1 || N < 1 || C < 1 || mt < 1 || nt < 1) return fail(MG3M_ERR_SHAPE, "sizes must be >= 1");
  const double Mp = (double)((M + mt - 1) / mt) * mt, Np = (double)((N + nt - 1) / nt) * nt;
  *flop_overhead = Mp * Np / ((double)M * N) - 1.0;
  *data_overhead = ((double)C * Mp + (double)C * Np + Mp * Np) /
                       ((double)C * M + (double)C * N + (double)M * N) - 1.0;
  return MG3M_OK;
}

const char* mg3m_status_string(int status) {
  switch (status) {
    case MG3M_OK: return "MG3M_OK: success";
    case MG3M_ERR_NULL: return "MG3M_ERR_NULL: a required pointer is NULL";
    case MG3M_ERR_SHAPE: return "MG3M_ERR_SHAPE: invalid dimensions, stride, pad or empty output";
    case MG3M_ERR_LAYOUT: return "MG3M_ERR_LAYOUT: unknown layout";
    case MG3M_ERR_TOO_LARGE: return "MG3M_ERR_TOO_LARGE: tensor too large for 32-bit indexing";
    case MG3M_ERR_ALIAS: return "MG3M_ERR_ALIAS: output overlaps an input";
    case MG3M_ERR_WORKSPACE: return "MG3M_ERR_WORKSPACE: workspace missing, misaligned or too small";
    case MG3M_ERR_PLAN: return "MG3M_ERR_PLAN: invalid plan override";
    case MG3M_ERR_HIP: return "MG3M_ERR_HIP: HIP runtime error";
    case MG3M_ERR_ALIGN: return "MG3M_ERR_ALIGN: pointer not 4-byte aligned";
    case MG3M_ERR_ARG: return "MG3M_ERR_ARG: bad auxiliary argument";
    default: return "MG3M: unknown status";
  }
}

const char* mg3m_last_error(void) { return g_last_error.c_str(); }

int mg3m_trim_workspace_pool(void) {
  g_last_error.clear();
  {
    // per-stream buffers: wait for the last call that used each, then give
    // it back (its stream may be gone, so not stream-ordered)
    WsCache& c = ws_cache();
    std::lock_guard<std::mutex> lock(c.mu);
    int cur = 0;
    hipError_t e = hipGetDevice(&cur);
    for (auto& en : c.entries) {
      if (e == hipSuccess) e = hipEventSynchronize(en.last);
      if (e == hipSuccess) e = hipSetDevice(en.dev);
      if (e == hipSuccess && en.ptr != nullptr) e = hipFreeAsync(en.ptr, nullptr);
      if (e == hipSuccess) e = hipStreamSynchronize(nullptr);
      if (e == hipSuccess) e = hipEventDestroy(en.last);
      if (e != hipSuccess) break;
      en.last = nullptr;
    }
    if (e == hipSuccess) e = hipSetDevice(cur);
    c.entries.erase(std::remove_if(c.entries.begin(), c.entries.end(),
                                   [](const WsCache::Entry& en) { return en.last == nullptr; }),
                    c.entries.end());
    if (e != hipSuccess) return fail(MG3M_ERR_HIP, std::string("freeing the per-stream workspaces: ") +
                                                       hipGetErrorString(e));
  }
  WsPools& wp = ws_pools();
  std::lock_guard<std::mutex> lock(wp.mu);
  for (auto& kv : wp.pools) {
    hipError_t e = hipMemPoolTrimTo(kv.second, 0);
    if (e != hipSuccess)
      return fail(MG3M_ERR_HIP, "hipMemPoolTrimTo (device " + std::to_string(kv.first) + "): " + hipGetErrorString(e));
  }
  return MG3M_OK;
}

}  // extern "C"
