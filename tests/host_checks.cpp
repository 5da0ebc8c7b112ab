// Host-side checks built with AddressSanitizer and UndefinedBehaviorSanitizer
// (tests/test_host_sanitizers.py compiles and runs this with g++): the
// planner, the C ABI's validation and dispatch path and the network
// executor's validation, on a seeded grid of shapes, plan overrides and
// malformed arguments; and the CPU oracle against its pins.  Nothing here
// touches a GPU: the five kernel launchers are replaced by stubs that check
// each launch's arguments against the plan and the buffers instead of
// launching, and the device pointers passed in are never dereferenced.  HIP
// runtime calls (workspace pool, events, allocations) fail on a host without
// a GPU, which exercises their error paths.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "mg3m.h"
#include "mg3m_internal.h"

extern "C" {
int oracle_out_dims(int h, int w, int r, int s, int std_h, int std_w, int pad_h, int pad_w, int* out_h,
                    int* out_w);
int oracle_conv2d_f64(const float* x, const float* wt, double* acc, double* mag, int n, int c, int h, int w,
                      int k, int r, int s, int std_h, int std_w, int pad_h, int pad_w, int layout);
int oracle_conv2d_points_f64(const float* x, const float* wt, const int64_t* idx, int64_t npts, double* acc,
                             double* mag, int n, int c, int h, int w, int k, int r, int s, int std_h, int std_w,
                             int pad_h, int pad_w, int layout);
}

static int g_failures = 0;
#define CHECK(cond, ...)                                  \
  do {                                                    \
    if (!(cond)) {                                        \
      ++g_failures;                                       \
      std::fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
      std::fprintf(stderr, __VA_ARGS__);                  \
      std::fprintf(stderr, "\n");                         \
    }                                                     \
  } while (0)

// ------------------------------------------------------------ launch stubs
// What the last stubbed launches saw, for the checks after each call.
struct Seen {
  int convs = 0, reduces = 0, copies = 0, pools = 0, swaps = 0;
  mg3m::Plan plan{};
  mg3m::KArgs args{};
  mg3m::RArgs rargs{};
} g_seen;

namespace mg3m {

int launch_conv(const Plan& p, const KArgs& a, void*, std::string* err, void*, void*) {
  ++g_seen.convs;
  g_seen.plan = p;
  g_seen.args = a;
  // the launch covers every tile once: whole tiles, then the tail runs
  const long long tiles = (long long)p.tiles_m * p.tiles_n;
  CHECK((long long)p.tiles_m * p.t.mt >= a.Mg && (long long)(p.tiles_m - 1) * p.t.mt < a.Mg, "tiles_m");
  CHECK((long long)p.tiles_n * p.t.nt >= a.Ng && (long long)(p.tiles_n - 1) * p.t.nt < a.Ng, "tiles_n");
  CHECK((long long)p.k_tiles * p.t.kt >= a.Kg && (long long)(p.k_tiles - 1) * p.t.kt < a.Kg, "k_tiles");
  CHECK(p.dp_tiles + p.tail_tiles == tiles, "dp + tail tiles %d + %d != %lld", p.dp_tiles, p.tail_tiles, tiles);
  if (p.persist) {
    CHECK(p.tail_wgs == 0 && p.grid >= 1 && p.grid <= p.dp_tiles, "persistent grid");
  } else {
    CHECK(p.grid == (long long)p.dp_tiles + p.tail_wgs, "grid");
  }
  if (p.tail_wgs > 0) {
    CHECK(a.ws != nullptr, "tail runs without a workspace");
    // the tail runs cover the tail tiles' k-steps exactly: tail_wgs runs of
    // sk_q steps, sk_r of them one longer (per tile for split plans)
    const long long steps = (long long)p.tail_tiles * p.k_tiles;
    const long long covered = p.sk_s > 0 ? (long long)p.tail_tiles * ((long long)p.sk_s * p.sk_q + p.sk_r)
                                         : (long long)p.tail_wgs * p.sk_q + p.sk_r;
    CHECK(covered == steps, "tail runs cover %lld of %lld steps", covered, steps);
    CHECK(p.sk_q >= 1 && p.sk_q <= p.k_tiles, "run length");
    const long long slots = (long long)p.tail_wgs + p.tail_tiles - 1;
    CHECK((size_t)slots * p.t.mt * p.t.nt * (p.acc64 ? 8 : 4) + p.wt_bytes + p.via_bytes <= p.ws_bytes,
          "partial slots");
  }
  // tensor sizes the kernel addresses through its buffer resources
  CHECK((long long)a.x_bytes == 4LL * a.N * a.C * a.H * a.W, "x_bytes");
  CHECK((long long)a.w_bytes == 4LL * a.Kg * a.Mg, "w_bytes");
  CHECK((long long)a.y_bytes == 4LL * a.Mg * a.Ng, "y_bytes");
  CHECK(a.mstride == (p.layout == kHWCN ? a.N : a.Ho * a.Wo), "mstride");
  *err = "";
  return MG3M_OK;
}

int launch_tail_reduce(const RArgs& r, void*, std::string*) {
  ++g_seen.reduces;
  g_seen.rargs = r;
  CHECK(r.tail_tiles > 0 && r.mt % 4 == 0 && r.nt % 4 == 0, "reduce shape");
  return MG3M_OK;
}

int launch_maxpool(const PArgs& p, void*, std::string*) {
  ++g_seen.pools;
  CHECK(p.Ho >= 1 && p.Wo >= 1, "pool output");
  return MG3M_OK;
}

int launch_filter_to_rsck(const float*, float* wt, int K, int C, int R, int S, void*, std::string*) {
  ++g_seen.copies;
  CHECK(wt != nullptr && (long long)K * C * R * S > 0, "filter copy");
  return MG3M_OK;
}

int launch_swap_outer_inner(const float* in, float* out, int A, int Cm, int B, void*, std::string*,
                            const float*, int relu) {
  ++g_seen.swaps;
  CHECK(in != nullptr && out != nullptr && in != out && A >= 1 && Cm >= 1 && B >= 1, "layout change");
  CHECK(relu == 0 || relu == 1, "layout change relu");
  return MG3M_OK;
}

int launch_swap_outer_inner_pair(const SwapJob jobs[2], unsigned tiles, void*, std::string*) {
  ++g_seen.swaps;
  CHECK(jobs[1].tile0 >= 1 && tiles > jobs[1].tile0, "layout change pair");
  return MG3M_OK;
}

int launch_swap_outer_inner_batch(const SwapJob* jobs, int n, unsigned tiles, void*, std::string*) {
  ++g_seen.swaps;
  CHECK(n == 0 || (jobs != nullptr && tiles >= 1), "layout change batch");
  return MG3M_OK;
}

}  // namespace mg3m

// ------------------------------------------------------------ helpers
static uint64_t g_rng = 0x2307049410000001ull;
static uint32_t rnd() {   // xorshift64*
  g_rng ^= g_rng >> 12;
  g_rng ^= g_rng << 25;
  g_rng ^= g_rng >> 27;
  return (uint32_t)((g_rng * 0x2545F4914F6CDD1Dull) >> 32);
}
static int rint_in(int lo, int hi) { return lo + (int)(rnd() % (uint32_t)(hi - lo + 1)); }

// fake, 256-byte aligned device addresses far apart: never dereferenced
static float* fake(int i) { return reinterpret_cast<float*>((uintptr_t)(0x100000000ull * (uint64_t)(i + 1))); }

// ------------------------------------------------------------ planner and ABI
static void check_plans() {
  const char* tiles[] = {"128x128", "64x256", "256x64", "64x128", "128x64", "64x64", "32x128", "32x64",
                         "128x32", "64x32", "256x128", "128x256", "128x128,kt=32", "16x64", "64x64,kt=32"};
  int calls = 0;
  for (int it = 0; it < 1500; ++it) {
    const int N = rint_in(1, 70), C = rint_in(1, 600), K = rint_in(1, 600);
    const int H = rint_in(1, 60), W = rint_in(1, 60), R = rint_in(1, 7), S = rint_in(1, 7);
    const int st = rint_in(1, 4), pd = rint_in(0, 4), layout = rint_in(0, 1);
    int Ho = 0, Wo = 0;
    if (conv2d_out_dims(H, W, R, S, st, pd, &Ho, &Wo) != MG3M_OK) continue;
    std::string plan;
    switch (it % 6) {
      case 0: break;
      case 1: plan = std::string("tile=") + tiles[rnd() % 15] + ",split=" + std::to_string(rint_in(1, 20)); break;
      case 2: plan = std::string("tile=") + tiles[rnd() % 15] + ",tail=" + std::to_string(rint_in(2, 9)); break;
      case 3: plan = "sk=" + std::to_string(rint_in(1, 5000)); break;
      case 4: plan = std::string("tile=") + tiles[rnd() % 15] + ",persist=" + std::to_string(rint_in(1, 6)); break;
      default: plan = "split=" + std::to_string(rint_in(1, 64)); break;
    }
    const char* pl = plan.empty() ? nullptr : plan.c_str();
    mg3m_plan_info info;
    const int rc = conv2d_fwd_f32_plan_info(N, C, H, W, K, R, S, st, pd, layout, pl, &info);
    CHECK(rc == MG3M_OK || rc == MG3M_ERR_PLAN || rc == MG3M_ERR_TOO_LARGE, "plan_info rc %d", rc);
    if (rc != MG3M_OK) continue;
    char buf[1024];
    CHECK(conv2d_fwd_f32_plan_string(N, C, H, W, K, R, S, st, pd, layout, pl, buf, sizeof buf) == MG3M_OK,
          "plan_string");
    CHECK(conv2d_fwd_f32_plan_string(N, C, H, W, K, R, S, st, pd, layout, pl, buf, 8) == MG3M_ERR_ARG,
          "short buffer");
    size_t ws = 0;
    CHECK(conv2d_fwd_f32_workspace_bytes(N, C, H, W, K, R, S, st, pd, layout, pl, &ws) == MG3M_OK &&
              ws == info.workspace_bytes, "workspace bytes");
    // full dispatch path on fake buffers: validation, plan, launch stubs
    const Seen before = g_seen;
    const int rc2 = conv2d_fwd_f32_ex(fake(0), fake(1), fake(2), N, C, H, W, K, R, S, st, pd, layout,
                                      ws ? fake(3) : nullptr, ws, pl, nullptr);
    CHECK(rc2 == MG3M_OK, "dispatch rc %d (%s)", rc2, mg3m_last_error());
    CHECK(g_seen.convs == before.convs + 1, "one main launch");
    CHECK(g_seen.reduces == before.reduces + (info.tail_tiles > 0 ? 1 : 0), "tail reduce launch");
    CHECK(g_seen.plan.grid == info.grid && g_seen.plan.dp_tiles == info.dp_tiles, "plan reaches the launch");
    if (info.tail_tiles > 0) {
      CHECK(g_seen.rargs.tail_tiles == info.tail_tiles && g_seen.rargs.dp_tiles == info.dp_tiles, "reduce args");
    }
    // too small a workspace is rejected before any launch
    if (ws > 0) {
      const Seen b2 = g_seen;
      CHECK(conv2d_fwd_f32_ex(fake(0), fake(1), fake(2), N, C, H, W, K, R, S, st, pd, layout, fake(3), ws - 1, pl,
                              nullptr) == MG3M_ERR_WORKSPACE, "short workspace");
      CHECK(g_seen.convs == b2.convs, "nothing launched on a rejected call");
    }
    // the plain call takes its workspace from the device pool: without a GPU
    // that fails (a HIP error) whenever the plan needs one
    const int rc3 = conv2d_fwd_f32(fake(0), fake(1), fake(2), N, C, H, W, K, R, S, st, pd, layout, nullptr);
    CHECK(rc3 == MG3M_OK || rc3 == MG3M_ERR_HIP, "plain call rc %d", rc3);
    ++calls;
  }
  CHECK(calls > 500, "too few valid shapes (%d)", calls);
  std::printf("plans: %d shapes dispatched to the launch stubs\n", calls);
}

static void check_errors() {
  const int g[] = {2, 8, 10, 10, 16, 3, 3, 1, 1};
  auto call = [&](const float* x, const float* w, float* y, int layout) {
    return conv2d_fwd_f32(x, w, y, g[0], g[1], g[2], g[3], g[4], g[5], g[6], g[7], g[8], layout, nullptr);
  };
  const int convs = g_seen.convs;
  CHECK(call(nullptr, fake(1), fake(2), 0) == MG3M_ERR_NULL, "null x");
  CHECK(call(fake(0), fake(1), nullptr, 0) == MG3M_ERR_NULL, "null y");
  CHECK(call(reinterpret_cast<float*>((uintptr_t)fake(0) + 2), fake(1), fake(2), 0) == MG3M_ERR_ALIGN, "align");
  CHECK(call(fake(0), fake(1), fake(2), 7) == MG3M_ERR_LAYOUT, "layout");
  CHECK(call(fake(0), fake(1), fake(0), 0) == MG3M_ERR_ALIAS, "alias");
  CHECK(conv2d_fwd_f32(fake(0), fake(1), fake(2), 0, 8, 10, 10, 16, 3, 3, 1, 1, 0, nullptr) == MG3M_ERR_SHAPE, "N=0");
  CHECK(conv2d_fwd_f32(fake(0), fake(1), fake(2), 2, 8, 1, 1, 16, 5, 5, 1, 1, 0, nullptr) == MG3M_ERR_SHAPE, "empty");
  CHECK(conv2d_fwd_f32(fake(0), fake(1), fake(2), 1 << 20, 1 << 12, 64, 64, 16, 3, 3, 1, 1, 0, nullptr) ==
            MG3M_ERR_TOO_LARGE, "too large");
  CHECK(conv2d_fwd_f32(fake(0), fake(1), fake(2), 2, 8, 1 << 30, 1 << 30, 16, 3, 3, 1, 1, 0, nullptr) ==
            MG3M_ERR_TOO_LARGE, "huge spatial size");
  CHECK(conv2d_fwd_f32(fake(0), fake(1), fake(2), 2, 8, 10, 10, 16, 3, 3, 0x7fffffff, 0x7fffffff, 0, nullptr) ==
            MG3M_ERR_TOO_LARGE, "huge stride and pad");
  CHECK(g_seen.convs == convs, "a rejected call launched");
  // malformed overrides, random and hand-written: rejected or accepted, never
  // read out of bounds
  const char* bad[] = {"tile=", "tile=x", "tile=64x64;kt=32", "split=", "split=0", "split=99", "kt=8", "tail=1",
                       "sk=0", "sk=-5", "persist=0", "persist=17", "=", ",,,", "tile=64x64,split=2,tail=3",
                       "tile=99999999999999999999x1", "bogus=1", "tile=64x64,", "tile=64x64,kt=32,persist=3,"};
  mg3m_plan_info info;
  for (const char* b : bad) {
    const int rc = conv2d_fwd_f32_plan_info(32, 512, 7, 7, 2048, 1, 1, 1, 0, 0, b, &info);
    CHECK(rc == MG3M_OK || rc == MG3M_ERR_PLAN, "override '%s' rc %d", b, rc);
  }
  const char alphabet[] = "tilesprkx=,0123456789-; ";
  for (int i = 0; i < 20000; ++i) {
    std::string s;
    const int n = rint_in(0, 40);
    for (int j = 0; j < n; ++j) s.push_back(alphabet[rnd() % (sizeof alphabet - 1)]);
    const int rc = conv2d_fwd_f32_plan_info(4, 64, 14, 14, 128, 3, 3, 1, 1, rint_in(0, 1), s.c_str(), &info);
    CHECK(rc == MG3M_OK || rc == MG3M_ERR_PLAN, "fuzzed override '%s' rc %d", s.c_str(), rc);
  }
  // pooling validation and the stubbed launch
  CHECK(maxpool2d_f32(fake(0), fake(1), 2, 3, 9, 9, 2, 2, 2, 2, 0, 0, 0, nullptr) == MG3M_OK, "pool");
  CHECK(maxpool2d_f32(fake(0), fake(1), 2, 3, 9, 9, 2, 2, 2, 2, 2, 0, 0, nullptr) == MG3M_ERR_SHAPE, "pool pad");
  // network executor: bad layer lists are rejected before any allocation
  mg3m_layer L[2];
  std::memset(L, 0, sizeof L);
  L[0].op = MG3M_OP_CONV; L[0].input = 0; L[0].add = -1; L[0].K = 8; L[0].R = L[0].S = 3;
  L[0].stride = 1; L[0].pad = 1; L[0].w = fake(4);
  L[1] = L[0];
  L[1].input = 5;                               // reads an activation that does not exist yet
  mg3m_net* net = nullptr;
  CHECK(mg3m_net_create(L, 2, 2, 4, 8, 8, 0, 0, &net) == MG3M_ERR_ARG && net == nullptr, "net input index");
  L[1].input = 1;
  L[1].add = 0;                                 // adds the input, whose shape differs
  CHECK(mg3m_net_create(L, 2, 2, 4, 8, 8, 0, 0, &net) != MG3M_OK && net == nullptr, "net add shape");
  CHECK(mg3m_net_create(nullptr, 2, 2, 4, 8, 8, 0, 0, &net) != MG3M_OK, "net null layers");
  CHECK(mg3m_net_destroy(nullptr) == MG3M_OK, "destroy null");
  // a batch of layout changes: each job's tiles follow the previous job's,
  // and the access widths follow the sizes and the alignments
  {
    mg3m::SwapJob jobs[3] = {};
    jobs[0].in = fake(0); jobs[0].out = fake(1); jobs[0].A = 64; jobs[0].Cm = 64; jobs[0].B = 9;    // 1 x 9 tiles
    jobs[1].in = fake(2) + 1; jobs[1].out = fake(3); jobs[1].A = 130; jobs[1].Cm = 3; jobs[1].B = 1;  // 3 x 1
    jobs[2].in = fake(4); jobs[2].out = fake(5) + 2; jobs[2].A = 8; jobs[2].Cm = 100; jobs[2].B = 49;  // 1 x 77
    unsigned tiles = 0;
    std::string err;
    CHECK(mg3m::prepare_swap_batch(jobs, 3, &tiles, &err) == MG3M_OK, "swap batch: %s", err.c_str());
    CHECK(tiles == 9 + 3 + 77, "swap batch tiles %u", tiles);
    CHECK(jobs[0].tile0 == 0 && jobs[1].tile0 == 9 && jobs[2].tile0 == 12, "swap batch tile0");
    CHECK(jobs[0].tiles_j == 9 && jobs[1].tiles_j == 1 && jobs[2].tiles_j == 77, "swap batch tiles_j");
    CHECK(jobs[0].vl && jobs[0].vs, "swap batch widths 0");
    CHECK(!jobs[1].vl && !jobs[1].vs, "swap batch widths 1");        // J = 3; A = 130
    CHECK(jobs[2].vl && !jobs[2].vs, "swap batch widths 2");        // out not 16-byte aligned
    jobs[1].A = 0;
    CHECK(mg3m::prepare_swap_batch(jobs, 3, &tiles, &err) == MG3M_ERR_SHAPE, "swap batch empty job");
    jobs[1].A = 130;
    jobs[2].Cm = 1 << 20; jobs[2].B = 1 << 12;                      // J = 2^32
    CHECK(mg3m::prepare_swap_batch(jobs, 3, &tiles, &err) == MG3M_ERR_TOO_LARGE, "swap batch J");
  }
  double fo = 0, dov = 0;
  CHECK(mg3m_padding_overhead(30, 44, 16, 4, 16, &fo, &dov) == MG3M_OK, "padding overhead");
  std::printf("errors: validation paths checked\n");
}

// ------------------------------------------------------------ oracle pins
// im2col with zero rows for taps outside the input, then a naive GEMM, both
// in fp64, written independently of the oracle (NCHW logical indexing).
static void im2col_gemm(const std::vector<float>& x, const std::vector<float>& w, std::vector<double>& y, int N,
                        int C, int H, int W, int K, int R, int S, int st, int pd, int Ho, int Wo) {
  const int rows = C * R * S, cols = Ho * Wo;
  std::vector<double> col((size_t)rows * cols);
  y.assign((size_t)N * K * cols, 0.0);
  for (int b = 0; b < N; ++b) {
    for (int c = 0; c < C; ++c)
      for (int r = 0; r < R; ++r)
        for (int s = 0; s < S; ++s)
          for (int oh = 0; oh < Ho; ++oh)
            for (int ow = 0; ow < Wo; ++ow) {
              const int ih = oh * st - pd + r, iw = ow * st - pd + s;
              const bool in = ih >= 0 && ih < H && iw >= 0 && iw < W;
              col[(size_t)((c * R + r) * S + s) * cols + oh * Wo + ow] =
                  in ? (double)x[(((size_t)b * C + c) * H + ih) * W + iw] : 0.0;
            }
    for (int k = 0; k < K; ++k)
      for (int j = 0; j < cols; ++j) {
        double acc = 0.0;
        for (int i = 0; i < rows; ++i) acc += (double)w[(size_t)k * rows + i] * col[(size_t)i * cols + j];
        y[((size_t)b * K + k) * cols + j] = acc;
      }
  }
}

static void check_oracle() {
  int cases = 0;
  for (int it = 0; it < 300; ++it) {
    const int N = rint_in(1, 3), C = rint_in(1, 5), K = rint_in(1, 4), H = rint_in(1, 7), W = rint_in(1, 7);
    const int R = rint_in(1, 5), S = rint_in(1, 5), st = rint_in(1, 3), pd = rint_in(0, 3);
    int Ho = 0, Wo = 0;
    if (oracle_out_dims(H, W, R, S, st, st, pd, pd, &Ho, &Wo) != 0) continue;
    std::vector<float> x((size_t)N * C * H * W), w((size_t)K * C * R * S);
    for (auto& v : x) v = (float)((int)(rnd() % 2001) - 1000) / 1000.0f;
    for (auto& v : w) v = (float)((int)(rnd() % 2001) - 1000) / 1000.0f;
    const size_t n_out = (size_t)N * K * Ho * Wo;
    std::vector<double> acc(n_out), mag(n_out), ref;
    CHECK(oracle_conv2d_f64(x.data(), w.data(), acc.data(), mag.data(), N, C, H, W, K, R, S, st, st, pd, pd, 1) == 0,
          "oracle rc");
    im2col_gemm(x, w, ref, N, C, H, W, K, R, S, st, pd, Ho, Wo);
    for (size_t i = 0; i < n_out; ++i)
      CHECK(std::fabs(acc[i] - ref[i]) <= 1e-12 * (mag[i] + 1e-300) + 0.0, "brute force at %zu: %g vs %g", i,
            acc[i], ref[i]);
    // selected points agree with the full evaluation
    std::vector<int64_t> idx;
    for (size_t i = 0; i < n_out; i += 3) idx.push_back((int64_t)i);
    std::vector<double> pa(idx.size()), pm(idx.size());
    CHECK(oracle_conv2d_points_f64(x.data(), w.data(), idx.data(), (int64_t)idx.size(), pa.data(), pm.data(), N, C,
                                   H, W, K, R, S, st, st, pd, pd, 1) == 0, "points rc");
    for (size_t j = 0; j < idx.size(); ++j) CHECK(pa[j] == acc[idx[j]] && pm[j] == mag[idx[j]], "points %zu", j);
    // out-of-range point indices are rejected
    int64_t badi = (int64_t)n_out;
    double d0, d1;
    CHECK(oracle_conv2d_points_f64(x.data(), w.data(), &badi, 1, &d0, &d1, N, C, H, W, K, R, S, st, st, pd, pd, 1) ==
              -1, "point index past the end");
    // delta filter (C == K, stride 1): a shift of the input by the tap's offset
    if (st == 1 && C == K) {
      const int r0 = rint_in(0, R - 1), s0 = rint_in(0, S - 1);
      std::vector<float> d((size_t)K * C * R * S, 0.0f);
      for (int k = 0; k < K; ++k) d[(((size_t)k * C + k) * R + r0) * S + s0] = 1.0f;
      std::vector<double> a2(n_out), m2(n_out);
      oracle_conv2d_f64(x.data(), d.data(), a2.data(), m2.data(), N, C, H, W, K, R, S, 1, 1, pd, pd, 1);
      for (int b = 0; b < N; ++b)
        for (int k = 0; k < K; ++k)
          for (int oh = 0; oh < Ho; ++oh)
            for (int ow = 0; ow < Wo; ++ow) {
              const int ih = oh + r0 - pd, iw = ow + s0 - pd;
              const double want = (ih >= 0 && ih < H && iw >= 0 && iw < W)
                                      ? (double)x[(((size_t)b * C + k) * H + ih) * W + iw] : 0.0;
              CHECK(a2[(((size_t)b * K + k) * Ho + oh) * Wo + ow] == want, "delta filter");
            }
    }
    ++cases;
  }
  // invalid shapes
  double a, m;
  float v = 0.f;
  CHECK(oracle_conv2d_f64(&v, &v, &a, &m, 1, 1, 1, 1, 1, 3, 3, 1, 1, 0, 0, 0) == -1, "empty output");
  CHECK(oracle_conv2d_f64(&v, &v, &a, &m, 1, 1, 1, 1, 1, 1, 1, 1, 1, 0, 0, 5) == -1, "bad layout");
  std::printf("oracle: %d shapes against im2col + GEMM\n", cases);
}

int main() {
  check_plans();
  check_errors();
  check_oracle();
  if (g_failures) {
    std::fprintf(stderr, "%d checks failed\n", g_failures);
    return 1;
  }
  std::printf("all host checks passed\n");
  return 0;
}
