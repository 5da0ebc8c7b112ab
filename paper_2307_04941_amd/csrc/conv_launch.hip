// Kernel launch: picks the instantiation for a plan's loader variant and
// tile, and the deterministic split-K reduction.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdlib>
#include <string>

#include "mg3m.h"
#include "mg3m_internal.h"

namespace mg3m {

typedef float f32x4r __attribute__((ext_vector_type(4)));
typedef double f64x2r __attribute__((ext_vector_type(2)));

// Stream-K plans: the run (see the kernel's tail_run) holding reduction
// step x of the tail; the first sk_r runs are sk_q + 1 steps long, the rest
// sk_q.
__device__ __forceinline__ int run_of_step(const RArgs& r, int x) {
  const int long_steps = r.sk_r * (r.sk_q + 1);
  return x < long_steps ? x / (r.sk_q + 1) : r.sk_r + (x - long_steps) / r.sk_q;
}

// Tail reduction: for every element of every tail tile, y = the sum of the
// tile's piece partials in run order (the runs covering the tile's steps,
// first to last), so the result does not depend on scheduling.  F64: the
// partials are fp64 (from the fp64-accumulating kernel), summed in fp64 and
// rounded to fp32 once.  One thread per four consecutive columns of one tile
// row; rows and columns past the output are skipped.
template <bool F64>
__global__ __launch_bounds__(256) void tail_reduce(RArgs r) {
  const long long tile_elems = (long long)r.mt * r.nt;
  const long long per_tile4 = tile_elems / 4;
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= per_tile4 * r.tail_tiles) return;
  const int t = (int)(i / per_tile4);
  const int e = (int)(i - (long long)t * per_tile4) * 4;
  const int row = e / r.nt, col = e - row * r.nt;
  // runs covering the tile: split plans give tile t the runs t*sk_s ... t*sk_s + sk_s - 1
  const int w0 = r.sk_s > 0 ? t * r.sk_s : run_of_step(r, t * r.k_tiles);
  const int w1 = r.sk_s > 0 ? w0 + r.sk_s - 1 : run_of_step(r, (t + 1) * r.k_tiles - 1);
  // the piece of run w in tail tile t sits in slot w + t.  Pieces are loaded
  // up to four at a time, all of them in flight before the first add, so a
  // thread waits out the memory latency once per four pieces, not once per
  // piece; the adds stay in run order.
  const long long off = ((long long)w0 + t) * tile_elems + e;
  f32x4r sum;
  if constexpr (F64) {
    const double* p = static_cast<const double*>(r.ws) + off;
    auto ld = [&](long long i) { return *reinterpret_cast<const f64x2r*>(p + i); };
    f64x2r lo = ld(0), hi = ld(2);
    for (int w = w0 + 1; w <= w1; w += 4, p += 4 * tile_elems) {
      const int n = min(4, w1 - w + 1);
      f64x2r l[4], h[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (u < n) {
          l[u] = ld((u + 1) * tile_elems);
          h[u] = ld((u + 1) * tile_elems + 2);
        }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (u < n) {
          lo += l[u];
          hi += h[u];
        }
    }
    sum = f32x4r{(float)lo[0], (float)lo[1], (float)hi[0], (float)hi[1]};
  } else {
    const float* p = static_cast<const float*>(r.ws) + off;
    auto ld = [&](long long i) { return *reinterpret_cast<const f32x4r*>(p + i); };
    sum = ld(0);
    for (int w = w0 + 1; w <= w1; w += 4, p += 4 * tile_elems) {
      const int n = min(4, w1 - w + 1);
      f32x4r v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (u < n) v[u] = ld((u + 1) * tile_elems);
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (u < n) sum += v[u];
    }
  }
  const int tile = r.dp_tiles + t;
  const int tm = tile % r.tiles_m, tn = tile / r.tiles_m;
  const int m = tm * r.mt + row;
  if (m >= r.Mg) return;
  const int n0 = tn * r.nt + col;
  auto index = [&](int n) -> long long {
    if (r.layout == kHWCN) {                 // y[Ho][Wo][K][N], n = pix*N + b
      const int pix = n / r.N, b = n - pix * r.N;
      return ((long long)pix * r.K + m) * r.N + b;
    }
    const int b = n / r.HoWo, pix = n - b * r.HoWo;   // y[N][K][Ho][Wo]
    return ((long long)b * r.K + m) * r.HoWo + pix;
  };
  auto finish = [&](float v, long long idx) {
    if (r.add != nullptr) v += r.add[idx];
    return (r.relu != 0 && v < 0.f) ? 0.f : v;
  };
  if (r.vec4 && n0 + 3 < r.Ng) {
    const long long i0 = index(n0);
    if ((r.add != nullptr) | (r.relu != 0)) {
#pragma unroll
      for (int q = 0; q < 4; ++q) sum[q] = finish(sum[q], i0 + q);
    }
    *reinterpret_cast<f32x4r*>(r.y + i0) = sum;
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (n0 + q < r.Ng) {
        const long long idx = index(n0 + q);
        r.y[idx] = finish(sum[q], idx);
      }
  }
}

static KernelFn kernel_for(int variant, int tile) {
  switch (variant) {
    case kVarHwcnVecN: return conv_kernel_hwcn_vecn(tile);
    case kVarHwcnVecNTap: return conv_kernel_hwcn_vecn_tap(tile);
    case kVarHwcnVecNTapDma: return conv_kernel_hwcn_vecn_tap_dma(tile);
    case kVarHwcnVecC: return conv_kernel_hwcn_vecc(tile);
    case kVarHwcnVecA: return conv_kernel_hwcn_veca(tile);
    case kVarHwcnScalar: return conv_kernel_hwcn_scalar(tile);
    case kVarNchwVecA:
    case kVarNchwScalar: return conv_kernel_nchw(variant, tile);
    case kVarNchwTap: return conv_kernel_nchw_tap(tile);
    default: return nullptr;
  }
}

static KernelFn kernel_fused_for(int variant, int tile) {
  switch (variant) {
    case kVarHwcnVecNTap: return conv_kernel_hwcn_vecn_tap_fused(tile);
    case kVarHwcnVecNTapDma: return conv_kernel_hwcn_vecn_tap_dma_fused(tile);
    case kVarHwcnVecN: return conv_kernel_hwcn_vecn_fused(tile);
    case kVarHwcnVecC:
    case kVarHwcnVecA:
    case kVarHwcnScalar: return conv_kernel_hwcn_other_fused(variant, tile);
    case kVarNchwVecA:
    case kVarNchwScalar: return conv_kernel_nchw_fused(variant, tile);
    case kVarNchwTap: return conv_kernel_nchw_tap_fused(tile);
    default: return nullptr;
  }
}

static KernelFn kernel64_for(int variant, int tile) {
  switch (variant) {
    case kVarHwcnVecNTap: return conv_kernel64_hwcn_vecn_tap(tile);
    case kVarHwcnVecN:
    case kVarHwcnVecC:
    case kVarHwcnVecA:
    case kVarHwcnScalar: return conv_kernel64_hwcn(variant, tile);
    case kVarNchwVecA:
    case kVarNchwScalar:
    case kVarNchwTap: return conv_kernel64_nchw(variant, tile);
    default: return nullptr;
  }
}

// Test hook: MG3M_TEST_FAIL_LAUNCH=1 makes every convolution launch fail as a
// rejected launch would (nothing is launched), so callers' error paths --
// the status, the message, the release of a stream-ordered workspace -- can
// be exercised without a faulty kernel.
static bool launch_failure_injected() {
  const char* v = std::getenv("MG3M_TEST_FAIL_LAUNCH");
  return v != nullptr && v[0] == '1' && v[1] == 0;
}

// One launch: dp_tiles work-groups of whole tiles, then tail_wgs of tail runs.
int launch_conv(const Plan& p, const KArgs& a, void* stream, std::string* err, void* start, void* stop) {
  if (launch_failure_injected()) {
    *err = "kernel launch: failure injected by MG3M_TEST_FAIL_LAUNCH";
    return MG3M_ERR_HIP;
  }
  const bool fused = (a.add != nullptr) | (a.relu != 0);
  if (p.acc64 && fused) {
    *err = "internal: the fp64-accumulating kernel has no fused output stage";
    return MG3M_ERR_PLAN;
  }
  // stream-K runs need the kernel's loop over pieces; other kernels take one
  // piece per work-group
  if (p.tail_wgs > 0 && p.sk_s == 0 && (p.acc64 || !tail_runs_multi(p.b_mode))) {
    *err = "internal: stream-K tail plan for a kernel without multi-piece runs";
    return MG3M_ERR_PLAN;
  }
  if (p.persist && (p.acc64 || p.tail_wgs != 0 || p.grid > p.dp_tiles)) {
    *err = "internal: persistent plans take whole tiles of the fp32 kernel only";
    return MG3M_ERR_PLAN;
  }
  if (p.dp_tiles < 0 || p.tail_wgs < 0 || (!p.persist && p.grid != (long long)p.dp_tiles + p.tail_wgs) ||
      p.grid < 1 || p.grid > 0x7fffffffLL || (p.tail_wgs > 0 && (a.ws == nullptr || p.sk_q < 1))) {
    *err = "internal: grid out of range or inconsistent";
    return MG3M_ERR_PLAN;
  }
  KernelFn fn = p.persist ? (fused ? conv_kernel_pt_fused(p.variant, p.tile) : conv_kernel_pt(p.variant, p.tile))
                : p.acc64 ? kernel64_for(p.variant, p.tile)
                          : (fused ? kernel_fused_for(p.variant, p.tile) : kernel_for(p.variant, p.tile));
  if (fn == nullptr) {
    *err = "internal: no kernel for this loader variant and tile";
    return MG3M_ERR_PLAN;
  }
  hipError_t e = hipSuccess;
  if (start != nullptr || stop != nullptr) {
    // the events take the kernel's own start and end times from its dispatch
    // (no separate event packets around it on the stream)
    KArgs ka = a;
    void* args[] = {&ka};
    e = hipExtLaunchKernel(reinterpret_cast<const void*>(fn), dim3((unsigned)p.grid), dim3(p.t.wm * p.t.wn * 64),
                           args, 0, static_cast<hipStream_t>(stream), static_cast<hipEvent_t>(start),
                           static_cast<hipEvent_t>(stop), 0);
    if (e == hipSuccess) e = hipGetLastError();
  } else {
    hipLaunchKernelGGL(fn, dim3((unsigned)p.grid), dim3(p.t.wm * p.t.wn * 64), 0, (hipStream_t)stream, a);
    e = hipGetLastError();
  }
  if (e != hipSuccess) {
    *err = std::string("kernel launch: ") + hipGetErrorString(e);
    return MG3M_ERR_HIP;
  }
  return MG3M_OK;
}

// wt[((r*S + s)*C + c)*K + k] = w[((k*C + c)*R + r)*S + s] is the layout
// change out[b][c][a] = in[a][c][b] with (A, Cm, B) = (K, C, R*S): its tiles
// read each filter row's C*R*S floats in order and write each (tap, c)'s K
// contiguous floats.
int launch_filter_to_rsck(const float* w, float* wt, int K, int C, int R, int S, void* stream,
                          std::string* err) {
  return launch_swap_outer_inner(w, wt, K, C, R * S, stream, err);
}

int launch_tail_reduce(const RArgs& r, void* stream, std::string* err) {
  const long long threads = (long long)r.mt * r.nt / 4 * r.tail_tiles;
  const long long blocks = (threads + 255) / 256;
  if (r.mt % 4 || r.nt % 4 || blocks < 1 || blocks > 0x7fffffffLL) {
    *err = "internal: tail reduction shape out of range";
    return MG3M_ERR_PLAN;
  }
  if (r.f64)
    hipLaunchKernelGGL(tail_reduce<true>, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, r);
  else
    hipLaunchKernelGGL(tail_reduce<false>, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, r);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    *err = std::string("tail reduction launch: ") + hipGetErrorString(e);
    return MG3M_ERR_HIP;
  }
  return MG3M_OK;
}

}  // namespace mg3m
