// Measurement kernels (include/mg3m_measure.h): an empty kernel, an
// fp32-MFMA-only kernel, and 16-byte copy / fill kernels.  They set the
// convolution's numbers against what the chip sustains; none of them is on
// the convolution's path.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>

#include "mg3m.h"
#include "mg3m_internal.h"
#include "mg3m_measure.h"

namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(64) void empty_kernel() {}

// Eight independent accumulator chains per wave keep the MFMA pipe issuing
// back to back (each 32x32x2 fp32 MFMA is 16 passes; a chain's next MFMA
// waits for its previous one).
__global__ __launch_bounds__(256) void mfma_probe(float* sink, int iters) {
  floatx16 acc[8];
#pragma unroll
  for (int c = 0; c < 8; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[c][e] = 0.f;
  const float a = 1e-3f * (float)(threadIdx.x & 63), b = 1e-3f * (float)(blockIdx.x & 63);
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < 8; ++c)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[c][e];
  sink[(size_t)blockIdx.x * 256 + threadIdx.x] = s;
}

// Streaming probes: each work-group covers 16 KB, each thread four 16-byte
// accesses 4 KB apart (every access instruction of a wave is 1 KB
// contiguous), all four issued before any completes; one pass over the
// buffer, no grid-stride loop.
constexpr int kUnroll = 4;
constexpr size_t kBlockVec = 256 * kUnroll;    // 16-byte vectors per work-group

__global__ __launch_bounds__(256) void copy_probe(const f32x4* __restrict__ src, f32x4* __restrict__ dst,
                                                  size_t n4) {
  const size_t base = (size_t)blockIdx.x * kBlockVec + threadIdx.x;
  f32x4 v[kUnroll];
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const size_t i = base + (size_t)u * 256;
    v[u] = i < n4 ? src[i] : f32x4{0.f, 0.f, 0.f, 0.f};
  }
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const size_t i = base + (size_t)u * 256;
    if (i < n4) dst[i] = v[u];
  }
}

__global__ __launch_bounds__(256) void fill_probe(f32x4* __restrict__ dst, size_t n4) {
  const size_t base = (size_t)blockIdx.x * kBlockVec + threadIdx.x;
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const size_t i = base + (size_t)u * 256;
    if (i < n4) dst[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
}

unsigned stream_blocks(size_t n4) { return (unsigned)((n4 + kBlockVec - 1) / kBlockVec); }

int launched(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return mg3m::set_error(MG3M_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
  return MG3M_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

}  // namespace

extern "C" {

int mg3m_launch_empty(void* stream) {
  mg3m::clear_error();
  hipLaunchKernelGGL(empty_kernel, dim3(1), dim3(64), 0, static_cast<hipStream_t>(stream));
  return launched("empty kernel launch");
}

int mg3m_probe_mfma_f32(float* sink, int blocks, int iters, void* stream, double* flops) {
  mg3m::clear_error();
  if (sink == nullptr || flops == nullptr) return mg3m::set_error(MG3M_ERR_NULL, "sink and flops must be non-NULL");
  if (blocks < 1 || blocks > (1 << 20) || iters < 1 || iters > (1 << 24))
    return mg3m::set_error(MG3M_ERR_ARG, "blocks must be 1..2^20 and iters 1..2^24");
  hipLaunchKernelGGL(mfma_probe, dim3((unsigned)blocks), dim3(256), 0, static_cast<hipStream_t>(stream), sink, iters);
  *flops = (double)blocks * 4.0 * (double)iters * 8.0 * 4096.0;
  return launched("MFMA probe launch");
}

int mg3m_probe_copy(const void* src, void* dst, size_t bytes, void* stream) {
  mg3m::clear_error();
  if (src == nullptr || dst == nullptr) return mg3m::set_error(MG3M_ERR_NULL, "src and dst must be non-NULL");
  if (bytes == 0 || bytes % 16 != 0) return mg3m::set_error(MG3M_ERR_ARG, "bytes must be a positive multiple of 16");
  if (!aligned16(src) || !aligned16(dst)) return mg3m::set_error(MG3M_ERR_ALIGN, "src and dst must be 16-byte aligned");
  const uintptr_t s = reinterpret_cast<uintptr_t>(src), d = reinterpret_cast<uintptr_t>(dst);
  if (s < d + bytes && d < s + bytes) return mg3m::set_error(MG3M_ERR_ALIAS, "src and dst overlap");
  if (bytes / 16 > (size_t)kBlockVec * 0x7fffffffULL) return mg3m::set_error(MG3M_ERR_ARG, "bytes too large");
  hipLaunchKernelGGL(copy_probe, dim3(stream_blocks(bytes / 16)), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<const f32x4*>(src), static_cast<f32x4*>(dst), bytes / 16);
  return launched("copy probe launch");
}

int mg3m_probe_fill(void* dst, size_t bytes, void* stream) {
  mg3m::clear_error();
  if (dst == nullptr) return mg3m::set_error(MG3M_ERR_NULL, "dst must be non-NULL");
  if (bytes == 0 || bytes % 16 != 0) return mg3m::set_error(MG3M_ERR_ARG, "bytes must be a positive multiple of 16");
  if (!aligned16(dst)) return mg3m::set_error(MG3M_ERR_ALIGN, "dst must be 16-byte aligned");
  if (bytes / 16 > (size_t)kBlockVec * 0x7fffffffULL) return mg3m::set_error(MG3M_ERR_ARG, "bytes too large");
  hipLaunchKernelGGL(fill_probe, dim3(stream_blocks(bytes / 16)), dim3(256), 0, static_cast<hipStream_t>(stream),
                     static_cast<f32x4*>(dst), bytes / 16);
  return launched("fill probe launch");
}

int mg3m_timing_event_create(void** event) {
  mg3m::clear_error();
  if (event == nullptr) return mg3m::set_error(MG3M_ERR_NULL, "event must be non-NULL");
  hipEvent_t e = nullptr;
  const hipError_t r = hipEventCreateWithFlags(&e, hipEventDisableSystemFence);
  if (r != hipSuccess) return mg3m::set_error(MG3M_ERR_HIP, std::string("hipEventCreateWithFlags: ") + hipGetErrorString(r));
  *event = e;
  return MG3M_OK;
}

int mg3m_timing_event_record(void* event, void* stream) {
  mg3m::clear_error();
  if (event == nullptr) return mg3m::set_error(MG3M_ERR_NULL, "event must be non-NULL");
  const hipError_t r = hipEventRecord(static_cast<hipEvent_t>(event), static_cast<hipStream_t>(stream));
  if (r != hipSuccess) return mg3m::set_error(MG3M_ERR_HIP, std::string("hipEventRecord: ") + hipGetErrorString(r));
  return MG3M_OK;
}

int mg3m_timing_event_elapsed_ms(void* start, void* stop, float* ms) {
  mg3m::clear_error();
  if (start == nullptr || stop == nullptr || ms == nullptr)
    return mg3m::set_error(MG3M_ERR_NULL, "start, stop and ms must be non-NULL");
  const hipError_t r = hipEventElapsedTime(ms, static_cast<hipEvent_t>(start), static_cast<hipEvent_t>(stop));
  if (r != hipSuccess) return mg3m::set_error(MG3M_ERR_HIP, std::string("hipEventElapsedTime: ") + hipGetErrorString(r));
  return MG3M_OK;
}

int mg3m_timing_event_destroy(void* event) {
  mg3m::clear_error();
  if (event == nullptr) return mg3m::set_error(MG3M_ERR_NULL, "event must be non-NULL");
  const hipError_t r = hipEventDestroy(static_cast<hipEvent_t>(event));
  if (r != hipSuccess) return mg3m::set_error(MG3M_ERR_HIP, std::string("hipEventDestroy: ") + hipGetErrorString(r));
  return MG3M_OK;
}

}  // extern "C"
