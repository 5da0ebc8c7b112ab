// Layout change for the network executor: out[b][c][a] = in[a][c][b].  With
// (A, Cm, B) = (N, C, H*W) it takes an NCHW tensor to HWCN; with (H*W, C, N)
// it takes HWCN back to NCHW.  NCHW networks run every layer in HWCN (the
// tuned layout) and change layout only at their input and output, and an
// NCHW call whose plan runs it as HWCN changes x, then y, the same way (with
// the fused output stage applied on the way back).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>

#include "mg3m.h"
#include "mg3m_internal.h"

namespace {

// The input is read as in[a][j] with j = c * B + b (J = Cm * B), and one
// work-group moves a 64 x 64 block of (a, j) through LDS: the reads run along
// j, 256 contiguous bytes per a; the writes run along a, 256 contiguous bytes
// per j at out[b][c][a0 .. a0 + 64).  Flattening (c, b) keeps both sides whole
// when B is small (a filter's R*S taps, a batch of one).  VL (J a multiple of
// 4, in 16-byte aligned): 16-byte loads; VS (A a multiple of 4, out and add
// 16-byte aligned): 16-byte stores.  The extra column keeps the transposed
// reads off one bank.  Tiles run j-fastest over a 1-D grid.
template <bool VL, bool VS>
__device__ __forceinline__ void swap_tile(float (&t)[64][65], const float* __restrict__ in, float* out, int A,
                                          int Cm, int B, const float* add, int relu, unsigned tiles_j,
                                          unsigned block) {
  const unsigned J = (unsigned)Cm * (unsigned)B;
  const unsigned tj = block % tiles_j, ta = block / tiles_j;
  const int a0 = (int)ta * 64;
  const unsigned j0 = tj * 64;
  const int tid = (int)threadIdx.x;
  if constexpr (VL) {
    const int q = tid & 15, r = tid >> 4;           // float4 q of a row, rows r, r + 16, ...
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int a = a0 + r + 16 * i;
      const unsigned j = j0 + 4 * q;
      if (a < A && j < J) {                         // J % 4 == 0: the whole float4 is inside
        const float4 v = *reinterpret_cast<const float4*>(in + (size_t)a * J + j);
        t[r + 16 * i][4 * q] = v.x;
        t[r + 16 * i][4 * q + 1] = v.y;
        t[r + 16 * i][4 * q + 2] = v.z;
        t[r + 16 * i][4 * q + 3] = v.w;
      }
    }
  } else {
    const int tx = tid & 63, ty = tid >> 6;
    for (int i = ty; i < 64; i += 4) {
      const int a = a0 + i;
      const unsigned j = j0 + tx;
      if (a < A && j < J) t[i][tx] = in[(size_t)a * J + j];
    }
  }
  __syncthreads();
  if constexpr (VS) {
    const int q = tid & 15, r = tid >> 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const unsigned j = j0 + r + 16 * i;
      const int a = a0 + 4 * q;
      if (a < A && j < J) {                         // A % 4 == 0: the whole float4 is inside
        const unsigned c = j / (unsigned)B, b = j - c * (unsigned)B;
        const size_t o = ((size_t)b * Cm + c) * A + a;
        const int row = r + 16 * i;
        float4 v = make_float4(t[4 * q][row], t[4 * q + 1][row], t[4 * q + 2][row], t[4 * q + 3][row]);
        if (add != nullptr) {                       // add may be out itself: read before the write
          const float4 d = *reinterpret_cast<const float4*>(add + o);
          v.x += d.x; v.y += d.y; v.z += d.z; v.w += d.w;
        }
        if (relu != 0) {                            // ReLU keeps NaN
          v.x = v.x < 0.f ? 0.f : v.x; v.y = v.y < 0.f ? 0.f : v.y;
          v.z = v.z < 0.f ? 0.f : v.z; v.w = v.w < 0.f ? 0.f : v.w;
        }
        *reinterpret_cast<float4*>(out + o) = v;
      }
    }
  } else {
    const int tx = tid & 63, ty = tid >> 6;
    for (int i = ty; i < 64; i += 4) {
      const unsigned j = j0 + i;
      const int a = a0 + tx;
      if (a < A && j < J) {
        const unsigned c = j / (unsigned)B, b = j - c * (unsigned)B;
        const size_t o = ((size_t)b * Cm + c) * A + a;
        float v = t[tx][i];
        if (add != nullptr) v += add[o];            // add may be out itself: read before the write
        out[o] = (relu != 0 && v < 0.f) ? 0.f : v;  // ReLU keeps NaN
      }
    }
  }
}

template <bool VL, bool VS>
__global__ __launch_bounds__(256) void swap_outer_inner(const float* __restrict__ in, float* out, int A, int Cm,
                                                        int B, const float* add, int relu, unsigned tiles_j) {
  __shared__ float t[64][65];
  swap_tile<VL, VS>(t, in, out, A, Cm, B, add, relu, tiles_j, blockIdx.x);
}

// A batch: work-group i runs tile i - tile0 of the job whose work-groups
// hold i (the last job with tile0 <= i).
__global__ __launch_bounds__(256) void swap_outer_inner_batch(const mg3m::SwapJob* __restrict__ jobs, int n) {
  __shared__ float t[64][65];
  const unsigned blk = blockIdx.x;
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (jobs[mid].tile0 <= blk) lo = mid;
    else hi = mid - 1;
  }
  const mg3m::SwapJob& j = jobs[lo];
  const unsigned local = blk - j.tile0;
  if (j.vl && j.vs) swap_tile<true, true>(t, j.in, j.out, j.A, j.Cm, j.B, nullptr, 0, j.tiles_j, local);
  else if (j.vl) swap_tile<true, false>(t, j.in, j.out, j.A, j.Cm, j.B, nullptr, 0, j.tiles_j, local);
  else if (j.vs) swap_tile<false, true>(t, j.in, j.out, j.A, j.Cm, j.B, nullptr, 0, j.tiles_j, local);
  else swap_tile<false, false>(t, j.in, j.out, j.A, j.Cm, j.B, nullptr, 0, j.tiles_j, local);
}

// Two jobs passed by value (an NCHW call run as HWCN: its x and its filter).
struct SwapPair {
  mg3m::SwapJob j[2];
};
__global__ __launch_bounds__(256) void swap_outer_inner_pair(SwapPair p) {
  __shared__ float t[64][65];
  const int k = blockIdx.x >= p.j[1].tile0 ? 1 : 0;
  const mg3m::SwapJob& j = p.j[k];
  const unsigned local = blockIdx.x - j.tile0;
  if (j.vl && j.vs) swap_tile<true, true>(t, j.in, j.out, j.A, j.Cm, j.B, nullptr, 0, j.tiles_j, local);
  else if (j.vl) swap_tile<true, false>(t, j.in, j.out, j.A, j.Cm, j.B, nullptr, 0, j.tiles_j, local);
  else if (j.vs) swap_tile<false, true>(t, j.in, j.out, j.A, j.Cm, j.B, nullptr, 0, j.tiles_j, local);
  else swap_tile<false, false>(t, j.in, j.out, j.A, j.Cm, j.B, nullptr, 0, j.tiles_j, local);
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

template <bool VL, bool VS>
void launch(unsigned blocks, unsigned tiles_j, const float* in, float* out, int A, int Cm, int B, const float* add,
            int relu, hipStream_t stream) {
  hipLaunchKernelGGL((swap_outer_inner<VL, VS>), dim3(blocks), dim3(256), 0, stream, in, out, A, Cm, B, add, relu,
                     tiles_j);
}

}  // namespace

namespace mg3m {

int launch_swap_outer_inner(const float* in, float* out, int A, int Cm, int B, void* stream, std::string* err,
                            const float* add, int relu) {
  if (A < 1 || Cm < 1 || B < 1) {
    *err = "internal: empty layout change";
    return MG3M_ERR_SHAPE;
  }
  const long long J = (long long)Cm * B;
  const long long tj = (J + 63) / 64, ta = (A + 63) / 64;
  // j and the block index are 32-bit in the kernel; a block count times 256
  // threads stays within the 32-bit launch size
  if (J > 0x7fffffffLL || tj * ta > (1LL << 24) - 1) {
    *err = "layout change: a dimension exceeds the launch grid";
    return MG3M_ERR_TOO_LARGE;
  }
  const bool vl = J % 4 == 0 && aligned16(in);
  const bool vs = A % 4 == 0 && aligned16(out) && (add == nullptr || aligned16(add));
  const unsigned blocks = (unsigned)(tj * ta), tiles_j = (unsigned)tj;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (vl && vs) launch<true, true>(blocks, tiles_j, in, out, A, Cm, B, add, relu, s);
  else if (vl) launch<true, false>(blocks, tiles_j, in, out, A, Cm, B, add, relu, s);
  else if (vs) launch<false, true>(blocks, tiles_j, in, out, A, Cm, B, add, relu, s);
  else launch<false, false>(blocks, tiles_j, in, out, A, Cm, B, add, relu, s);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    *err = std::string("layout change launch: ") + hipGetErrorString(e);
    return MG3M_ERR_HIP;
  }
  return MG3M_OK;
}

int launch_swap_outer_inner_batch(const SwapJob* dev_jobs, int n, unsigned tiles, void* stream, std::string* err) {
  if (n < 1 || tiles < 1) return MG3M_OK;
  hipLaunchKernelGGL(swap_outer_inner_batch, dim3(tiles), dim3(256), 0, static_cast<hipStream_t>(stream), dev_jobs,
                     n);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    *err = std::string("layout change launch: ") + hipGetErrorString(e);
    return MG3M_ERR_HIP;
  }
  return MG3M_OK;
}

int launch_swap_outer_inner_pair(const SwapJob jobs[2], unsigned tiles, void* stream, std::string* err) {
  SwapPair p;
  p.j[0] = jobs[0];
  p.j[1] = jobs[1];
  hipLaunchKernelGGL(swap_outer_inner_pair, dim3(tiles), dim3(256), 0, static_cast<hipStream_t>(stream), p);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    *err = std::string("layout change launch: ") + hipGetErrorString(e);
    return MG3M_ERR_HIP;
  }
  return MG3M_OK;
}

}  // namespace mg3m
