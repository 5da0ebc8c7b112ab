// Implicit-GEMM forward convolution for gfx950 (MI355X): the device templates
// -- conv_igemm_f32 on fp32 MFMA (plain, or with the fused output stage
// y = act(conv + add)) and conv_igemm_acc64 on fp64 MFMA (the paper's fp64
// arithmetic on fp32 data).  Included by the instantiation files
// (conv_hwcn_*.hip, conv_nchw*.hip, conv_acc64_*.hip); not part of the
// public interface.
//
// The convolution of Eq. 1 (Sec. 2.1) is computed as the matrix product of
// Eq. 2 / Alg. 1 (Sec. 4.1.1), without materialising the patch matrix:
//
//   OUT[m][n] = sum_k A[m][k] * B[k][n]
//   m = output channel                  (Mg = OC)
//   n = (output pixel, image)           (Ng = B*outH*outW)
//   k = (filter tap, input channel)     (Kg = IC*fltH*fltW)
//
// In the paper's HWCN storage (Sec. 4.1.1) the filter is already the dense
// Kg x OC matrix A^T (each FLT_mtx of Alg. 1 is one IC x OC slab of it, k
// ordered (fh, fw, ic)), and column n of B at row k is one element of the
// IN_mtx at pixel (ih, iw), so a k-slab of B is a gather of contiguous IN_mtx
// rows.  In NCHW the reduction runs in (ic, fh, fw) order, or tap-major like
// HWCN on a [R][S][C][K] copy of the filter when C is a multiple of kt.
//
// How the paper's design maps onto CDNA4:
//  * Multi-grained mapping (Sec. 4.1.2): the work-group tile (mt x nt) and the
//    split of the reduction are chosen per shape by the host planner; small
//    tiles play the role of TB(1,1), tiles whose waves share one operand that
//    of TB(1,8), 2-D wave grids that of TB(8,8).
//  * On-chip sharing (Sec. 4.2, Eq. 4/5): the waves of a work-group share the
//    staged A and B tiles through LDS instead of register broadcasts.
//  * Filter reuse (Alg. 2): one staged A tile serves all nt columns.
//  * Double buffering (Alg. 3): two LDS stages; the next tile's global loads
//    are in flight while the MFMAs consume the current stage.  Staged rows
//    are XOR-swizzled rather than padded, so each lane reads its fragments
//    without bank conflicts from one base address.
//  * Register blocking (Sec. 4.4.1, Eq. 9): each wave holds a (mt/wm) x
//    (nt/wn) accumulator block as 32x32 MFMA blocks in AccVGPRs; each lane
//    reads one A and one B value from LDS per 4096-flop MFMA.
//  * Remainders (Sec. 4.4.2): instead of sixteen remainder kernels, edge
//    tiles and padding taps are zero-filled by the buffer hardware (an
//    out-of-range offset reads as 0) and stores are masked.
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>
#include <utility>

#include "mg3m_internal.h"

namespace mg3m {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Byte offset that is past the end of every buffer the kernels read (tensors
// are limited to kMaxTensorBytes): a raw buffer load there returns zero.
constexpr unsigned kOOB = 0xFFFFFFC0u;

typedef double f64x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const float* p, unsigned bytes) {
  // stride 0 (raw buffer), num_records = bytes, 32-bit data format.
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(p), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ f32x4 bload4(__amdgpu_buffer_rsrc_t r, unsigned off) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
__device__ __forceinline__ float bload1(__amdgpu_buffer_rsrc_t r, unsigned off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
__device__ __forceinline__ void st4(float* p, f32x4 v) { *reinterpret_cast<f32x4*>(p) = v; }
// Buffer store at byte offset voff + soff: one per-lane offset register
// serves a whole tile of stores, the constant part riding in soff.
__device__ __forceinline__ void bstore1(__amdgpu_buffer_rsrc_t r, unsigned voff, unsigned soff, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), r, voff, soff, 0);
}

// Placement of one staged operand tile (rows of DIM floats) in LDS: the row
// stride, and the column swizzle that keeps the rows one fragment read
// touches on disjoint banks (see lds_row_stride).  The swizzle permutes
// 16-float groups inside each 64-float block, so 16-byte stores stay whole,
// and it depends on the row only through row % 2 (fp32) or row % 4 (fp64).
template <int DIM, bool ACC64>
struct LdsLayout {
  static constexpr int kStride = ACC64 ? lds_row_stride64(DIM) : lds_row_stride(DIM);
  static constexpr bool kSwz = DIM % 64 == 0;
  __device__ static constexpr int col(int row, int c) {
    if constexpr (!kSwz) return c;
    else if constexpr (ACC64) return c ^ ((row & 3) << 4);
    else return c ^ ((row & 1) << 5);
  }
};

// Tile geometry.  ACC64 selects the fp64-accumulating kernel's LDS layout.
template <int MT, int NT, int KT, int WM, int WN, bool ACC64 = false>
struct Cfg {
  static constexpr int T = WM * WN * 64;        // threads per work-group
  static constexpr int WTM = MT / WM;           // wave tile rows
  static constexpr int WTN = NT / WN;           // wave tile columns
  static constexpr int TM = WTM / 32;           // 32x32 MFMA blocks per wave, rows
  static constexpr int TN = WTN / 32;           // ... columns
  static constexpr int TM16 = WTM / 16;         // 16x16 MFMA blocks per wave (fp64), rows
  static constexpr int TN16 = WTN / 16;         // ... columns
  using LA = LdsLayout<MT, ACC64>;
  using LB = LdsLayout<NT, ACC64>;
  static constexpr int AS = LA::kStride;
  static constexpr int BS = LB::kStride;
  static constexpr int A_STAGE = KT * AS;
  static constexpr int B_STAGE = KT * BS;
  static constexpr int LDS_FLOATS = 2 * A_STAGE + 2 * B_STAGE;
  static constexpr int A_ELEMS = KT * MT / T;    // A elements each thread loads per stage
  static constexpr int B_ELEMS = KT * NT / T;
  static_assert(ACC64 || (WTM % 32 == 0 && WTN % 32 == 0), "wave tile must be whole 32x32 blocks");
  static_assert(!ACC64 || (WTM % 16 == 0 && WTN % 16 == 0), "wave tile must be whole 16x16 blocks");
  static_assert(KT % 4 == 0, "MFMA steps consume 2 (fp32) or 4 (fp64) reduction rows");
  static_assert(LDS_FLOATS * 4 == (ACC64 ? lds_bytes_for64(TileDesc{MT, NT, KT, WM, WN, 0, 0.0})
                                         : lds_bytes_for(TileDesc{MT, NT, KT, WM, WN, 0, 0.0})),
                "LDS size model");
};

// Reduction index k -> (filter row r, filter column s, input channel c).
template <int LAYOUT>
__device__ __forceinline__ void split_k(const KArgs& a, int k, int& r, int& s, int& c) {
  if constexpr (LAYOUT == kHWCN) {           // k = (r*S + s)*C + c
    c = k % a.C; int rs = k / a.C; s = rs % a.S; r = rs / a.S;
  } else {                                   // k = (c*R + r)*S + s
    s = k % a.S; int cr = k / a.S; r = cr % a.R; c = cr / a.R;
  }
}

// Move (r, s, c) forward by one step of qs*C + rc reduction rows (rc < C),
// HWCN order (c fastest): in closed form, where a loop of one carry per C
// rows took up to KT/C passes per row and stage (18-20% of the time of the
// three-channel stems).
struct RscStep {
  int qs, rc;
  __device__ void init(const KArgs& a, int step) {
    qs = step / a.C;
    rc = step - qs * a.C;
  }
};
__device__ __forceinline__ void step_rsc(const KArgs& a, const RscStep& st, int& r, int& s, int& c) {
  c += st.rc;
  s += st.qs;
  if (c >= a.C) {
    c -= a.C;
    ++s;
  }
  while (s >= a.S) {
    s -= a.S;
    ++r;
  }
}

// ------------------------------------------------------------ A (filter)
// HWCN filter w[R][S][C][K] is A^T[k][m] (OC contiguous): each thread owns a
// 4-wide OC vector and NV rows of the KT x MT tile.  Element offsets advance
// by KT*K per stage.
template <class C, int MT, int KT>
struct AVecM {
  static constexpr int MC4 = MT / 4;
  static constexpr int RSTEP = C::T / MC4;
  static constexpr int NV = KT / RSTEP;
  static_assert(C::T % MC4 == 0 && KT % RSTEP == 0 && NV * 4 == C::A_ELEMS, "A vec-M split");
  int m4, kr0, k0, off0;
  bool m_ok;
  f32x4 v[NV];

  __device__ void init(const KArgs& a, int t, int m0, int kbeg) {
    m4 = t % MC4;
    kr0 = t / MC4;
    const int m = m0 + m4 * 4;
    m_ok = m < a.Mg;
    k0 = kbeg + kr0;
    off0 = k0 * a.K + m;
  }
  __device__ void advance(const KArgs& a) {
    k0 += KT;
    off0 += KT * a.K;
  }
  __device__ void load(const KArgs& a, __amdgpu_buffer_rsrc_t wr) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const bool ok = m_ok & (k0 + i * RSTEP < a.Kg);
      const unsigned off = (unsigned)(off0 + i * RSTEP * a.K) * 4u;
      v[i] = bload4(wr, ok ? off : kOOB);
    }
  }
  __device__ void store(float* As) const {
    static_assert(RSTEP % 4 == 0, "a thread's rows share their swizzle");
    const int col = C::LA::col(kr0, m4 * 4);
#pragma unroll
    for (int i = 0; i < NV; ++i) st4(As + (kr0 + i * RSTEP) * C::AS + col, v[i]);
  }
};

// HWCN filter for the one-tap-per-slab path: rows of a stage are channels
// c0..c0+KT-1 of tap (r, s), in the same stage order as the patch loader.
template <class C, int MT, int KT>
struct AVecMTap {
  static constexpr int MC4 = MT / 4;
  static constexpr int RSTEP = C::T / MC4;
  static constexpr int NV = KT / RSTEP;
  static_assert(C::T % MC4 == 0 && KT % RSTEP == 0 && NV * 4 == C::A_ELEMS, "A vec-M split");
  int m4, kr0, base;
  bool m_ok;
  int r, s, c0;
  f32x4 v[NV];

  __device__ void init(const KArgs& a, int t, int m0, int kbeg) {
    m4 = t % MC4;
    kr0 = t / MC4;
    const int m = m0 + m4 * 4;
    m_ok = m < a.Mg;
    base = kr0 * a.K + m;
    const int t0 = kbeg / KT, rs = a.R * a.S;
    const int slab = t0 / rs, tap = t0 - slab * rs;
    c0 = slab * KT;
    r = tap / a.S;
    s = tap - r * a.S;
  }
  __device__ void advance(const KArgs& a) {
    if (++s == a.S) {
      s = 0;
      if (++r == a.R) { r = 0; c0 += KT; }
    }
  }
  __device__ void load(const KArgs& a, __amdgpu_buffer_rsrc_t wr) {
    const int o = base + ((r * a.S + s) * a.C + c0) * a.K;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const unsigned off = (unsigned)(o + i * RSTEP * a.K) * 4u;
      v[i] = bload4(wr, m_ok ? off : kOOB);
    }
  }
  __device__ void store(float* As) const {
    static_assert(RSTEP % 4 == 0, "a thread's rows share their swizzle");
    const int col = C::LA::col(kr0, m4 * 4);
#pragma unroll
    for (int i = 0; i < NV; ++i) st4(As + (kr0 + i * RSTEP) * C::AS + col, v[i]);
  }
};

// NCHW filter w[K][C][R][S] is A[m][k] (Kg contiguous): 4-wide k vectors,
// transposed into the k-major LDS tile.
template <class C, int MT, int KT>
struct AVecK {
  static constexpr int KV = KT / 4;
  static constexpr int MSTEP = C::T / KV;
  static constexpr int NV = MT / MSTEP;
  static_assert(C::T % KV == 0 && MT % MSTEP == 0 && NV * 4 == C::A_ELEMS, "A vec-K split");
  int k4, mr0, k, m_base;
  f32x4 v[NV];

  __device__ void init(const KArgs&, int t, int m0, int kbeg) {
    k4 = t % KV;
    mr0 = t / KV;
    k = kbeg + 4 * k4;
    m_base = m0;
  }
  __device__ void advance(const KArgs&) { k += KT; }
  __device__ void load(const KArgs& a, __amdgpu_buffer_rsrc_t wr) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int m = m_base + mr0 + i * MSTEP;
      const bool ok = (m < a.Mg) & (k < a.Kg);
      const unsigned off = (unsigned)(m * a.Kg + k) * 4u;
      v[i] = bload4(wr, ok ? off : kOOB);
    }
  }
  __device__ void store(float* As) const {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int mm = mr0 + i * MSTEP;
#pragma unroll
      for (int e = 0; e < 4; ++e) As[(4 * k4 + e) * C::AS + C::LA::col(4 * k4 + e, mm)] = v[i][e];
    }
  }
};

// Any layout, any alignment: single elements, coalesced along the
// contiguous axis of the filter (m for HWCN, k for NCHW).
template <int LAYOUT, class C, int MT, int KT>
struct AScalar {
  static constexpr int NE = C::A_ELEMS;
  int t_, m0_, kbase;
  float v[NE];

  __device__ void init(const KArgs&, int t, int m0, int kbeg) { t_ = t; m0_ = m0; kbase = kbeg; }
  __device__ void advance(const KArgs&) { kbase += KT; }
  __device__ static void coords(int e, int& m, int& kr) {
    if constexpr (LAYOUT == kHWCN) { m = e % MT; kr = e / MT; }
    else { kr = e % KT; m = e / KT; }
  }
  __device__ void load(const KArgs& a, __amdgpu_buffer_rsrc_t wr) {
#pragma unroll
    for (int i = 0; i < NE; ++i) {
      int m, kr;
      coords(t_ + i * C::T, m, kr);
      const int mg = m0_ + m, k = kbase + kr;
      const bool ok = (mg < a.Mg) & (k < a.Kg);
      const int idx = (LAYOUT == kHWCN) ? k * a.K + mg : mg * a.Kg + k;
      v[i] = bload1(wr, ok ? (unsigned)idx * 4u : kOOB);
    }
  }
  __device__ void store(float* As) const {
#pragma unroll
    for (int i = 0; i < NE; ++i) {
      int m, kr;
      coords(t_ + i * C::T, m, kr);
      As[kr * C::AS + C::LA::col(kr, m)] = v[i];
    }
  }
};

// ------------------------------------------------------ B (input patches)
// HWCN, N % 4 == 0, C % KT == 0: a KT-row slab of the reduction then lies
// inside one filter tap (r, s) -- the per-pixel IN_mtx of Alg. 1 -- so the tap
// is the same for the whole work-group and kept in scalar registers; each
// thread tests its column against the padding once per stage and its NV rows
// are consecutive channel offsets of one input pixel.  Stages run the taps
// inside each channel slab (Alg. 1's fh, fw loops inside the IC blocks), so
// a neighbouring output pixel's shifted reuse of an input pixel comes one
// stage later and still hits in L2.
template <class C, int NT, int KT>
struct BVecNTap {
  static constexpr int NC4 = NT / 4;
  static constexpr int RSTEP = C::T / NC4;
  static constexpr int NV = KT / RSTEP;
  static_assert(C::T % NC4 == 0 && KT % RSTEP == 0 && NV * 4 == C::B_ELEMS, "B vec-N split");
  int n4, kr0, ih0, iw0, base;
  bool col_ok;
  int r, s, c0;            // uniform: tap and first channel of the slab
  f32x4 v[NV];

  __device__ void init(const KArgs& a, int t, int n0, int kbeg) {
    n4 = t % NC4;
    kr0 = t / NC4;
    const int n = n0 + n4 * 4;
    col_ok = n < a.Ng;
    const int pix = n / a.N;
    const int b = n - pix * a.N;
    const int ho = pix / a.Wo, wo = pix - ho * a.Wo;
    ih0 = ho * a.sh - a.ph;
    iw0 = wo * a.sw - a.pw;
    // element offset of (ih0, iw0, channel kr0, image b); only used when the
    // tap lands inside the input
    base = ((ih0 * a.W + iw0) * a.C + kr0) * a.N + b;
    // stage t covers channels c0..c0+KT-1 of tap (r, s); stages run taps
    // inner, channel slabs outer: t = (c0 / KT) * R*S + r*S + s
    const int t0 = kbeg / KT, rs = a.R * a.S;
    const int slab = t0 / rs, tap = t0 - slab * rs;
    c0 = slab * KT;
    r = tap / a.S;
    s = tap - r * a.S;
  }
  __device__ void advance(const KArgs& a) {
    if (++s == a.S) {
      s = 0;
      if (++r == a.R) { r = 0; c0 += KT; }
    }
  }
  __device__ void load(const KArgs& a, __amdgpu_buffer_rsrc_t xr) {
    const bool ok = col_ok & ((unsigned)(ih0 + r) < (unsigned)a.H) &
                    ((unsigned)(iw0 + s) < (unsigned)a.W);
    const int o = base + ((r * a.W + s) * a.C + c0) * a.N;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const unsigned off = (unsigned)(o + i * RSTEP * a.N) * 4u;
      v[i] = bload4(xr, ok ? off : kOOB);
    }
  }
  __device__ void store(float* Bs) const {
    static_assert(RSTEP % 4 == 0, "a thread's rows share their swizzle");
    const int col = C::LB::col(kr0, n4 * 4);
#pragma unroll
    for (int i = 0; i < NV; ++i) st4(Bs + (kr0 + i * RSTEP) * C::BS + col, v[i]);
  }
};

// ------------------------------------- direct global->LDS loaders (one tap)
// The one-tap HWCN loaders in a form that loads straight into LDS
// (buffer_load_dwordx4 ... lds): a wave's 16-byte load puts lane l's data at
// the wave's LDS address + 16*l, so thread t's slot in a stage is float
// 4*t, its row and physical column follow from t as in the register-staged
// loaders, and the thread loads the logical column that the XOR swizzle
// places in that slot (the swizzle is its own inverse).  No VGPRs hold the
// staged data and no LDS stores are issued; the loaded rows are visible to
// the work-group after the loads complete and a barrier.
typedef __attribute__((address_space(3))) void* lds_addr_t;

__device__ __forceinline__ void bload_lds16(__amdgpu_buffer_rsrc_t r, float* lds, unsigned off) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_addr_t)lds, 16, off, 0, 0, 0);
}

template <class C, int MT, int KT>
struct AVecMTapDma {
  static constexpr int MC4 = MT / 4;
  static constexpr int RSTEP = C::T / MC4;
  static constexpr int NV = KT / RSTEP;
  static_assert(C::T % MC4 == 0 && KT % RSTEP == 0 && NV * 4 == C::A_ELEMS, "A vec-M split");
  static_assert(C::AS == MT, "unpadded rows: thread t's slot is float 4*t");
  static_assert(RSTEP % 2 == 0, "a thread's rows share their swizzle");
  int base, wslot;          // element offset at tap (0, 0) and channel 0; the wave's first slot
  bool m_ok;
  int r, s, c0;

  __device__ void init(const KArgs& a, int t, int m0, int kbeg) {
    const int kr0 = t / MC4;
    const int col = C::LA::col(kr0, (t % MC4) * 4);   // logical column of the thread's slot
    const int m = m0 + col;
    m_ok = m < a.Mg;
    base = kr0 * a.K + m;
    wslot = __builtin_amdgcn_readfirstlane((t >> 6) * 256);
    const int t0 = kbeg / KT, rs = a.R * a.S;
    const int slab = t0 / rs, tap = t0 - slab * rs;
    c0 = slab * KT;
    r = tap / a.S;
    s = tap - r * a.S;
  }
  __device__ void advance(const KArgs& a) {
    if (++s == a.S) {
      s = 0;
      if (++r == a.R) { r = 0; c0 += KT; }
    }
  }
  __device__ void load(const KArgs& a, __amdgpu_buffer_rsrc_t wr, float* As) {
    const int o = base + ((r * a.S + s) * a.C + c0) * a.K;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const unsigned off = (unsigned)(o + i * RSTEP * a.K) * 4u;
      bload_lds16(wr, As + wslot + i * RSTEP * MT, m_ok ? off : kOOB);
    }
  }
};

template <class C, int NT, int KT>
struct BVecNTapDma {
  static constexpr int NC4 = NT / 4;
  static constexpr int RSTEP = C::T / NC4;
  static constexpr int NV = KT / RSTEP;
  static_assert(C::T % NC4 == 0 && KT % RSTEP == 0 && NV * 4 == C::B_ELEMS, "B vec-N split");
  static_assert(C::BS == NT, "unpadded rows: thread t's slot is float 4*t");
  static_assert(RSTEP % 2 == 0, "a thread's rows share their swizzle");
  int ih0, iw0, base, wslot;
  bool col_ok;
  int r, s, c0;

  __device__ void init(const KArgs& a, int t, int n0, int kbeg) {
    const int kr0 = t / NC4;
    const int n = n0 + C::LB::col(kr0, (t % NC4) * 4);   // first of the four logical columns
    col_ok = n < a.Ng;
    const int pix = n / a.N;
    const int b = n - pix * a.N;
    const int ho = pix / a.Wo, wo = pix - ho * a.Wo;
    ih0 = ho * a.sh - a.ph;
    iw0 = wo * a.sw - a.pw;
    base = ((ih0 * a.W + iw0) * a.C + kr0) * a.N + b;
    wslot = __builtin_amdgcn_readfirstlane((t >> 6) * 256);
    const int t0 = kbeg / KT, rs = a.R * a.S;
    const int slab = t0 / rs, tap = t0 - slab * rs;
    c0 = slab * KT;
    r = tap / a.S;
    s = tap - r * a.S;
  }
  __device__ void advance(const KArgs& a) {
    if (++s == a.S) {
      s = 0;
      if (++r == a.R) { r = 0; c0 += KT; }
    }
  }
  __device__ void load(const KArgs& a, __amdgpu_buffer_rsrc_t xr, float* Bs) {
    const bool ok = col_ok & ((unsigned)(ih0 + r) < (unsigned)a.H) & ((unsigned)(iw0 + s) < (unsigned)a.W);
    const int o = base + ((r * a.W + s) * a.C + c0) * a.N;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const unsigned off = (unsigned)(o + i * RSTEP * a.N) * 4u;
      bload_lds16(xr, Bs + wslot + i * RSTEP * NT, ok ? off : kOOB);
    }
  }
};

// Debug build (-DMG3M_LDS_POISON=1, `build --lds-poison`): at the start of
// every stage the LDS buffer that the previous stage consumed is filled with
// NaN, behind a barrier, before it is staged again.  A read that some missing
// barrier lets through then returns NaN (and the output shows it) instead of
// a stale stage's values.  Off in the product build.
#ifndef MG3M_LDS_POISON
#define MG3M_LDS_POISON 0
#endif
template <class C>
__device__ __forceinline__ void poison_stage(float* As, float* Bs) {
  if constexpr (MG3M_LDS_POISON != 0) {
    const float nan = __builtin_nanf("");
    for (int i = (int)threadIdx.x; i < C::A_STAGE; i += C::T) As[i] = nan;
    for (int i = (int)threadIdx.x; i < C::B_STAGE; i += C::T) Bs[i] = nan;
    __syncthreads();
  }
}

// s_waitcnt with only the vector-memory count at zero (gfx9 encoding:
// vmcnt[3:0] in bits 3:0 and vmcnt[5:4] in bits 15:14 = 0, expcnt bits 6:4
// and lgkmcnt bits 11:8 at their maxima, i.e. not waited on).
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// The stage pipeline of run_stages with direct-to-LDS loaders: stage it+1's
// loads go straight into the other buffer (last read in iteration it-1, which
// every wave finished before that iteration's barrier) while stage it's MFMAs
// run; each iteration ends by waiting for this wave's loads and a barrier.
template <class C, class AL, class BL, class F>
__device__ __forceinline__ void run_stages_dma(const KArgs& a, AL& al, BL& bl, float* As0, float* Bs0, int nk,
                                               __amdgpu_buffer_rsrc_t xr, __amdgpu_buffer_rsrc_t wr,
                                               F&& compute) {
  if (nk <= 0) return;
  al.load(a, wr, As0);
  bl.load(a, xr, Bs0);
  wait_vmem();
  __syncthreads();
  auto step = [&](auto cur_c) {
    constexpr int CUR = decltype(cur_c)::value;
    poison_stage<C>(As0 + (CUR ^ 1) * C::A_STAGE, Bs0 + (CUR ^ 1) * C::B_STAGE);
    al.advance(a);
    bl.advance(a);
    al.load(a, wr, As0 + (CUR ^ 1) * C::A_STAGE);
    bl.load(a, xr, Bs0 + (CUR ^ 1) * C::B_STAGE);
    __builtin_amdgcn_sched_barrier(0);
    compute(As0 + CUR * C::A_STAGE, Bs0 + CUR * C::B_STAGE);
    __builtin_amdgcn_sched_barrier(0);
    wait_vmem();
    __syncthreads();
  };
  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;
  int it = 0;
  for (; it + 2 <= nk - 1; it += 2) {
    step(B0{});
    step(B1{});
  }
  if (it < nk - 1) {
    step(B0{});
    ++it;
  }
  const int last = it & 1;
  compute(As0 + last * C::A_STAGE, Bs0 + last * C::B_STAGE);
}

// NCHW input x[N][C][H][W] (Eq. 1's order), reduction order k = (c*R + r)*S + s.
// Each thread owns four consecutive output columns n..n+3 (consecutive output
// pixels of one image) and NV consecutive rows of the KT x NT tile.  With
// stride_w == 1 the four columns of one output row read four consecutive
// inputs along W: one 16-byte load covers them, and elements that fall off
// the left or right edge of the image row (padding) are zeroed afterwards --
// the load itself only has to stay inside the tensor.  Otherwise (a group
// that wraps to the next output row, any stride_w > 1, the tensor's first or
// last words) the four elements are loaded one by one from per-column bases
// computed once per work-group.  The row index (c, r, s) advances by
// carries, with no division in the main loop.
template <class C, int NT, int KT>
struct BVecW {
  static constexpr int NC4 = NT / 4;
  static constexpr int RG = C::T / NC4;      // threads sharing one column group
  static constexpr int NV = KT / RG;         // consecutive rows per thread
  static_assert(C::T % NC4 == 0 && KT % RG == 0 && NV * 4 == C::B_ELEMS, "B vec-W split");
  int n4, kr0;
  int cb[4], ih0[4], iw0[4];   // per column: x index at (c, r, s) = 0, and the tap origin
  bool vrow;                   // the four columns are one run of one output row (stride_w 1)
  int c, r, s;                 // reduction index of the thread's first row
  int dc, dr, ds;              // KT in the mixed radix (C, R, S)
  f32x4 v[NV], e4[NV];         // row loaded as one vector, or element by element
  bool fast_[NV];              // row i took the vector load
  unsigned keep;               // bits 4i..4i+3: elements of row i's vector inside the image row

  __device__ void init(const KArgs& a, int t, int n0, int kbeg) {
    n4 = t % NC4;
    kr0 = (t / NC4) * NV;
    const int n = n0 + n4 * 4, hw = a.Ho * a.Wo;
    int wo_first = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int ne = n + e;
      const int b = ne / hw, pix = ne - b * hw;
      const int ho = pix / a.Wo, wo = pix - ho * a.Wo;
      if (e == 0) wo_first = wo;
      const bool live = ne < a.Ng;
      ih0[e] = live ? ho * a.sh - a.ph : -(1 << 30);   // columns past the end read nothing
      iw0[e] = wo * a.sw - a.pw;
      cb[e] = live ? (b * a.C * a.H + ih0[e]) * a.W + iw0[e] : 0;
    }
    vrow = (a.sw == 1) & (n + 3 < a.Ng) & (wo_first + 3 < a.Wo);
    const int rs = a.R * a.S, k0 = kbeg + kr0;
    c = k0 / rs;
    r = (k0 - c * rs) / a.S;
    s = k0 - c * rs - r * a.S;
    dc = KT / rs;
    dr = (KT - dc * rs) / a.S;
    ds = KT - dc * rs - dr * a.S;
    // e4 is carried from stage to stage (stale in rows that take the vector
    // load, where it is not used), so it never shares registers with v
#pragma unroll
    for (int i = 0; i < NV; ++i) e4[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  __device__ void advance(const KArgs& a) {
    s += ds;
    r += dr;
    c += dc;
    if (s >= a.S) { s -= a.S; ++r; }
    if (r >= a.R) { r -= a.R; ++c; }
  }
  __device__ void load(const KArgs& a, __amdgpu_buffer_rsrc_t xr) {
    const int hw = a.H * a.W;
    const int x_elems = (int)(a.x_bytes / 4u);
    int ci = c, ri = r, si = s;
    keep = 0;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      if (i > 0) {
        if (++si == a.S) {
          si = 0;
          if (++ri == a.R) { ri = 0; ++ci; }
        }
      }
      const int rel = ci * hw + ri * a.W + si;
      const bool k_ok = ci < a.C;
      const int iw = iw0[0] + si, off = cb[0] + rel;
      const bool fast = vrow & k_ok & ((unsigned)(ih0[0] + ri) < (unsigned)a.H) & (off >= 0) &
                        (off + 3 < x_elems);
      keep |= (((unsigned)iw < (unsigned)a.W) | (((unsigned)(iw + 1) < (unsigned)a.W) << 1) |
               (((unsigned)(iw + 2) < (unsigned)a.W) << 2) | (((unsigned)(iw + 3) < (unsigned)a.W) << 3))
              << (4 * i);
      fast_[i] = fast;
      v[i] = bload4(xr, fast ? (unsigned)off * 4u : kOOB);
      // separate registers: writing v[i] again would make the compiler wait
      // for the vector load here, inside the load phase
      if (!fast) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const bool ok = k_ok & ((unsigned)(ih0[e] + ri) < (unsigned)a.H) &
                          ((unsigned)(iw0[e] + si) < (unsigned)a.W);
          e4[i][e] = bload1(xr, ok ? (unsigned)(cb[e] + rel) * 4u : kOOB);
        }
      }
    }
  }
  __device__ void store(float* Bs) const {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      f32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = fast_[i] ? (((keep >> (4 * i + e)) & 1u) ? v[i][e] : 0.f) : e4[i][e];
      st4(Bs + (kr0 + i) * C::BS + C::LB::col(kr0 + i, n4 * 4), o);
    }
  }
};

// NCHW with the reduction taken tap-major, k = (r*S + s)*C + c, and C % KT ==
// 0: a KT-row slab is one filter tap (r, s) over KT consecutive channels, the
// same for the whole work-group, and stages run the taps inside each channel
// slab (as BVecNTap does for HWCN).  The filter is read from its [R][S][C][K]
// copy by AVecMTap.  Columns as in BVecW; a thread's NV consecutive rows are
// consecutive channels, H*W apart in x, so the image-bounds test, the border
// mask and the choice between one 16-byte load per row and element loads are
// made once per stage.
template <class C, int NT, int KT>
struct BVecWTap {
  static constexpr int NC4 = NT / 4;
  static constexpr int RG = C::T / NC4;
  static constexpr int NV = KT / RG;
  static_assert(C::T % NC4 == 0 && KT % RG == 0 && NV * 4 == C::B_ELEMS, "B vec-W split");
  int n4, kr0;
  int cb[4], ih0[4], iw0[4];
  bool vrow;
  int r, s, c0;                // uniform: tap and first channel of the slab
  f32x4 v[NV], e4[NV];
  bool fast;
  unsigned keep;

  __device__ void init(const KArgs& a, int t, int n0, int kbeg) {
    n4 = t % NC4;
    kr0 = (t / NC4) * NV;
    const int n = n0 + n4 * 4, hw = a.Ho * a.Wo;
    int wo_first = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int ne = n + e;
      const int b = ne / hw, pix = ne - b * hw;
      const int ho = pix / a.Wo, wo = pix - ho * a.Wo;
      if (e == 0) wo_first = wo;
      const bool live = ne < a.Ng;
      ih0[e] = live ? ho * a.sh - a.ph : -(1 << 30);
      iw0[e] = wo * a.sw - a.pw;
      // x index of (b, channel kr0, ih0, iw0)
      cb[e] = live ? ((b * a.C + kr0) * a.H + ih0[e]) * a.W + iw0[e] : 0;
    }
    vrow = (a.sw == 1) & (n + 3 < a.Ng) & (wo_first + 3 < a.Wo);
    const int t0 = kbeg / KT, rs = a.R * a.S;
    const int slab = t0 / rs, tap = t0 - slab * rs;
    c0 = slab * KT;
    r = tap / a.S;
    s = tap - r * a.S;
#pragma unroll
    for (int i = 0; i < NV; ++i) e4[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  __device__ void advance(const KArgs& a) {
    if (++s == a.S) {
      s = 0;
      if (++r == a.R) { r = 0; c0 += KT; }
    }
  }
  __device__ void load(const KArgs& a, __amdgpu_buffer_rsrc_t xr) {
    const int hw = a.H * a.W;
    const int rel = c0 * hw + r * a.W + s;
    const int iw = iw0[0] + s, off = cb[0] + rel;
    fast = vrow & ((unsigned)(ih0[0] + r) < (unsigned)a.H) & (off >= 0) &
           (off + (NV - 1) * hw + 3 < (int)(a.x_bytes / 4u));
    keep = ((unsigned)iw < (unsigned)a.W) | (((unsigned)(iw + 1) < (unsigned)a.W) << 1) |
           (((unsigned)(iw + 2) < (unsigned)a.W) << 2) | (((unsigned)(iw + 3) < (unsigned)a.W) << 3);
#pragma unroll
    for (int i = 0; i < NV; ++i) v[i] = bload4(xr, fast ? (unsigned)(off + i * hw) * 4u : kOOB);
    if (!fast) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const bool ok = ((unsigned)(ih0[e] + r) < (unsigned)a.H) & ((unsigned)(iw0[e] + s) < (unsigned)a.W);
#pragma unroll
        for (int i = 0; i < NV; ++i) e4[i][e] = bload1(xr, ok ? (unsigned)(cb[e] + rel + i * hw) * 4u : kOOB);
      }
    }
  }
  __device__ void store(float* Bs) const {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      f32x4 o;
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = fast ? (((keep >> e) & 1u) ? v[i][e] : 0.f) : e4[i][e];
      st4(Bs + (kr0 + i) * C::BS + C::LB::col(kr0 + i, n4 * 4), o);
    }
  }
};

// HWCN, N % 4 == 0: each thread owns one 4-wide batch vector of one output
// pixel (a fixed column group) and NV rows of the KT x NT tile.
template <class C, int NT, int KT>
struct BVecN {
  static constexpr int NC4 = NT / 4;
  static constexpr int RSTEP = C::T / NC4;
  static constexpr int NV = KT / RSTEP;
  static_assert(C::T % NC4 == 0 && KT % RSTEP == 0 && NV * 4 == C::B_ELEMS, "B vec-N split");
  int n4, kr0, ih0, iw0, b;
  bool col_ok;
  RscStep st;
  int k[NV], r[NV], s[NV], c[NV];
  f32x4 v[NV];

  __device__ void init(const KArgs& a, int t, int n0, int kbeg) {
    n4 = t % NC4;
    kr0 = t / NC4;
    // with a whole wave per tile row (NC4 a multiple of 64) a thread's rows
    // are its wave's: k, r, s and c then live in scalar registers
    if constexpr (NC4 % 64 == 0) kr0 = __builtin_amdgcn_readfirstlane(kr0);
    const int n = n0 + n4 * 4;
    col_ok = n < a.Ng;
    const int pix = n / a.N;
    b = n - pix * a.N;
    const int ho = pix / a.Wo, wo = pix - ho * a.Wo;
    ih0 = ho * a.sh - a.ph;
    iw0 = wo * a.sw - a.pw;
    st.init(a, KT);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      k[i] = kbeg + kr0 + i * RSTEP;
      split_k<kHWCN>(a, k[i], r[i], s[i], c[i]);
    }
  }
  __device__ void advance(const KArgs& a) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      k[i] += KT;
      step_rsc(a, st, r[i], s[i], c[i]);
    }
  }
  __device__ void load(const KArgs& a, __amdgpu_buffer_rsrc_t xr) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int ih = ih0 + r[i], iw = iw0 + s[i];
      const bool ok = col_ok & (k[i] < a.Kg) & ((unsigned)ih < (unsigned)a.H) &
                      ((unsigned)iw < (unsigned)a.W);
      const unsigned off = (unsigned)(((ih * a.W + iw) * a.C + c[i]) * a.N + b) * 4u;
      v[i] = bload4(xr, ok ? off : kOOB);
    }
  }
  __device__ void store(float* Bs) const {
    static_assert(RSTEP % 4 == 0, "a thread's rows share their swizzle");
    const int col = C::LB::col(kr0, n4 * 4);
#pragma unroll
    for (int i = 0; i < NV; ++i) st4(Bs + (kr0 + i * RSTEP) * C::BS + col, v[i]);
  }
};

// HWCN, N == 1, C % 4 == 0: each thread owns one 4-deep channel vector of
// one filter tap (a fixed row group) and NV output pixels.
template <class C, int NT, int KT>
struct BVecC {
  static constexpr int KV = KT / 4;
  static constexpr int NSTEP = C::T / KV;
  static constexpr int NV = NT / NSTEP;
  static_assert(C::T % KV == 0 && NT % NSTEP == 0 && NV * 4 == C::B_ELEMS, "B vec-C split");
  int k4, nc0, k, r, s, c;
  RscStep st;
  int ih0[NV], iw0[NV];
  bool col_ok[NV];
  f32x4 v[NV];

  __device__ void init(const KArgs& a, int t, int n0, int kbeg) {
    k4 = t % KV;
    nc0 = t / KV;
    k = kbeg + 4 * k4;
    split_k<kHWCN>(a, k, r, s, c);
    st.init(a, KT);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int n = n0 + nc0 + i * NSTEP;          // N == 1: n is the output pixel
      col_ok[i] = n < a.Ng;
      const int ho = n / a.Wo, wo = n - ho * a.Wo;
      ih0[i] = ho * a.sh - a.ph;
      iw0[i] = wo * a.sw - a.pw;
    }
  }
  __device__ void advance(const KArgs& a) {
    k += KT;
    step_rsc(a, st, r, s, c);
  }
  __device__ void load(const KArgs& a, __amdgpu_buffer_rsrc_t xr) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int ih = ih0[i] + r, iw = iw0[i] + s;
      const bool ok = col_ok[i] & (k < a.Kg) & ((unsigned)ih < (unsigned)a.H) &
                      ((unsigned)iw < (unsigned)a.W);
      const unsigned off = (unsigned)((ih * a.W + iw) * a.C + c) * 4u;
      v[i] = bload4(xr, ok ? off : kOOB);
    }
  }
  __device__ void store(float* Bs) const {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int n = nc0 + i * NSTEP;
#pragma unroll
      for (int e = 0; e < 4; ++e) Bs[(4 * k4 + e) * C::BS + C::LB::col(4 * k4 + e, n)] = v[i][e];
    }
  }
};

// Any layout, any alignment: single elements, indices decomposed per stage.
template <int LAYOUT, class C, int NT, int KT>
struct BScalar {
  static constexpr int NE = C::B_ELEMS;
  int t_, n0_, kbase;
  float v[NE];

  __device__ void init(const KArgs&, int t, int n0, int kbeg) { t_ = t; n0_ = n0; kbase = kbeg; }
  __device__ void advance(const KArgs&) { kbase += KT; }
  __device__ void load(const KArgs& a, __amdgpu_buffer_rsrc_t xr) {
#pragma unroll
    for (int i = 0; i < NE; ++i) {
      const int e = t_ + i * C::T;
      const int n = n0_ + e % NT, k = kbase + e / NT;
      unsigned off = kOOB;
      if (n < a.Ng && k < a.Kg) {
        int r, s, c;
        split_k<LAYOUT>(a, k, r, s, c);
        int b, pix;
        if constexpr (LAYOUT == kHWCN) { pix = n / a.N; b = n - pix * a.N; }
        else { const int hw = a.Ho * a.Wo; b = n / hw; pix = n - b * hw; }
        const int ho = pix / a.Wo, wo = pix - ho * a.Wo;
        const int ih = ho * a.sh - a.ph + r, iw = wo * a.sw - a.pw + s;
        if ((unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W) {
          const int idx = (LAYOUT == kHWCN) ? ((ih * a.W + iw) * a.C + c) * a.N + b
                                            : ((b * a.C + c) * a.H + ih) * a.W + iw;
          off = (unsigned)idx * 4u;
        }
      }
      v[i] = bload1(xr, off);
    }
  }
  __device__ void store(float* Bs) const {
#pragma unroll
    for (int i = 0; i < NE; ++i) {
      const int e = t_ + i * C::T;
      Bs[(e / NT) * C::BS + C::LB::col(e / NT, e % NT)] = v[i];
    }
  }
};

template <int LAYOUT, int AM, class C, int MT, int KT, int BM = -1>
struct ASel;
template <class C, int MT, int KT, int BM>
struct ASel<kHWCN, kAVecM, C, MT, KT, BM> { using type = AVecM<C, MT, KT>; };
template <class C, int MT, int KT>
struct ASel<kHWCN, kAVecM, C, MT, KT, kBVecNTap> { using type = AVecMTap<C, MT, KT>; };
template <class C, int MT, int KT>
struct ASel<kHWCN, kAVecM, C, MT, KT, kBVecNTapDma> { using type = AVecMTapDma<C, MT, KT>; };
template <class C, int MT, int KT>
struct ASel<kNCHW, kAVecM, C, MT, KT, kBVecWTap> { using type = AVecMTap<C, MT, KT>; };
template <class C, int MT, int KT, int BM>
struct ASel<kNCHW, kAVecK, C, MT, KT, BM> { using type = AVecK<C, MT, KT>; };
template <int LAYOUT, class C, int MT, int KT, int BM>
struct ASel<LAYOUT, kAScalar, C, MT, KT, BM> { using type = AScalar<LAYOUT, C, MT, KT>; };

template <int LAYOUT, int BM, class C, int NT, int KT>
struct BSel;
template <class C, int NT, int KT>
struct BSel<kHWCN, kBVecN, C, NT, KT> { using type = BVecN<C, NT, KT>; };
template <class C, int NT, int KT>
struct BSel<kHWCN, kBVecNTap, C, NT, KT> { using type = BVecNTap<C, NT, KT>; };
template <class C, int NT, int KT>
struct BSel<kHWCN, kBVecNTapDma, C, NT, KT> { using type = BVecNTapDma<C, NT, KT>; };
template <class C, int NT, int KT>
struct BSel<kHWCN, kBVecC, C, NT, KT> { using type = BVecC<C, NT, KT>; };
template <class C, int NT, int KT>
struct BSel<kNCHW, kBVecW, C, NT, KT> { using type = BVecW<C, NT, KT>; };
template <class C, int NT, int KT>
struct BSel<kNCHW, kBVecWTap, C, NT, KT> { using type = BVecWTap<C, NT, KT>; };
template <int LAYOUT, class C, int NT, int KT>
struct BSel<LAYOUT, kBScalar, C, NT, KT> { using type = BScalar<LAYOUT, C, NT, KT>; };

// --------------------------------------------------------- MFMA on a stage
// 32x32x2 fp32 MFMA operand layout: lane (hh, q) = (lane / 32, lane % 32)
// supplies A[row q][k = hh] and B[k = hh][column q].
template <class C, int KT>
__device__ __forceinline__ void mma_stage(floatx16 (&acc)[C::TM][C::TN], const float* As,
                                          const float* Bs, int wm, int wn, int hh, int q) {
  // Row 2*kk + hh, logical column c + q with c a multiple of 32: the
  // swizzle depends on the row only through hh and leaves q (< 32) alone.
  int ca[C::TM], cb[C::TN];
#pragma unroll
  for (int i = 0; i < C::TM; ++i) ca[i] = hh * C::AS + C::LA::col(hh, wm * C::WTM + i * 32) + q;
#pragma unroll
  for (int j = 0; j < C::TN; ++j) cb[j] = hh * C::BS + C::LB::col(hh, wn * C::WTN + j * 32) + q;
  float av[KT / 2][C::TM], bv[KT / 2][C::TN];
#pragma unroll
  for (int kk = 0; kk < KT / 2; ++kk) {
#pragma unroll
    for (int i = 0; i < C::TM; ++i) av[kk][i] = As[ca[i] + 2 * kk * C::AS];
#pragma unroll
    for (int j = 0; j < C::TN; ++j) bv[kk][j] = Bs[cb[j] + 2 * kk * C::BS];
  }
#pragma unroll
  for (int kk = 0; kk < KT / 2; ++kk)
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
      for (int j = 0; j < C::TN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[kk][i], bv[kk][j], acc[i][j], 0, 0, 0);
}

// fp64 16x16x4 MFMA operand layout (checked on gfx950): lane (g, q) =
// (lane / 16, lane % 16) supplies A[row q][k = g] and B[k = g][column q].  The fp32 operands are
// widened exactly, so every product is exact and only the fp64 additions
// round.
template <class C, int KT>
__device__ __forceinline__ void mma_stage64(f64x4 (&acc)[C::TM16][C::TN16], const float* As,
                                            const float* Bs, int wm, int wn, int g, int q) {
  // Row 4*kk + g, logical column c + q with c a multiple of 16: the
  // swizzle depends on the row only through g and leaves q (< 16) alone.
  int ca[C::TM16], cb[C::TN16];
#pragma unroll
  for (int i = 0; i < C::TM16; ++i) ca[i] = g * C::AS + C::LA::col(g, wm * C::WTM + i * 16) + q;
#pragma unroll
  for (int j = 0; j < C::TN16; ++j) cb[j] = g * C::BS + C::LB::col(g, wn * C::WTN + j * 16) + q;
#pragma unroll
  for (int kk = 0; kk < KT / 4; ++kk) {
    double av[C::TM16], bv[C::TN16];
#pragma unroll
    for (int i = 0; i < C::TM16; ++i) av[i] = (double)As[ca[i] + 4 * kk * C::AS];
#pragma unroll
    for (int j = 0; j < C::TN16; ++j) bv[j] = (double)Bs[cb[j] + 4 * kk * C::BS];
#pragma unroll
    for (int i = 0; i < C::TM16; ++i)
#pragma unroll
      for (int j = 0; j < C::TN16; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[i], bv[j], acc[i][j], 0, 0, 0);
  }
}

// fp32 16x16x4 MFMA, for 16-row tiles: the same operand layout as the fp64
// 16x16x4 (lane (g, q) supplies A[row q][k = g] and B[k = g][column q]) on
// the same LDS layout, with fp32 operands and accumulators.
template <class C, int KT>
__device__ __forceinline__ void mma_stage16(f32x4 (&acc)[C::TM16][C::TN16], const float* As,
                                            const float* Bs, int wm, int wn, int g, int q) {
  int ca[C::TM16], cb[C::TN16];
#pragma unroll
  for (int i = 0; i < C::TM16; ++i) ca[i] = g * C::AS + C::LA::col(g, wm * C::WTM + i * 16) + q;
#pragma unroll
  for (int j = 0; j < C::TN16; ++j) cb[j] = g * C::BS + C::LB::col(g, wn * C::WTN + j * 16) + q;
  float av[KT / 4][C::TM16], bv[KT / 4][C::TN16];
#pragma unroll
  for (int kk = 0; kk < KT / 4; ++kk) {
#pragma unroll
    for (int i = 0; i < C::TM16; ++i) av[kk][i] = As[ca[i] + 4 * kk * C::AS];
#pragma unroll
    for (int j = 0; j < C::TN16; ++j) bv[kk][j] = Bs[cb[j] + 4 * kk * C::BS];
  }
#pragma unroll
  for (int kk = 0; kk < KT / 4; ++kk)
#pragma unroll
    for (int i = 0; i < C::TM16; ++i)
#pragma unroll
      for (int j = 0; j < C::TN16; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[kk][i], bv[kk][j], acc[i][j], 0, 0, 0);
}

// ------------------------------------------------------ stage pipeline
// Runs nk stages of the reduction through the two LDS buffers, calling
// compute(As, Bs) on each staged pair.  The loads of stage it+1 are issued
// before stage it's MFMAs and land in the other buffer after them; one
// barrier per stage.  Buffer cur^1 was last read in iteration it-1, which
// every wave finished before the barrier that ended it.  Stages alternate
// between the two buffers, so the loop is unrolled by two to make the buffer
// offsets compile-time constants.
template <class C, class AL, class BL, class F>
__device__ __forceinline__ void run_stages(const KArgs& a, AL& al, BL& bl, float* As0, float* Bs0,
                                           int nk, __amdgpu_buffer_rsrc_t xr,
                                           __amdgpu_buffer_rsrc_t wr, F&& compute) {
  if (nk <= 0) return;
  al.load(a, wr);
  bl.load(a, xr);
  al.store(As0);
  bl.store(Bs0);
  __syncthreads();
  auto step = [&](auto cur_c) {
    constexpr int CUR = decltype(cur_c)::value;
    poison_stage<C>(As0 + (CUR ^ 1) * C::A_STAGE, Bs0 + (CUR ^ 1) * C::B_STAGE);
    al.advance(a);
    bl.advance(a);
    al.load(a, wr);
    bl.load(a, xr);
    // keep the global loads ahead of the MFMAs (the scheduler would
    // otherwise sink them next to their LDS stores and expose their latency)
    __builtin_amdgcn_sched_barrier(0);
    compute(As0 + CUR * C::A_STAGE, Bs0 + CUR * C::B_STAGE);
    __builtin_amdgcn_sched_barrier(0);
    al.store(As0 + (CUR ^ 1) * C::A_STAGE);
    bl.store(Bs0 + (CUR ^ 1) * C::B_STAGE);
    __syncthreads();
  };
  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;
  int it = 0;
  for (; it + 2 <= nk - 1; it += 2) {
    step(B0{});
    step(B1{});
  }
  if (it < nk - 1) {
    step(B0{});
    ++it;
  }
  const int last = it & 1;
  compute(As0 + last * C::A_STAGE, Bs0 + last * C::B_STAGE);
}

// ------------------------------------------------------ tile mapping
// XCD grouping of the whole tiles: work-group i runs on XCD i % 8, so the G
// whole tiles are renumbered to give each XCD a contiguous run of them (tiles
// sharing a patch tile or halo rows then share one L2).  The runs differ in
// length by at most one.  Work-groups at or past G keep their number.
__device__ __forceinline__ int xcd_group(int L, int G) {
  if (L >= G) return L;
  const int q8 = G >> 3, r8 = G & 7, xcd = L & 7, loc = L >> 3;
  return (xcd < r8) ? xcd * (q8 + 1) + loc : r8 * (q8 + 1) + (xcd - r8) * q8 + loc;
}

// Tail work.  The reduction steps of the tail tiles (tail_tiles * k_tiles
// of them, tile by tile) are dealt out to the tail work-groups as runs of
// consecutive steps, in one of two ways:
//  * split (sk_s > 0): each tail tile's k_tiles steps are cut into sk_s runs
//    of sk_q steps, one more for the first sk_r of them; run w is piece
//    w % sk_s of tail tile w / sk_s.  A run never leaves its tile.
//  * stream-K (sk_s == 0): all the steps are cut into tail_wgs runs of sk_q
//    steps, one more for the first sk_r; run w starts at w*sk_q + min(w,
//    sk_r).  No run is longer than a tile, so a run holds the end of one tail
//    tile and the start of the next at most.
struct TailRun {
  int it, end;   // current step and end of the run (steps counted from the first tail tile)
};

// Run taken by the tail work-group launched w-th.  Split: consecutive
// work-groups take the same piece of consecutive tiles, so they work on the
// same k-slab at the same time and neighbouring tiles share input rows and
// filter columns in L2.  Stream-K: launch order.
__device__ __forceinline__ int tail_wg(const KArgs& a, int w) {
  return a.sk_s > 0 ? (w % a.tail_tiles) * a.sk_s + w / a.tail_tiles : w;
}

__device__ __forceinline__ TailRun tail_run(const KArgs& a, int w) {
  if (a.sk_s > 0) {
    const int t = w / a.sk_s, j = w - t * a.sk_s;
    const int it = t * a.k_tiles + j * a.sk_q + min(j, a.sk_r);
    return TailRun{it, it + a.sk_q + (j < a.sk_r ? 1 : 0)};
  }
  const int it = w * a.sk_q + min(w, a.sk_r);
  return TailRun{it, it + a.sk_q + (w < a.sk_r ? 1 : 0)};
}

// The piece of a run in one tail tile: tile index relative to the first
// tail tile, its first k-tile and its length.
__device__ __forceinline__ void tail_piece(const KArgs& a, const TailRun& r, int* rel, int* kt0, int* nk) {
  *rel = r.it / a.k_tiles;
  *kt0 = r.it - *rel * a.k_tiles;
  *nk = min(r.end - r.it, a.k_tiles - *kt0);
}

// Split plans only: the run of the tail work-group launched L-th is piece j
// = L / tail_tiles of tail tile rel = L % tail_tiles (tail_wg), run number
// w = rel * sk_s + j; the same as tail_run and tail_piece, computed directly.
__device__ __forceinline__ void split_piece(const KArgs& a, int L, int* w, int* rel, int* kt0, int* nk) {
  const int j = L / a.tail_tiles;
  *rel = L - j * a.tail_tiles;
  *w = *rel * a.sk_s + j;
  *kt0 = j * a.sk_q + min(j, a.sk_r);
  *nk = a.sk_q + (j < a.sk_r ? 1 : 0);
}

// Partial slot of the piece of run w in tail tile rel.  Along the order of
// the steps both w and rel never decrease and one of them grows from piece to
// piece, so w + rel is unique; the slots run to tail_wgs + tail_tiles - 2.
__device__ __forceinline__ long long tail_slot(int w, int rel) { return (long long)w + rel; }

// Output element (m, n) sits at out_colbase(n) + m * mstride in either layout.
template <int LAYOUT>
__device__ __forceinline__ int out_colbase(const KArgs& a, int n) {
  if constexpr (LAYOUT == kHWCN) {
    const int pix = n / a.N, b = n - pix * a.N;
    return pix * a.K * a.N + b;
  } else {
    const int hw = a.Ho * a.Wo, b = n / hw, pix = n - b * hw;
    return b * a.K * hw + pix;
  }
}

// Fused output stage: y = act(conv + add), for the network executor.
__device__ __forceinline__ float finish1(const KArgs& a, float v, int idx) {
  if (a.add != nullptr) v += a.add[idx];
  return (a.relu != 0 && v < 0.f) ? 0.f : v;
}

// ----------------------------------------------------------------- kernels
// One tile's product over the k-tiles [kt0, kt0 + nk): stage the operands
// through LDS, run the MFMAs, and hand the accumulators to store(acc, m0, n0,
// wm, wn, hh, q) with the tile's origin and the lane's place in it.  Every
// per-lane value is derived here from the thread index t.
template <int LAYOUT, int AM, int BM, int MT, int NT, int KT, int WM, int WN, class Store>
__device__ __forceinline__ void tile_product_f32(const KArgs& a, float* lds, int t, int tile, int kt0,
                                                 int nk, Store&& store) {
  using C = Cfg<MT, NT, KT, WM, WN>;
  const int tm = tile % a.tiles_m;
  const int tn = tile / a.tiles_m;
  const int m0 = tm * MT, n0 = tn * NT;
  const int kbeg = kt0 * KT;

  float* const As0 = lds;
  float* const Bs0 = lds + 2 * C::A_STAGE;

  const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, a.x_bytes);
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(a.w, a.w_bytes);

  typename ASel<LAYOUT, AM, C, MT, KT, BM>::type al;
  typename BSel<LAYOUT, BM, C, NT, KT>::type bl;
  al.init(a, t, m0, kbeg);
  bl.init(a, t, n0, kbeg);

  const int wave = t >> 6, lane = t & 63;
  const int wm = wave % WM, wn = wave / WM;
  const int hh = lane >> 5, q = lane & 31;

  floatx16 acc[C::TM][C::TN];
#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  auto mma = [&](const float* As, const float* Bs) { mma_stage<C, KT>(acc, As, Bs, wm, wn, hh, q); };
  if constexpr (BM == kBVecNTapDma) run_stages_dma<C>(a, al, bl, As0, Bs0, nk, xr, wr, mma);
  else run_stages<C>(a, al, bl, As0, Bs0, nk, xr, wr, mma);
  store(acc, m0, n0, wm, wn, hh, q);
}

// Tail work-groups: the one launched `launched`-th computes its run and
// stores each piece's tile-local partial sums (row-major mt x nt) in the
// piece's slot; the tail reduction adds them up and applies any fused output
// stage.  MULTI (one-tap HWCN loader, tail_runs_multi): stream-K runs, one
// piece per tail tile the run touches (two at most), taken in a loop whose
// thread index is made opaque per piece (hoisted out of the loop, the
// loaders' and stores' per-lane offsets would stay live across the main loop
// and cost occupancy).  Otherwise: split plans, one piece per run.
template <int LAYOUT, int AM, int BM, int MT, int NT, int KT, int WM, int WN, bool MULTI>
__device__ __forceinline__ void tail_runs_f32(const KArgs& a, float* lds, int launched) {
  using C = Cfg<MT, NT, KT, WM, WN>;
  if constexpr (!MULTI) {
    int w, rel, kt0, nk;
    split_piece(a, launched, &w, &rel, &kt0, &nk);
    float* const part = a.ws + tail_slot(w, rel) * (MT * NT);
    tile_product_f32<LAYOUT, AM, BM, MT, NT, KT, WM, WN>(
        a, lds, threadIdx.x, a.dp_tiles + rel, kt0, nk,
        [&](floatx16 (&acc)[C::TM][C::TN], int, int, int wm, int wn, int hh, int q) {
#pragma unroll
          for (int j = 0; j < C::TN; ++j) {
            const int col = wn * C::WTN + j * 32 + q;
#pragma unroll
            for (int i = 0; i < C::TM; ++i)
#pragma unroll
              for (int e = 0; e < 16; ++e)
                part[(wm * C::WTM + i * 32 + 8 * (e >> 2) + 4 * hh + (e & 3)) * NT + col] = acc[i][j][e];
          }
        });
  } else {
    const int w = tail_wg(a, launched);
    TailRun run = tail_run(a, w);
    for (;;) {
      int rel, kt0, nk;
      tail_piece(a, run, &rel, &kt0, &nk);
      int t = threadIdx.x;
      asm volatile("" : "+v"(t));
      // buffer stores: one per-lane offset register serves all of the piece's
      // stores (with plain stores the loop keeps a 64-bit address per store)
      const __amdgpu_buffer_rsrc_t pr = make_rsrc(a.ws + tail_slot(w, rel) * (MT * NT), MT * NT * 4);
      tile_product_f32<LAYOUT, AM, BM, MT, NT, KT, WM, WN>(
          a, lds, t, a.dp_tiles + rel, kt0, nk,
          [&](floatx16 (&acc)[C::TM][C::TN], int, int, int wm, int wn, int hh, int q) {
            const unsigned lane_b = 4u * ((wm * C::WTM + 4 * hh) * NT + wn * C::WTN + q);
#pragma unroll
            for (int j = 0; j < C::TN; ++j)
#pragma unroll
              for (int i = 0; i < C::TM; ++i)
#pragma unroll
                for (int e = 0; e < 16; ++e)
                  bstore1(pr, lane_b, 4u * ((i * 32 + 8 * (e >> 2) + (e & 3)) * NT + j * 32), acc[i][j][e]);
          });
      run.it += nk;
      if (run.it >= run.end) return;
      __syncthreads();   // the next piece restages the LDS buffers
    }
  }
}

// Epilogue of a whole tile, straight from the accumulators into y (with the
// fused output stage when FUSE).  32x32 accumulator layout: register e of
// lane (hh, q) holds row 8*(e/4) + 4*hh + e%4, column q.
template <int LAYOUT, class C, bool FUSE>
__device__ __forceinline__ void store_tile_f32(const KArgs& a, floatx16 (&acc)[C::TM][C::TN], int m0, int n0,
                                               int wm, int wn, int hh, int q) {
  float* const out = a.y;
#pragma unroll
  for (int j = 0; j < C::TN; ++j) {
    const int n = n0 + wn * C::WTN + j * 32 + q;
    if (n >= a.Ng) continue;
    const int colbase = out_colbase<LAYOUT>(a, n);
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int row0 = m0 + wm * C::WTM + i * 32 + 8 * g + 4 * hh;
        if (a.e_mode == kEVecM) {
          // four consecutive output channels, contiguous when mstride == 1
          if (row0 < a.Mg) {
            f32x4 v{acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]};
            if constexpr (FUSE) {
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] = finish1(a, v[e], colbase + row0 + e);
            }
            st4(out + colbase + row0, v);
          }
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (row0 + e < a.Mg) {
              const int idx = colbase + (row0 + e) * a.mstride;
              if constexpr (FUSE) out[idx] = finish1(a, acc[i][j][4 * g + e], idx);
              else out[idx] = acc[i][j][4 * g + e];
            }
        }
      }
  }
}

// Epilogue of a whole tile through a buffer resource on y, element stores
// (the layouts where output channel m and m+1 are mstride apart, any
// mstride): a per-lane base offset per 32-column block plus the row's part,
// and elements outside the output sent to the out-of-range offset (with a
// zero scalar offset, as the loaders do), which the buffer hardware drops --
// no branches and no 64-bit address per store.
template <int LAYOUT, class C, bool FUSE = false>
__device__ __forceinline__ void store_tile_f32_buf(const KArgs& a, floatx16 (&acc)[C::TM][C::TN], int m0, int n0,
                                                   int wm, int wn, int hh, int q) {
  const __amdgpu_buffer_rsrc_t yr = make_rsrc(a.y, a.y_bytes);
  const bool has_add = FUSE && a.add != nullptr;
  const __amdgpu_buffer_rsrc_t ar = make_rsrc(has_add ? a.add : a.y, a.y_bytes);
  // opaque here, so that the row offsets below are formed where the stores
  // use them (hoisted out of the persistent kernel's loop over tiles, their
  // products spilled scalar registers)
  unsigned rs4 = 4u * (unsigned)a.mstride;
  asm volatile("" : "+s"(rs4));
  const int row_l = m0 + wm * C::WTM + 4 * hh;      // lane's first row
  const int rows_left = a.Mg - row_l;                // rows r of the wave tile with r < rows_left exist
#pragma unroll
  for (int j = 0; j < C::TN; ++j) {
    const int n = n0 + wn * C::WTN + j * 32 + q;
    const bool col_ok = n < a.Ng;
    const unsigned voff = 4u * (unsigned)(out_colbase<LAYOUT>(a, n) + row_l * a.mstride);
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const unsigned o = voff + (unsigned)(i * 32 + 8 * g) * rs4;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = i * 32 + 8 * g + e;         // row offset from the lane's first row
          const bool ok = col_ok & (r < rows_left);
          const unsigned off = ok ? o + (unsigned)e * rs4 : kOOB;
          float v = acc[i][j][4 * g + e];
          if constexpr (FUSE) {
            // fused output stage: add (same layout as y) read through its own
            // buffer resource at the store's offset; ReLU keeps NaN
            if (has_add) v += bload1(ar, off);
            if (a.relu != 0 && v < 0.f) v = 0.f;
          }
          bstore1(yr, off, 0u, v);
        }
      }
  }
}

// Work-groups [0, dp_tiles) compute whole tiles (tile xcd_group(i)) over
// the full reduction and store them to y; the work-groups after them run the
// tail (tail_runs_f32) in the same launch, starting as the last round of
// whole tiles drains.  Stream-K runs (a loop over pieces) only with the
// one-tap HWCN loader (tail_runs_multi): for the other loaders the loop would
// cost the whole tiles registers and occupancy.  FUSE: the output stage
// applies y = act(conv + add) (KArgs::add, relu).  A separate instantiation:
// the fused stage works on the accumulators in VGPRs, and the compiler copies
// all of them out of the AGPRs at once, which in a shared kernel would cost
// the plain convolution a wave per SIMD.
// Waves per SIMD that the tile's plain kernel reaches with its registers and
// LDS (the planner's occupancy model).  The fused direct-to-LDS kernels are
// held to the same (left alone, the add loads of their epilogue took them to
// 140 registers, a wave per SIMD fewer); they need no staging registers, so
// the bound costs no spills.
constexpr int plain_waves_per_simd(int mt, int nt, int kt, int wm, int wn) {
  for (int i = 0; i < kNumTiles; ++i) {
    const TileDesc& d = kTiles[i];
    if (d.mt == mt && d.nt == nt && d.kt == kt && d.wm == wm && d.wn == wn && d.m16 == 0) {
      const int by_regs = 512 / ((d.regs + 7) / 8 * 8);
      const int by_lds = 160 * 1024 / lds_bytes_for(d) * d.wm * d.wn / 4;
      const int w = by_regs < by_lds ? by_regs : by_lds;
      return w < 1 ? 1 : (w < 8 ? w : 8);
    }
  }
  return 1;
}

template <int LAYOUT, int AM, int BM, int MT, int NT, int KT, int WM, int WN, bool FUSE>
__global__ __launch_bounds__(WM * WN * 64)
__attribute__((amdgpu_waves_per_eu(FUSE && BM == kBVecNTapDma ? plain_waves_per_simd(MT, NT, KT, WM, WN) : 1)))
void conv_igemm_f32(KArgs a) {
  using C = Cfg<MT, NT, KT, WM, WN>;
  __shared__ __attribute__((aligned(16))) float lds[C::LDS_FLOATS];

  if ((int)blockIdx.x >= a.dp_tiles) {
    tail_runs_f32<LAYOUT, AM, BM, MT, NT, KT, WM, WN, tail_runs_multi(BM)>(a, lds, blockIdx.x - a.dp_tiles);
    return;
  }
  const int tile = xcd_group(blockIdx.x, a.dp_tiles);
  tile_product_f32<LAYOUT, AM, BM, MT, NT, KT, WM, WN>(
      a, lds, threadIdx.x, tile, 0, a.k_tiles,
      [&](floatx16 (&acc)[C::TM][C::TN], int m0, int n0, int wm, int wn, int hh, int q) {
        // the direct-to-LDS path (HWCN, N % 4 == 0: element stores) stores
        // through a buffer resource: branch-free, 2.4% faster on VGG-16 conv3
        if constexpr (BM == kBVecNTapDma) store_tile_f32_buf<LAYOUT, C, FUSE>(a, acc, m0, n0, wm, wn, hh, q);
        else store_tile_f32<LAYOUT, C, FUSE>(a, acc, m0, n0, wm, wn, hh, q);
      });
}

// ------------------------------------------------- persistent whole tiles
// mma_stage over the first nkk k-pairs of a stage only (rows 2*nkk and up are
// past Kg: their zero-filled products are skipped, not computed).
template <class C, int KT>
__device__ __forceinline__ void mma_stage_upto(floatx16 (&acc)[C::TM][C::TN], const float* As,
                                               const float* Bs, int wm, int wn, int hh, int q, int nkk) {
  int ca[C::TM], cb[C::TN];
#pragma unroll
  for (int i = 0; i < C::TM; ++i) ca[i] = hh * C::AS + C::LA::col(hh, wm * C::WTM + i * 32) + q;
#pragma unroll
  for (int j = 0; j < C::TN; ++j) cb[j] = hh * C::BS + C::LB::col(hh, wn * C::WTN + j * 32) + q;
#pragma unroll
  for (int kk = 0; kk < KT / 2; ++kk) {
    if (kk < nkk) {   // uniform: a scalar branch per k-pair
      float av[C::TM], bv[C::TN];
#pragma unroll
      for (int i = 0; i < C::TM; ++i) av[i] = As[ca[i] + 2 * kk * C::AS];
#pragma unroll
      for (int j = 0; j < C::TN; ++j) bv[j] = Bs[cb[j] + 2 * kk * C::BS];
#pragma unroll
      for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
  }
}

// Persistent whole tiles, for layers whose reduction is only a few stages
// deep (the three-channel stems: Kg = 27 for a 3x3 filter): there a
// work-group's life is a stage or two of MFMAs and then a burst of output
// stores, and work-groups that start together compute together and store
// together, so the chip alternates between the two instead of overlapping
// them.  Here gridDim.x work-groups each take every cnt-th tile of their
// XCD's contiguous run of tiles (below), and the stages of all of a
// work-group's tiles form one pipeline, one stage's loads in flight while
// the previous stage's MFMAs run; the last stage of a tile loads the first
// stage of the next one.  A tile's output stores are issued one stage later,
// right after the loads of the next tile's second stage (or of the tile after
// it when a tile has one stage), and before that stage's MFMAs.  On gfx9 one
// memory counter counts loads and stores, so the wait that ends the stage
// (for its loads) covers the stores as well, but only after a stage of MFMAs
// has run beside them.  The loaders stage through registers or, for the
// one-tap HWCN path, load straight into LDS.  The last stage of each tile
// computes only the k-pairs that hold rows below Kg.
template <int LAYOUT, int AM, int BM, int MT, int NT, int KT, int WM, int WN, bool FUSE>
__global__ __launch_bounds__(WM * WN * 64)
void conv_igemm_f32_pt(KArgs a) {
  using C = Cfg<MT, NT, KT, WM, WN>;
  __shared__ __attribute__((aligned(16))) float lds[C::LDS_FLOATS];
  // Work-group i runs on XCD i % 8.  Each XCD takes one contiguous run of the
  // tiles, in proportion to its work-groups, and its work-groups walk that
  // run together: tiles lo + loc, lo + loc + cnt, ...  A band of cnt
  // consecutive tiles is in flight per XCD at a time, and the next band
  // starts where it ends, so the input rows the two share (a filter's halo)
  // are still in that XCD's L2.
  const int G = (int)gridDim.x;
  const int q8 = G >> 3, r8 = G & 7, xcd = (int)(blockIdx.x & 7), loc = (int)(blockIdx.x >> 3);
  const int cnt = q8 + (xcd < r8 ? 1 : 0);                               // work-groups on this XCD
  const int rank0 = xcd < r8 ? xcd * (q8 + 1) : r8 * (q8 + 1) + (xcd - r8) * q8;
  const int hi = (int)((long long)a.dp_tiles * (rank0 + cnt) / G);
  int tile = (int)((long long)a.dp_tiles * rank0 / G) + loc;
  if (tile >= hi) return;

  const int t = threadIdx.x;
  float* const As0 = lds;
  float* const Bs0 = lds + 2 * C::A_STAGE;
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, a.x_bytes);
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(a.w, a.w_bytes);
  typename ASel<LAYOUT, AM, C, MT, KT, BM>::type al;
  typename BSel<LAYOUT, BM, C, NT, KT>::type bl;
  // A stage's loads into buffer b go straight into LDS with the direct-to-LDS
  // loaders, or into registers that commit(b) writes to LDS after the
  // current stage's MFMAs.  A stage ends when its loads have landed (with the
  // direct loads: this wave's memory count at zero, then the barrier) and
  // every wave is done with the buffer it consumed.
  constexpr bool kDma = BM == kBVecNTapDma;
  auto issue = [&](int b) {
    if constexpr (kDma) {
      al.load(a, wr, As0 + b * C::A_STAGE);
      bl.load(a, xr, Bs0 + b * C::B_STAGE);
    } else {
      al.load(a, wr);
      bl.load(a, xr);
    }
  };
  auto commit = [&](int b) {
    if constexpr (!kDma) {
      al.store(As0 + b * C::A_STAGE);
      bl.store(Bs0 + b * C::B_STAGE);
    }
  };
  auto stage_end = [&]() {
    if constexpr (kDma) wait_vmem();
    __syncthreads();
  };

  int m0 = (tile % a.tiles_m) * MT, n0 = (tile / a.tiles_m) * NT;
  al.init(a, t, m0, 0);
  bl.init(a, t, n0, 0);
  const int wave = t >> 6, lane = t & 63;
  const int wm = wave % WM, wn = wave / WM;
  const int hh = lane >> 5, q = lane & 31;
  // k-pairs of the last stage that hold a row below Kg
  const int last_kk = (a.Kg - (a.k_tiles - 1) * KT + 1) / 2;
  const int nk = a.k_tiles;

  issue(0);
  commit(0);
  stage_end();
  int cur = 0;
  int pm0 = 0, pn0 = 0;          // origin of the tile whose stores are pending
  bool pending = false;
  floatx16 acc[C::TM][C::TN];
  auto clear = [&]() {
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
      for (int j = 0; j < C::TN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
  };
  for (;;) {
    const int next = tile + cnt;
    if (nk > 1) {
      // stage 0 (staged in buffer cur), stage 1's loads in flight; then the
      // previous tile's stores
      poison_stage<C>(As0 + (cur ^ 1) * C::A_STAGE, Bs0 + (cur ^ 1) * C::B_STAGE);
      al.advance(a);
      bl.advance(a);
      issue(cur ^ 1);
      if (pending) store_tile_f32_buf<LAYOUT, C, FUSE>(a, acc, pm0, pn0, wm, wn, hh, q);
      // the stores read acc before it is cleared (else both stay live)
      __builtin_amdgcn_sched_barrier(0);
      clear();
      mma_stage<C, KT>(acc, As0 + cur * C::A_STAGE, Bs0 + cur * C::B_STAGE, wm, wn, hh, q);
      __builtin_amdgcn_sched_barrier(0);
      commit(cur ^ 1);
      stage_end();
      cur ^= 1;
      // stages 1 .. nk-2
      for (int it = 1; it + 1 < nk; ++it) {
        poison_stage<C>(As0 + (cur ^ 1) * C::A_STAGE, Bs0 + (cur ^ 1) * C::B_STAGE);
        al.advance(a);
        bl.advance(a);
        issue(cur ^ 1);
        __builtin_amdgcn_sched_barrier(0);
        mma_stage<C, KT>(acc, As0 + cur * C::A_STAGE, Bs0 + cur * C::B_STAGE, wm, wn, hh, q);
        __builtin_amdgcn_sched_barrier(0);
        commit(cur ^ 1);
        stage_end();
        cur ^= 1;
      }
    }
    // the last stage: its loads are the next tile's first stage; with one
    // stage per tile, the previous tile's stores go out after them
    const bool fetch = next < hi;
    poison_stage<C>(As0 + (cur ^ 1) * C::A_STAGE, Bs0 + (cur ^ 1) * C::B_STAGE);
    if (fetch) {
      al.init(a, t, (next % a.tiles_m) * MT, 0);
      bl.init(a, t, (next / a.tiles_m) * NT, 0);
      issue(cur ^ 1);
    }
    if (nk == 1) {
      if (pending) store_tile_f32_buf<LAYOUT, C, FUSE>(a, acc, pm0, pn0, wm, wn, hh, q);
      __builtin_amdgcn_sched_barrier(0);
      clear();
    }
    __builtin_amdgcn_sched_barrier(0);
    mma_stage_upto<C, KT>(acc, As0 + cur * C::A_STAGE, Bs0 + cur * C::B_STAGE, wm, wn, hh, q, last_kk);
    __builtin_amdgcn_sched_barrier(0);
    if (fetch) commit(cur ^ 1);
    stage_end();
    cur ^= 1;
    pm0 = m0;
    pn0 = n0;
    pending = true;
    if (!fetch) break;
    tile = next;
    m0 = (tile % a.tiles_m) * MT;
    n0 = (tile / a.tiles_m) * NT;
  }
  store_tile_f32_buf<LAYOUT, C, FUSE>(a, acc, pm0, pn0, wm, wn, hh, q);
}

template <int LAYOUT, int AM, int BM, bool FUSE, int TI>
constexpr KernelFn kernel_pt_at() {
  constexpr TileDesc d = kTiles[TI];
  if constexpr (d.m16 != 0) return nullptr;     // 16-row tiles: not built persistent
  else return &conv_igemm_f32_pt<LAYOUT, AM, BM, d.mt, d.nt, d.kt, d.wm, d.wn, FUSE>;
}

template <int LAYOUT, int AM, int BM, bool FUSE, int... TI>
KernelFn pick_tile_pt(int tile, std::integer_sequence<int, TI...>) {
  KernelFn fn = nullptr;
  ((fn = (tile == TI ? kernel_pt_at<LAYOUT, AM, BM, FUSE, TI>() : fn)), ...);
  return fn;
}

template <int LAYOUT, int AM, int BM, bool FUSE = false>
KernelFn kernel_pt_for_tile(int tile) {
  if (tile < 0 || tile >= kNumTiles) return nullptr;
  return pick_tile_pt<LAYOUT, AM, BM, FUSE>(tile, std::make_integer_sequence<int, kNumTiles>{});
}

// ------------------------------------------------------ 16-row tiles
// Layers with 16 or 48 output channels leave a half or a quarter of every
// 32x32 MFMA block idle.  Their tiles run on 16x16x4 MFMAs instead, with the
// operands staged in the 16x16-block LDS layout (as the fp64-accumulating
// kernel does).  16x16x4 fp32 accumulator layout: element e of lane (g, q)
// holds row 4*g + e, column q.
__device__ __forceinline__ constexpr int m16_row(int g, int e) { return 4 * g + e; }

template <int LAYOUT, int AM, int BM, int MT, int NT, int KT, int WM, int WN, class Store>
__device__ __forceinline__ void tile_product_f32m16(const KArgs& a, float* lds, int t, int tile, int kt0,
                                                    int nk, Store&& store) {
  using C = Cfg<MT, NT, KT, WM, WN, true>;
  const int tm = tile % a.tiles_m;
  const int tn = tile / a.tiles_m;
  const int m0 = tm * MT, n0 = tn * NT;
  const int kbeg = kt0 * KT;

  float* const As0 = lds;
  float* const Bs0 = lds + 2 * C::A_STAGE;
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, a.x_bytes);
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(a.w, a.w_bytes);

  typename ASel<LAYOUT, AM, C, MT, KT, BM>::type al;
  typename BSel<LAYOUT, BM, C, NT, KT>::type bl;
  al.init(a, t, m0, kbeg);
  bl.init(a, t, n0, kbeg);

  const int wave = t >> 6, lane = t & 63;
  const int wm = wave % WM, wn = wave / WM;
  const int g = lane >> 4, q = lane & 15;

  f32x4 acc[C::TM16][C::TN16];
#pragma unroll
  for (int i = 0; i < C::TM16; ++i)
#pragma unroll
    for (int j = 0; j < C::TN16; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  run_stages<C>(a, al, bl, As0, Bs0, nk, xr, wr, [&](const float* As, const float* Bs) {
    mma_stage16<C, KT>(acc, As, Bs, wm, wn, g, q);
  });
  store(acc, m0, n0, wm, wn, g, q);
}

// Work-groups [0, dp_tiles): whole tiles, stored to y (with the fused output
// stage when FUSE); the rest: one split piece each, whose tile-local partial
// sums (row-major mt x nt, fp32) the tail reduction adds up.  Runs crossing a
// tile boundary (stream-K) are not taken by these tiles.
template <int LAYOUT, int AM, int BM, int MT, int NT, int KT, int WM, int WN, bool FUSE>
__global__ __launch_bounds__(WM * WN * 64)
void conv_igemm_f32_m16(KArgs a) {
  using C = Cfg<MT, NT, KT, WM, WN, true>;
  __shared__ __attribute__((aligned(16))) float lds[C::LDS_FLOATS];

  int tile, kt0 = 0, nk = a.k_tiles, w = 0, rel = 0;
  const bool partial = (int)blockIdx.x >= a.dp_tiles;
  if (!partial) {
    tile = xcd_group(blockIdx.x, a.dp_tiles);
  } else {
    split_piece(a, blockIdx.x - a.dp_tiles, &w, &rel, &kt0, &nk);
    tile = a.dp_tiles + rel;
  }
  tile_product_f32m16<LAYOUT, AM, BM, MT, NT, KT, WM, WN>(
      a, lds, threadIdx.x, tile, kt0, nk,
      [&](f32x4 (&acc)[C::TM16][C::TN16], int m0, int n0, int wm, int wn, int g, int q) {
        if (partial) {
          float* const part = a.ws + tail_slot(w, rel) * (MT * NT);
#pragma unroll
          for (int j = 0; j < C::TN16; ++j) {
            const int col = wn * C::WTN + j * 16 + q;
#pragma unroll
            for (int i = 0; i < C::TM16; ++i)
#pragma unroll
              for (int e = 0; e < 4; ++e) part[(wm * C::WTM + i * 16 + m16_row(g, e)) * NT + col] = acc[i][j][e];
          }
          return;
        }
        float* const out = a.y;
#pragma unroll
        for (int j = 0; j < C::TN16; ++j) {
          const int n = n0 + wn * C::WTN + j * 16 + q;
          if (n >= a.Ng) continue;
          const int colbase = out_colbase<LAYOUT>(a, n);
#pragma unroll
          for (int i = 0; i < C::TM16; ++i)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const int row = m0 + wm * C::WTM + i * 16 + m16_row(g, e);
              if (row < a.Mg) {
                const int idx = colbase + row * a.mstride;
                if constexpr (FUSE) out[idx] = finish1(a, acc[i][j][e], idx);
                else out[idx] = acc[i][j][e];
              }
            }
        }
      });
}

template <int LAYOUT, int AM, int BM, bool FUSE, int TI>
constexpr KernelFn kernel_at() {
  constexpr TileDesc d = kTiles[TI];
  if constexpr (d.m16 != 0 && BM == kBVecNTapDma) return nullptr;   // not built: 16-row tiles stage through VGPRs
  else if constexpr (d.m16 != 0) return &conv_igemm_f32_m16<LAYOUT, AM, BM, d.mt, d.nt, d.kt, d.wm, d.wn, FUSE>;
  else return &conv_igemm_f32<LAYOUT, AM, BM, d.mt, d.nt, d.kt, d.wm, d.wn, FUSE>;
}

template <int LAYOUT, int AM, int BM, bool FUSE, int... TI>
KernelFn pick_tile(int tile, std::integer_sequence<int, TI...>) {
  KernelFn fn = nullptr;
  ((fn = (tile == TI ? kernel_at<LAYOUT, AM, BM, FUSE, TI>() : fn)), ...);
  return fn;
}

template <int LAYOUT, int AM, int BM, bool FUSE = false>
KernelFn kernel_for_tile(int tile) {
  if (tile < 0 || tile >= kNumTiles) return nullptr;
  return pick_tile<LAYOUT, AM, BM, FUSE>(tile, std::make_integer_sequence<int, kNumTiles>{});
}

// ------------------------------------------------- fp64-accumulating kernels
// Same operand staging and tile schedule as the fp32 kernels (fp32 tiles in
// LDS; whole tiles, then runs over the tail tiles); the MFMAs take the
// operands widened to fp64 and accumulate in fp64.  A whole tile rounds each
// output to fp32 once, at the store.  A piece stores its fp64 partial sums,
// which the tail reduction adds in fp64 and then rounds once, so the sum
// never leaves fp64 before that one rounding.
template <int LAYOUT, int AM, int BM, int MT, int NT, int KT, int WM, int WN, class Store>
__device__ __forceinline__ void tile_product_f64(const KArgs& a, float* lds, int t, int tile, int kt0,
                                                 int nk, Store&& store) {
  using C = Cfg<MT, NT, KT, WM, WN, true>;
  const int tm = tile % a.tiles_m;
  const int tn = tile / a.tiles_m;
  const int m0 = tm * MT, n0 = tn * NT;
  const int kbeg = kt0 * KT;

  float* const As0 = lds;
  float* const Bs0 = lds + 2 * C::A_STAGE;
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(a.x, a.x_bytes);
  const __amdgpu_buffer_rsrc_t wr = make_rsrc(a.w, a.w_bytes);

  typename ASel<LAYOUT, AM, C, MT, KT, BM>::type al;
  typename BSel<LAYOUT, BM, C, NT, KT>::type bl;
  al.init(a, t, m0, kbeg);
  bl.init(a, t, n0, kbeg);

  const int wave = t >> 6, lane = t & 63;
  const int wm = wave % WM, wn = wave / WM;
  const int g = lane >> 4, q = lane & 15;

  f64x4 acc[C::TM16][C::TN16];
#pragma unroll
  for (int i = 0; i < C::TM16; ++i)
#pragma unroll
    for (int j = 0; j < C::TN16; ++j) acc[i][j] = f64x4{0.0, 0.0, 0.0, 0.0};

  run_stages<C>(a, al, bl, As0, Bs0, nk, xr, wr, [&](const float* As, const float* Bs) {
    mma_stage64<C, KT>(acc, As, Bs, wm, wn, g, q);
  });
  store(acc, m0, n0, wm, wn, g, q);
}

// Work-groups [0, dp_tiles): whole tiles rounded to fp32 at the store; the
// rest: one split piece each (tail plans of the fp64 kernel are always
// split), stored as fp64 partials.  16x16 fp64 accumulator layout: element e
// of lane (g, q) holds row g + 4*e, column q.  A lane's four rows are not
// adjacent, so the stores are single elements (lanes g = 0..3 together cover
// four adjacent rows).
template <int LAYOUT, int AM, int BM, int MT, int NT, int KT, int WM, int WN>
__global__ __launch_bounds__(WM * WN * 64)
void conv_igemm_acc64(KArgs a) {
  using C = Cfg<MT, NT, KT, WM, WN, true>;
  __shared__ __attribute__((aligned(16))) float lds[C::LDS_FLOATS];

  int tile, kt0 = 0, nk = a.k_tiles, w = 0, rel = 0;
  const bool partial = (int)blockIdx.x >= a.dp_tiles;
  if (!partial) {
    tile = xcd_group(blockIdx.x, a.dp_tiles);
  } else {
    split_piece(a, blockIdx.x - a.dp_tiles, &w, &rel, &kt0, &nk);
    tile = a.dp_tiles + rel;
  }
  tile_product_f64<LAYOUT, AM, BM, MT, NT, KT, WM, WN>(
      a, lds, threadIdx.x, tile, kt0, nk,
      [&](f64x4 (&acc)[C::TM16][C::TN16], int m0, int n0, int wm, int wn, int g, int q) {
        if (partial) {
          // tile-local fp64 partial sums, row-major mt x nt, in the piece's slot
          double* const part = reinterpret_cast<double*>(a.ws) + tail_slot(w, rel) * (MT * NT);
#pragma unroll
          for (int j = 0; j < C::TN16; ++j) {
            const int col = wn * C::WTN + j * 16 + q;
#pragma unroll
            for (int i = 0; i < C::TM16; ++i)
#pragma unroll
              for (int e = 0; e < 4; ++e) part[(wm * C::WTM + i * 16 + g + 4 * e) * NT + col] = acc[i][j][e];
          }
          return;
        }
        float* const out = a.y;
#pragma unroll
        for (int j = 0; j < C::TN16; ++j) {
          const int n = n0 + wn * C::WTN + j * 16 + q;
          if (n >= a.Ng) continue;
          const int colbase = out_colbase<LAYOUT>(a, n);
#pragma unroll
          for (int i = 0; i < C::TM16; ++i)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const int row = m0 + wm * C::WTM + i * 16 + g + 4 * e;
              if (row < a.Mg) out[colbase + row * a.mstride] = (float)acc[i][j][e];
            }
        }
      });
}

template <int LAYOUT, int AM, int BM, int TI>
constexpr KernelFn kernel64_at() {
  constexpr TileDesc d = kTiles64[TI];
  return &conv_igemm_acc64<LAYOUT, AM, BM, d.mt, d.nt, d.kt, d.wm, d.wn>;
}

template <int LAYOUT, int AM, int BM, int... TI>
KernelFn pick_tile64(int tile, std::integer_sequence<int, TI...>) {
  KernelFn fn = nullptr;
  ((fn = (tile == TI ? kernel64_at<LAYOUT, AM, BM, TI>() : fn)), ...);
  return fn;
}

template <int LAYOUT, int AM, int BM>
KernelFn kernel64_for_tile(int tile) {
  if (tile < 0 || tile >= kNumTiles64) return nullptr;
  return pick_tile64<LAYOUT, AM, BM>(tile, std::make_integer_sequence<int, kNumTiles64>{});
}

}  // namespace mg3m
