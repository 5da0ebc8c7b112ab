// Implicit-GEMM forward convolution on fp32 MFMA for gfx950 (MI355X).
//
// The convolution of Eq. 1 (Sec. 2.1) is computed as the matrix product of
// Eq. 2 / Alg. 1 (Sec. 4.1.1), without materialising the patch matrix:
//
//   OUT[m][n] = sum_k A[m][k] * B[k][n]
//   m = output channel (Mg = OC)
//   n = (pixel, batch)  (Ng = B*outH*outW)
//   k = filter tap and input channel (Kg = IC*fltH*fltW)
//
// In the paper's HWCN storage (Sec. 4.1.1) the filter is already the dense
// Kg x OC matrix A^T (each FLT_mtx of Alg. 1 is one IC x OC slab of it, k
// ordered (fh, fw, ic)), and column n of B at row k is one element of the
// IN_mtx at pixel (ih, iw), so a k-slab of B is a gather of contiguous IN_mtx
// rows.  In NCHW the reduction runs in (ic, fh, fw) order.
//
// Mapping of the paper's design onto CDNA4:
//  * Multi-grained mapping (Sec. 4.1.2): the work-group tile (mt x nt) and the
//    split-K factor are picked per shape by the planner; small tiles play the
//    role of TB(1,1), wide single-operand-sharing tiles of TB(1,8), 2-D wave
//    grids of TB(8,8).
//  * On-chip sharing (Sec. 4.2, Eq. 4/5): the waves of a work-group share the
//    staged A and B tiles through LDS instead of register broadcasts.
//  * Filter reuse (Alg. 2): one staged A tile serves all nt columns.
//  * Double buffering (Alg. 3): two LDS stages; the next tile's global loads
//    are in flight while the MFMAs consume the current one.
//  * Register blocking (Sec. 4.4.1, Eq. 9): each wave holds a (mt/wm) x
//    (nt/wn) accumulator block as 32x32 MFMA blocks in AccVGPRs; each lane
//    reads one A and one B value per 4096-flop MFMA.
//  * Remainders (Sec. 4.4.2): edge tiles are zero-filled on load and masked
//    on store, instead of sixteen remainder kernels.
#include <hip/hip_runtime.h>

#include <string>
#include <utility>

#include "mg3m_internal.h"

namespace mg3m {

typedef float floatx16 __attribute__((ext_vector_type(16)));

template <int MT, int NT, int KT, int WM, int WN>
struct Cfg {
  static constexpr int T = WM * WN * 64;        // threads per work-group
  static constexpr int WTM = MT / WM;           // wave tile rows
  static constexpr int WTN = NT / WN;           // wave tile columns
  static constexpr int TM = WTM / 32;           // 32x32 MFMA blocks per wave, rows
  static constexpr int TN = WTN / 32;           // ... columns
  static constexpr int AS = lds_row_stride(MT);
  static constexpr int BS = lds_row_stride(NT);
  static constexpr int CS = lds_c_stride(NT);
  static constexpr int A_STAGE = KT * AS;
  static constexpr int B_STAGE = KT * BS;
  static constexpr int AB_FLOATS = 2 * A_STAGE + 2 * B_STAGE;
  static constexpr int C_FLOATS = MT * CS;
  static constexpr int LDS_FLOATS = AB_FLOATS > C_FLOATS ? AB_FLOATS : C_FLOATS;
  static constexpr int A_ELEMS = KT * MT / T;    // A elements each thread loads per stage
  static constexpr int B_ELEMS = KT * NT / T;
  static_assert(WTM % 32 == 0 && WTN % 32 == 0, "wave tile must be whole 32x32 blocks");
  static_assert(A_ELEMS % 4 == 0 && B_ELEMS % 4 == 0, "each thread loads whole 16-byte vectors");
  static_assert(T % (MT / 4) == 0 && T % (NT / 4) == 0, "vector columns must divide the threads");
  static_assert(KT % 4 == 0 && T % (KT / 4) == 0, "k vectors must divide the threads");
  static_assert(LDS_FLOATS * 4 == lds_bytes_for(TileDesc{MT, NT, KT, WM, WN}), "LDS size model");
};

__device__ __forceinline__ float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ void st4(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }

// Index of output element (m, n) in the layout's y array.
template <int LAYOUT>
__device__ __forceinline__ int out_index(const KArgs& a, int m, int n) {
  if constexpr (LAYOUT == kHWCN) {          // y[Ho][Wo][K][N], n = pix*N + b
    int pix = n / a.N, b = n - pix * a.N;
    return (pix * a.K + m) * a.N + b;
  } else {                                   // y[N][K][Ho][Wo], n = b*HoWo + pix
    int hw = a.Ho * a.Wo;
    int b = n / hw, pix = n - b * hw;
    return (b * a.K + m) * hw + pix;
  }
}

// ---------------------------------------------------------------- A (filter)
template <int LAYOUT, class C, int MT, int KT>
struct ALoader {
  static constexpr int NE = C::A_ELEMS;
  static constexpr int NV = NE / 4;
  float v[NE];
  int kbase;

  __device__ void init(int kbeg) { kbase = kbeg; }
  __device__ void advance() { kbase += KT; }

  __device__ void load(const KArgs& a, int t, int m0) {
    if (a.a_mode == kAVecM) {                // HWCN: A^T[k][m] = w[k*K + m], vectors along m
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        int vv = t + i * C::T;
        int m4 = vv % (MT / 4), kr = vv / (MT / 4);
        int k = kbase + kr, m = m0 + m4 * 4;
        float4 r = make_float4(0.f, 0.f, 0.f, 0.f);
        if (k < a.Kg && m < a.Mg) r = ld4(a.w + k * a.K + m);
        v[4 * i + 0] = r.x; v[4 * i + 1] = r.y; v[4 * i + 2] = r.z; v[4 * i + 3] = r.w;
      }
    } else if (a.a_mode == kAVecK) {         // NCHW: A[m][k] = w[m*Kg + k], vectors along k
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        int vv = t + i * C::T;
        int k4 = vv % (KT / 4), mm = vv / (KT / 4);
        int k = kbase + k4 * 4, m = m0 + mm;
        float4 r = make_float4(0.f, 0.f, 0.f, 0.f);
        if (k < a.Kg && m < a.Mg) r = ld4(a.w + m * a.Kg + k);
        v[4 * i + 0] = r.x; v[4 * i + 1] = r.y; v[4 * i + 2] = r.z; v[4 * i + 3] = r.w;
      }
    } else {
#pragma unroll
      for (int i = 0; i < NE; ++i) {
        int e = t + i * C::T;
        int m, kr;
        if constexpr (LAYOUT == kHWCN) { m = e % MT; kr = e / MT; }
        else { kr = e % KT; m = e / KT; }
        int k = kbase + kr, mg = m0 + m;
        float r = 0.f;
        if (k < a.Kg && mg < a.Mg)
          r = (LAYOUT == kHWCN) ? a.w[k * a.K + mg] : a.w[mg * a.Kg + k];
        v[i] = r;
      }
    }
  }

  __device__ void store(const KArgs& a, float* As, int t) const {
    if (a.a_mode == kAVecM) {
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        int vv = t + i * C::T;
        int m4 = vv % (MT / 4), kr = vv / (MT / 4);
        st4(As + kr * C::AS + m4 * 4, make_float4(v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]));
      }
    } else if (a.a_mode == kAVecK) {
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        int vv = t + i * C::T;
        int k4 = vv % (KT / 4), mm = vv / (KT / 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) As[(k4 * 4 + e) * C::AS + mm] = v[4 * i + e];
      }
    } else {
#pragma unroll
      for (int i = 0; i < NE; ++i) {
        int e = t + i * C::T;
        int m, kr;
        if constexpr (LAYOUT == kHWCN) { m = e % MT; kr = e / MT; }
        else { kr = e % KT; m = e / KT; }
        As[kr * C::AS + m] = v[i];
      }
    }
  }
};

// ------------------------------------------------------ B (input patches)
// Decompose a reduction index into (fh, fw, ic) for the layout's k order.
template <int LAYOUT>
__device__ __forceinline__ void split_k(const KArgs& a, int k, int& r, int& s, int& c) {
  if constexpr (LAYOUT == kHWCN) {           // k = (r*S + s)*C + c
    c = k % a.C; int rs = k / a.C; s = rs % a.S; r = rs / a.S;
  } else {                                   // k = (c*R + r)*S + s
    s = k % a.S; int cr = k / a.S; r = cr % a.R; c = cr / a.R;
  }
}

// HWCN, N % 4 == 0: each thread owns one 4-wide batch vector of one pixel
// (a fixed column) and walks KT*NT/(4T) rows of the tile.
template <class C, int NT, int KT>
struct BLoaderVecN {
  static constexpr int NV = C::B_ELEMS / 4;
  static constexpr int NC4 = NT / 4;
  static constexpr int RSTEP = C::T / NC4;
  int n4, ih0, iw0, bcol;
  bool col_ok;
  int k[NV], r[NV], s[NV], c[NV];
  float4 v[NV];

  __device__ void init(const KArgs& a, int t, int n0, int kbeg) {
    n4 = t % NC4;
    int n = n0 + n4 * 4;
    col_ok = n < a.Ng;
    int pix = n / a.N;
    bcol = n - pix * a.N;
    int ho = pix / a.Wo, wo = pix - ho * a.Wo;
    ih0 = ho * a.sh - a.ph;
    iw0 = wo * a.sw - a.pw;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      k[i] = kbeg + t / NC4 + i * RSTEP;
      split_k<kHWCN>(a, k[i], r[i], s[i], c[i]);
    }
  }
  __device__ void advance(const KArgs& a) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      k[i] += KT;
      c[i] += KT;
      while (c[i] >= a.C) {
        c[i] -= a.C;
        if (++s[i] == a.S) { s[i] = 0; ++r[i]; }
      }
    }
  }
  __device__ void load(const KArgs& a, int) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      int ih = ih0 + r[i], iw = iw0 + s[i];
      float4 val = make_float4(0.f, 0.f, 0.f, 0.f);
      if (col_ok && k[i] < a.Kg && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W)
        val = ld4(a.x + ((ih * a.W + iw) * a.C + c[i]) * a.N + bcol);
      v[i] = val;
    }
  }
  __device__ void store(float* Bs, int t) const {
#pragma unroll
    for (int i = 0; i < NV; ++i) st4(Bs + (t / NC4 + i * RSTEP) * C::BS + n4 * 4, v[i]);
  }
};

// HWCN, N == 1, C % 4 == 0: each thread owns one 4-deep channel vector (a
// fixed row group, one filter tap) and walks KT*NT/(4T) pixels.
template <class C, int NT, int KT>
struct BLoaderVecC {
  static constexpr int NV = C::B_ELEMS / 4;
  static constexpr int KV = KT / 4;
  static constexpr int NSTEP = C::T / KV;
  int k4, k, r, s, c;
  int ih0[NV], iw0[NV];
  bool col_ok[NV];
  float4 v[NV];

  __device__ void init(const KArgs& a, int t, int n0, int kbeg) {
    k4 = t % KV;
    k = kbeg + k4 * 4;
    split_k<kHWCN>(a, k, r, s, c);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      int n = n0 + t / KV + i * NSTEP;        // N == 1: n is the pixel
      col_ok[i] = n < a.Ng;
      int ho = n / a.Wo, wo = n - ho * a.Wo;
      ih0[i] = ho * a.sh - a.ph;
      iw0[i] = wo * a.sw - a.pw;
    }
  }
  __device__ void advance(const KArgs& a) {
    k += KT;
    c += KT;
    while (c >= a.C) {
      c -= a.C;
      if (++s == a.S) { s = 0; ++r; }
    }
  }
  __device__ void load(const KArgs& a, int) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      int ih = ih0[i] + r, iw = iw0[i] + s;
      float4 val = make_float4(0.f, 0.f, 0.f, 0.f);
      if (col_ok[i] && k < a.Kg && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W)
        val = ld4(a.x + (ih * a.W + iw) * a.C + c);
      v[i] = val;
    }
  }
  __device__ void store(float* Bs, int t) const {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      int n = t / KV + i * NSTEP;
      Bs[(k4 * 4 + 0) * C::BS + n] = v[i].x;
      Bs[(k4 * 4 + 1) * C::BS + n] = v[i].y;
      Bs[(k4 * 4 + 2) * C::BS + n] = v[i].z;
      Bs[(k4 * 4 + 3) * C::BS + n] = v[i].w;
    }
  }
};

// Any layout, any alignment: single elements, indices decomposed per stage.
template <int LAYOUT, class C, int NT, int KT>
struct BLoaderScalar {
  static constexpr int NE = C::B_ELEMS;
  int kbase, n0;
  float v[NE];

  __device__ void init(const KArgs& a, int t, int n0_, int kbeg) { kbase = kbeg; n0 = n0_; }
  __device__ void advance(const KArgs& a) { kbase += KT; }
  __device__ void load(const KArgs& a, int t) {
#pragma unroll
    for (int i = 0; i < NE; ++i) {
      int e = t + i * C::T;
      int n = n0 + e % NT, k = kbase + e / NT;
      float val = 0.f;
      if (n < a.Ng && k < a.Kg) {
        int r, s, c;
        split_k<LAYOUT>(a, k, r, s, c);
        int b, pix;
        if constexpr (LAYOUT == kHWCN) { pix = n / a.N; b = n - pix * a.N; }
        else { int hw = a.Ho * a.Wo; b = n / hw; pix = n - b * hw; }
        int ho = pix / a.Wo, wo = pix - ho * a.Wo;
        int ih = ho * a.sh - a.ph + r, iw = wo * a.sw - a.pw + s;
        if ((unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W) {
          int idx = (LAYOUT == kHWCN) ? ((ih * a.W + iw) * a.C + c) * a.N + b
                                      : ((b * a.C + c) * a.H + ih) * a.W + iw;
          val = a.x[idx];
        }
      }
      v[i] = val;
    }
  }
  __device__ void store(float* Bs, int t) const {
#pragma unroll
    for (int i = 0; i < NE; ++i) {
      int e = t + i * C::T;
      Bs[(e / NT) * C::BS + e % NT] = v[i];
    }
  }
};

template <int LAYOUT, int BMODE, class C, int NT, int KT>
struct BSel;
template <class C, int NT, int KT>
struct BSel<kHWCN, kBVecN, C, NT, KT> { using type = BLoaderVecN<C, NT, KT>; };
template <class C, int NT, int KT>
struct BSel<kHWCN, kBVecC, C, NT, KT> { using type = BLoaderVecC<C, NT, KT>; };
template <int LAYOUT, class C, int NT, int KT>
struct BSel<LAYOUT, kBScalar, C, NT, KT> { using type = BLoaderScalar<LAYOUT, C, NT, KT>; };

// ------------------------------------------------------------------ kernel
template <int LAYOUT, int BMODE, int MT, int NT, int KT, int WM, int WN>
__global__ __launch_bounds__(WM * WN * 64)
void conv_igemm_f32(KArgs a) {
  using C = Cfg<MT, NT, KT, WM, WN>;
  __shared__ __attribute__((aligned(16))) float lds[C::LDS_FLOATS];

  const int t = threadIdx.x;

  // Work-group -> tile.  Consecutive hardware work-group ids go to different
  // XCDs (round robin over 8); remap so that each XCD receives a contiguous
  // run of tiles, which share filter and halo input rows in its L2.
  int L = blockIdx.x;
  if (a.xcd_remap) {
    const int G = gridDim.x, q = G >> 3, r8 = G & 7, xcd = L & 7, loc = L >> 3;
    L = (xcd < r8) ? xcd * (q + 1) + loc : r8 * (q + 1) + (xcd - r8) * q + loc;
  }
  const int tm = L % a.tiles_m;
  const int rest = L / a.tiles_m;
  const int tn = rest % a.tiles_n;
  const int ks = rest / a.tiles_n;
  const int m0 = tm * MT, n0 = tn * NT;
  const int kt0 = ks * a.kps;
  const int nk = max(0, min(a.kps, a.k_tiles - kt0));
  const int kbeg = kt0 * KT;

  // Stage buffers: A stage i at lds + i*A_STAGE, B stage i after both A stages.
  float* const As0 = lds;
  float* const Bs0 = lds + 2 * C::A_STAGE;

  ALoader<LAYOUT, C, MT, KT> al;
  typename BSel<LAYOUT, BMODE, C, NT, KT>::type bl;
  al.init(kbeg);
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

  if (nk > 0) {
    al.load(a, t, m0);
    bl.load(a, t);
    al.store(a, As0, t);
    bl.store(Bs0, t);
  }
  __syncthreads();

  for (int it = 0; it < nk; ++it) {
    const int cur = it & 1;
    const bool more = it + 1 < nk;
    if (more) {
      al.advance();
      bl.advance(a);
      al.load(a, t, m0);
      bl.load(a, t);
    }
    const float* Ac = As0 + cur * C::A_STAGE + wm * C::WTM + q;
    const float* Bc = Bs0 + cur * C::B_STAGE + wn * C::WTN + q;
#pragma unroll
    for (int kk = 0; kk < KT; kk += 2) {
      float av[C::TM], bv[C::TN];
#pragma unroll
      for (int i = 0; i < C::TM; ++i) av[i] = Ac[(kk + hh) * C::AS + i * 32];
#pragma unroll
      for (int j = 0; j < C::TN; ++j) bv[j] = Bc[(kk + hh) * C::BS + j * 32];
#pragma unroll
      for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
      al.store(a, As0 + (cur ^ 1) * C::A_STAGE, t);
      bl.store(Bs0 + (cur ^ 1) * C::B_STAGE, t);
    }
    __syncthreads();
  }

  // Epilogue: stage the tile through LDS so that global stores are 16-byte
  // vectors along whichever axis is contiguous in the output layout.
  // 32x32 MFMA accumulator layout: register e of lane (hh, q) holds
  // row 8*(e/4) + 4*hh + e%4, column q of the block.
  float* Cs = lds;
#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        int row = wm * C::WTM + i * 32 + 8 * (e >> 2) + 4 * hh + (e & 3);
        int col = wn * C::WTN + j * 32 + q;
        Cs[row * C::CS + col] = acc[i][j][e];
      }
  __syncthreads();

  float* out = a.out + (long long)ks * a.out_split_stride;
  if (a.e_mode == kEVecN) {
    constexpr int NC4 = NT / 4, EV = MT * NT / (4 * C::T);
#pragma unroll
    for (int i = 0; i < EV; ++i) {
      int vv = t + i * C::T;
      int n4 = vv % NC4, mr = vv / NC4;
      int m = m0 + mr, n = n0 + n4 * 4;
      if (m < a.Mg && n < a.Ng) st4(out + out_index<LAYOUT>(a, m, n), ld4(Cs + mr * C::CS + n4 * 4));
    }
  } else if (a.e_mode == kEVecM) {
    constexpr int MC4 = MT / 4, EV = MT * NT / (4 * C::T);
#pragma unroll
    for (int i = 0; i < EV; ++i) {
      int vv = t + i * C::T;
      int m4 = vv % MC4, nc = vv / MC4;
      int m = m0 + m4 * 4, n = n0 + nc;
      if (m < a.Mg && n < a.Ng) {
        float4 val = make_float4(Cs[(m4 * 4 + 0) * C::CS + nc], Cs[(m4 * 4 + 1) * C::CS + nc],
                                 Cs[(m4 * 4 + 2) * C::CS + nc], Cs[(m4 * 4 + 3) * C::CS + nc]);
        st4(out + out_index<LAYOUT>(a, m, n), val);
      }
    }
  } else {
    constexpr int ES = MT * NT / C::T;
#pragma unroll 4
    for (int i = 0; i < ES; ++i) {
      int e = t + i * C::T;
      int nc = e % NT, mr = e / NT;
      int m = m0 + mr, n = n0 + nc;
      if (m < a.Mg && n < a.Ng) out[out_index<LAYOUT>(a, m, n)] = Cs[mr * C::CS + nc];
    }
  }
}

// Split-K reduction: y = sum over splits of the partials, in split order.
__global__ __launch_bounds__(256) void splitk_reduce_f32(const float* __restrict__ ws,
                                                         float* __restrict__ y, long long elems,
                                                         int split, int vec4) {
  long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (vec4) {
    long long e = i * 4;
    if (e >= elems) return;
    float4 s = ld4(ws + e);
    for (int p = 1; p < split; ++p) {
      float4 u = ld4(ws + (long long)p * elems + e);
      s.x += u.x; s.y += u.y; s.z += u.z; s.w += u.w;
    }
    st4(y + e, s);
  } else {
    if (i >= elems) return;
    float s = ws[i];
    for (int p = 1; p < split; ++p) s += ws[(long long)p * elems + i];
    y[i] = s;
  }
}

// ------------------------------------------------------------- dispatch
using KernelFn = void (*)(KArgs);

template <int LAYOUT, int BMODE, int TI>
constexpr KernelFn kernel_at() {
  constexpr TileDesc d = kTiles[TI];
  return &conv_igemm_f32<LAYOUT, BMODE, d.mt, d.nt, d.kt, d.wm, d.wn>;
}

template <int LAYOUT, int BMODE, int... TI>
constexpr void fill_row(KernelFn* row, std::integer_sequence<int, TI...>) {
  ((row[TI] = kernel_at<LAYOUT, BMODE, TI>()), ...);
}

struct KernelTable {
  KernelFn fn[2][kNumBModes][kNumTiles] = {};
  KernelTable() {
    auto seq = std::make_integer_sequence<int, kNumTiles>{};
    fill_row<kHWCN, kBVecN>(fn[kHWCN][kBVecN], seq);
    fill_row<kHWCN, kBVecC>(fn[kHWCN][kBVecC], seq);
    fill_row<kHWCN, kBScalar>(fn[kHWCN][kBScalar], seq);
    fill_row<kNCHW, kBScalar>(fn[kNCHW][kBScalar], seq);
  }
};

static const KernelTable& table() {
  static const KernelTable t;
  return t;
}

int launch_conv(const Plan& p, const KArgs& a, void* stream, std::string* err) {
  if (p.layout < 0 || p.layout > 1 || p.b_mode < 0 || p.b_mode >= kNumBModes || p.tile < 0 ||
      p.tile >= kNumTiles) {
    *err = "internal: plan out of range";
    return 7;
  }
  KernelFn fn = table().fn[p.layout][p.b_mode][p.tile];
  if (fn == nullptr) {
    *err = "internal: no kernel for this layout and loader mode";
    return 7;
  }
  if (p.grid < 1 || p.grid > 0x7fffffffLL) {
    *err = "internal: grid size out of range";
    return 7;
  }
  hipLaunchKernelGGL(fn, dim3((unsigned)p.grid), dim3(p.t.wm * p.t.wn * 64), 0,
                     (hipStream_t)stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    *err = std::string("kernel launch: ") + hipGetErrorString(e);
    return 8;
  }
  return 0;
}

int launch_splitk_reduce(const float* ws, float* y, long long elems, int split, bool vec4,
                         void* stream, std::string* err) {
  long long threads = vec4 ? (elems + 3) / 4 : elems;
  long long blocks = (threads + 255) / 256;
  if (blocks < 1 || blocks > 0x7fffffffLL) {
    *err = "internal: reduction grid out of range";
    return 7;
  }
  hipLaunchKernelGGL(splitk_reduce_f32, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream,
                     ws, y, elems, split, vec4 ? 1 : 0);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    *err = std::string("split-K reduction launch: ") + hipGetErrorString(e);
    return 8;
  }
  return 0;
}

}  // namespace mg3m
