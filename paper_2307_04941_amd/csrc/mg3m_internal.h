// Private declarations shared by the planner (host C++), the ABI layer and
// the HIP kernels.  Not part of the public interface.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>

namespace mg3m {

enum Layout : int { kHWCN = 0, kNCHW = 1 };

// Filter (A operand) loader: 16-byte vectors along OC (HWCN, K % 4 == 0),
// along the reduction axis (NCHW, Kg % 4 == 0), or single elements.
enum AMode : int { kAVecM = 0, kAVecK = 1, kAScalar = 2 };
// Input-patch (B operand) gather: 16-byte vectors along the batch
// (HWCN, N % 4 == 0), along channels (HWCN, N == 1, C % 4 == 0), or single
// elements (any layout).
enum BMode : int { kBVecN = 0, kBVecC = 1, kBScalar = 2, kNumBModes = 3 };
// Epilogue store: 16-byte vectors along Ng (contiguous output runs of 4),
// along OC (HWCN, N == 1, K % 4 == 0), or single elements.
enum EMode : int { kEVecN = 0, kEVecM = 1, kEScalar = 2 };

struct ConvShape {
  int N, C, H, W, K, R, S;
  int sh, sw, ph, pw;
  int Ho, Wo;
  int layout;
  long long Mg, Ng, Kg;
};

// A kernel tile shape: one work-group computes an mt x nt block of the
// output matrix, stepping the reduction kt at a time, with wm x wn waves.
struct TileDesc {
  int mt, nt, kt, wm, wn;
};

// The tile menu.  Every entry is instantiated for each layout / loader mode.
constexpr int kNumTiles = 10;
inline constexpr TileDesc kTiles[kNumTiles] = {
    {128, 128, 16, 2, 2},   // 0: 2-D wave grid sharing both operands (TB(8,8)-like)
    {64, 256, 16, 1, 4},    // 1: four waves sharing one filter tile (TB(1,8)-like)
    {256, 64, 16, 4, 1},    // 2: four waves sharing one patch tile
    {64, 128, 16, 1, 2},    // 3
    {128, 64, 16, 2, 1},    // 4
    {64, 64, 16, 1, 1},     // 5: one wave per work-group (TB(1,1)-like)
    {32, 128, 16, 1, 2},    // 6
    {32, 64, 16, 1, 1},     // 7
    {128, 32, 16, 2, 1},    // 8
    {64, 32, 16, 1, 1},     // 9
};

// LDS row strides (floats) of the staged operand tiles.  The two half-waves of
// an MFMA operand read hit rows k and k+1; a stride of 32 (mod 64) floats keeps
// them on disjoint banks.
constexpr int lds_row_stride(int dim) { return dim % 64 == 0 ? dim + 32 : dim; }
constexpr int lds_c_stride(int nt) { return nt + 8; }   // epilogue staging
// LDS bytes per work-group: two stages of A and B tiles, reused for the
// epilogue's output tile.
constexpr int lds_bytes_for(const TileDesc& t) {
  const int ab = 2 * t.kt * lds_row_stride(t.mt) + 2 * t.kt * lds_row_stride(t.nt);
  const int c = t.mt * lds_c_stride(t.nt);
  return 4 * (ab > c ? ab : c);
}

struct Plan {
  int layout;
  int tile;                 // index into kTiles
  TileDesc t;
  int split;                // split-K factor
  int kps;                  // k-tiles per split
  int k_tiles;              // total k-tiles
  int tiles_m, tiles_n;
  long long grid;
  int a_mode, b_mode, e_mode;
  int xcd_remap;
  size_t ws_bytes;
  int lds_bytes;
  double pad_eff;
  double est_us;
};

// Kernel arguments (passed by value).
struct KArgs {
  const float* x;
  const float* w;
  float* out;               // y, or the split-K workspace
  int N, C, H, W, K, R, S;
  int sh, sw, ph, pw, Ho, Wo;
  int Mg, Ng, Kg;
  int tiles_m, tiles_n, kps, k_tiles;
  int a_mode, e_mode, xcd_remap;
  long long out_split_stride;   // elements between split-K partials
};

// Planner (host only, no HIP calls).  Returns 0 or an mg3m_status code and
// fills *err with a message on failure.
int make_shape(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
               int layout, ConvShape* s, std::string* err);
int make_plan(const ConvShape& s, const char* override_text, bool x16, bool w16, bool y16,
              Plan* p, std::string* err);
std::string plan_to_string(const ConvShape& s, const Plan& p);

// Kernel launchers (conv_igemm.hip).
int launch_conv(const Plan& p, const KArgs& a, void* stream, std::string* err);
int launch_splitk_reduce(const float* ws, float* y, long long elems, int split, bool vec4,
                         void* stream, std::string* err);

}  // namespace mg3m
