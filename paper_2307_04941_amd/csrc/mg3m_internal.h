// Private declarations shared by the planner (host C++), the ABI layer and
// the HIP kernels.  Not part of the public interface.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>

namespace mg3m {

enum Layout : int { kHWCN = 0, kNCHW = 1 };

// Operand loader variants.  Each is a separate kernel instantiation, so the
// main loop carries no run-time branch on the mode.
//   A (filter):        kAVecM   16-byte vectors along OC   (HWCN, K % 4 == 0)
//                      kAVecK   16-byte vectors along Kg   (NCHW, Kg % 4 == 0)
//                      kAScalar single elements            (any)
//   B (input patches): kBVecNTap 16-byte vectors along the batch, one filter tap
//                               per staged slab (HWCN, N % 4 == 0, C % kt == 0)
//                      kBVecN   16-byte vectors along the batch (HWCN, N % 4 == 0)
//                      kBVecC   16-byte vectors along channels  (HWCN, N == 1, C % 4 == 0)
//                      kBScalar single elements                 (HWCN, any)
//                      kBVecW   16-byte vectors along W where four columns of one
//                               output row allow it, else per-column elements (NCHW)
//                      kBVecWTap the same with one filter tap per staged slab of
//                               channels (NCHW, C % kt == 0; the filter is first
//                               copied to [R][S][C][K] and read by kAVecM)
enum AMode : int { kAVecM = 0, kAVecK = 1, kAScalar = 2 };
enum BMode : int { kBVecN = 0, kBVecC = 1, kBScalar = 2, kBVecNTap = 3, kBVecW = 4, kBVecWTap = 5,
                   kBVecNTapDma = 6 };
// The loader pairs that are instantiated.
enum Variant : int {
  kVarHwcnVecN = 0,     // HWCN, A vec-M, B vec-N
  kVarHwcnVecC = 1,     // HWCN, A vec-M, B vec-C
  kVarHwcnVecA = 2,     // HWCN, A vec-M, B scalar
  kVarHwcnScalar = 3,   // HWCN, A scalar, B scalar
  kVarNchwVecA = 4,     // NCHW, A vec-K, B vec-W
  kVarNchwScalar = 5,   // NCHW, A scalar, B vec-W
  kVarHwcnVecNTap = 6,  // HWCN, A vec-M, B vec-N with one tap per slab (the tuned path)
  kVarNchwTap = 7,      // NCHW, A vec-M on the [R][S][C][K] filter copy, B vec-W one tap per slab
  kVarHwcnVecNTapDma = 8,  // kVarHwcnVecNTap with both operands loaded straight into LDS
  kNumVariants = 9
};
// Epilogue store: single elements, or 16-byte vectors of four consecutive
// output channels (HWCN with N == 1 and K % 4 == 0, where they are contiguous).
enum EMode : int { kEElem = 0, kEVecM = 1 };

struct ConvShape {
  int N, C, H, W, K, R, S;
  int sh, sw, ph, pw;
  int Ho, Wo;
  int layout;
  long long Mg, Ng, Kg;
};

// A kernel tile shape: one work-group computes an mt x nt block of the
// output matrix, stepping the reduction kt at a time, with wm x wn waves.
// regs and eff feed the planner's cost model.  regs is the per-lane register
// count (VGPR + AGPR) of the tuned loader variant as compiled for gfx950: the
// .vgpr_count of its code object metadata.  A CPU test compares the two after
// every build, so a kernel change that moves the count fails until this
// table follows.  eff is the fraction of the fp32 MFMA peak the model charges
// the tile when a layer keeps every CU full.  The eff values started as measured full-occupancy
// efficiencies and were then fitted: every tile x schedule the planner can
// choose (10141 plans) was timed on MI355X over the VGG-16, ResNet-50,
// AlexNet/inception and scene-sweep layers, and eff was moved until the
// model's pick per layer came closest to the fastest measured plan (summed
// per-workload excess time 8.8% -> 4.8%; VGG-16 1.2% -> 0.5%).  128x32 keeps its
// measured value: a lower one traded it for 32x128 on ResNet-50 layers where
// interleaved re-timing showed 32x128 1-5% slower.  The 16-row tile's eff was
// fitted the same way after its plans were timed on those layers and on the
// 48 channel scenes (IC, OC from 16 to 1024 at N=128): the model then gives
// it exactly the K=16 layers (1.4-1.65x faster at N >= 32); with 48 output
// channels the 32-row tiles measured faster.
// m16: the tile runs on 16x16x4 fp32 MFMAs (16-row blocks; otherwise
// 32x32x2) and stages its operands in the 16x16-block LDS layout.
struct TileDesc {
  int mt, nt, kt, wm, wn;
  int regs;
  double eff;
  int m16 = 0;
  int forced_only = 0;   // reached only through a plan override, never by the selector
  // factor on eff for layers with more than one filter tap and more than two
  // kt-deep channel slabs per tap (1 = no difference)
  double eff_multitap = 1.0;
  // registers of the persistent kernel (conv_igemm_f32_pt) with the kBVecN,
  // kBVecNTap and kBVecNTapDma patch loaders, as compiled (0: not built)
  int regs_pt[3] = {0, 0, 0};
};

// The tile menu.  Every entry is instantiated for every loader variant.
constexpr int kNumTiles = 15;
inline constexpr TileDesc kTiles[kNumTiles] = {
    // mt,  nt, kt, wm, wn, regs, eff,  m16, forced, eff_multitap, regs_pt {vec_n, vec_n_tap, vec_n_tap_dma}
    {128, 128, 16, 2, 2, 116, 0.913, 0, 0, 1.0, {136, 121, 105}},  // 0: 2-D wave grid sharing both operands (TB(8,8)-like)
    {64, 256, 16, 1, 4, 116, 0.865, 0, 0, 1.0, {126, 125, 104}},   // 1: four waves sharing one filter tile (TB(1,8)-like)
    {256, 64, 16, 4, 1, 120, 0.891, 0, 0, 1.0, {134, 125, 104}},   // 2: four waves sharing one patch tile
    {64, 128, 16, 1, 2, 120, 0.890, 0, 0, 1.0, {161, 129, 104}},   // 3
    {128, 64, 16, 2, 1, 128, 0.823, 0, 0, 1.0, {145, 129, 104}},   // 4
    {64, 64, 16, 1, 1, 128, 0.740, 0, 0, 1.0, {163, 132, 100}},    // 5: one wave per work-group (TB(1,1)-like)
    {32, 128, 16, 1, 2, 88, 0.799, 0, 0, 1.0, {124, 91, 69}},     // 6
    {32, 64, 16, 1, 1, 92, 0.652, 0, 0, 1.0, {126, 93, 67}},      // 7
    {128, 32, 16, 2, 1, 88, 0.808, 0, 0, 1.0, {99, 90, 68}},     // 8
    {64, 32, 16, 1, 1, 92, 0.750, 0, 0, 1.0, {109, 92, 66}},      // 9
    {256, 128, 16, 4, 2, 111, 0.886, 0, 0, 1.0, {127, 119, 106}},  // 10: eight waves
    {128, 256, 16, 2, 4, 111, 0.832, 0, 0, 1.0, {120, 119, 106}},  // 11: eight waves
    {128, 128, 32, 2, 2, 140, 0.785, 0, 0, 1.0, {169, 137, 105}},  // 12: deeper reduction step
    {16, 64, 16, 1, 1, 88, 0.50, 1, 0, 1.0, {0, 0, 0}},          // 13: 16-row tile (16x16x4 MFMAs): 16 output channels
    {64, 64, 32, 2, 2, 60, 0.78, 0, 0, 0.9, {86, 71, 55}},        // 14: four 32x32 waves, deep step
};

// LDS row strides (floats) of the staged operand tiles.  An MFMA fragment
// read touches 2 (fp32 32x32x2) or 4 (fp64 16x16x4) consecutive k-rows at the
// same columns.  Rows whose length is a multiple of 64 floats are stored
// unpadded and XOR-swizzled in the kernels (bit 5 of the column flipped on odd
// rows for fp32, bits 4-5 by the row mod 4 for fp64), which puts those rows
// on disjoint banks.  32-float rows need nothing for fp32 (rows already 32
// banks apart) and 16 floats of padding for fp64.
constexpr int lds_row_stride(int dim) { return dim; }
constexpr int lds_row_stride64(int dim) { return (dim % 64 != 0 && dim % 32 == 0) ? dim + 16 : dim; }
// LDS bytes per work-group: two stages of the A and B tiles.
constexpr int lds_bytes_for(const TileDesc& t) {
  return 4 * (2 * t.kt * lds_row_stride(t.mt) + 2 * t.kt * lds_row_stride(t.nt));
}
constexpr int lds_bytes_for64(const TileDesc& t) {
  return 4 * (2 * t.kt * lds_row_stride64(t.mt) + 2 * t.kt * lds_row_stride64(t.nt));
}

// Tile menu of the fp64-accumulating kernel (fp32 operands, every product and
// partial sum in fp64, one rounding to fp32 at the store: the numerics of the
// paper's kernel, Sec. 4.1.1 and Alg. 2).  Split tiles keep fp64 partials.  regs
// as above.  eff is not a measured fraction here: it is fitted so that the
// cost model's pick per layer (tile and schedule) matches the fastest plan
// measured on MI355X over the VGG-16 and ResNet-50 layers (within 0.3% in
// total time).  On full layers the large tiles sustain 80-87% of the fp64
// MFMA peak, the one-wave tiles (64x64, 32x64, 64x32) 75-80%; the model's
// occupancy term already credits the latter with more resident waves.  The
// four-wave 64x64 tile (74 registers, 6 work-groups per CU) came later: its
// eff puts every ResNet-50 layer and VGG-16 conv2 and conv11-13 on it and
// keeps VGG-16's other layers on the large tiles (measured: ResNet-50's
// layers 2780 -> 2513 us in total, VGG-16's 29039 -> 28867 us).
constexpr int kNumTiles64 = 9;
inline constexpr TileDesc kTiles64[kNumTiles64] = {
    {128, 128, 16, 2, 2, 202, 0.925},  // 0
    {64, 256, 16, 1, 4, 206, 0.900},   // 1
    {256, 64, 16, 4, 1, 206, 0.800},   // 2
    {64, 128, 16, 1, 2, 210, 0.800},   // 3
    {128, 64, 16, 2, 1, 210, 0.800},   // 4
    {64, 64, 16, 1, 1, 212, 0.500},    // 5
    {32, 64, 16, 1, 2, 80, 0.500},     // 6
    {64, 32, 16, 2, 1, 78, 0.500},     // 7
    {64, 64, 16, 2, 2, 74, 0.64},      // 8: four 32x32 waves
};

// Largest tensor the kernels address: byte offsets are 32-bit and 0xFFFFFFC0
// is reserved as the out-of-range offset that reads as zero.
constexpr long long kMaxTensorBytes = 0xFFFFFFC0LL;

// How the output tiles are scheduled.  Tiles are numbered tm + tiles_m * tn.
// One launch: its first dp_tiles work-groups compute one whole tile each and
// write it to y; the remaining tail_wgs work-groups share the reduction steps
// of the other tail_tiles tiles (tail_tiles * k_tiles steps, tile by tile) in
// contiguous runs, each piece of a run (its part in one tile) writing
// tile-local partials to the workspace; a second kernel sums each tile's
// pieces in run order into y (deterministic).  Split plans (sk_s > 0) cut
// every tail tile into sk_s runs; stream-K plans (sk_s == 0) cut all the
// steps into tail_wgs equal runs, a run then spanning up to two tiles.  Pure
// data parallel: tail_tiles = 0.  Split-K: dp_tiles = 0.  Hybrid: dp_tiles is
// a whole number of rounds of resident work-groups and the leftover tiles'
// steps fill the last round evenly instead of leaving it mostly empty.
struct Plan {
  int layout;
  int acc64;                // 1: the fp64-accumulating kernel (tile indexes kTiles64)
  int tile;                 // index into kTiles (kTiles64 when acc64)
  TileDesc t;
  int k_tiles;              // ceil(Kg / kt)
  int tiles_m, tiles_n;
  int dp_tiles, tail_tiles;
  int tail_wgs;             // work-groups sharing the tail tiles' reduction steps (0 without a tail)
  int sk_s;                 // split plans: runs per tail tile (tail_wgs = sk_s * tail_tiles); stream-K: 0
  int sk_q, sk_r;           // steps per run: sk_q, one more for the first sk_r (of each tile when split)
  int split;                // tail work-groups per tail tile, rounded up (1 without a tail)
  int persist;              // 1: whole tiles only, grid work-groups looping over them (conv_igemm_f32_pt)
  long long grid;           // dp_tiles + tail_wgs (persistent plans: at most dp_tiles)
  int a_mode, b_mode, e_mode;
  int variant;
  size_t ws_bytes;          // workspace: the filter copy (wt_bytes), then the partials
  size_t wt_bytes;          // [R][S][C][K] copy of an NCHW filter (kVarNchwTap), 256-byte rounded; else 0
  int via_hwcn;             // 1: an NCHW call run as HWCN on copies of x, w and y in the workspace
  size_t via_bytes;         // those copies (x, then w, then y, each 256-byte rounded) at the workspace's front
  int lds_bytes;
  double pad_eff;
  double est_us;
};

// Kernel arguments (passed by value).
struct KArgs {
  const float* x;
  const float* w;
  float* y;
  float* ws;                // tile-local partials of the tail tiles (fp64 in the fp64-accumulating kernel)
  unsigned x_bytes, w_bytes;
  unsigned y_bytes;         // bytes of y (the persistent kernel stores through a buffer resource)
  int N, C, H, W, K, R, S;
  int sh, sw, ph, pw, Ho, Wo;
  int Mg, Ng, Kg;
  int tiles_m, k_tiles;
  int dp_tiles, tail_tiles;
  int sk_q, sk_r;           // tail runs (see Plan)
  int sk_s;                 // split plans: runs per tail tile; stream-K plans: 0
  int e_mode;
  int mstride;              // output elements between output channels m and m+1
  const float* add;         // added to each output before the activation (y's layout), or null
  int relu;                 // 1: y = max(y, 0) (NaN kept)
};

// Arguments of the tail reduction.
struct RArgs {
  const void* ws;           // fp32 partials, or fp64 ones when f64
  float* y;
  int mt, nt;               // tile shape
  int tiles_m, dp_tiles, tail_tiles;
  int k_tiles, sk_q, sk_r, sk_s;  // the tail runs, as in KArgs
  int layout, N, K, HoWo, Mg, Ng;
  int vec4;                 // four consecutive columns are contiguous in y
  int f64;                  // the partials are fp64
  const float* add;         // as in KArgs
  int relu;
};

// Arguments of max pooling.
struct PArgs {
  const float* x;
  float* y;
  int N, C, H, W, R, S;
  int sh, sw, ph, pw, Ho, Wo;
  int layout;
  int aligned16;            // x and y are 16-byte aligned
};

// A convolution's arguments as the entry points receive them, and which
// kernel family computes it (fp32 or fp64 accumulation).
struct ConvGeom {
  int N, C, H, W, K, R, S;
  int sh, sw, ph, pw;
  int layout;
  bool acc64;
  size_t ws_cap = SIZE_MAX;   // largest workspace a plan may use (the no-allocation entry point's scratch)
};

// Planner (host only, no HIP calls).  Returns 0 or an mg3m_status code and
// fills *err with a message on failure.
int make_shape(int N, int C, int H, int W, int K, int R, int S, int stride_h, int stride_w,
               int pad_h, int pad_w, int layout, ConvShape* s, std::string* err);
// ws_cap: only plans whose workspace fits are considered; when none does,
// MG3M_ERR_WORKSPACE.
int make_plan(const ConvShape& s, const char* override_text, bool acc64, bool x16, bool w16,
              bool y16, Plan* p, std::string* err, size_t ws_cap = SIZE_MAX);
std::string plan_to_string(const ConvShape& s, const Plan& p);

// Whether the fp32 kernel of a patch loader runs stream-K tail plans (runs
// spanning two tiles, taken in a loop).  Only the one-tap HWCN loader does
// so without losing occupancy on its whole tiles; the others, and the
// fp64-accumulating kernel, take split tail plans (one piece per run).
constexpr bool tail_runs_multi(int b_mode) { return b_mode == kBVecNTap || b_mode == kBVecNTapDma; }

// Kernel entry points by (variant, tile): conv_hwcn_*.hip, conv_nchw.hip.
using KernelFn = void (*)(KArgs);
KernelFn conv_kernel_hwcn_vecn(int tile);
KernelFn conv_kernel_hwcn_vecn_tap(int tile);
KernelFn conv_kernel_hwcn_vecn_tap_dma(int tile);   // conv_hwcn_vecn_tap_dma.hip
KernelFn conv_kernel_hwcn_vecn_tap_dma_fused(int tile);   // conv_hwcn_vecn_tap_dma_fused.hip
KernelFn conv_kernel_hwcn_vecc(int tile);
KernelFn conv_kernel_hwcn_veca(int tile);
KernelFn conv_kernel_hwcn_scalar(int tile);
KernelFn conv_kernel_nchw(int variant, int tile);
// The same with the fused output stage: conv_*_fused.hip.
KernelFn conv_kernel_hwcn_vecn_tap_fused(int tile);
KernelFn conv_kernel_hwcn_vecn_fused(int tile);
KernelFn conv_kernel_hwcn_other_fused(int variant, int tile);
KernelFn conv_kernel_nchw_fused(int variant, int tile);
KernelFn conv_kernel_nchw_tap(int tile);            // conv_nchw_tap.hip
// Persistent whole-tile kernels by (variant, tile): conv_hwcn_persist.hip;
// null where not built (other variants, 16-row tiles).
KernelFn conv_kernel_pt(int variant, int tile);
KernelFn conv_kernel_pt_fused(int variant, int tile);   // conv_hwcn_persist_fused.hip
constexpr bool persist_built(int variant, const TileDesc& t) {
  return (variant == kVarHwcnVecN || variant == kVarHwcnVecNTap || variant == kVarHwcnVecNTapDma) && t.m16 == 0;
}
KernelFn conv_kernel_nchw_tap_fused(int tile);      // conv_nchw_tap_fused.hip
// fp64-accumulating kernels by (variant, tile): conv_acc64_*.hip.
KernelFn conv_kernel64_hwcn_vecn_tap(int tile);
KernelFn conv_kernel64_hwcn(int variant, int tile);
KernelFn conv_kernel64_nchw(int variant, int tile);

// Kernel launchers (conv_launch.hip, pool.hip).
// start / stop: hipEvent_t handles (or null) that take the main kernel's own
// start and end times (mg3m_time_next_kernel).
int launch_conv(const Plan& p, const KArgs& a, void* stream, std::string* err, void* start = nullptr,
                void* stop = nullptr);
int launch_tail_reduce(const RArgs& r, void* stream, std::string* err);
int launch_maxpool(const PArgs& p, void* stream, std::string* err);
// wt[R][S][C][K] = w[K][C][R][S] (conv_launch.hip).
// out[b][c][a] = in[a][c][b] (layout.hip): NCHW -> HWCN with (A, Cm, B) =
// (N, C, H*W), HWCN -> NCHW with (H*W, C, N).  A and Cm at most 65535 tiles
// of 64 and 65535, else MG3M_ERR_TOO_LARGE.
// With add (same layout and size as out) and relu: out = act(in' + add), the
// fused output stage of an NCHW call run as HWCN.
int launch_swap_outer_inner(const float* in, float* out, int A, int Cm, int B, void* stream, std::string* err,
                            const float* add = nullptr, int relu = 0);
int launch_filter_to_rsck(const float* w, float* wt, int K, int C, int R, int S, void* stream,
                          std::string* err);
// A batch of layout changes in one launch (an NCHW network's filter copies):
// the caller fills in, out, A, Cm and B; prepare_swap_batch checks each
// change against the single launch's limits and fills in the rest (its
// 64 x 64 tiles along j = c * B + b, its first work-group, its access widths)
// and the batch's work-groups.  The launch takes the jobs in device memory.
struct SwapJob {
  const float* in;
  float* out;
  int A, Cm, B;
  unsigned tiles_j;   // 64-wide tiles along j
  unsigned tile0;     // the job's first work-group
  int vl, vs;         // 16-byte loads (J % 4 == 0, in aligned); 16-byte stores (A % 4 == 0, out aligned)
};
int prepare_swap_batch(SwapJob* jobs, int n, unsigned* tiles, std::string* err);
int launch_swap_outer_inner_batch(const SwapJob* dev_jobs, int n, unsigned tiles, void* stream, std::string* err);
// Two prepared jobs passed by value: no table in device memory.
int launch_swap_outer_inner_pair(const SwapJob jobs[2], unsigned tiles, void* stream, std::string* err);

// Shared by the C entry points and the network executor (abi.cpp): validate,
// plan and launch one convolution (y = act(conv + add)).  own_workspace: take
// a split plan's partials from the library's stream-ordered pool for the
// stream's device (allocated and freed on `stream`) instead of `workspace`.  Returns an mg3m_status and records the message for
// mg3m_last_error().
int conv_run(const float* x, const float* w, float* y, const ConvGeom& g, void* workspace,
             size_t workspace_bytes, bool own_workspace, const char* plan, const float* add, int relu,
             void* stream);
int conv_plan(const ConvGeom& g, const char* plan, ConvShape* s, Plan* p);   // host only
// Validate and launch one max pooling; pads at most half the window.
int maxpool_run(const float* x, float* y, int N, int C, int H, int W, int R, int S, int sh, int sw,
                int ph, int pw, int layout, void* stream);
int maxpool_dims(int H, int W, int R, int S, int sh, int sw, int ph, int pw, int* Ho, int* Wo,
                 std::string* err);
// Record a status and message for mg3m_last_error() (calling thread); returns status.
int set_error(int status, const std::string& msg);
void clear_error();

}  // namespace mg3m
