/*
 * mg3m.h -- C ABI of the MI355X (gfx950) forward 2-D convolution library.
 *
 * The operation is the single-precision forward convolution of Eq. 1 of the
 * MG3MConv paper (Sec. 2.1), with the symbols of its Table 1:
 *
 *   OUT[b,oc,oh,ow] = sum_{ic,fh,fw} IN[b,ic,ih,iw] * FLT[oc,ic,fh,fw],
 *   ih = oh*stride + fh - pad,  iw = ow*stride + fw - pad,
 *
 * taps outside the input contributing nothing (zero padding; the skip rule
 * of Alg. 2, Sec. 4.3.1).  No filter flip (cross-correlation).  The output
 * size is outH = floor((inH + 2*pad - fltH)/stride) + 1, likewise outW.
 * It is computed as an implicit matrix multiplication (Sec. 4.1.1, Eq. 2,
 * Alg. 1): Mg = OC rows, Ng = B*outH*outW columns, Kg = IC*fltH*fltW depth,
 * on fp32 MFMA, with a per-shape tile / split-K plan standing in for the
 * paper's multi-grained thread-block mapping (Sec. 4.1.2).
 *
 * Symbols in the argument lists: N = B (batch), C = IC, K = OC, H,W =
 * inH,inW, R,S = fltH,fltW.
 *
 * Layouts (argument `layout`):
 *   MG3M_LAYOUT_HWCN (0): the paper's storage order (Sec. 4.1.1)
 *       x[H][W][C][N], w[R][S][C][K], y[Ho][Wo][K][N]  -- the tuned path
 *   MG3M_LAYOUT_NCHW (1): Eq. 1's index order
 *       x[N][C][H][W], w[K][C][R][S], y[N][K][Ho][Wo]
 * All tensors are dense, fp32, row-major in the order written.
 *
 * Pointers: x, w, y and workspace are DEVICE pointers on the current HIP
 * device; stream is a hipStream_t (NULL = the default stream).  Every
 * compute call is asynchronous and stream-ordered: it returns once the work
 * is queued.  The caller owns every buffer; the library never frees or keeps
 * a caller pointer.  y is overwritten (no accumulation, bias or activation).
 *
 * Errors: every entry point returns an mg3m_status.  Argument validation is
 * synchronous and happens before anything is launched, so a rejected call
 * writes nothing.  Checked: dimensions >= 1, stride >= 1, pad >= 0, a
 * non-empty output, non-NULL pointers, 4-byte aligned pointers, every tensor
 * at most 4 GiB - 64 bytes (the kernels use 32-bit byte offsets), y not
 * overlapping x or w, a known layout, a large enough workspace, a valid plan
 * override.  HIP launch failures return
 * MG3M_ERR_HIP with the HIP error text in mg3m_last_error(); setting the
 * environment variable MG3M_TEST_FAIL_LAUNCH=1 makes every convolution
 * launch fail that way (nothing is launched), for testing callers' error
 * paths.  No C++ exception crosses this interface.  Calls on different streams may run
 * concurrently from different host threads.
 *
 * Environment (read at each call that plans a shape):
 *   MG3M_FORCE_PLAN=<override>  applied wherever a call passes no override
 *       (plan NULL, and the plain entry points): the override syntax of
 *       conv2d_fwd_f32_ex.  A forced plan that does not apply to a shape
 *       fails that call with MG3M_ERR_PLAN, naming the variable.
 *   MG3M_LOG=1  prints each plan once to stderr, when the library first
 *       makes it for a shape, alignment and override.
 */
#ifndef MG3M_H
#define MG3M_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

enum mg3m_layout {
    MG3M_LAYOUT_HWCN = 0,
    MG3M_LAYOUT_NCHW = 1
};

enum mg3m_status {
    MG3M_OK = 0,
    MG3M_ERR_NULL = 1,        /* a required pointer is NULL */
    MG3M_ERR_SHAPE = 2,       /* a dimension < 1, stride < 1, pad < 0 or empty output */
    MG3M_ERR_LAYOUT = 3,      /* unknown layout */
    MG3M_ERR_TOO_LARGE = 4,   /* a tensor is larger than 4 GiB - 64 bytes */
    MG3M_ERR_ALIAS = 5,       /* y overlaps x or w */
    MG3M_ERR_WORKSPACE = 6,   /* workspace missing or too small for the plan */
    MG3M_ERR_PLAN = 7,        /* malformed or inapplicable plan override */
    MG3M_ERR_HIP = 8,         /* HIP runtime or launch error (see mg3m_last_error) */
    MG3M_ERR_ALIGN = 9,       /* a pointer is not 4-byte aligned */
    MG3M_ERR_ARG = 10         /* bad auxiliary argument (output buffer, length) */
};

/* Output size by the floor formula above.  Ho, Wo: host out-parameters.
 * Returns MG3M_OK or MG3M_ERR_SHAPE / MG3M_ERR_NULL. */
int conv2d_out_dims(int H, int W, int R, int S, int stride, int pad, int *Ho, int *Wo);

/* y = conv(x, w) in `layout`.  Plan chosen by the per-shape selector.  When
 * the plan shares the Kg reduction of some output tiles out among several
 * work-groups (all tiles, or only those left over after whole rounds of
 * work-groups; each work-group takes an equal run of their k-tiles, stream-K
 * fashion), the pieces' partial sums go to a workspace that the library keeps
 * for `stream` (one buffer per stream, reused by every later call there and
 * replaced by a larger one, stream-ordered, when a plan needs more; taken
 * from the library's stream-ordered pool for the stream's device; a call
 * being captured into a graph takes a pool block inside the graph instead;
 * see mg3m_trim_workspace_pool) and a second kernel
 * sums them in a fixed order, so results are
 * deterministic run to run.  NCHW plans with C a multiple of the plan's kt, K a multiple of 4,
 * a filter of more than one tap and stride_w 1 take the reduction tap-major: a
 * first kernel copies the filter to [R][S][C][K] in that workspace.  An NCHW
 * call may instead run as HWCN (the selector weighs both; see via= below):
 * x and the filter are copied to HWCN and [R][S][C][K] in the workspace, the
 * HWCN kernels write an HWCN copy of y there, and a last kernel writes y in
 * NCHW (applying the fused output stage, for conv2d_fwd_f32_fused). */
int conv2d_fwd_f32(const float *x, const float *w, float *y,
                   int N, int C, int H, int W, int K, int R, int S,
                   int stride, int pad, int layout, void *stream);

/* Bytes of workspace the plan for this shape needs: the piece partials when
 * tiles' reductions are shared out, plus, for NCHW plans taken tap-major (C a multiple of the
 * plan's kt, K a multiple of 4, R*S > 1, stride_w 1), a [R][S][C][K] copy of
 * the filter that the call makes first; 0 when neither applies.
 * plan: NULL for the selector's choice, or an override string (below).
 * bytes: host out-parameter. */
int conv2d_fwd_f32_workspace_bytes(int N, int C, int H, int W, int K, int R, int S,
                                   int stride, int pad, int layout,
                                   const char *plan, size_t *bytes);

/* As conv2d_fwd_f32, with a caller-owned device workspace (may be NULL when
 * the plan needs none; must be 16-byte aligned and at least
 * conv2d_fwd_f32_workspace_bytes() long otherwise) and an optional plan
 * override.  Override syntax: comma-separated key=value pairs,
 *   tile=<MT>x<NT>   one of the kernel tile shapes: 128x128, 64x256, 256x64,
 *                    64x128, 128x64, 64x64, 32x128, 32x64, 128x32, 64x32,
 *                    256x128, 128x256, 128x128 with kt=32, 16x64 (16x16x4
 *                    MFMAs; the selector takes it only when K mod 32 is 1..16),
 *                    and 64x64 with kt=32 (four 32x32 waves)
 *   via=hwcn|none    NCHW calls of the fp32 kernel: run as HWCN on copies of x, w and
 *                    y in the workspace (hwcn), or in NCHW (none); by default the
 *                    selector weighs both.  via=hwcn on HWCN or fp64 calls ->
 *                    MG3M_ERR_PLAN
 *   waves=<WM>x<WN>  the work-group's wave grid (1..8 each), to pick among tiles
 *                    of one shape (64x64 comes as 1x1 with kt=16 and 2x2 with
 *                    kt=32), so the tile, waves and kt of a plan string read back
 *                    as an override for the same tile
 *   kt=16|32         reduction depth staged per step (default 16 with a tile)
 *   split=<n>        share every tile's reduction out over n work-groups per tile
 *                    (1..64, clamped to the tile's k-tiles; 1 = no split)
 *   tail=<n>         the same for the tiles left over after whole rounds of resident
 *                    work-groups only (2..64); the other tiles run whole
 *   persist=<w>      every tile whole, computed by min(tiles, 256*w) work-groups that
 *                    each loop over tiles (1..16); the next tile's first loads and
 *                    MFMAs overlap the previous tile's output stores.  HWCN with the
 *                    batch-vector patch loaders (N and K multiples of 4, aligned
 *                    buffers) and 32x32x2-MFMA tiles only, else MG3M_ERR_PLAN
 *   dma=0|1          the one-tap HWCN loaders (HWCN, N and K multiples of 4, C a
 *                    multiple of kt, aligned buffers) load straight into LDS (1, the
 *                    default where it applies: 32x32x2-MFMA tiles of the fp32
 *                    kernel, persistent plans included) or stage through VGPRs (0);
 *                    dma=1 where it does not apply -> MG3M_ERR_PLAN
 *   sk=<g>           the left-over tiles' k-tiles dealt out to g work-groups in equal
 *                    runs (stream-K); g from the number of left-over tiles to their
 *                    k-tiles in total, else MG3M_ERR_PLAN.  Runs that span two tiles
 *                    need the one-tap HWCN loader (HWCN, N and K multiples of 4, C a
 *                    multiple of kt, aligned buffers) of this fp32 call and a
 *                    32x32x2-MFMA tile (not 16x64); other
 *                    shapes accept only g that cuts every left-over tile into equal
 *                    runs (a split), else MG3M_ERR_PLAN
 * e.g. "tile=128x128,kt=32,split=2".  At most one of split, tail, sk and persist.
 * Unknown keys or shapes -> MG3M_ERR_PLAN. */
int conv2d_fwd_f32_ex(const float *x, const float *w, float *y,
                      int N, int C, int H, int W, int K, int R, int S,
                      int stride, int pad, int layout,
                      void *workspace, size_t workspace_bytes,
                      const char *plan, void *stream);

/* Separate vertical and horizontal stride and padding (Table 1's stdH, stdW,
 * padH, padW).  Output size: Ho = floor((H + 2*pad_h - R)/stride_h) + 1,
 * Wo = floor((W + 2*pad_w - S)/stride_w) + 1.  Ho, Wo: host out-parameters.
 * Returns MG3M_OK or MG3M_ERR_SHAPE / MG3M_ERR_NULL / MG3M_ERR_TOO_LARGE. */
int conv2d_out_dims_hw(int H, int W, int R, int S, int stride_h, int stride_w,
                       int pad_h, int pad_w, int *Ho, int *Wo);

/* As conv2d_fwd_f32_ex with separate vertical and horizontal stride and
 * padding (everything else, including the workspace rules and the plan
 * override, is the same). */
int conv2d_fwd_f32_hw(const float *x, const float *w, float *y,
                      int N, int C, int H, int W, int K, int R, int S,
                      int stride_h, int stride_w, int pad_h, int pad_w, int layout,
                      void *workspace, size_t workspace_bytes,
                      const char *plan, void *stream);

/* Workspace bytes of conv2d_fwd_f32_hw's plan (host only). */
int conv2d_fwd_f32_hw_workspace_bytes(int N, int C, int H, int W, int K, int R, int S,
                                      int stride_h, int stride_w, int pad_h, int pad_w,
                                      int layout, const char *plan, size_t *bytes);

/* y = conv(x, w) with the numerics of the paper's kernel: fp32 operands,
 * every product and partial sum in fp64, and one round-to-nearest-even to
 * fp32 per output (Sec. 4.1.1, Alg. 2, which converts each staged tile to
 * double and computes in double).  Each output is therefore within one fp32
 * rounding of its fp64 sum.  On fp64 MFMA (half the fp32 peak).  Separate
 * vertical and horizontal stride and padding as in conv2d_fwd_f32_hw.  When
 * the plan shares out the reduction of some tiles, their pieces' fp64 partial
 * sums go to the workspace the library keeps for `stream` (as for
 * conv2d_fwd_f32) and a second kernel adds them
 * in a fixed order in fp64 before the one rounding, so results are
 * deterministic run to run.  plan: NULL, or an override with the keys of
 * conv2d_fwd_f32_ex: tile=<MT>x<NT> (one of 128x128, 64x256, 256x64,
 * 64x128, 128x64, 64x64, 32x64, 64x32), split=<n>, tail=<n>, sk=<g> (a split
 * only); kt other than 16 -> MG3M_ERR_PLAN.  Pointers, ownership, validation and errors as for
 * conv2d_fwd_f32. */
int conv2d_fwd_f32_acc64(const float *x, const float *w, float *y,
                         int N, int C, int H, int W, int K, int R, int S,
                         int stride_h, int stride_w, int pad_h, int pad_w, int layout,
                         const char *plan, void *stream);

/* The plan of conv2d_fwd_f32_acc64 for this shape, as text (host only; buffer
 * rules as conv2d_fwd_f32_plan_string). */
int conv2d_fwd_f32_acc64_plan_string(int N, int C, int H, int W, int K, int R, int S,
                                     int stride_h, int stride_w, int pad_h, int pad_w,
                                     int layout, const char *plan, char *buf, size_t len);

/* y = act(conv(x, w) + add): the convolution of conv2d_fwd_f32_hw with the
 * network's elementwise steps fused into its output stage (whole tiles store
 * the finished value; split tiles finish it in the reduction), so the
 * activation never makes an extra trip through HBM.  add: NULL, or a device
 * tensor with y's shape and layout (a residual connection); it may be y
 * itself (in place) but may not partly overlap it.  relu: 0 = none, 1 =
 * max(v, 0) with NaN kept.  Workspace, plan override and errors as for
 * conv2d_fwd_f32_hw (workspace size from conv2d_fwd_f32_hw_workspace_bytes). */
int conv2d_fwd_f32_fused(const float *x, const float *w, float *y, const float *add, int relu,
                         int N, int C, int H, int W, int K, int R, int S,
                         int stride_h, int stride_w, int pad_h, int pad_w, int layout,
                         void *workspace, size_t workspace_bytes,
                         const char *plan, void *stream);

/* Max pooling over R x S windows with stride and padding per axis, padded
 * taps ignored (the pooling layers of VGG, AlexNet and ResNet), in either
 * layout: x[H][W][C][N] -> y[Ho][Wo][C][N], or x[N][C][H][W] ->
 * y[N][C][Ho][Wo].  Ho, Wo by the convolution's floor formula.  Padding is
 * at most half the window on each axis, so every window holds an input.  A
 * NaN in a window gives NaN.  Device pointers, stream-ordered; errors as for
 * conv2d_fwd_f32 (MG3M_ERR_SHAPE also for padding over half the window). */
int maxpool2d_f32(const float *x, float *y, int N, int C, int H, int W, int R, int S,
                  int stride_h, int stride_w, int pad_h, int pad_w, int layout, void *stream);

/* Output size of maxpool2d_f32 (host only). */
int maxpool2d_out_dims(int H, int W, int R, int S, int stride_h, int stride_w,
                       int pad_h, int pad_w, int *Ho, int *Wo);

/* ---------------------------------------------------------------------------
 * Network executor: a chain of convolution and pooling layers run back to
 * back on the device (the convolution stacks of the real networks of
 * Sec. 5.2), activations kept in one device arena, all launches on one
 * stream, optionally replayed from a captured HIP graph.
 *
 * Activations are numbered: 0 is the network input, i >= 1 the output of
 * layer i-1; the last layer writes the caller's y.  A layer reads any earlier
 * activation, so branches and residual connections are expressed by `input`
 * and `add`. */
enum mg3m_op {
    MG3M_OP_CONV = 0,        /* y = act(conv(in, w) + add) */
    MG3M_OP_MAXPOOL = 1      /* y = maxpool(in) */
};

typedef struct mg3m_layer {
    int op;                  /* MG3M_OP_* */
    int input;               /* activation read (0 .. layer index) */
    int add;                 /* CONV: activation added before the ReLU (same shape as the output), -1 = none */
    int relu;                /* CONV: 1 = ReLU, 0 = none */
    int K;                   /* CONV: output channels */
    int R, S;                /* filter (CONV) or window (MAXPOOL) height and width */
    int stride, pad;         /* both axes */
    const float *w;          /* CONV: device filter in the network's layout (HWCN [R][S][C][K], NCHW [K][C][R][S]),
                                owned by the caller and kept alive while the network is used */
} mg3m_layer;

typedef struct mg3m_net mg3m_net;

/* Validate the chain for an input of N images of C x H x W, infer every
 * activation's shape, plan every convolution, and allocate (hipMalloc, on the
 * current device) one arena for the activations and one split-K workspace.
 * keep_all = 0: activations share arena space once no later layer reads
 * them (liveness); 1: every activation keeps its own space, for inspection.
 * On success *net is set; on failure nothing is allocated and the status
 * (MG3M_ERR_ARG for a bad layer list, _SHAPE, _LAYOUT, _TOO_LARGE, _HIP) is
 * returned with the failing layer in mg3m_last_error(). */
int mg3m_net_create(const mg3m_layer *layers, int n_layers, int N, int C, int H, int W,
                    int layout, int keep_all, mg3m_net **net);

/* Shape of activation id (0 .. n_layers) and, for 1 .. n_layers-1, its device
 * pointer in the arena (NULL for the input and the output, which the caller
 * owns).  Stored activations are HWCN ([H][W][C][N]) in every network: an
 * NCHW network runs its layers in HWCN and changes layout only for x, y and
 * its filters (copied once per forward pass).  Host only.  ptr may be NULL. */
int mg3m_net_activation(const mg3m_net *net, int id, int *C, int *H, int *W, const float **ptr);

/* Bytes of the activation arena (for an NCHW network including the HWCN
 * copies of its input and output) and of the workspace (the split-K partials
 * and, for an NCHW network, the [R][S][C][K] copies of its filters).  Host
 * only. */
int mg3m_net_memory(const mg3m_net *net, size_t *arena_bytes, size_t *workspace_bytes);

/* Run the whole chain: x (activation 0) -> y (the last activation), both
 * device tensors in the network's layout, on `stream` (NULL = default).
 * Calls on one network must not overlap (they share the arena). */
int mg3m_net_forward(mg3m_net *net, const float *x, float *y, void *stream);

/* As mg3m_net_forward, replayed from a HIP graph captured on the first call
 * (and again whenever x, y or stream differ from the captured ones).  stream
 * must not be the default stream (it cannot be captured): MG3M_ERR_ARG. */
int mg3m_net_forward_graph(mg3m_net *net, const float *x, float *y, void *stream);

/* Free the arena, the workspace and any captured graph (NULL is accepted). */
int mg3m_net_destroy(mg3m_net *net);

/* The plan the selector (or the override) picks for this shape, as text,
 * e.g. "tile=128x128,waves=2x2,kt=16,split=1,grid=1568,...".  Host only; no
 * HIP call.  buf: host buffer of `len` bytes, always NUL-terminated on
 * success; MG3M_ERR_ARG if it is too short. */
int conv2d_fwd_f32_plan_string(int N, int C, int H, int W, int K, int R, int S,
                               int stride, int pad, int layout, const char *plan,
                               char *buf, size_t len);

/* Numbers behind a plan, for tests and benchmarks.  Host only. */
typedef struct mg3m_plan_info {
    int mt, nt, kt;           /* work-group tile: rows (OC), columns (B*outH*outW), depth step */
    int waves_m, waves_n;     /* waves per work-group along rows / columns */
    int split;                /* tail work-groups per tail tile, rounded up (1 = no tail) */
    int k_tiles;              /* ceil(Kg / kt) */
    int k_tiles_per_wg;       /* most k-tiles one work-group computes */
    int dp_tiles;             /* tiles computed whole, one per work-group */
    int tail_tiles;           /* tiles whose reduction is shared out (their partials are summed) */
    int tail_wgs;             /* work-groups sharing the tail tiles' k-tiles in equal runs */
    int tiles_m, tiles_n;     /* ceil(Mg / mt), ceil(Ng / nt) */
    long long grid;           /* work-groups launched by the main kernel */
    long long Mg, Ng, Kg;     /* implicit-GEMM sizes */
    size_t workspace_bytes;
    int lds_bytes;            /* LDS per work-group */
    double pad_efficiency;    /* Mg*Ng*Kg / (padded tile volume), in (0, 1] */
    double est_us;            /* the selector's predicted time */
    int layout;               /* MG3M_LAYOUT_* */
    int a_mode, b_mode;       /* operand loader variant of the main kernel (its template arguments) */
    int e_mode;               /* epilogue store mode */
    int persistent;           /* 1: grid work-groups loop over the dp_tiles whole tiles */
    int via_hwcn;             /* 1: an NCHW call run as HWCN on copies in the workspace (layout, a_mode,
                                 b_mode and e_mode are then the HWCN kernels') */
} mg3m_plan_info;

int conv2d_fwd_f32_plan_info(int N, int C, int H, int W, int K, int R, int S,
                             int stride, int pad, int layout, const char *plan,
                             mg3m_plan_info *info);

/* Measurement hook for timing the main convolution kernel alone with HIP
 * events on the stream it runs on.  start and stop are hipEvent_t handles
 * created by the caller (both non-NULL), or both NULL to clear the hook.  The
 * next compute call (conv2d_fwd_f32, _ex, _hw or _acc64) made on the calling host thread
 * launches its main kernel with the two events attached (hipExtLaunchKernel):
 * start takes the kernel's start time and stop its end time -- before any
 * split-K reduction, with no separate event packets on the stream -- and then
 * clears the hook; a call rejected by validation leaves it set.  The library
 * keeps only the handles: both events must stay alive until that call has
 * returned (or the hook is cleared).  Returns MG3M_OK, or MG3M_ERR_ARG if
 * exactly one handle is NULL. */
int mg3m_time_next_kernel(void *start, void *stop);

/* Padding overhead of computing an M x N (x C deep) product in whole
 * mt x nt register blocks, as in the remainder analysis of Sec. 4.4.2:
 *   flop_overhead = (ceil(M/mt)*mt * ceil(N/nt)*nt) / (M*N) - 1
 *   data_overhead = (C*Mp + C*Np + Mp*Np) / (C*M + C*N + M*N) - 1
 * with Mp, Np the padded sizes.  Host only.  Out-parameters may not be NULL. */
int mg3m_padding_overhead(int M, int N, int C, int mt, int nt,
                          double *flop_overhead, double *data_overhead);

/* Fixed text for a status code (never NULL). */
const char *mg3m_status_string(int status);

/* Detail of the last error on the calling host thread ("" if none). */
const char *mg3m_last_error(void);

/* For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  The same
 * convolution as conv2d_fwd_f32 (same arguments, layouts, validation and
 * errors), but it allocates nothing: a plan's workspace (split-K partials,
 * the [R][S][C][K] filter copy of tap-major NCHW plans) lives in a fixed
 * device array of MG3M_NOALLOC_SCRATCH_BYTES that each device holds from the
 * first such call on it (the array's address is looked up then) until the
 * process ends.  The selector only considers plans whose workspace fits, so
 * a plan may differ from conv2d_fwd_f32's (results then differ by rounding
 * only, and agree exactly on small-integer data).  No plan fits only when a
 * tap-major NCHW filter copy alone exceeds the array: MG3M_ERR_WORKSPACE,
 * with nothing launched.  Nothing in the array needs clearing: every value a
 * call reads there was written earlier by the same call.  All calls on one
 * device share its array, so calls that may overlap in time on one device
 * (other streams, other host threads) race and must be ordered by the
 * caller; calls on one stream are ordered already. */
#define MG3M_NOALLOC_SCRATCH_BYTES (128ull * 1024ull * 1024ull)
int conv2d_fwd_f32_noalloc(const float *x, const float *w, float *y,
                           int N, int C, int H, int W, int K, int R, int S,
                           int stride, int pad, int layout, void *stream);

/* The workspaces that conv2d_fwd_f32 and conv2d_fwd_f32_acc64 take for
 * themselves come from one stream-ordered memory pool per device, which the
 * library creates at the first such call on that device.  Each stream that is
 * not being captured keeps one buffer from it (the largest its calls needed)
 * for its later calls, up to 32 streams per device; calls on further streams,
 * and captured calls, take a block per call and give it back on the stream.
 * Freed blocks stay in the pool for the next call (mapping tens of MB afresh
 * per call costs microseconds).  This call waits for the last call that used
 * each such buffer, gives the buffers back to their pools (the next call on
 * each stream takes a new one), then returns to the system every
 * block of every pool that no call is using, and keeps the pools for later
 * calls.  Blocking host call.  Returns MG3M_OK, or MG3M_ERR_HIP with the HIP
 * error text in mg3m_last_error(). */
int mg3m_trim_workspace_pool(void);

#ifdef __cplusplus
}
#endif

#endif /* MG3M_H */
