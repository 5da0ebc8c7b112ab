/*
 * The C ABI used from plain C, with no Python and no torch: HIP runtime calls
 * for memory and streams, include/mg3m.h for the convolution.  Built by the
 * package build (paper_2307_04941_amd/debug/c_abi_gpu) and run by
 * tests/test_c_abi_gpu.py on a GPU.
 *
 * Small-integer data (x, w in {-2..2}) makes every partial sum an integer far
 * below 2^24, so fp32 is exact in any order: each output must equal the sum
 * of Eq. 1 computed here with integer arithmetic, bit for bit.  Checked: the
 * plain call on the default stream and on a created stream, a forced split
 * plan with a caller workspace, the entry point that allocates nothing, and
 * validation errors that are reported before anything is launched.
 * Prints "c abi ok" and exits 0, or names the first failure and exits 1.
 */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "mg3m.h"

#define N 4
#define C 32
#define H 13
#define W 11
#define K 36
#define R 3
#define S 3
#define STRIDE 1
#define PAD 1

static int fails = 0;

#define EXPECT(cond, ...)            \
  do {                               \
    if (!(cond)) {                   \
      fprintf(stderr, __VA_ARGS__);  \
      fputc('\n', stderr);           \
      ++fails;                       \
    }                                \
  } while (0)

#define HIP(call)                                                                    \
  do {                                                                               \
    hipError_t e_ = (call);                                                          \
    if (e_ != hipSuccess) {                                                          \
      fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_));            \
      exit(1);                                                                       \
    }                                                                                \
  } while (0)

/* splitmix64: a small seeded generator for the test data */
static uint64_t rng_state = 20231202u;
static int next_small(void) {
  uint64_t z = (rng_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  z ^= z >> 31;
  return (int)(z % 5) - 2;
}

/* HWCN: x[h][w][c][n], w[r][s][c][k], y[ho][wo][k][n] */
static void reference(const int* x, const int* w, long long* y, int Ho, int Wo) {
  for (int ho = 0; ho < Ho; ++ho)
    for (int wo = 0; wo < Wo; ++wo)
      for (int k = 0; k < K; ++k)
        for (int n = 0; n < N; ++n) {
          long long acc = 0;
          for (int c = 0; c < C; ++c)
            for (int r = 0; r < R; ++r)
              for (int s = 0; s < S; ++s) {
                const int ih = ho * STRIDE - PAD + r, iw = wo * STRIDE - PAD + s;
                if (ih < 0 || ih >= H || iw < 0 || iw >= W) continue;
                acc += (long long)x[((ih * W + iw) * C + c) * N + n] * w[((r * S + s) * C + c) * K + k];
              }
          y[((ho * Wo + wo) * K + k) * N + n] = acc;
        }
}

static void check(const char* what, const float* got, const long long* ref, size_t n) {
  for (size_t i = 0; i < n; ++i)
    if (got[i] != (float)ref[i]) {
      EXPECT(0, "%s: output %zu is %.1f, expected %lld", what, i, got[i], ref[i]);
      return;
    }
}

int main(void) {
  int Ho = 0, Wo = 0;
  EXPECT(conv2d_out_dims(H, W, R, S, STRIDE, PAD, &Ho, &Wo) == MG3M_OK && Ho == 13 && Wo == 11,
         "conv2d_out_dims: %d x %d", Ho, Wo);
  const size_t nx = (size_t)N * C * H * W, nw = (size_t)K * C * R * S, ny = (size_t)N * K * Ho * Wo;
  int* xi = malloc(nx * sizeof(int));
  int* wi = malloc(nw * sizeof(int));
  float* xf = malloc(nx * sizeof(float));
  float* wf = malloc(nw * sizeof(float));
  float* yf = malloc(ny * sizeof(float));
  long long* ref = malloc(ny * sizeof(long long));
  if (!xi || !wi || !xf || !wf || !yf || !ref) return 1;
  for (size_t i = 0; i < nx; ++i) xf[i] = (float)(xi[i] = next_small());
  for (size_t i = 0; i < nw; ++i) wf[i] = (float)(wi[i] = next_small());
  reference(xi, wi, ref, Ho, Wo);

  float *dx, *dw, *dy;
  HIP(hipMalloc((void**)&dx, nx * sizeof(float)));
  HIP(hipMalloc((void**)&dw, nw * sizeof(float)));
  HIP(hipMalloc((void**)&dy, ny * sizeof(float)));
  HIP(hipMemcpy(dx, xf, nx * sizeof(float), hipMemcpyHostToDevice));
  HIP(hipMemcpy(dw, wf, nw * sizeof(float), hipMemcpyHostToDevice));

  /* the selector's plan on the default stream */
  HIP(hipMemset(dy, 0xFF, ny * sizeof(float)));
  int rc = conv2d_fwd_f32(dx, dw, dy, N, C, H, W, K, R, S, STRIDE, PAD, MG3M_LAYOUT_HWCN, NULL);
  EXPECT(rc == MG3M_OK, "conv2d_fwd_f32: %s (%s)", mg3m_status_string(rc), mg3m_last_error());
  HIP(hipDeviceSynchronize());
  HIP(hipMemcpy(yf, dy, ny * sizeof(float), hipMemcpyDeviceToHost));
  check("conv2d_fwd_f32, default stream", yf, ref, ny);

  /* a created stream */
  hipStream_t st;
  HIP(hipStreamCreate(&st));
  HIP(hipMemsetAsync(dy, 0xFF, ny * sizeof(float), st));
  rc = conv2d_fwd_f32(dx, dw, dy, N, C, H, W, K, R, S, STRIDE, PAD, MG3M_LAYOUT_HWCN, st);
  EXPECT(rc == MG3M_OK, "conv2d_fwd_f32 on a stream: %s (%s)", mg3m_status_string(rc), mg3m_last_error());
  HIP(hipStreamSynchronize(st));
  HIP(hipMemcpy(yf, dy, ny * sizeof(float), hipMemcpyDeviceToHost));
  check("conv2d_fwd_f32, created stream", yf, ref, ny);

  /* a forced split plan with a caller workspace */
  const char* plan = "tile=64x64,split=3";
  size_t wsb = 0;
  rc = conv2d_fwd_f32_workspace_bytes(N, C, H, W, K, R, S, STRIDE, PAD, MG3M_LAYOUT_HWCN, plan, &wsb);
  EXPECT(rc == MG3M_OK && wsb > 0, "workspace_bytes: %s, %zu bytes", mg3m_status_string(rc), wsb);
  void* dws = NULL;
  HIP(hipMalloc(&dws, wsb > 0 ? wsb : 16));
  char text[512];
  rc = conv2d_fwd_f32_plan_string(N, C, H, W, K, R, S, STRIDE, PAD, MG3M_LAYOUT_HWCN, plan, text, sizeof text);
  EXPECT(rc == MG3M_OK && strncmp(text, "tile=64x64,", 11) == 0 && strstr(text, "split=3") != NULL,
         "plan_string: %s", text);
  HIP(hipMemsetAsync(dy, 0xFF, ny * sizeof(float), st));
  rc = conv2d_fwd_f32_ex(dx, dw, dy, N, C, H, W, K, R, S, STRIDE, PAD, MG3M_LAYOUT_HWCN, dws, wsb, plan, st);
  EXPECT(rc == MG3M_OK, "conv2d_fwd_f32_ex: %s (%s)", mg3m_status_string(rc), mg3m_last_error());
  HIP(hipStreamSynchronize(st));
  HIP(hipMemcpy(yf, dy, ny * sizeof(float), hipMemcpyDeviceToHost));
  check("conv2d_fwd_f32_ex, tile=64x64,split=3", yf, ref, ny);

  /* the entry point that allocates nothing */
  HIP(hipMemsetAsync(dy, 0xFF, ny * sizeof(float), st));
  rc = conv2d_fwd_f32_noalloc(dx, dw, dy, N, C, H, W, K, R, S, STRIDE, PAD, MG3M_LAYOUT_HWCN, st);
  EXPECT(rc == MG3M_OK, "conv2d_fwd_f32_noalloc: %s (%s)", mg3m_status_string(rc), mg3m_last_error());
  HIP(hipStreamSynchronize(st));
  HIP(hipMemcpy(yf, dy, ny * sizeof(float), hipMemcpyDeviceToHost));
  check("conv2d_fwd_f32_noalloc", yf, ref, ny);

  /* validation: reported before anything is launched, y untouched */
  HIP(hipMemset(dy, 0, ny * sizeof(float)));
  rc = conv2d_fwd_f32(NULL, dw, dy, N, C, H, W, K, R, S, STRIDE, PAD, MG3M_LAYOUT_HWCN, st);
  EXPECT(rc == MG3M_ERR_NULL, "NULL x: %s", mg3m_status_string(rc));
  rc = conv2d_fwd_f32(dx, dw, dy, N, C, H, W, K, R, S, STRIDE, PAD, 7, st);
  EXPECT(rc == MG3M_ERR_LAYOUT, "bad layout: %s", mg3m_status_string(rc));
  rc = conv2d_fwd_f32(dx, dw, dy, N, C, 1, 1, K, R, S, 1, 0, MG3M_LAYOUT_HWCN, st);
  EXPECT(rc == MG3M_ERR_SHAPE, "empty output: %s", mg3m_status_string(rc));
  rc = conv2d_fwd_f32(dx, dw, dx, N, C, H, W, K, R, S, STRIDE, PAD, MG3M_LAYOUT_HWCN, st);
  EXPECT(rc == MG3M_ERR_ALIAS, "y over x: %s", mg3m_status_string(rc));
  rc = conv2d_fwd_f32_ex(dx, dw, dy, N, C, H, W, K, R, S, STRIDE, PAD, MG3M_LAYOUT_HWCN, dws, 4, plan, st);
  EXPECT(rc == MG3M_ERR_WORKSPACE, "short workspace: %s", mg3m_status_string(rc));
  rc = conv2d_fwd_f32_ex(dx, dw, dy, N, C, H, W, K, R, S, STRIDE, PAD, MG3M_LAYOUT_HWCN, dws, wsb,
                         "tile=48x48", st);
  EXPECT(rc == MG3M_ERR_PLAN, "bad plan: %s", mg3m_status_string(rc));
  HIP(hipStreamSynchronize(st));
  HIP(hipMemcpy(yf, dy, ny * sizeof(float), hipMemcpyDeviceToHost));
  for (size_t i = 0; i < ny; ++i)
    if (yf[i] != 0.0f) {
      EXPECT(0, "a rejected call wrote output %zu", i);
      break;
    }

  HIP(hipStreamDestroy(st));
  HIP(hipFree(dws));
  HIP(hipFree(dx));
  HIP(hipFree(dw));
  HIP(hipFree(dy));
  free(xi); free(wi); free(xf); free(wf); free(yf); free(ref);
  if (fails) {
    fprintf(stderr, "c abi: %d failure(s)\n", fails);
    return 1;
  }
  printf("c abi ok\n");
  return 0;
}
