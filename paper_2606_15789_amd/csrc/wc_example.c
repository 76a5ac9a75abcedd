/* wc_example.c -- libwc used from plain C: no Python, no PyTorch.
 *
 * Device memory comes from hipMalloc, the blob from wc_encode on the host.
 * The program decodes a bf16 matrix on the GPU (wc_decode) and checks it
 * byte for byte.  It then multiplies the same weights, stored as 16-row
 * column-block tiles, by one row of activations without ever writing them out
 * (wc_gemv), and checks y against an fp64 dot product within the fp32
 * summation bound.  Exit status 0 on success.
 *
 * Built next to libwc.so by the package's build; run as ./wc_example.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../../include/wc.h"

#define ROWS 256
#define COLS 2048

static int fail(const char* what, int code) {
  fprintf(stderr, "wc_example: %s failed (%d)\n", what, code);
  return 1;
}

/* bf16 storage word of a float, round to nearest even */
static uint16_t bf16_of(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

static double value_of(uint16_t h) {
  const uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

/* roughly Normal(0, sigma): a sum of 12 uniforms from a 64-bit LCG */
static uint64_t lcg = 0x853C49E6748FEA9Bull;
static float normalish(float sigma) {
  float s = 0.0f;
  for (int i = 0; i < 12; i++) {
    lcg = lcg * 6364136223846793005ull + 1442695040888963407ull;
    s += (float)(lcg >> 40) / 16777216.0f;
  }
  return sigma * (s - 6.0f);
}

int main(void) {
  const uint64_t n = (uint64_t)ROWS * COLS, nbytes = 2 * n;
  uint16_t* w = malloc(nbytes);
  uint16_t* back = malloc(nbytes);
  uint16_t x[COLS];
  float y[ROWS];
  if (!w || !back) return fail("malloc", 0);
  for (uint64_t i = 0; i < n; i++) w[i] = bf16_of(normalish(0.02f));
  for (int k = 0; k < COLS; k++) x[k] = bf16_of(normalish(1.0f));

  /* 1. decode: 64 KiB byte-run chunks */
  const wc_tensor t = {w, nbytes, WC_BF16, 0, ROWS, COLS};
  wc_params p = {65536, 64, 12, 0, 0, 0, WC_CODEBOOK_TENSOR, WC_TILE_ROWS};
  wc_blob* blob = NULL;
  wc_status rc = wc_encode(&t, 1, &p, &blob);
  if (rc != WC_OK) return fail("wc_encode", rc);
  wc_stats st;
  rc = wc_analyze(&t, &st);
  if (rc != WC_OK) return fail("wc_analyze", rc);

  void *dblob = NULL, *dout = NULL, *dx = NULL, *dy = NULL;
  int32_t* derr = NULL;
  if (hipMalloc(&dblob, blob->size) != hipSuccess || hipMalloc(&dout, nbytes) != hipSuccess ||
      hipMalloc((void**)&derr, 4) != hipSuccess)
    return fail("hipMalloc", 0);
  if (hipMemcpy(dblob, blob->data, blob->size, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemset(derr, 0, 4) != hipSuccess)
    return fail("hipMemcpy", 0);
  void* dst[1] = {dout};
  rc = wc_decode(blob, dblob, dst, 1, NULL, derr);
  if (rc != WC_OK) return fail("wc_decode", rc);
  int32_t err = -1;
  if (hipDeviceSynchronize() != hipSuccess ||
      hipMemcpy(back, dout, nbytes, hipMemcpyDeviceToHost) != hipSuccess ||
      hipMemcpy(&err, derr, 4, hipMemcpyDeviceToHost) != hipSuccess)
    return fail("hipMemcpy back", 0);
  if (err != 0) return fail("device error bits", err);
  if (memcmp(back, w, nbytes)) return fail("decoded bytes differ", 0);
  printf("wc_example: decoded %llu bf16 bit-exact; blob %llu bytes, %.4f x smaller, %.3f %% over "
         "the order-0 bound\n",
         (unsigned long long)n, (unsigned long long)blob->size, (double)nbytes / blob->size,
         100.0 * ((double)blob->size / st.bound_bytes - 1.0));
  wc_free(blob);
  hipFree(dblob);

  /* 2. fused decode-GEMV: 16-row column-block tiles of 16 x 2048 */
  p.tile_rows = 16;
  p.tile_cols = 2048;
  p.tile_order = WC_TILE_COLUMN_BLOCKS;
  rc = wc_encode(&t, 1, &p, &blob);
  if (rc != WC_OK) return fail("wc_encode (tiles)", rc);
  if (hipMalloc(&dblob, blob->size) != hipSuccess || hipMalloc(&dx, sizeof x) != hipSuccess ||
      hipMalloc(&dy, sizeof y) != hipSuccess)
    return fail("hipMalloc", 0);
  if (hipMemcpy(dblob, blob->data, blob->size, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(dx, x, sizeof x, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemset(dy, 0, sizeof y) != hipSuccess || hipMemset(derr, 0, 4) != hipSuccess)
    return fail("hipMemcpy", 0);
  const uint32_t tensor = 0;
  const void* xs[1] = {dx};
  float* ys[1] = {dy};
  rc = wc_gemv(blob, dblob, 1, &tensor, xs, 1, ys, NULL, derr);
  if (rc != WC_OK) return fail("wc_gemv", rc);
  if (hipDeviceSynchronize() != hipSuccess ||
      hipMemcpy(y, dy, sizeof y, hipMemcpyDeviceToHost) != hipSuccess ||
      hipMemcpy(&err, derr, 4, hipMemcpyDeviceToHost) != hipSuccess)
    return fail("hipMemcpy back", 0);
  if (err != 0) return fail("device error bits (gemv)", err);
  double worst = 0.0;
  for (int r = 0; r < ROWS; r++) {
    double s = 0.0, a = 0.0;
    for (int k = 0; k < COLS; k++) {
      const double q = value_of(x[k]) * value_of(w[(uint64_t)r * COLS + k]);
      s += q;
      a += fabs(q);
    }
    /* fp32 sums of exact bf16 products: at most COLS roundings of 2^-24 */
    const double bound = 2.0 * COLS * ldexp(1.0, -24) * a;
    const double d = fabs(y[r] - s);
    if (d > bound) return fail("gemv outside the fp32 summation bound", r);
    if (a > 0 && d / a > worst) worst = d / a;
  }
  printf("wc_example: fused decode-GEMV of %d x %d bf16 matches fp64 (largest error %.2e of "
         "sum |x w|)\n",
         ROWS, COLS, worst);
  wc_free(blob);
  hipFree(dblob);
  hipFree(dout);
  hipFree(dx);
  hipFree(dy);
  hipFree(derr);
  free(w);
  free(back);
  return 0;
}
