/*
 * Plain-C client of libquake: allocates device memory with the HIP runtime,
 * calls the C ABI declared in include/quake.h, and checks properties that hold
 * exactly or within a known bound (no Python, no torch involved): softmax rows
 * (also split over workgroups that exchange through a caller-owned
 * workspace), exact powers of two, attention of equal scores, the product with an identity
 * matrix, and argument validation.
 *
 * Built by paper_2412_00408_amd/build.py (build_c_client) with gcc against
 * include/quake.h and the HIP runtime only; run by tests/test_gpu_c_client.py.
 * Exit status 0 on success, 1 on a failed check, 2 on a HIP error; prints one
 * line per check.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "quake.h"

static int failures = 0;

static void check(int ok, const char* what) {
  printf("%s: %s\n", ok ? "ok  " : "FAIL", what);
  if (!ok) failures++;
}

#define HIPCHECK(x)                                                   \
  do {                                                                \
    hipError_t e_ = (x);                                              \
    if (e_ != hipSuccess) {                                           \
      printf("FAIL: %s -> %s\n", #x, hipGetErrorString(e_));          \
      return 2;                                                       \
    }                                                                 \
  } while (0)

int main(void) {
  int ndev = 0;
  HIPCHECK(hipGetDeviceCount(&ndev));
  if (ndev < 1) {
    printf("FAIL: no GPU\n");
    return 2;
  }
  check(quake_abi_version() == QUAKE_ABI_VERSION, "abi version matches the header");

  /* softmax of 8 rows x 1000 binary32 values: rows sum to 1 */
  const int rows = 8, cols = 1000;
  float* hx = (float*)malloc(sizeof(float) * rows * cols);
  float* hy = (float*)malloc(sizeof(float) * rows * cols);
  uint32_t s = 12345u;
  for (int i = 0; i < rows * cols; ++i) {
    s = s * 1664525u + 1013904223u;
    hx[i] = ((float)(s >> 8) / 16777216.0f - 0.5f) * 8.0f;
  }
  void *dx = NULL, *dy = NULL;
  HIPCHECK(hipMalloc(&dx, sizeof(float) * rows * cols));
  HIPCHECK(hipMalloc(&dy, sizeof(float) * rows * cols));
  HIPCHECK(hipMemcpy(dx, hx, sizeof(float) * rows * cols, hipMemcpyHostToDevice));
  quake_status st = quake_softmax(dx, dy, rows, cols, cols, cols, QUAKE_F32, QUAKE_2, 1.0f, NULL);
  check(st == QUAKE_OK, "quake_softmax returns QUAKE_OK");
  HIPCHECK(hipDeviceSynchronize());
  HIPCHECK(hipMemcpy(hy, dy, sizeof(float) * rows * cols, hipMemcpyDeviceToHost));
  int sums_ok = 1;
  for (int r = 0; r < rows; ++r) {
    double sum = 0.0;
    for (int j = 0; j < cols; ++j) sum += hy[r * cols + j];
    if (fabs(sum - 1.0) > cols * 6e-8) sums_ok = 0;
  }
  check(sums_ok, "every softmax row sums to 1 within n * 2^-24");

  /* rows of 40000 binary32 values with a workspace the caller allocates and
   * zero-fills: the split-row path, whose chunks exchange their maxima and
   * sums through it. Rows sum to 1, agree with the workspace-free kernel
   * within the softmax tolerance, and the slots are zero again afterwards.
   * Then rows of 40001 values, which start at every offset from 16 bytes:
   * the same paths in their shifted forms. */
  for (int pass = 0; pass < 2; ++pass) {
    const int R = 4, C = pass ? 40001 : 40000;
    float* lx = (float*)malloc(sizeof(float) * R * C);
    float* la = (float*)malloc(sizeof(float) * R * C);
    float* lb = (float*)malloc(sizeof(float) * R * C);
    for (int i = 0; i < R * C; ++i) {
      s = s * 1664525u + 1013904223u;
      lx[i] = ((float)(s >> 8) / 16777216.0f - 0.5f) * 12.0f;
    }
    int64_t nb = 0;
    check(quake_softmax_workspace_size(R, C, QUAKE_F32, &nb) == QUAKE_OK && nb > 256,
          "workspace size query");
    void *lxd = NULL, *lad = NULL, *lbd = NULL, *wsd = NULL;
    HIPCHECK(hipMalloc(&lxd, sizeof(float) * R * C));
    HIPCHECK(hipMalloc(&lad, sizeof(float) * R * C));
    HIPCHECK(hipMalloc(&lbd, sizeof(float) * R * C));
    HIPCHECK(hipMalloc(&wsd, (size_t)nb));
    HIPCHECK(hipMemset(wsd, 0, (size_t)nb));
    HIPCHECK(hipMemcpy(lxd, lx, sizeof(float) * R * C, hipMemcpyHostToDevice));
    check(quake_softmax_ws(lxd, lad, R, C, C, C, QUAKE_F32, QUAKE_2, 1.0f, wsd, nb - 1, NULL) ==
              QUAKE_EINVAL, "a workspace smaller than the query is rejected");
    st = quake_softmax_ws(lxd, lad, R, C, C, C, QUAKE_F32, QUAKE_2, 1.0f, wsd, nb, NULL);
    check(st == QUAKE_OK, "quake_softmax_ws with a caller workspace returns QUAKE_OK");
    st = quake_softmax(lxd, lbd, R, C, C, C, QUAKE_F32, QUAKE_2, 1.0f, NULL);
    check(st == QUAKE_OK, "quake_softmax on the same long rows returns QUAKE_OK");
    HIPCHECK(hipDeviceSynchronize());
    HIPCHECK(hipMemcpy(la, lad, sizeof(float) * R * C, hipMemcpyDeviceToHost));
    HIPCHECK(hipMemcpy(lb, lbd, sizeof(float) * R * C, hipMemcpyDeviceToHost));
    int lsum_ok = 1, agree = 1;
    for (int r = 0; r < R; ++r) {
      double sum = 0.0;
      for (int j = 0; j < C; ++j) {
        const double a = la[r * C + j], b = lb[r * C + j];
        sum += a;
        if (fabs(a - b) > 1e-6 * fabs(b) + 1.2e-38) agree = 0;
      }
      if (fabs(sum - 1.0) > C * 6e-8) lsum_ok = 0;
    }
    check(lsum_ok, "split rows sum to 1 within n * 2^-24");
    check(agree, "split and workspace-free rows agree within 1e-6 relative");
    unsigned char* hws = (unsigned char*)malloc((size_t)nb);
    HIPCHECK(hipMemcpy(hws, wsd, (size_t)nb, hipMemcpyDeviceToHost));
    int zero = 1;
    for (int64_t i = 256; i < nb; ++i) zero &= hws[i] == 0;
    check(zero, "the workspace slots are zero again after the call");
    free(hws);
    free(lx);
    free(la);
    free(lb);
    HIPCHECK(hipFree(lxd));
    HIPCHECK(hipFree(lad));
    HIPCHECK(hipFree(lbd));
    HIPCHECK(hipFree(wsd));
  }

  /* QuAKE2 is exact at integer powers of two (Sec. III-B): with a = fl32(ln2),
   * c0 = fl32(2^23 * a / ln2) = 2^23 and c1 = 127 * 2^23, so l = (k + 127) * 2^23
   * exactly, the mantissa field is 0, y_m = 1 and the result is exactly 2^k. */
  float hk[64], he[64];
  for (int k = 0; k < 64; ++k) hk[k] = (float)(k - 32);
  HIPCHECK(hipMemcpy(dx, hk, sizeof(hk), hipMemcpyHostToDevice));
  st = quake_exp(dx, dy, 64, QUAKE_F32, QUAKE_2, 0.693147180559945309f, 0.0f, NULL);
  check(st == QUAKE_OK, "quake_exp returns QUAKE_OK");
  HIPCHECK(hipDeviceSynchronize());
  HIPCHECK(hipMemcpy(he, dy, sizeof(he), hipMemcpyDeviceToHost));
  int pow_ok = 1;
  for (int k = 0; k < 64; ++k)
    if (he[k] != ldexpf(1.0f, k - 32)) pow_ok = 0;
  check(pow_ok, "QuAKE2 of x = k with a = ln2 is exactly 2^k");

  /* attention with all-zero queries: every score is 0, every probability
   * exactly 1, so each output is the plain mean of the values the query may
   * use (causal: keys 0..i). With v[j][d] = j + 1 (exact in bfloat16) the mean
   * over keys 0..i is (i + 2) / 2, exact in bfloat16 for i < 255. */
  {
    const int heads = 2, seq = 40, dim = 64;
    const size_t nq = (size_t)heads * seq * dim;
    uint16_t* hq = (uint16_t*)calloc(nq, 2);
    uint16_t* hv = (uint16_t*)malloc(nq * 2);
    uint16_t* ho = (uint16_t*)malloc(nq * 2);
    for (int h = 0; h < heads; ++h)
      for (int d = 0; d < dim; ++d)
        for (int j = 0; j < seq; ++j) {
          float f = (float)(j + 1);
          uint32_t b;
          memcpy(&b, &f, 4);
          hv[((size_t)h * dim + d) * seq + j] = (uint16_t)(b >> 16);   /* v^T, exact */
        }
    void *dq = NULL, *dv = NULL, *dout = NULL;
    HIPCHECK(hipMalloc(&dq, nq * 2));
    HIPCHECK(hipMalloc(&dv, nq * 2));
    HIPCHECK(hipMalloc(&dout, nq * 2));
    HIPCHECK(hipMemcpy(dq, hq, nq * 2, hipMemcpyHostToDevice));
    HIPCHECK(hipMemcpy(dv, hv, nq * 2, hipMemcpyHostToDevice));
    st = quake_attention(dq, dq, dv, dout, heads, seq, dim, seq, QUAKE_BF16, QUAKE_2, 0.125f, 1,
                         NULL);
    check(st == QUAKE_OK, "quake_attention returns QUAKE_OK");
    HIPCHECK(hipDeviceSynchronize());
    HIPCHECK(hipMemcpy(ho, dout, nq * 2, hipMemcpyDeviceToHost));
    int mean_ok = 1;
    for (int h = 0; h < heads; ++h)
      for (int i = 0; i < seq; ++i)
        for (int d = 0; d < dim; ++d) {
          uint32_t b = (uint32_t)ho[((size_t)h * seq + i) * dim + d] << 16;
          float f;
          memcpy(&f, &b, 4);
          if (f != 0.5f * (float)(i + 2)) mean_ok = 0;
        }
    check(mean_ok, "causal attention of equal scores is the mean of the allowed values");
    check(quake_attention(dq, dq, dv, dout, heads, seq, 128, seq, QUAKE_BF16, QUAKE_2, 0.125f, 1,
                          NULL) == QUAKE_EINVAL, "attention head dim other than 64 rejected");
    HIPCHECK(hipFree(dq));
    HIPCHECK(hipFree(dv));
    HIPCHECK(hipFree(dout));
    free(hq);
    free(hv);
    free(ho);
  }

  /* x w^T with x the identity and no GELU: each output is one product with
     1.0 plus products with zero, so y = w^T bit for bit (128 x 192 x 128, one
     full tile of the matrix-core kernel); with the GELU, zero weights give 0. */
  {
    const int64_t m = 128, k = 128, n = 192;
    uint16_t* hx2 = (uint16_t*)calloc((size_t)(m * k), 2);
    uint16_t* hw2 = (uint16_t*)malloc((size_t)(n * k) * 2);
    uint16_t* hy2 = (uint16_t*)malloc((size_t)(m * n) * 2);
    for (int64_t i = 0; i < m; ++i) hx2[i * k + i] = 0x3F80; /* bfloat16 1.0 */
    for (int64_t r = 0; r < n; ++r)
      for (int64_t c = 0; c < k; ++c) {
        float f = (float)((r * 131 + c * 71) % 200 - 100) / 16.0f; /* exact in bfloat16 */
        uint32_t b;
        memcpy(&b, &f, 4);
        hw2[r * k + c] = (uint16_t)(b >> 16);
      }
    void *dx2 = NULL, *dw2 = NULL, *dy2 = NULL;
    HIPCHECK(hipMalloc(&dx2, (size_t)(m * k) * 2));
    HIPCHECK(hipMalloc(&dw2, (size_t)(n * k) * 2));
    HIPCHECK(hipMalloc(&dy2, (size_t)(m * n) * 2));
    HIPCHECK(hipMemcpy(dx2, hx2, (size_t)(m * k) * 2, hipMemcpyHostToDevice));
    HIPCHECK(hipMemcpy(dw2, hw2, (size_t)(n * k) * 2, hipMemcpyHostToDevice));
    st = quake_linear_gelu(dx2, dw2, dy2, m, n, k, k, k, n, QUAKE_BF16, QUAKE_2, 0, NULL);
    check(st == QUAKE_OK, "quake_linear_gelu returns QUAKE_OK");
    HIPCHECK(hipDeviceSynchronize());
    HIPCHECK(hipMemcpy(hy2, dy2, (size_t)(m * n) * 2, hipMemcpyDeviceToHost));
    int id_ok = 1;
    for (int64_t i = 0; i < m; ++i)
      for (int64_t j = 0; j < n; ++j)
        if (hy2[i * n + j] != hw2[j * k + i]) id_ok = 0;
    check(id_ok, "identity x gives y = w^T exactly");
    st = quake_linear_gelu(dx2, dw2, dy2, m, n, k, k, k, n, QUAKE_BF16, QUAKE_2, 1, NULL);
    HIPCHECK(hipDeviceSynchronize());
    HIPCHECK(hipMemcpy(hy2, dy2, (size_t)(m * n) * 2, hipMemcpyDeviceToHost));
    int zero_ok = st == QUAKE_OK;
    for (int64_t i = 0; i < m; ++i)
      for (int64_t j = 0; j < n; ++j)
        if (hw2[j * k + i] == 0 && hy2[i * n + j] != 0) zero_ok = 0;
    check(zero_ok, "GELU of a zero product is 0");
    check(quake_linear_gelu(dx2, dw2, dy2, m, n, 12, k, k, n, QUAKE_BF16, QUAKE_2, 1, NULL) ==
              QUAKE_EINVAL, "linear k not a multiple of 8 rejected");
    HIPCHECK(hipFree(dx2));
    HIPCHECK(hipFree(dw2));
    HIPCHECK(hipFree(dy2));
    free(hx2);
    free(hw2);
    free(hy2);
  }

  /* argument validation happens before any HIP call */
  check(quake_gelu(NULL, NULL, 5, QUAKE_F32, QUAKE_2, NULL) == QUAKE_EINVAL, "NULL buffers rejected");
  check(quake_sigmoid(dx, dy, 5, (quake_dtype)7, QUAKE_2, 0, NULL) == QUAKE_EDTYPE, "bad dtype rejected");
  check(quake_softmax(dx, dy, 2, 8, 4, 8, QUAKE_F32, QUAKE_2, 1.0f, NULL) == QUAKE_EINVAL,
        "ldx < cols rejected");
  check(strncmp(quake_status_str(QUAKE_EMODE), "QUAKE_EMODE", 11) == 0, "status strings");

  HIPCHECK(hipFree(dx));
  HIPCHECK(hipFree(dy));
  free(hx);
  free(hy);
  printf("%s\n", failures ? "abi smoke FAILED" : "abi smoke passed");
  return failures ? 1 : 0;
}
