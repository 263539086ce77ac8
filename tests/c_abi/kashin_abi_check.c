/*
 * A C consumer of the library: the boundary used with plain pointers and the HIP runtime only,
 * no Python.  Test infrastructure (driven by tests/test_abi_host.py and tests/test_c_abi_gpu.py).
 *
 *   kashin_abi_check host   host-side calls: the supported-length set, the sign mask against the
 *                           published splitmix64 outputs, argument validation and error strings
 *   kashin_abi_check gpu    on the current device: decompose a few rows and check
 *                           w = u + P vhat + r through kashin_apply_p (Alg. 2's identity, fp32
 *                           rounding), then quantise and reconstruct them and check the codes'
 *                           range and the dequantisation error against the rows' scale
 * Prints one line per check and exits non-zero on the first failure.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "kashin.h"

#define CHECK(cond, ...)                      \
  do {                                        \
    if (!(cond)) {                            \
      fprintf(stderr, "FAIL: " __VA_ARGS__);  \
      fprintf(stderr, "\n");                  \
      return 1;                               \
    }                                         \
  } while (0)

static int host_checks(void) {
  static const int lengths[] = {64,   96,   172,  256,  512,   768,   1024,  2048,  3072,
                                4096, 5120, 6144, 8192, 10000, 11008, 13824, 14336, 16384};
  const int nl = (int)(sizeof(lengths) / sizeof(lengths[0]));
  int count = 0;
  for (int n = 0; n <= 20000; ++n) {
    int listed = 0;
    for (int i = 0; i < nl; ++i) listed |= lengths[i] == n;
    CHECK(kashin_supported_n(n) == listed, "kashin_supported_n(%d) = %d", n, kashin_supported_n(n));
    count += listed;
  }
  CHECK(count == nl, "supported count %d", count);
  printf("supported lengths: %d, exactly the documented set\n", count);

  /* eps_j = -1 iff the top bit of splitmix64 output j is set; outputs of state 0 start
   * 0xe220a8397b1dcdaf (top bit set), 0x6e789e6aa1b965f4, 0x06c45d188009454f (top bits clear) */
  int8_t eps[64];
  CHECK(kashin_signs(64, 0, eps) == KASHIN_OK, "kashin_signs");
  CHECK(eps[0] == -1 && eps[1] == 1 && eps[2] == 1, "signs %d %d %d", eps[0], eps[1], eps[2]);
  for (int i = 0; i < 64; ++i) CHECK(eps[i] == 1 || eps[i] == -1, "sign %d = %d", i, eps[i]);
  printf("sign mask of seed 0 starts -1 +1 +1\n");

  kashin_plan_t plan = NULL;
  CHECK(kashin_plan(NULL, 512, 1, 4) == KASHIN_E_INVALID, "null out-pointer accepted");
  CHECK(strlen(kashin_last_error()) > 0, "no error message");
  CHECK(kashin_plan(&plan, 500, 1, 4) == KASHIN_E_UNSUPPORTED_N, "length 500 accepted");
  CHECK(kashin_plan(&plan, 512, 1, 0) == KASHIN_E_INVALID, "zero blocks accepted");
  CHECK(kashin_rotate(5120, 1, 0, NULL, KASHIN_F32, 0, 5120, NULL, 5120, NULL) == KASHIN_E_UNSUPPORTED_N,
        "rotation of odd part 5 accepted");
  CHECK(kashin_quantize(NULL, NULL, KASHIN_F32, 1, 512, 0, NULL, NULL, NULL, NULL) == KASHIN_E_INVALID,
        "null plan accepted");
  CHECK(kashin_optq_workspace_bytes(4096, 4096, 129) == -1, "chunk 129 accepted");
  CHECK(kashin_optq_workspace_bytes(4096, 4096, 128) > 0, "workspace size");
  CHECK(strcmp(kashin_status_string(KASHIN_OK), kashin_status_string(KASHIN_E_HIP)) != 0, "status strings");
  printf("validation: null, unsupported and out-of-range arguments rejected with messages\n");
  return 0;
}

#define HIPCHECK(x) CHECK((x) == hipSuccess, "%s: %s", #x, hipGetErrorString(x))

static int gpu_checks(void) {
  enum { N = 512, M = 7, K = 20, NBY = N / 4 };
  float* h_w = (float*)malloc(sizeof(float) * M * N);
  float* h_out = (float*)malloc(sizeof(float) * M * N * 4);
  uint8_t* h_codes = (uint8_t*)malloc(2 * M * NBY);
  float h_ce[M * 8];
  /* deterministic rows: a scaled sum of incommensurate sines, one outlier per row */
  for (int i = 0; i < M; ++i)
    for (int j = 0; j < N; ++j)
      h_w[i * N + j] = 0.02f * (float)(sin(0.37 * (i + 1) * j + 0.5 * i) + 0.5 * sin(2.1 * ((j * j) % 97))) +
                       (j == (37 * i) % N ? 0.3f : 0.f);
  float *w, *u, *vh, *r, *pv, *what, *ce;
  uint8_t *cu, *cv;
  const size_t bytes = sizeof(float) * M * N;
  HIPCHECK(hipMalloc((void**)&w, bytes));
  HIPCHECK(hipMalloc((void**)&u, bytes));
  HIPCHECK(hipMalloc((void**)&vh, bytes));
  HIPCHECK(hipMalloc((void**)&r, bytes));
  HIPCHECK(hipMalloc((void**)&pv, bytes));
  HIPCHECK(hipMalloc((void**)&what, bytes));
  HIPCHECK(hipMalloc((void**)&ce, sizeof(float) * M * 8));
  HIPCHECK(hipMalloc((void**)&cu, M * NBY));
  HIPCHECK(hipMalloc((void**)&cv, M * NBY));
  HIPCHECK(hipMemcpy(w, h_w, bytes, hipMemcpyHostToDevice));

  kashin_plan_t plan = NULL;
  CHECK(kashin_plan(&plan, N, 11, K) == KASHIN_OK, "kashin_plan: %s", kashin_last_error());
  CHECK(kashin_decompose(plan, w, KASHIN_F32, M, N, u, vh, r, NULL, NULL, NULL) == KASHIN_OK, "decompose: %s",
        kashin_last_error());
  CHECK(kashin_apply_p(plan, vh, pv, M, NULL) == KASHIN_OK, "apply_p: %s", kashin_last_error());
  CHECK(kashin_quantize(plan, w, KASHIN_F32, M, N, 0, cu, cv, ce, NULL) == KASHIN_OK, "quantize: %s",
        kashin_last_error());
  CHECK(kashin_reconstruct(plan, cu, cv, ce, M, what, N, NULL) == KASHIN_OK, "reconstruct: %s",
        kashin_last_error());
  HIPCHECK(hipDeviceSynchronize());
  HIPCHECK(hipMemcpy(h_out, u, bytes, hipMemcpyDeviceToHost));
  HIPCHECK(hipMemcpy(h_out + M * N, pv, bytes, hipMemcpyDeviceToHost));
  HIPCHECK(hipMemcpy(h_out + 2 * M * N, r, bytes, hipMemcpyDeviceToHost));
  HIPCHECK(hipMemcpy(h_out + 3 * M * N, what, bytes, hipMemcpyDeviceToHost));
  HIPCHECK(hipMemcpy(h_codes, cu, M * NBY, hipMemcpyDeviceToHost));
  HIPCHECK(hipMemcpy(h_codes + M * NBY, cv, M * NBY, hipMemcpyDeviceToHost));
  HIPCHECK(hipMemcpy(h_ce, ce, sizeof(h_ce), hipMemcpyDeviceToHost));

  double worst_id = 0, worst_q = 0;
  for (int i = 0; i < M; ++i) {
    double winf = 0, id = 0, q = 0;
    for (int j = 0; j < N; ++j) winf = fmax(winf, fabs(h_w[i * N + j]));
    for (int j = 0; j < N; ++j) {
      const int k = i * N + j;
      id = fmax(id, fabs(h_w[k] - h_out[k] - h_out[M * N + k] - h_out[2 * M * N + k]));
      q = fmax(q, fabs(h_w[k] - h_out[3 * M * N + k]));
    }
    worst_id = fmax(worst_id, id / winf);
    worst_q = fmax(worst_q, q / winf);
    for (int f = 0; f < 2; ++f)
      for (int c = 1; c < 4; ++c) CHECK(h_ce[i * 8 + 4 * f + c - 1] <= h_ce[i * 8 + 4 * f + c], "centres unsorted");
  }
  printf("w = u + P vhat + r within %.2e of ||w||_inf\n", worst_id);
  printf("dequantised rows within %.2e of ||w||_inf\n", worst_q);
  CHECK(worst_id <= 1e-5, "decomposition identity off by %.3e", worst_id);
  /* 2-bit codes per factor: the dequantisation error is a fraction of the row scale, not noise */
  CHECK(worst_q < 0.5, "dequantisation error %.3e", worst_q);
  CHECK(kashin_plan_destroy(plan) == KASHIN_OK, "destroy");
  (void)hipFree(w), (void)hipFree(u), (void)hipFree(vh), (void)hipFree(r), (void)hipFree(pv);
  (void)hipFree(what), (void)hipFree(ce), (void)hipFree(cu), (void)hipFree(cv);
  free(h_w), free(h_out), free(h_codes);
  return 0;
}

int main(int argc, char** argv) {
  if (argc != 2 || (strcmp(argv[1], "host") != 0 && strcmp(argv[1], "gpu") != 0)) {
    fprintf(stderr, "usage: %s host|gpu\n", argv[0]);
    return 2;
  }
  const int rc = strcmp(argv[1], "host") == 0 ? host_checks() : gpu_checks();
  if (rc == 0) printf("ok\n");
  return rc;
}
