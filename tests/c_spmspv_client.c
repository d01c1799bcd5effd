/* A C99 client of the device path with no PyTorch in the process: it encodes
 * a matrix with the host encoder, copies the three format arrays and x to
 * device memory from hipMalloc, zero-fills the workspace with
 * celty_spmspv_workspace_init, runs celty_spmspv on the null stream and
 * writes y back.  Built by the package's build step; the GPU tests feed it
 * seeded problems and compare y with the oracle.
 *
 * usage: c_spmspv_client IN OUT
 *   IN : int32 M, K, R; float32 tau; fp16 W[M*K] (row-major); uint8 mask[M*K];
 *        fp16 x[K]
 *   OUT: fp16 y[M]
 * Exit status 0 on success; 2 bad usage or input; 3 encoder error; 4 HIP
 * runtime error; 5 SpMSpV error (the status string goes to stderr). */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include <hip/hip_runtime_api.h>

#include "celty.h"

static void* read_exact(FILE* f, size_t n) {
  void* p = malloc(n ? n : 1);
  if (p && n && fread(p, 1, n, f) != n) {
    free(p);
    return NULL;
  }
  return p;
}

#define HIP_OK(call)                                                        \
  do {                                                                      \
    hipError_t e_ = (call);                                                 \
    if (e_ != hipSuccess) {                                                 \
      fprintf(stderr, "%s: %s\n", #call, hipGetErrorString(e_));            \
      return 4;                                                             \
    }                                                                       \
  } while (0)

int main(int argc, char** argv) {
  if (argc != 3) return 2;
  FILE* f = fopen(argv[1], "rb");
  if (!f) return 2;
  int32_t dims[3];
  float tau;
  if (fread(dims, sizeof dims, 1, f) != 1 || fread(&tau, sizeof tau, 1, f) != 1) return 2;
  const int32_t M = dims[0], K = dims[1], R = dims[2];
  if (M < 1 || K < 1 || R < 1) return 2;
  const size_t MK = (size_t)M * (size_t)K;
  uint16_t* W = (uint16_t*)read_exact(f, MK * 2);
  uint8_t* mask = (uint8_t*)read_exact(f, MK);
  uint16_t* x = (uint16_t*)read_exact(f, (size_t)K * 2);
  fclose(f);
  if (!W || !mask || !x) return 2;

  int64_t G = 0, nnz = 0, pad = 0;
  celty_status st = celty_encode_plan(W, K, mask, K, M, K, R, CELTY_LAYOUT_RLC, &G, &nnz, &pad);
  if (st != CELTY_OK) return 3;
  const int32_t T = (M + R - 1) / R;
  const size_t n_gptr = (size_t)T * (size_t)K + 1;
  uint32_t* gptr = (uint32_t*)malloc(n_gptr * 4);
  uint16_t* values = NULL;
  if (posix_memalign((void**)&values, 16, (size_t)(8 * G + 8) * 2) != 0) return 3;
  uint32_t* runs = (uint32_t*)malloc((size_t)(G + 1) * 4);
  uint16_t* colmax = (uint16_t*)malloc((size_t)K * 2 + 4);
  celty_rlc_csc enc;
  if (!gptr || !runs || !colmax) return 3;
  st = celty_encode(W, K, mask, K, M, K, R, CELTY_LAYOUT_RLC, gptr, values, runs, colmax, G, &enc, 0);
  if (st != CELTY_OK) return 3;

  void *d_gptr, *d_values, *d_runs, *d_colmax, *d_x, *d_y, *d_ws;
  const size_t ws_bytes = celty_spmspv_workspace_bytes(M, K, R);
  HIP_OK(hipMalloc(&d_gptr, n_gptr * 4));
  HIP_OK(hipMalloc(&d_values, (size_t)(8 * G + 8) * 2));
  HIP_OK(hipMalloc(&d_runs, (size_t)(G + 1) * 4));
  HIP_OK(hipMalloc(&d_colmax, (size_t)K * 2));
  HIP_OK(hipMalloc(&d_x, (size_t)K * 2));
  HIP_OK(hipMalloc(&d_y, (size_t)M * 2));
  HIP_OK(hipMalloc(&d_ws, ws_bytes));
  HIP_OK(hipMemcpy(d_gptr, gptr, n_gptr * 4, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_values, values, (size_t)(8 * G) * 2, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_runs, runs, (size_t)G * 4, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_colmax, colmax, (size_t)K * 2, hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(d_x, x, (size_t)K * 2, hipMemcpyHostToDevice));

  celty_rlc_csc dev = enc;   /* same header, device arrays */
  dev.gptr = (const uint32_t*)d_gptr;
  dev.values = (const uint16_t*)d_values;
  dev.runs = (const uint32_t*)d_runs;
  dev.colmax = (const uint16_t*)d_colmax;
  st = celty_spmspv_workspace_init(d_ws, ws_bytes, NULL);
  if (st == CELTY_OK) st = celty_spmspv(&dev, d_x, tau, d_y, d_ws, ws_bytes, NULL);
  if (st != CELTY_OK) {
    fprintf(stderr, "celty: %s\n", celty_status_string(st));
    return 5;
  }
  HIP_OK(hipDeviceSynchronize());
  uint16_t* y = (uint16_t*)malloc((size_t)M * 2);
  if (!y) return 2;
  HIP_OK(hipMemcpy(y, d_y, (size_t)M * 2, hipMemcpyDeviceToHost));
  FILE* o = fopen(argv[2], "wb");
  if (!o || fwrite(y, 2, (size_t)M, o) != (size_t)M) return 2;
  fclose(o);
  HIP_OK(hipFree(d_gptr));
  HIP_OK(hipFree(d_values));
  HIP_OK(hipFree(d_runs));
  HIP_OK(hipFree(d_colmax));
  HIP_OK(hipFree(d_x));
  HIP_OK(hipFree(d_y));
  HIP_OK(hipFree(d_ws));
  free(W); free(mask); free(x); free(gptr); free(values); free(runs); free(colmax); free(y);
  return 0;
}
