/*
 * A plain C11 caller of the library: no Python, no torch.  It reads a set of
 * matrices and step scalars from a file, places them in hipMalloc'd device
 * buffers, vets them with muon_check_buffers, runs one muon_step_debug and
 * writes W, M and the orthogonalised update O back to a file, which the test
 * compares with the fp64 oracle.
 *
 * Input (little-endian): int32 n, float lr, momentum, weight_decay, int32
 * ns_steps, nesterov; then per matrix int64 rows, cols, int32 param_dtype,
 * grad_dtype (MUON_F32 / MUON_BF16), followed by W, G (their dtypes) and M
 * (fp32), each rows x cols row-major.
 * Output: per matrix W (param dtype), M (fp32), O (fp32).
 * Exit status 0 on success; otherwise the failing call and muon_last_error()
 * are printed.
 */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "muon.h"

static size_t esize(int32_t dt) { return dt == MUON_BF16 ? 2 : 4; }

static int read_all(FILE* f, void* p, size_t bytes) { return fread(p, 1, bytes, f) == bytes; }

#define NEED(cond, msg)                                  \
  do {                                                   \
    if (!(cond)) {                                       \
      fprintf(stderr, "c_abi_step: %s\n", msg);          \
      return 1;                                          \
    }                                                    \
  } while (0)

#define MUON(call)                                                                  \
  do {                                                                              \
    muon_status s_ = (call);                                                        \
    if (s_ != MUON_OK) {                                                            \
      fprintf(stderr, "c_abi_step: %s -> %s: %s\n", #call, muon_status_string(s_), \
              muon_last_error());                                                   \
      return 1;                                                                     \
    }                                                                               \
  } while (0)

#define HIP(call)                                                                       \
  do {                                                                                  \
    hipError_t e_ = (call);                                                             \
    if (e_ != hipSuccess) {                                                             \
      fprintf(stderr, "c_abi_step: %s -> %s\n", #call, hipGetErrorString(e_));          \
      return 1;                                                                         \
    }                                                                                   \
  } while (0)

int main(int argc, char** argv) {
  NEED(argc == 3, "usage: c_abi_step INPUT OUTPUT");
  FILE* in = fopen(argv[1], "rb");
  NEED(in, "cannot open the input");
  int32_t n = 0, ns_steps = 0, nesterov = 0;
  float lr = 0.f, mu = 0.f, wd = 0.f;
  NEED(read_all(in, &n, 4) && read_all(in, &lr, 4) && read_all(in, &mu, 4) && read_all(in, &wd, 4) &&
           read_all(in, &ns_steps, 4) && read_all(in, &nesterov, 4),
       "short header");
  NEED(n >= 1 && n <= 1024, "matrix count out of range");

  muon_matrix_desc* d = calloc((size_t)n, sizeof(muon_matrix_desc));
  void** host = calloc((size_t)n * 3, sizeof(void*));
  void** dev = calloc((size_t)n * 4, sizeof(void*)); /* W, G, M, O per matrix */
  NEED(d && host && dev, "out of host memory");
  for (int32_t i = 0; i < n; ++i) {
    NEED(read_all(in, &d[i].rows, 8) && read_all(in, &d[i].cols, 8) && read_all(in, &d[i].param_dtype, 4) &&
             read_all(in, &d[i].grad_dtype, 4),
         "short matrix header");
    NEED(d[i].rows >= 1 && d[i].cols >= 1 && d[i].rows * d[i].cols <= ((int64_t)1 << 28), "matrix size out of range");
    d[i].momentum_dtype = MUON_F32;
    d[i].tile_hint = 0;
    const size_t el = (size_t)(d[i].rows * d[i].cols);
    const size_t bytes[3] = {el * esize(d[i].param_dtype), el * esize(d[i].grad_dtype), el * 4};
    for (int k = 0; k < 3; ++k) {
      host[3 * i + k] = malloc(bytes[k]);
      NEED(host[3 * i + k] && read_all(in, host[3 * i + k], bytes[k]), "short matrix data");
      HIP(hipMalloc(&dev[4 * i + k], bytes[k]));
      HIP(hipMemcpy(dev[4 * i + k], host[3 * i + k], bytes[k], hipMemcpyHostToDevice));
    }
    HIP(hipMalloc(&dev[4 * i + 3], el * 4));
  }
  fclose(in);

  muon_plan_opts opts;
  MUON(muon_plan_opts_default(&opts));
  muon_plan plan = NULL;
  MUON(muon_plan_create(d, n, &opts, &plan));
  size_t ws_bytes = 0;
  MUON(muon_plan_workspace_bytes(plan, &ws_bytes));
  void* ws = NULL;
  HIP(hipMalloc(&ws, ws_bytes));

  void** params = calloc((size_t)n, sizeof(void*));
  const void** grads = calloc((size_t)n, sizeof(void*));
  void** moms = calloc((size_t)n, sizeof(void*));
  float** outs = calloc((size_t)n, sizeof(float*));
  NEED(params && grads && moms && outs, "out of host memory");
  for (int32_t i = 0; i < n; ++i) {
    params[i] = dev[4 * i];
    grads[i] = dev[4 * i + 1];
    moms[i] = dev[4 * i + 2];
    outs[i] = (float*)dev[4 * i + 3];
  }
  MUON(muon_check_buffers(plan, params, grads, moms, ws, ws_bytes, outs));
  MUON(muon_step_debug(plan, params, grads, moms, lr, mu, wd, ns_steps, nesterov, ws, ws_bytes, NULL, outs));
  HIP(hipDeviceSynchronize());

  FILE* out = fopen(argv[2], "wb");
  NEED(out, "cannot open the output");
  for (int32_t i = 0; i < n; ++i) {
    const size_t el = (size_t)(d[i].rows * d[i].cols);
    const size_t bytes[3] = {el * esize(d[i].param_dtype), el * 4, el * 4};
    const int src[3] = {0, 2, 3};
    for (int k = 0; k < 3; ++k) {
      void* buf = malloc(bytes[k]);
      NEED(buf, "out of host memory");
      HIP(hipMemcpy(buf, dev[4 * i + src[k]], bytes[k], hipMemcpyDeviceToHost));
      NEED(fwrite(buf, 1, bytes[k], out) == bytes[k], "short write");
      free(buf);
    }
  }
  NEED(fclose(out) == 0, "cannot close the output");

  MUON(muon_plan_destroy(plan));
  HIP(hipFree(ws));
  for (int32_t i = 0; i < n; ++i) {
    for (int k = 0; k < 4; ++k) HIP(hipFree(dev[4 * i + k]));
    for (int k = 0; k < 3; ++k) free(host[3 * i + k]);
  }
  free(d);
  free(host);
  free(dev);
  free(params);
  free(grads);
  free(moms);
  free(outs);
  return 0;
}
