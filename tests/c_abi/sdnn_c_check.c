/*
 * sdnn_c_check.c -- the C ABI (include/sdnn.h) driven from plain C99 with the HIP
 * runtime's C API, as a C caller would: host CSR in, device B / C / bias / workspace,
 * sdnn_plan_create (Sec. 2.1 preparation), sdnn_spmm and sdnn_spmm_split (Sec. 3.2.2
 * execution), results copied back.  Test infrastructure: the inputs are raw files that
 * the test writes from the seeded input generators, and the outputs go back to the
 * test, which checks them against the CPU oracle.
 *
 *   sdnn_c_check -sizes
 *     prints sizeof(sdnn_plan_opts) and sizeof(sdnn_plan_info_t) as compiled (no GPU)
 *   sdnn_c_check DIR M K N
 *     reads  DIR/row_ptr.i32 (M+1), DIR/col_idx.i32 (nnz), DIR/values.f32 (nnz),
 *            DIR/B.f32 (K*N), DIR/bias.f32 (M)
 *     writes DIR/C_plain.f32 and DIR/C_split.f32 (M*N each), DIR/perm.i32 (M)
 *   exit status 0 on success; otherwise a message on stderr naming the failing call.
 */
#include <stdio.h>
#include <stdlib.h>

#include <hip/hip_runtime_api.h>

#include "sdnn.h"

static void* read_file(const char* dir, const char* name, size_t bytes) {
  char path[4096];
  snprintf(path, sizeof path, "%s/%s", dir, name);
  FILE* f = fopen(path, "rb");
  if (!f) return NULL;
  void* buf = malloc(bytes ? bytes : 1);
  size_t got = buf ? fread(buf, 1, bytes, f) : 0;
  fclose(f);
  if (got != bytes) {
    free(buf);
    return NULL;
  }
  return buf;
}

static int write_file(const char* dir, const char* name, const void* data, size_t bytes) {
  char path[4096];
  snprintf(path, sizeof path, "%s/%s", dir, name);
  FILE* f = fopen(path, "wb");
  if (!f) return 0;
  size_t put = fwrite(data, 1, bytes, f);
  fclose(f);
  return put == bytes;
}

#define CHECK_SDNN(call)                                                          \
  do {                                                                            \
    sdnn_status st_ = (call);                                                     \
    if (st_ != SDNN_OK) {                                                         \
      fprintf(stderr, "%s failed: %s\n", #call, sdnn_status_str(st_));            \
      return 1;                                                                   \
    }                                                                             \
  } while (0)
#define CHECK_HIP(call)                                                           \
  do {                                                                            \
    if ((call) != hipSuccess) {                                                   \
      fprintf(stderr, "%s failed\n", #call);                                      \
      return 1;                                                                   \
    }                                                                             \
  } while (0)

int main(int argc, char** argv) {
  if (argc == 2 && argv[1][0] == '-' && argv[1][1] == 's') {  /* -sizes: no device work */
    printf("%zu %zu\n", sizeof(sdnn_plan_opts), sizeof(sdnn_plan_info_t));
    return 0;
  }
  if (argc != 5) {
    fprintf(stderr, "usage: %s DIR M K N\n", argv[0]);
    return 2;
  }
  const char* dir = argv[1];
  const int32_t M = atoi(argv[2]), K = atoi(argv[3]), N = atoi(argv[4]);
  int32_t* row_ptr = read_file(dir, "row_ptr.i32", sizeof(int32_t) * (size_t)(M + 1));
  if (!row_ptr) return 3;
  const size_t nnz = (size_t)row_ptr[M];
  int32_t* col_idx = read_file(dir, "col_idx.i32", sizeof(int32_t) * nnz);
  float* values = read_file(dir, "values.f32", sizeof(float) * nnz);
  float* B = read_file(dir, "B.f32", sizeof(float) * (size_t)K * N);
  float* bias = read_file(dir, "bias.f32", sizeof(float) * (size_t)M);
  if (!col_idx || !values || !B || !bias) return 3;

  /* segments of 2 chunks (64 rows of B) so that the split call has several */
  sdnn_plan_opts opts = {0, 1, 0, 2, NULL, 0, 0};
  sdnn_plan plan = NULL;
  CHECK_SDNN(sdnn_plan_create(row_ptr, col_idx, values, M, K, &opts, &plan));
  sdnn_plan_info_t info;
  CHECK_SDNN(sdnn_plan_info(plan, &info));

  float *dB = NULL, *dC = NULL, *dbias = NULL, *dws = NULL;
  const size_t ws_floats = (size_t)(info.splits > 0 ? info.splits : 1) * M * N;
  CHECK_HIP(hipMalloc((void**)&dB, sizeof(float) * (size_t)K * N + 16));
  CHECK_HIP(hipMalloc((void**)&dC, sizeof(float) * (size_t)M * N + 16));
  CHECK_HIP(hipMalloc((void**)&dbias, sizeof(float) * (size_t)M + 16));
  CHECK_HIP(hipMalloc((void**)&dws, sizeof(float) * ws_floats + 16));
  CHECK_HIP(hipMemcpy(dB, B, sizeof(float) * (size_t)K * N, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(dbias, bias, sizeof(float) * (size_t)M, hipMemcpyHostToDevice));

  float* C = malloc(sizeof(float) * (size_t)M * N + 4);
  int32_t* perm = malloc(sizeof(int32_t) * (size_t)M + 4);
  if (!C || !perm) return 3;
  CHECK_SDNN(sdnn_spmm(plan, dB, dC, N, dbias, SDNN_EPI_GELU, NULL));
  CHECK_HIP(hipDeviceSynchronize());
  CHECK_HIP(hipMemcpy(C, dC, sizeof(float) * (size_t)M * N, hipMemcpyDeviceToHost));
  if (!write_file(dir, "C_plain.f32", C, sizeof(float) * (size_t)M * N)) return 4;

  CHECK_SDNN(sdnn_spmm_split(plan, dB, dC, N, dbias, SDNN_EPI_GELU, 0, dws,
                             (int64_t)ws_floats, NULL));
  CHECK_HIP(hipDeviceSynchronize());
  CHECK_HIP(hipMemcpy(C, dC, sizeof(float) * (size_t)M * N, hipMemcpyDeviceToHost));
  if (!write_file(dir, "C_split.f32", C, sizeof(float) * (size_t)M * N)) return 4;

  CHECK_SDNN(sdnn_plan_get_perm(plan, perm));
  if (!write_file(dir, "perm.i32", perm, sizeof(int32_t) * (size_t)M)) return 4;

  /* the same product from a plan fixed to 128-column tiles (used when N % 4 == 0) */
  sdnn_plan_opts nopts = {0, 1, 0, 0, NULL, 0, 128};
  sdnn_plan nplan = NULL;
  int32_t tile = 0;
  CHECK_SDNN(sdnn_plan_create(row_ptr, col_idx, values, M, K, &nopts, &nplan));
  CHECK_SDNN(sdnn_plan_launch_tile(nplan, N, &tile));
  CHECK_SDNN(sdnn_spmm(nplan, dB, dC, N, dbias, SDNN_EPI_GELU, NULL));
  CHECK_HIP(hipDeviceSynchronize());
  CHECK_HIP(hipMemcpy(C, dC, sizeof(float) * (size_t)M * N, hipMemcpyDeviceToHost));
  if (!write_file(dir, "C_narrow.f32", C, sizeof(float) * (size_t)M * N)) return 4;
  sdnn_plan_destroy(nplan);

  sdnn_plan_destroy(plan);
  hipFree(dB);
  hipFree(dC);
  hipFree(dbias);
  hipFree(dws);
  free(row_ptr);
  free(col_idx);
  free(values);
  free(B);
  free(bias);
  free(C);
  free(perm);
  printf("sdnn_c_check ok: M=%d K=%d N=%d nnz=%zu segments=%d tile=%d\n", M, K, N, nnz,
         info.splits, tile);
  return 0;
}
