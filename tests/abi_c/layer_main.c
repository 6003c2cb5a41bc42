/* Calls the layer through the C ABI alone (no Python, no torch): reads a layer descriptor and
 * its inputs from a binary file, runs omnimoe_layer_forward on the first GPU and writes y, idx
 * and gates back. Used by the GPU tests to show the boundary works from plain C.
 *
 * Input file:  omnimoe_layer_desc (48 bytes), then x, keys_row, keys_col, u, v in the layer's
 *              storage dtype (row-major, sizes from the descriptor).
 * Output file: y [T, d] fp32, idx [T, H, K] int32, gates [T, H, K] fp32.
 * Exit status 0 on success; otherwise the failing call is printed. */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "../../include/omnimoe.h"

#define HIP_OK(call)                                                                    \
  do {                                                                                  \
    hipError_t e_ = (call);                                                             \
    if (e_ != hipSuccess) {                                                             \
      fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_));                \
      return 2;                                                                         \
    }                                                                                   \
  } while (0)

static int read_exact(FILE* f, void* p, size_t n) { return fread(p, 1, n, f) == n ? 0 : -1; }

static int upload(FILE* f, size_t bytes, void** dev) {
  void* h = malloc(bytes ? bytes : 1);
  if (!h || read_exact(f, h, bytes)) {
    free(h);
    return -1;
  }
  if (hipMalloc(dev, bytes ? bytes : 16) != hipSuccess ||
      hipMemcpy(*dev, h, bytes, hipMemcpyHostToDevice) != hipSuccess) {
    free(h);
    return -1;
  }
  free(h);
  return 0;
}

int main(int argc, char** argv) {
  if (argc != 3) {
    fprintf(stderr, "usage: %s input.bin output.bin\n", argv[0]);
    return 2;
  }
  printf("%s\n", omnimoe_status_string(OMNIMOE_OK));
  FILE* in = fopen(argv[1], "rb");
  if (!in) return 2;
  omnimoe_layer_desc d;
  if (read_exact(in, &d, sizeof d)) return 2;
  const size_t s = d.dtype == OMNIMOE_BF16 ? 2 : 4;
  const size_t N = (size_t)d.n_rows * d.n_cols;
  const size_t M = (size_t)d.T * d.H * d.K;
  void *x, *kr, *kc, *u, *v, *y, *idx, *gates, *ws;
  if (upload(in, (size_t)d.T * d.d * s, &x) || upload(in, (size_t)d.H * d.n_rows * d.d_key * s, &kr) ||
      upload(in, (size_t)d.H * d.n_cols * d.d_key * s, &kc) || upload(in, N * d.d * s, &u) ||
      upload(in, N * d.d * s, &v)) {
    fprintf(stderr, "reading or uploading the inputs failed\n");
    return 2;
  }
  fclose(in);
  size_t ws_bytes = 0;
  omnimoe_status st = omnimoe_workspace_size(&d, OMNIMOE_STAGE_LAYER, &ws_bytes);
  if (st != OMNIMOE_OK) {
    fprintf(stderr, "omnimoe_workspace_size: %s\n", omnimoe_status_string(st));
    return 3;
  }
  HIP_OK(hipMalloc(&y, (size_t)d.T * d.d * 4));
  HIP_OK(hipMalloc(&idx, M * 4));
  HIP_OK(hipMalloc(&gates, M * 4));
  HIP_OK(hipMalloc(&ws, ws_bytes));
  hipStream_t stream;
  HIP_OK(hipStreamCreate(&stream));
  /* A call that must fail on the host, before any launch: a workspace one byte short. */
  st = omnimoe_layer_forward(&d, x, kr, kc, u, v, (float*)y, (int32_t*)idx, (float*)gates, ws,
                             ws_bytes - 1, stream);
  if (st != OMNIMOE_ERR_WORKSPACE) {
    fprintf(stderr, "short workspace not rejected: %s\n", omnimoe_status_string(st));
    return 4;
  }
  st = omnimoe_layer_forward(&d, x, kr, kc, u, v, (float*)y, (int32_t*)idx, (float*)gates, ws,
                             ws_bytes, stream);
  if (st != OMNIMOE_OK) {
    fprintf(stderr, "omnimoe_layer_forward: %s\n", omnimoe_status_string(st));
    return 3;
  }
  HIP_OK(hipStreamSynchronize(stream));
  FILE* out = fopen(argv[2], "wb");
  if (!out) return 2;
  const size_t sizes[3] = {(size_t)d.T * d.d * 4, M * 4, M * 4};
  void* bufs[3] = {y, idx, gates};
  for (int i = 0; i < 3; ++i) {
    void* h = malloc(sizes[i] ? sizes[i] : 1);
    if (!h) return 2;
    HIP_OK(hipMemcpy(h, bufs[i], sizes[i], hipMemcpyDeviceToHost));
    if (fwrite(h, 1, sizes[i], out) != sizes[i]) return 2;
    free(h);
  }
  fclose(out);
  HIP_OK(hipStreamDestroy(stream));
  void* all[9] = {x, kr, kc, u, v, y, idx, gates, ws};
  for (int i = 0; i < 9; ++i) HIP_OK(hipFree(all[i]));
  printf("layer ok\n");
  return 0;
}
