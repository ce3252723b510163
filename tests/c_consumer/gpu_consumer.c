/* A plain C11 program that runs convolution passes through the C ABI with
 * device memory of its own (hipMalloc), no Python or PyTorch involved.
 *
 * Usage: gpu_consumer IN OUT N H W C K R STRIDE PAD
 * IN holds the fp16 bit patterns of x (N*H*W*C), w (K*R*R*C) and dy
 * (N*P*Q*K), in that order; OUT receives y = conv2d_fwd(x, w) (N*P*Q*K),
 * dx = conv2d_bwd_data(dy, w) (N*H*W*C) and dw = conv2d_bwd_weight(x, dy)
 * (K*R*R*C), in that order. Exit status 0 on success; a failing call
 * prints its status string. */
#include <stdio.h>
#include <stdlib.h>

#include "fcngrad.h"

static int check_hip(hipError_t e, const char *what) {
  if (e != hipSuccess) {
    fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
    return 1;
  }
  return 0;
}

static int check_fg(fg_status s, const char *what) {
  if (s != FG_OK) {
    fprintf(stderr, "%s: %s\n", what, fg_status_string(s));
    return 1;
  }
  return 0;
}

int main(int argc, char **argv) {
  if (argc != 11) {
    fprintf(stderr, "usage: %s IN OUT N H W C K R STRIDE PAD\n", argv[0]);
    return 2;
  }
  const int n = atoi(argv[3]), h = atoi(argv[4]), w = atoi(argv[5]), c = atoi(argv[6]);
  const int k = atoi(argv[7]), r = atoi(argv[8]), st = atoi(argv[9]), pd = atoi(argv[10]);
  fg_conv_desc d = {n, h, w, c, k, r, r, st, st, pd, pd, 0, 0};
  int32_t p, q;
  if (check_fg(fg_conv_out_dims(&d, 0, &p, &q), "fg_conv_out_dims")) return 1;
  const size_t nx = (size_t)n * h * w * c, nw = (size_t)k * r * r * c;
  const size_t ny = (size_t)n * p * q * k;
  const size_t total_in = nx + nw + ny, total_out = ny + nx + nw;
  uint16_t *hin = malloc(total_in * 2), *hout = malloc(total_out * 2);
  if (!hin || !hout) return 1;
  FILE *f = fopen(argv[1], "rb");
  if (!f || fread(hin, 2, total_in, f) != total_in) {
    fprintf(stderr, "cannot read %s\n", argv[1]);
    return 1;
  }
  fclose(f);

  size_t ws_bytes = 0;
  const int ops[3] = {FG_OP_FWD, FG_OP_BWD_DATA, FG_OP_BWD_WEIGHT};
  for (int i = 0; i < 3; ++i) {
    const size_t b = fg_conv_workspace_bytes(&d, ops[i]);
    if (b > ws_bytes) ws_bytes = b;
  }
  void *din = NULL, *dout = NULL, *ws = NULL;
  if (check_hip(hipMalloc(&din, total_in * 2), "hipMalloc in") ||
      check_hip(hipMalloc(&dout, total_out * 2), "hipMalloc out") ||
      (ws_bytes && check_hip(hipMalloc(&ws, ws_bytes), "hipMalloc ws")) ||
      check_hip(hipMemcpy(din, hin, total_in * 2, hipMemcpyHostToDevice), "copy in"))
    return 1;
  const uint16_t *x = din, *wt = (const uint16_t *)din + nx, *dy = (const uint16_t *)din + nx + nw;
  uint16_t *y = dout, *dx = (uint16_t *)dout + ny, *dw = (uint16_t *)dout + ny + nx;
  if (check_fg(conv2d_fwd(&d, x, wt, y, FG_EPI_NONE, NULL, ws, ws_bytes, 0), "conv2d_fwd") ||
      check_fg(conv2d_bwd_data(&d, dy, wt, dx, FG_EPI_NONE, NULL, ws, ws_bytes, 0),
               "conv2d_bwd_data") ||
      check_fg(conv2d_bwd_weight(&d, x, dy, dw, ws, ws_bytes, 0), "conv2d_bwd_weight") ||
      check_hip(hipDeviceSynchronize(), "synchronize") ||
      check_hip(hipMemcpy(hout, dout, total_out * 2, hipMemcpyDeviceToHost), "copy out"))
    return 1;
  f = fopen(argv[2], "wb");
  if (!f || fwrite(hout, 2, total_out, f) != total_out) return 1;
  fclose(f);
  hipFree(din);
  hipFree(dout);
  if (ws) hipFree(ws);
  free(hin);
  free(hout);
  printf("ok %zu %zu %zu\n", ny, nx, nw);
  return 0;
}
