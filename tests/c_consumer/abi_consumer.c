/* A plain C11 consumer of the library's C ABI (include/fcngrad.h), built by
 * the CPU tests with gcc and linked against libfcngrad.so. It calls only
 * host-side entry points and argument checks that fail before any device
 * work, so it runs without a GPU.
 *
 * Usage: abi_consumer CAP_BYTES ALIGN_BYTES < numels
 * Reads tensor sizes (backward-completion order) from stdin, then prints
 *   plan NGROUPS
 *   group_of offset_of        (one line per tensor)
 *   group_numel               (one line per group)
 *   out_dims P Q PT QT        (a 3x3 stride-2 pad-1 conv on 4x256x256x256
 *                              and its transposed 4x4 stride-2 pad-1 form)
 *   ws BYTES                  (workspace of that conv's kernel gradient)
 *   kernel NAME               (the kernel its kernel gradient runs)
 *   einval OK|BAD             (null pointers and an unknown op are rejected)
 *   status NAME               (fg_status_string of FG_EUNSUPPORTED)
 */
#include <stdio.h>
#include <stdlib.h>

#include "fcngrad.h"

#define MAX_TENSORS 4096

int main(int argc, char **argv) {
  if (argc != 3) {
    fprintf(stderr, "usage: %s CAP_BYTES ALIGN_BYTES < numels\n", argv[0]);
    return 2;
  }
  const uint64_t cap = strtoull(argv[1], NULL, 10);
  const uint32_t align = (uint32_t)strtoul(argv[2], NULL, 10);
  static uint64_t numel[MAX_TENSORS], offset_of[MAX_TENSORS], group_numel[MAX_TENSORS];
  static int32_t group_of[MAX_TENSORS];
  int32_t n = 0, ngroups = 0;
  unsigned long long v;
  while (n < MAX_TENSORS && scanf("%llu", &v) == 1) numel[n++] = (uint64_t)v;

  fg_status st = grad_group_plan(numel, n, cap, align, 2, group_of, offset_of,
                                 &ngroups, group_numel);
  if (st != FG_OK) {
    printf("plan_error %s\n", fg_status_string(st));
    return 1;
  }
  printf("plan %d\n", ngroups);
  for (int32_t i = 0; i < n; ++i)
    printf("%d %llu\n", group_of[i], (unsigned long long)offset_of[i]);
  for (int32_t g = 0; g < ngroups; ++g)
    printf("%llu\n", (unsigned long long)group_numel[g]);

  /* n, h, w, c, k, r, s, stride_h, stride_w, pad_h, pad_w, x_ld, y_ld */
  fg_conv_desc d = {4, 256, 256, 256, 512, 3, 3, 2, 2, 1, 1, 0, 0};
  fg_conv_desc t = {4, 128, 128, 512, 256, 4, 4, 2, 2, 1, 1, 0, 0};
  int32_t p, q, pt, qt;
  if (fg_conv_out_dims(&d, 0, &p, &q) != FG_OK || fg_conv_out_dims(&t, 1, &pt, &qt) != FG_OK)
    return 1;
  printf("out_dims %d %d %d %d\n", p, q, pt, qt);
  printf("ws %zu\n", fg_conv_workspace_bytes(&d, FG_OP_BWD_WEIGHT));
  printf("kernel %s\n", fg_conv_kernel_name(&d, FG_OP_BWD_WEIGHT));

  /* rejected on the host: no device pointer is touched */
  const int bad =
      conv2d_fwd(&d, NULL, NULL, NULL, FG_EPI_NONE, NULL, NULL, 0, 0) != FG_EINVAL ||
      conv2d_bwd_weight(NULL, NULL, NULL, NULL, NULL, 0, 0) != FG_EINVAL ||
      grad_unscale_check(NULL, 16, 1.0f, NULL, NULL, 0) != FG_EINVAL ||
      fg_conv_out_dims(&d, 2, &p, &q) != FG_EINVAL;
  printf("einval %s\n", bad ? "BAD" : "OK");
  printf("status %s\n", fg_status_string(FG_EUNSUPPORTED));
  return 0;
}
