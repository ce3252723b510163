// Host-side interface between the C-ABI layer (abi.hip) and the kernel
// launchers. Not part of the public API.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <algorithm>

#include "fcngrad.h"

namespace fg {

// One output phase of a data convolution (forward, input gradient or
// transposed forward) written as an implicit GEMM over the taps that reach
// it. Output positions (a, b) of the phase land at image position
// (a*ostr + ooh, b*ostr + oow); tap (i, j) reads the input at
// (a*istr + dh0 + dstep*i, b*istr + dw0 + dstep*j) and the kernel element
// (r0 + rstep*i, s0 + rstep*j).
struct Phase {
  int32_t mh, mw;
  int32_t ooh, oow;
  int32_t nr, ns;
  int32_t dh0, dw0, dstep;
  int32_t r0, s0, rstep;
};

struct DataConvArgs {
  const uint16_t *act;   // input image  [n][hi][wi][cr]
  const uint16_t *wgt;   // weights (layout per w_kmajor)
  uint16_t *out;         // output image [n][ho][wo][co], pixel stride ldo
  const uint16_t *gate;  // laid out like out (FG_EPI_GATE) or null
  int32_t n, hi, wi, cr;
  int32_t ldi;           // pixel stride of act, elements (>= cr)
  int32_t ho, wo, co;
  int32_t ldo;           // pixel stride of out (and gate), elements (>= co)
  int32_t istr, ostr;
  int32_t s;             // kernel width
  // weight element (co, r, s, cr):
  //   k-major:  wgt[co*ldw + (r*S + s)*cr_stride + cr]
  //   mn-major: wgt[cr*w_red + (r*S + s)*w_tap + co]
  int32_t ldw, w_red, w_tap;
  int32_t wbytes;        // size of the weight tensor in bytes
  int32_t epi;
  int32_t nphase;
  int32_t nsplit;        // reduction split (set by the launcher)
  float *part;           // [nsplit][n*ho*wo*co] fp32 partials (nsplit > 1)
  Phase ph[4];
};

// Tile and split choice for a data convolution (pure host logic).
struct DataPlan {
  bool big;              // 256 x 256 tiles (else 128 x 128)
  int32_t nsplit;
  size_t ws_bytes;
};
DataPlan plan_data_conv(const DataConvArgs &a);

// Bytes from the first element of act to the last one a convolution reads
// (the span a buffer resource must cover).
__host__ __device__ inline size_t act_span_bytes(const DataConvArgs &a) {
  const size_t npix = (size_t)a.n * a.hi * a.wi;
  return npix ? ((npix - 1) * (size_t)a.ldi + (size_t)a.cr) * 2 : 0;
}

struct WgradArgs {
  const uint16_t *x;     // [n][h][w][c]
  const uint16_t *dy;    // [n][p][q][k]
  uint16_t *dw;          // [k][r][s][c] fp16 (single split)
  float *part;           // [nsplit][k][r*s*c] fp32 partials (nsplit > 1)
  int32_t n, h, w, c, k, r, s, p, q;
  int32_t ldx;           // pixel stride of x, elements (>= c)
  int32_t sh, sw, ph, pw;
  int32_t mtot;          // n*p*q
  int32_t mchunk;        // reduction rows per split, multiple of 64
  int32_t nsplit;
  int32_t *flag;         // set to 1 if an fp16 dW value is +-inf/NaN, or null
};

// Kernel selection for a shape; pure host logic, shared by the workspace
// query and the launchers so both always agree.
struct WgradPlan {
  bool big;              // 256 x 256 tiles (else 128 x 128)
  int32_t nsplit, mchunk;
  size_t ws_bytes;
};
// Split and tile plan of a kernel gradient; the fp32 partials of a split take
// ws_bytes <= max_ws_bytes (fewer splits when the best plan needs more).
WgradPlan plan_wgrad(const fg_conv_desc &d, int32_t p, int32_t q,
                     size_t max_ws_bytes = SIZE_MAX);

// The same span for the kernel gradient's x.
__host__ __device__ inline size_t x_span_bytes(const WgradArgs &a) {
  const size_t npix = (size_t)a.n * a.h * a.w;
  return npix ? ((npix - 1) * (size_t)a.ldx + (size_t)a.c) * 2 : 0;
}
size_t head_wgrad_ws_bytes(const fg_conv_desc &d);

hipError_t launch_data_conv(const DataConvArgs &a, bool w_kmajor,
                            hipStream_t st);
const char *data_conv_kernel_name(const DataConvArgs &a, bool w_kmajor);
const char *wgrad_kernel_name(const fg_conv_desc &d);
hipError_t launch_wgrad(const WgradArgs &a, bool big, hipStream_t st);

// LDS-DMA kernels (256 x 256 tiles): applicability and launchers.
bool data_dma_ok(const DataConvArgs &a);
// Stride-1 3x3 data convolution whose tile is whole output rows: the
// input-reuse kernel (conv_dma.hip) applies.
bool data_halo_ok(const DataConvArgs &a);
hipError_t launch_data_conv_halo(const DataConvArgs &a, bool w_kmajor,
                                 hipStream_t st);
bool wgrad_dma_ok(const WgradArgs &a);
// The same with 128 x 128 tiles (two workgroups per CU).
hipError_t launch_data_conv_dma_small(const DataConvArgs &a, bool w_kmajor,
                                      hipStream_t st);
hipError_t launch_data_conv_dma(const DataConvArgs &a, bool w_kmajor,
                                hipStream_t st);
hipError_t launch_wgrad_dma(const WgradArgs &a, hipStream_t st);
hipError_t launch_head_fwd(const uint16_t *x, const uint16_t *w, uint16_t *y,
                           int64_t npix, int32_t c, int32_t epi,
                           const uint16_t *gate, hipStream_t st);
hipError_t launch_head_bwd_data(const uint16_t *dy, const uint16_t *w,
                                uint16_t *dx, int64_t npix, int32_t c,
                                int32_t epi, const uint16_t *gate,
                                hipStream_t st);
size_t lars_adam_ws_bytes(const fg_opt_tensor *ts, int32_t n);
hipError_t launch_lars_adam_norms(const fg_opt_tensor *ts, int32_t n, int32_t first,
                                  int32_t count, const fg_opt_params &p, bool fp16_grad,
                                  float inv_scale, const int32_t *step_count, void *ws,
                                  hipStream_t st);
hipError_t launch_lars_adam_apply(const fg_opt_tensor *ts, int32_t n, int32_t first,
                                  int32_t count, bool with_ratio, const fg_opt_params &p,
                                  bool fp16_grad, float inv_scale, const int32_t *flags,
                                  int32_t nflags, int32_t *step_count, void *ws,
                                  hipStream_t st);
hipError_t launch_huber_head_grad(const uint16_t *y, const float *t, uint64_t numel,
                                  double scale, double delta, uint16_t *dy,
                                  hipStream_t st);
hipError_t launch_avg_pool2d_fwd(const uint16_t *x, int32_t n, int32_t h, int32_t w,
                                 int32_t c, uint16_t *y, hipStream_t st);
hipError_t launch_avg_pool2d_bwd(const uint16_t *dy, const uint16_t *gate, int32_t n,
                                 int32_t h, int32_t w, int32_t c, uint16_t *dx,
                                 hipStream_t st);
hipError_t launch_channel_slice_copy(const uint16_t *src, int32_t src_ld,
                                     const uint16_t *gate, int32_t gate_ld, uint16_t *dst,
                                     int32_t dst_ld, int64_t npix, int32_t nch,
                                     bool accumulate, hipStream_t st);
hipError_t launch_head_wgrad(const uint16_t *x, const uint16_t *dy,
                             uint16_t *dw, int64_t npix, int32_t c,
                             float *ws, int32_t *flag, hipStream_t st);

// One-shot profiling events (fg_profile_next_launch): prof_begin records the
// armed start event on the stream, prof_end the stop event, then disarms.
// Both do nothing when no events are armed.
hipError_t prof_begin(hipStream_t st);
hipError_t prof_end(hipStream_t st);

// Register-only MFMA chains (fg_mfma_loop): blocks x 256 threads, each
// writing one float to out.
hipError_t launch_mfma_loop(float *out, int32_t blocks, int32_t iters, int32_t mode,
                            hipStream_t st);

hipError_t launch_flags_clear(int32_t *flags, int32_t n, hipStream_t st);
hipError_t launch_pack(const fg_segment *segs, int32_t nseg, uint16_t *group,
                       uint64_t group_numel, hipStream_t st);
hipError_t launch_unscale(const uint16_t *group, uint64_t numel,
                          float inv_scale, float *out, int32_t *flag,
                          hipStream_t st);
hipError_t launch_unpack(const float *group, const fg_segment *segs,
                         int32_t nseg, hipStream_t st);
hipError_t launch_head_grad(const uint16_t *y, const float *t, uint64_t numel,
                            double scale, uint16_t *dy, hipStream_t st);
hipError_t launch_relu_backward(const uint16_t *dy, const uint16_t *act,
                                uint64_t numel, uint16_t *out,
                                hipStream_t st);

}  // namespace fg
