// Bandwidth-bound glue of the FC-DenseNet variant of the network (Section
// 6.2, Neural Network Architecture: dense blocks with growth rate 256,
// average pooling in place of max pooling; Model Implementation: Huber
// loss). All of them compute a value with a plain definition exactly (or in
// fp64) and round it once to fp16, nearest-even:
//   * huber_head_grad: dy = S/numel * clamp(y - t, -delta, delta), the
//     gradient of the loss-scaled mean Huber loss;
//   * avg_pool2d 2x2 stride 2 (NHWC): forward mean of the four inputs;
//     backward a quarter of the output gradient to each input, optionally
//     gated by a ReLU output (zero where the gate is <= 0);
//   * channel_slice_copy: per pixel, nch channels from one NHWC buffer to
//     another with other pixel strides (dense concatenation forward and its
//     slice gradients backward), optionally gated and optionally added to
//     what the destination holds.
// Threads move 8 channels (16 bytes) at a time: every channel count and
// pixel stride is a multiple of 8 and every pointer 16-byte aligned.
#include "common.h"
#include "internal.h"

namespace fg {

constexpr int kDenseThreads = 256;

typedef uint16_t h8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ h8 load8(const uint16_t *p) {
  return *reinterpret_cast<const h8 *>(p);
}
__device__ __forceinline__ void store8(uint16_t *p, const h8 &v) {
  *reinterpret_cast<h8 *>(p) = v;
}

static unsigned grid_for(uint64_t items) {
  uint64_t b = (items + kDenseThreads - 1) / kDenseThreads;
  return (unsigned)(b > 8192 ? 8192 : (b ? b : 1));
}

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kDenseThreads) void huber_head_grad_kernel(
    const uint16_t *y, const float *t, uint32_t numel, double scale, double delta,
    uint16_t *dy) {
  const uint32_t stride = gridDim.x * kDenseThreads;
  for (uint32_t i = blockIdx.x * kDenseThreads + threadIdx.x; i < numel; i += stride) {
    double d = (double)h_to_f32(y[i]) - (double)t[i];
    d = d > delta ? delta : (d < -delta ? -delta : d);
    dy[i] = f64_to_h(d * scale);
  }
}

hipError_t launch_huber_head_grad(const uint16_t *y, const float *t, uint64_t numel,
                                  double scale, double delta, uint16_t *dy,
                                  hipStream_t st) {
  hipLaunchKernelGGL(huber_head_grad_kernel, dim3(grid_for(numel)), dim3(kDenseThreads),
                     0, st, y, t, (uint32_t)numel, scale, delta, dy);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// One item: 8 channels of one output pixel.
__global__ __launch_bounds__(kDenseThreads) void avg_pool2d_fwd_kernel(
    const uint16_t *x, uint32_t h, uint32_t w, uint32_t c, uint32_t items,
    uint16_t *y) {
  const uint32_t c8 = c / 8, q = w / 2, p = h / 2;
  const uint32_t stride = gridDim.x * kDenseThreads;
  for (uint32_t it = blockIdx.x * kDenseThreads + threadIdx.x; it < items; it += stride) {
    const uint32_t cc = (it % c8) * 8;
    uint32_t pix = it / c8;
    const uint32_t oq = pix % q;
    pix /= q;
    const uint32_t op = pix % p;
    const uint32_t n = pix / p;
    const uint16_t *x0 = x + ((uint64_t)(n * h + 2 * op) * w + 2 * oq) * c + cc;
    const h8 a = load8(x0), b = load8(x0 + c), d = load8(x0 + (uint64_t)w * c),
             e = load8(x0 + (uint64_t)w * c + c);
    h8 o;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      // four fp16 values add exactly in fp64; the quarter is exact too
      const double s = ((double)h_to_f32(a[k]) + (double)h_to_f32(b[k])) +
                       ((double)h_to_f32(d[k]) + (double)h_to_f32(e[k]));
      o[k] = f64_to_h(s * 0.25);
    }
    store8(y + (uint64_t)it * 8, o);
  }
}

__global__ __launch_bounds__(kDenseThreads) void avg_pool2d_bwd_kernel(
    const uint16_t *dy, const uint16_t *gate, uint32_t h, uint32_t w, uint32_t c,
    uint32_t items, uint16_t *dx) {
  const uint32_t c8 = c / 8, q = w / 2, p = h / 2;
  const uint32_t stride = gridDim.x * kDenseThreads;
  for (uint32_t it = blockIdx.x * kDenseThreads + threadIdx.x; it < items; it += stride) {
    const uint32_t cc = (it % c8) * 8;
    uint32_t pix = it / c8;
    const uint32_t oq = pix % q;
    pix /= q;
    const uint32_t op = pix % p;
    const uint32_t n = pix / p;
    const h8 g = load8(dy + (uint64_t)it * 8);
    h8 v;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      // a quarter of an fp16 value is exact in fp32; one rounding to fp16
      const _Float16 r = (_Float16)(h_to_f32(g[k]) * 0.25f);
      v[k] = __builtin_bit_cast(uint16_t, r);
    }
    const uint64_t base = ((uint64_t)(n * h + 2 * op) * w + 2 * oq) * c + cc;
    const uint64_t off[4] = {0, c, (uint64_t)w * c, (uint64_t)w * c + c};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      h8 o = v;
      if (gate) {
        const h8 gt = load8(gate + base + off[j]);
#pragma unroll
        for (int k = 0; k < 8; ++k) o[k] = h_to_f32(gt[k]) > 0.f ? v[k] : (uint16_t)0;
      }
      store8(dx + base + off[j], o);
    }
  }
}

hipError_t launch_avg_pool2d_fwd(const uint16_t *x, int32_t n, int32_t h, int32_t w,
                                 int32_t c, uint16_t *y, hipStream_t st) {
  const uint64_t items = (uint64_t)n * (h / 2) * (w / 2) * (c / 8);
  hipLaunchKernelGGL(avg_pool2d_fwd_kernel, dim3(grid_for(items)), dim3(kDenseThreads), 0,
                     st, x, (uint32_t)h, (uint32_t)w, (uint32_t)c, (uint32_t)items, y);
  return hipGetLastError();
}

hipError_t launch_avg_pool2d_bwd(const uint16_t *dy, const uint16_t *gate, int32_t n,
                                 int32_t h, int32_t w, int32_t c, uint16_t *dx,
                                 hipStream_t st) {
  const uint64_t items = (uint64_t)n * (h / 2) * (w / 2) * (c / 8);
  hipLaunchKernelGGL(avg_pool2d_bwd_kernel, dim3(grid_for(items)), dim3(kDenseThreads), 0,
                     st, dy, gate, (uint32_t)h, (uint32_t)w, (uint32_t)c, (uint32_t)items,
                     dx);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
template <bool ACC>
__global__ __launch_bounds__(kDenseThreads) void channel_slice_copy_kernel(
    const uint16_t *src, uint32_t src_ld, const uint16_t *gate, uint32_t gate_ld,
    uint16_t *dst, uint32_t dst_ld, uint32_t nch, uint32_t items) {
  const uint32_t c8 = nch / 8;
  const uint32_t stride = gridDim.x * kDenseThreads;
  for (uint32_t it = blockIdx.x * kDenseThreads + threadIdx.x; it < items; it += stride) {
    const uint32_t cc = (it % c8) * 8;
    const uint64_t px = it / c8;
    h8 v = load8(src + px * src_ld + cc);
    if (gate) {
      const h8 g = load8(gate + px * gate_ld + cc);
#pragma unroll
      for (int k = 0; k < 8; ++k) v[k] = h_to_f32(g[k]) > 0.f ? v[k] : (uint16_t)0;
    }
    uint16_t *d = dst + px * dst_ld + cc;
    if constexpr (ACC) {
      const h8 o = load8(d);
#pragma unroll
      for (int k = 0; k < 8; ++k)
        v[k] = f64_to_h((double)h_to_f32(o[k]) + (double)h_to_f32(v[k]));
    }
    store8(d, v);
  }
}

hipError_t launch_channel_slice_copy(const uint16_t *src, int32_t src_ld,
                                     const uint16_t *gate, int32_t gate_ld, uint16_t *dst,
                                     int32_t dst_ld, int64_t npix, int32_t nch,
                                     bool accumulate, hipStream_t st) {
  const uint64_t items = (uint64_t)npix * (nch / 8);
  if (accumulate)
    hipLaunchKernelGGL(channel_slice_copy_kernel<true>, dim3(grid_for(items)),
                       dim3(kDenseThreads), 0, st, src, (uint32_t)src_ld, gate,
                       (uint32_t)gate_ld, dst, (uint32_t)dst_ld, (uint32_t)nch,
                       (uint32_t)items);
  else
    hipLaunchKernelGGL(channel_slice_copy_kernel<false>, dim3(grid_for(items)),
                       dim3(kDenseThreads), 0, st, src, (uint32_t)src_ld, gate,
                       (uint32_t)gate_ld, dst, (uint32_t)dst_ld, (uint32_t)nch,
                       (uint32_t)items);
  return hipGetLastError();
}

}  // namespace fg
