// Layer-wise adaptive Adam update of the fp32 master weights (Section 6.2,
// Model Implementation: LARS layer-wise rates used with Adam, beta1 0.9 and
// beta2 0.999, L2 weight decay). Per layer, with t the count of applied
// steps including this one:
//   g~ = g + wd w;  m = b1 m + (1-b1) g~;  v = b2 v + (1-b2) g~^2;
//   u = (m / (1-b1^t)) / (sqrt(v / (1-b2^t)) + eps);
//   tau = ||w|| / ||u|| over the layer (1 if either is 0);
//   w = w - lr tau u, and the fp16 working copy = w rounded nearest-even.
// The gradient g is either the fp32 unscaled gradient, or the fp16
// loss-scaled gradient (a group-buffer slot) times 1/S, which is the same
// fp32 value the unscale kernel writes.
//
// Three launches, all bandwidth-bound:
//   1. norms: reads w, m, v, g and sums u^2 and w^2 per workgroup (fixed
//      shape) into the workspace; writes nothing else, so it may run for a
//      group of layers as soon as their gradients exist, while the backward
//      pass still runs;
//   2. ratio: one workgroup per layer adds its partial sums in a fixed order
//      (fp64) and forms tau; the first advances the step count;
//   3. apply: recomputes the new moments and u with the same fp32 operations
//      and writes m, v, w and the fp16 copy; it may run per range of layers
//      (e.g. each just before the next forward pass reads that layer).
// A step whose gradient groups were flagged non-finite is skipped on the
// device: the ratio and apply kernels read the flags and return, so the host
// never waits.
#include <cmath>

#include "common.h"
#include "internal.h"

namespace fg {

constexpr int kOptThreads = 256;
constexpr int kOptIters = 4;                            // 4-element chunks per thread
constexpr int kOptElems = kOptThreads * 4 * kOptIters;  // per workgroup

struct OptPiece {
  uint64_t w32, w16, m, v, g;
  uint32_t numel, block0;
};
struct OptTable {
  int32_t n;
  uint32_t nblocks;
  OptPiece p[FG_MAX_SEGMENTS];
};
struct OptParams {
  float lr, b1, b2, eps, wd;
};

__device__ __forceinline__ int opt_piece(const OptTable &t, uint32_t b) {
  int lo = 0, hi = t.n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (t.p[mid].block0 <= b) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__device__ __forceinline__ bool opt_skip(const int32_t *flags, int nflags) {
  bool any = false;
  for (int i = 0; i < nflags; ++i) any |= flags[i] != 0;
  return any;
}

// Per-step constants. The bias corrections 1 - b^t are formed in fp64 (in
// fp32 the rounding of b^t would be amplified ~1/(1-b2) times for small t)
// and enter as reciprocals; u uses the hardware square root and reciprocal
// (about one ulp each), a few ulps from the correctly rounded quotient.
struct OptStep {
  float b1, c1, b2, c2, eps, wd, rbc1, rbc2;
  __device__ __forceinline__ void moments(float g, float w, float &m, float &v) const {
    const float gt = g + wd * w;
    m = b1 * m + c1 * gt;
    v = b2 * v + c2 * (gt * gt);
  }
  __device__ __forceinline__ float u(float m, float v) const {
    const float den = __builtin_amdgcn_sqrtf(v * rbc2) + eps;
    return (m * rbc1) * __builtin_amdgcn_rcpf(den);
  }
};

__device__ __forceinline__ OptStep opt_step(const OptParams &p, int t) {
  const double bc1 = 1.0 - pow((double)p.b1, (double)t);
  const double bc2 = 1.0 - pow((double)p.b2, (double)t);
  return OptStep{p.b1, 1.f - p.b1, p.b2, 1.f - p.b2, p.eps, p.wd,
                 (float)(1.0 / bc1), (float)(1.0 / bc2)};
}

// The fp16 copy must be the rounding of the fp32 weight as stored. Without a
// barrier the compiler folds the conversion into the update's fma (a mixed
// fma that rounds the exact result once, to fp16), which differs from the
// two-step rounding on fp32 ties.
__device__ __forceinline__ uint16_t stored_f32_to_h(float v) {
  asm volatile("" : "+v"(v));
  return f32_to_h(v);
}

// Gradient access: fp32 as stored, or fp16 times 1/S (materialised before
// use, so that the update sees the same fp32 value in both forms).
template <bool H>
struct Grad {
  uint64_t p;
  float inv;
  __device__ __forceinline__ f32x4 load4(uint32_t i) const {
    if constexpr (H) {
      const u32x2 h = *reinterpret_cast<const u32x2 *>(
          reinterpret_cast<const uint16_t *>(p) + i);
      f32x4 g;
      g[0] = h_to_f32((uint16_t)h[0]) * inv;
      g[1] = h_to_f32((uint16_t)(h[0] >> 16)) * inv;
      g[2] = h_to_f32((uint16_t)h[1]) * inv;
      g[3] = h_to_f32((uint16_t)(h[1] >> 16)) * inv;
#pragma unroll
      for (int e = 0; e < 4; ++e) asm volatile("" : "+v"(g[e]));
      return g;
    } else {
      return *reinterpret_cast<const f32x4 *>(reinterpret_cast<const float *>(p) + i);
    }
  }
  __device__ __forceinline__ float load1(uint32_t j) const {
    if constexpr (H) {
      float g = h_to_f32(reinterpret_cast<const uint16_t *>(p)[j]) * inv;
      asm volatile("" : "+v"(g));
      return g;
    } else {
      return reinterpret_cast<const float *>(p)[j];
    }
  }
};

// One 4-element chunk of a layer's arrays, zero beyond the layer's end
// (zeros add nothing to either sum).
template <bool H>
__device__ __forceinline__ void load_chunk(const OptPiece &pc, const Grad<H> &gr,
                                           uint32_t i, uint32_t end, f32x4 &g,
                                           f32x4 &w, f32x4 &m, f32x4 &v) {
  const float *wp = reinterpret_cast<const float *>(pc.w32);
  const float *mp = reinterpret_cast<const float *>(pc.m);
  const float *vp = reinterpret_cast<const float *>(pc.v);
  if (i + 4 <= end) {
    g = gr.load4(i);
    w = *reinterpret_cast<const f32x4 *>(wp + i);
    m = *reinterpret_cast<const f32x4 *>(mp + i);
    v = *reinterpret_cast<const f32x4 *>(vp + i);
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bool in = i + e < end;
      g[e] = in ? gr.load1(i + e) : 0.f;
      w[e] = in ? wp[i + e] : 0.f;
      m[e] = in ? mp[i + e] : 0.f;
      v[e] = in ? vp[i + e] : 0.f;
    }
  }
}

// sums of two values over the workgroup, fixed order: wave shuffles, then
// the four wave results in order (thread 0 holds the result)
template <typename T>
__device__ __forceinline__ void block_sum2(T &a, T &b) {
  __shared__ T red[2][kOptThreads / 64];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    a += __shfl_down(a, o, 64);
    b += __shfl_down(b, o, 64);
  }
  if ((threadIdx.x & 63) == 0) {
    red[0][threadIdx.x >> 6] = a;
    red[1][threadIdx.x >> 6] = b;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    a = red[0][0];
    b = red[1][0];
#pragma unroll
    for (int wv = 1; wv < kOptThreads / 64; ++wv) {
      a += red[0][wv];
      b += red[1][wv];
    }
  }
}

// Workgroup b0 + blockIdx.x of the table: sum of u^2 and of w^2 over its
// kOptElems elements into part[2b], part[2b+1].
template <bool H>
__global__ __launch_bounds__(kOptThreads) void lars_adam_norms_kernel(
    OptTable t, OptParams p, float inv, const int32_t *step_count, uint32_t b0,
    float *part) {
  const uint32_t b = b0 + blockIdx.x;
  const OptPiece pc = t.p[opt_piece(t, b)];
  const OptStep s = opt_step(p, *step_count + 1);
  const Grad<H> gr{pc.g, inv};
  const uint32_t beg = (b - pc.block0) * (uint32_t)kOptElems;
  const uint32_t end = min(pc.numel, beg + (uint32_t)kOptElems);
  f32x4 g[kOptIters], w[kOptIters], m[kOptIters], v[kOptIters];
#pragma unroll
  for (int c = 0; c < kOptIters; ++c) {
    const uint32_t i = beg + (c * kOptThreads + threadIdx.x) * 4;
    load_chunk<H>(pc, gr, i, end, g[c], w[c], m[c], v[c]);
  }
  float su = 0.f, sw = 0.f;
#pragma unroll
  for (int c = 0; c < kOptIters; ++c) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float mm = m[c][e], vv = v[c][e];
      s.moments(g[c][e], w[c][e], mm, vv);
      const float u = s.u(mm, vv);
      su += u * u;
      sw += w[c][e] * w[c][e];
    }
  }
  block_sum2(su, sw);
  if (threadIdx.x == 0) {
    part[2 * b] = su;
    part[2 * b + 1] = sw;
  }
}

// One workgroup per layer: tau from the layer's partial sums (fp64, fixed
// order). Workgroup 0 advances the step count.
__global__ __launch_bounds__(kOptThreads) void lars_adam_ratio_kernel(
    OptTable t, const int32_t *flags, int nflags, int32_t *step_count,
    const float *part, float *ratio, int32_t *t_cur) {
  if (opt_skip(flags, nflags)) return;
  const int l = blockIdx.x;
  const uint32_t b0 = t.p[l].block0;
  const uint32_t b1 = l + 1 < t.n ? t.p[l + 1].block0 : t.nblocks;
  double su = 0.0, sw = 0.0;
  for (uint32_t b = b0 + threadIdx.x; b < b1; b += kOptThreads) {
    su += (double)part[2 * b];
    sw += (double)part[2 * b + 1];
  }
  block_sum2(su, sw);
  if (threadIdx.x == 0) {
    ratio[l] = su > 0.0 && sw > 0.0 ? (float)(sqrt(sw) / sqrt(su)) : 1.f;
    if (l == 0) {
      const int32_t tn = *step_count + 1;
      *t_cur = tn;
      *step_count = tn;
    }
  }
}

// Workgroup b0 + blockIdx.x of the table.
template <bool H>
__global__ __launch_bounds__(kOptThreads) void lars_adam_apply_kernel(
    OptTable t, OptParams p, float inv, const int32_t *flags, int nflags,
    const float *ratio, const int32_t *t_cur, uint32_t b0) {
  if (opt_skip(flags, nflags)) return;
  const uint32_t b = b0 + blockIdx.x;
  const int pi = opt_piece(t, b);
  const OptPiece pc = t.p[pi];
  const OptStep s = opt_step(p, *t_cur);
  const float step = p.lr * ratio[pi];
  const Grad<H> gr{pc.g, inv};
  float *wp = reinterpret_cast<float *>(pc.w32);
  float *mp = reinterpret_cast<float *>(pc.m);
  float *vp = reinterpret_cast<float *>(pc.v);
  uint16_t *hp = reinterpret_cast<uint16_t *>(pc.w16);
  const uint32_t beg = (b - pc.block0) * (uint32_t)kOptElems;
  const uint32_t end = min(pc.numel, beg + (uint32_t)kOptElems);
  f32x4 g[kOptIters], w[kOptIters], m[kOptIters], v[kOptIters];
#pragma unroll
  for (int c = 0; c < kOptIters; ++c) {
    const uint32_t i = beg + (c * kOptThreads + threadIdx.x) * 4;
    load_chunk<H>(pc, gr, i, end, g[c], w[c], m[c], v[c]);
  }
#pragma unroll
  for (int c = 0; c < kOptIters; ++c) {
    const uint32_t i = beg + (c * kOptThreads + threadIdx.x) * 4;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float mm = m[c][e], vv = v[c][e];
      s.moments(g[c][e], w[c][e], mm, vv);
      m[c][e] = mm;
      v[c][e] = vv;
      w[c][e] = w[c][e] - step * s.u(mm, vv);
    }
    if (i + 4 <= end) {
      *reinterpret_cast<f32x4 *>(mp + i) = m[c];
      *reinterpret_cast<f32x4 *>(vp + i) = v[c];
      *reinterpret_cast<f32x4 *>(wp + i) = w[c];
      u32x2 h;
      h[0] = (uint32_t)stored_f32_to_h(w[c][0]) |
             ((uint32_t)stored_f32_to_h(w[c][1]) << 16);
      h[1] = (uint32_t)stored_f32_to_h(w[c][2]) |
             ((uint32_t)stored_f32_to_h(w[c][3]) << 16);
      *reinterpret_cast<u32x2 *>(hp + i) = h;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (i + e < end) {
          mp[i + e] = m[c][e];
          vp[i + e] = v[c][e];
          wp[i + e] = w[c][e];
          hp[i + e] = stored_f32_to_h(w[c][e]);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
static void opt_table(const fg_opt_tensor *ts, int32_t n, OptTable &t) {
  uint32_t nb = 0;
  t.n = n;
  for (int i = 0; i < n; ++i) {
    t.p[i] = OptPiece{ts[i].w32, ts[i].w16, ts[i].m, ts[i].v, ts[i].g,
                      (uint32_t)ts[i].numel, nb};
    nb += (uint32_t)((ts[i].numel + kOptElems - 1) / kOptElems);
  }
  t.nblocks = nb;
}

struct OptWs {
  float *part, *ratio;
  int32_t *t_cur;
};

// workspace: [2 * nblocks floats of partial sums][ratio per layer][t]
static OptWs opt_ws(void *ws, uint32_t nb) {
  float *part = reinterpret_cast<float *>(ws);
  float *ratio = part + 2 * (size_t)nb;
  return OptWs{part, ratio, reinterpret_cast<int32_t *>(ratio + FG_MAX_SEGMENTS)};
}

size_t lars_adam_ws_bytes(const fg_opt_tensor *ts, int32_t n) {
  OptTable t;
  opt_table(ts, n, t);
  return (size_t)t.nblocks * 2 * sizeof(float) + (size_t)FG_MAX_SEGMENTS * sizeof(float) +
         16;
}

static OptParams opt_params(const fg_opt_params &p) {
  return OptParams{p.lr, p.beta1, p.beta2, p.eps, p.weight_decay};
}

// blocks of layers [first, first + count)
static void block_range(const OptTable &t, int32_t first, int32_t count, uint32_t &b0,
                        uint32_t &b1) {
  b0 = t.p[first].block0;
  b1 = first + count < t.n ? t.p[first + count].block0 : t.nblocks;
}

hipError_t launch_lars_adam_norms(const fg_opt_tensor *ts, int32_t n, int32_t first,
                                  int32_t count, const fg_opt_params &pp, bool fp16_grad,
                                  float inv_scale, const int32_t *step_count, void *ws,
                                  hipStream_t st) {
  OptTable t;
  opt_table(ts, n, t);
  const OptParams p = opt_params(pp);
  uint32_t b0, b1;
  block_range(t, first, count, b0, b1);
  const OptWs w = opt_ws(ws, t.nblocks);
  if (fp16_grad)
    hipLaunchKernelGGL(lars_adam_norms_kernel<true>, dim3(b1 - b0), dim3(kOptThreads), 0,
                       st, t, p, inv_scale, step_count, b0, w.part);
  else
    hipLaunchKernelGGL(lars_adam_norms_kernel<false>, dim3(b1 - b0), dim3(kOptThreads), 0,
                       st, t, p, inv_scale, step_count, b0, w.part);
  return hipGetLastError();
}

hipError_t launch_lars_adam_apply(const fg_opt_tensor *ts, int32_t n, int32_t first,
                                  int32_t count, bool with_ratio, const fg_opt_params &pp,
                                  bool fp16_grad, float inv_scale, const int32_t *flags,
                                  int32_t nflags, int32_t *step_count, void *ws,
                                  hipStream_t st) {
  OptTable t;
  opt_table(ts, n, t);
  const OptParams p = opt_params(pp);
  const OptWs w = opt_ws(ws, t.nblocks);
  if (with_ratio) {
    hipLaunchKernelGGL(lars_adam_ratio_kernel, dim3(n), dim3(kOptThreads), 0, st, t,
                       flags, nflags, step_count, w.part, w.ratio, w.t_cur);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  uint32_t b0, b1;
  block_range(t, first, count, b0, b1);
  if (fp16_grad)
    hipLaunchKernelGGL(lars_adam_apply_kernel<true>, dim3(b1 - b0), dim3(kOptThreads), 0,
                       st, t, p, inv_scale, flags, nflags, w.ratio, w.t_cur, b0);
  else
    hipLaunchKernelGGL(lars_adam_apply_kernel<false>, dim3(b1 - b0), dim3(kOptThreads), 0,
                       st, t, p, inv_scale, flags, nflags, w.ratio, w.t_cur, b0);
  return hipGetLastError();
}

}  // namespace fg
