// Layer-wise adaptive Adam update of the fp32 master weights (Section 6.2,
// Model Implementation: LARS layer-wise rates used with Adam, beta1 0.9 and
// beta2 0.999), consuming the unscaled fp32 gradients the unpack writes.
// Per layer, with t the count of applied steps including this one:
//   g~ = g + wd w;  m = b1 m + (1-b1) g~;  v = b2 v + (1-b2) g~^2;
//   u = (m / (1-b1^t)) / (sqrt(v / (1-b2^t)) + eps);
//   tau = ||w|| / ||u|| over the layer (1 if either is 0);
//   w = w - lr tau u, and the fp16 working copy = w rounded nearest-even.
// A step whose gradient groups were flagged non-finite is skipped on the
// device: every kernel reads the flags and returns, so the host never waits.
// Three launches, all bandwidth-bound:
//   1. moments: new m, v; per-workgroup sums of u^2 and w^2 (fixed-shape
//      reduction) into the workspace;
//   2. ratio: one thread per layer adds its workgroups' sums in order (fp64)
//      and forms tau; thread 0 advances the step count;
//   3. apply: recomputes u from the stored moments (the same fp32
//      operations, so the same value) and writes w and its fp16 copy.
#include <cmath>

#include "common.h"
#include "internal.h"

namespace fg {

constexpr int kOptThreads = 256;
constexpr int kOptIters = 4;                            // float4 per thread
constexpr int kOptElems = kOptThreads * 4 * kOptIters;  // per workgroup

struct OptPiece {
  uint64_t w32, w16, m, v, g;
  uint32_t numel, block0;
};
struct OptTable {
  int32_t n;
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

struct OptStep {
  float lr, b1, b2, eps, wd, bc1, bc2;
  __device__ __forceinline__ float u(float m, float v) const {
    return (m / bc1) / (sqrtf(v / bc2) + eps);
  }
};

// The fp16 copy must be the rounding of the fp32 weight as stored. Without a
// barrier the compiler folds the conversion into the update's fma (a mixed
// fma that rounds the exact result once, to fp16), which differs from the
// two-step rounding on fp32 ties.
__device__ __forceinline__ uint16_t stored_f32_to_h(float v) {
  asm volatile("" : "+v"(v));
  return f32_to_h(v);
}

__device__ __forceinline__ OptStep opt_step(const OptParams &p, int t) {
  return OptStep{p.lr, p.b1, p.b2, p.eps, p.wd,
                 1.f - powf(p.b1, (float)t), 1.f - powf(p.b2, (float)t)};
}

// sums of two values over the workgroup, fixed order: wave shuffles, then
// the four wave results in order
__device__ __forceinline__ void block_sum2(float &a, float &b) {
  __shared__ float red[2][kOptThreads / 64];
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

__global__ __launch_bounds__(kOptThreads) void lars_adam_moments_kernel(
    OptTable t, OptParams p, const int32_t *flags, int nflags,
    const int32_t *step_count, float *part) {
  if (opt_skip(flags, nflags)) return;
  const OptPiece pc = t.p[opt_piece(t, blockIdx.x)];
  const OptStep s = opt_step(p, *step_count + 1);
  const float *g = reinterpret_cast<const float *>(pc.g);
  const float *w = reinterpret_cast<const float *>(pc.w32);
  float *m = reinterpret_cast<float *>(pc.m);
  float *v = reinterpret_cast<float *>(pc.v);
  const uint32_t beg = (blockIdx.x - pc.block0) * (uint32_t)kOptElems;
  const uint32_t end = min(pc.numel, beg + (uint32_t)kOptElems);
  float su = 0.f, sw = 0.f;
  for (uint32_t i = beg + threadIdx.x * 4; i < end; i += kOptThreads * 4) {
    if (i + 4 <= end) {
      const f32x4 gv = *reinterpret_cast<const f32x4 *>(g + i);
      const f32x4 wv = *reinterpret_cast<const f32x4 *>(w + i);
      f32x4 mv = *reinterpret_cast<const f32x4 *>(m + i);
      f32x4 vv = *reinterpret_cast<const f32x4 *>(v + i);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float gt = gv[e] + s.wd * wv[e];
        mv[e] = s.b1 * mv[e] + (1.f - s.b1) * gt;
        vv[e] = s.b2 * vv[e] + (1.f - s.b2) * gt * gt;
        const float u = s.u(mv[e], vv[e]);
        su += u * u;
        sw += wv[e] * wv[e];
      }
      *reinterpret_cast<f32x4 *>(m + i) = mv;
      *reinterpret_cast<f32x4 *>(v + i) = vv;
    } else {
      for (uint32_t j = i; j < end; ++j) {
        const float gt = g[j] + s.wd * w[j];
        const float mj = s.b1 * m[j] + (1.f - s.b1) * gt;
        const float vj = s.b2 * v[j] + (1.f - s.b2) * gt * gt;
        const float u = s.u(mj, vj);
        m[j] = mj;
        v[j] = vj;
        su += u * u;
        sw += w[j] * w[j];
      }
    }
  }
  block_sum2(su, sw);
  if (threadIdx.x == 0) {
    part[2 * blockIdx.x] = su;
    part[2 * blockIdx.x + 1] = sw;
  }
}

__global__ __launch_bounds__(64) void lars_adam_ratio_kernel(
    OptTable t, const int32_t *flags, int nflags, int32_t *step_count,
    const float *part, uint32_t nblocks, float *ratio, int32_t *t_cur) {
  if (opt_skip(flags, nflags)) return;
  const int l = threadIdx.x;
  if (l < t.n) {
    const uint32_t b0 = t.p[l].block0;
    const uint32_t b1 = l + 1 < t.n ? t.p[l + 1].block0 : nblocks;
    double su = 0.0, sw = 0.0;
    for (uint32_t b = b0; b < b1; ++b) {
      su += (double)part[2 * b];
      sw += (double)part[2 * b + 1];
    }
    ratio[l] = su > 0.0 && sw > 0.0 ? (float)(sqrt(sw) / sqrt(su)) : 1.f;
  }
  if (l == 0) {
    const int32_t tn = *step_count + 1;
    *t_cur = tn;
    *step_count = tn;
  }
}

__global__ __launch_bounds__(kOptThreads) void lars_adam_apply_kernel(
    OptTable t, OptParams p, const int32_t *flags, int nflags,
    const float *ratio, const int32_t *t_cur) {
  if (opt_skip(flags, nflags)) return;
  const int pi = opt_piece(t, blockIdx.x);
  const OptPiece pc = t.p[pi];
  const OptStep s = opt_step(p, *t_cur);
  const float step = s.lr * ratio[pi];
  const float *m = reinterpret_cast<const float *>(pc.m);
  const float *v = reinterpret_cast<const float *>(pc.v);
  float *w = reinterpret_cast<float *>(pc.w32);
  uint16_t *w16 = reinterpret_cast<uint16_t *>(pc.w16);
  const uint32_t beg = (blockIdx.x - pc.block0) * (uint32_t)kOptElems;
  const uint32_t end = min(pc.numel, beg + (uint32_t)kOptElems);
  for (uint32_t i = beg + threadIdx.x * 4; i < end; i += kOptThreads * 4) {
    if (i + 4 <= end) {
      const f32x4 mv = *reinterpret_cast<const f32x4 *>(m + i);
      const f32x4 vv = *reinterpret_cast<const f32x4 *>(v + i);
      f32x4 wv = *reinterpret_cast<const f32x4 *>(w + i);
#pragma unroll
      for (int e = 0; e < 4; ++e) wv[e] = wv[e] - step * s.u(mv[e], vv[e]);
      *reinterpret_cast<f32x4 *>(w + i) = wv;
      u32x2 h;
      h[0] = (uint32_t)stored_f32_to_h(wv[0]) |
             ((uint32_t)stored_f32_to_h(wv[1]) << 16);
      h[1] = (uint32_t)stored_f32_to_h(wv[2]) |
             ((uint32_t)stored_f32_to_h(wv[3]) << 16);
      *reinterpret_cast<u32x2 *>(w16 + i) = h;
    } else {
      for (uint32_t j = i; j < end; ++j) {
        const float wj = w[j] - step * s.u(m[j], v[j]);
        w[j] = wj;
        w16[j] = stored_f32_to_h(wj);
      }
    }
  }
}

// ---------------------------------------------------------------------------
static uint32_t opt_table(const fg_opt_tensor *ts, int32_t n, OptTable &t) {
  uint32_t nb = 0;
  t.n = n;
  for (int i = 0; i < n; ++i) {
    t.p[i] = OptPiece{ts[i].w32, ts[i].w16, ts[i].m, ts[i].v, ts[i].g,
                      (uint32_t)ts[i].numel, nb};
    nb += (uint32_t)((ts[i].numel + kOptElems - 1) / kOptElems);
  }
  return nb;
}

// workspace: [2 * nblocks floats of partial sums][ratio per layer][t]
size_t lars_adam_ws_bytes(const fg_opt_tensor *ts, int32_t n) {
  OptTable t;
  const uint32_t nb = opt_table(ts, n, t);
  return (size_t)nb * 2 * sizeof(float) + (size_t)FG_MAX_SEGMENTS * sizeof(float) + 16;
}

hipError_t launch_lars_adam(const fg_opt_tensor *ts, int32_t n, float lr, float b1,
                            float b2, float eps, float wd, const int32_t *flags,
                            int32_t nflags, int32_t *step_count, void *ws,
                            hipStream_t st) {
  OptTable t;
  const uint32_t nb = opt_table(ts, n, t);
  const OptParams p{lr, b1, b2, eps, wd};
  float *part = reinterpret_cast<float *>(ws);
  float *ratio = part + 2 * (size_t)nb;
  int32_t *t_cur = reinterpret_cast<int32_t *>(ratio + FG_MAX_SEGMENTS);
  hipLaunchKernelGGL(lars_adam_moments_kernel, dim3(nb), dim3(kOptThreads), 0, st,
                     t, p, flags, nflags, step_count, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(lars_adam_ratio_kernel, dim3(1), dim3(64), 0, st, t, flags,
                     nflags, step_count, part, nb, ratio, t_cur);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(lars_adam_apply_kernel, dim3(nb), dim3(kOptThreads), 0, st,
                     t, p, flags, nflags, ratio, t_cur);
  return hipGetLastError();
}

}  // namespace fg
