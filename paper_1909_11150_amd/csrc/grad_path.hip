// Bandwidth-bound kernels of the gradient path: fusion-buffer pack and
// unpack, loss-scale removal with a non-finite check, the loss-scaled L2
// head gradient and a standalone ReLU backward.
//
// Pack and unpack are one launch each over all members of a group: the host
// turns the members (and, for pack, the gaps between them) into "pieces",
// gives every piece a contiguous range of workgroups, and each workgroup
// finds its piece by binary search over the piece table passed by value.
#include "common.h"
#include "internal.h"

namespace fg {

// Streaming knobs: 16-byte vectors in flight per thread (fp16; twice as many
// for the fp32 copy), and non-temporal loads / stores. Measured on MI355X
// with the caches evicted, the nine 25 MiB groups back to back: 2 vectors
// gave pack 4.46, unscale 4.18, unpack 4.86 TB/s; 4 gave 4.27 / 4.07 / 3.35;
// 8 gave 2.74 / 2.91 / 4.61. Non-temporal stores gained nothing, and
// interleaving the workgroups' chunks changed nothing.
#ifndef FG_GRAD_VECS
#define FG_GRAD_VECS 2
#endif
#ifndef FG_GRAD_NT_LOAD
#define FG_GRAD_NT_LOAD 0
#endif
#ifndef FG_GRAD_NT_STORE
#define FG_GRAD_NT_STORE 0
#endif

constexpr int kGradThreads = 256;
// fp16 elements per workgroup of the copy kernel (FG_GRAD_VECS 16-byte
// vectors per thread for fp16; twice as many for fp32)
constexpr int kPieceElems = kGradThreads * 8 * FG_GRAD_VECS;

template <class T>
__device__ __forceinline__ T ld_stream(const T *p) {
#if FG_GRAD_NT_LOAD
  return __builtin_nontemporal_load(p);
#else
  return *p;
#endif
}

template <class T>
__device__ __forceinline__ void st_stream(T *p, const T &v) {
#if FG_GRAD_NT_STORE
  __builtin_nontemporal_store(v, p);
#else
  *p = v;
#endif
}

struct Piece {
  uint64_t src;      // device address of the source (0: zero fill)
  uint64_t dst;      // device address of the destination
  uint32_t numel;    // elements (< 2^31, checked by the caller)
  uint32_t block0;   // first workgroup of this piece
};

constexpr int kMaxPieces = 2 * FG_MAX_SEGMENTS + 1;
struct PieceTable {
  int32_t npiece;
  Piece p[kMaxPieces];
};

__device__ __forceinline__ int find_piece(const PieceTable &t, uint32_t b) {
  int lo = 0, hi = t.npiece - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (t.p[mid].block0 <= b) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Bit copy of ESZ-byte elements (2: fp16 pack, 4: fp32 unpack); a piece with
// src == 0 is zero filled. Workgroup b of a piece copies elements
// [b * kPieceElems, (b + 1) * kPieceElems); every thread issues all of its NV
// 16-byte loads (256 threads apart) before its first store.
template <int ESZ>
__global__ __launch_bounds__(kGradThreads) void copy_pieces_kernel(
    PieceTable t) {
  const int pi = find_piece(t, blockIdx.x);
  const Piece pc = t.p[pi];
  constexpr int EPV = 16 / ESZ;                           // elements per vector
  constexpr int NV = kPieceElems / (kGradThreads * EPV);  // vectors per thread
  const uint64_t beg = (uint64_t)(blockIdx.x - pc.block0) * kPieceElems;
  if (beg >= pc.numel) return;
  const uint64_t end =
      beg + kPieceElems < pc.numel ? beg + kPieceElems : (uint64_t)pc.numel;
  if (((pc.src | pc.dst) & 15) == 0) {
    const uint64_t nvec_end = end / EPV * EPV;  // beg is a multiple of EPV
    u32x4 v[NV];
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const uint64_t i =
          beg + ((uint64_t)j * kGradThreads + threadIdx.x) * EPV;
      v[j] = u32x4{0, 0, 0, 0};
      if (pc.src && i < nvec_end)
        v[j] = ld_stream(reinterpret_cast<const u32x4 *>(pc.src + i * ESZ));
    }
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const uint64_t i =
          beg + ((uint64_t)j * kGradThreads + threadIdx.x) * EPV;
      if (i < nvec_end) st_stream(reinterpret_cast<u32x4 *>(pc.dst + i * ESZ), v[j]);
    }
    // the last (< EPV) elements of the piece
    const uint64_t i = nvec_end + threadIdx.x;
    if (i < end) {
      if (ESZ == 2) {
        uint16_t e = pc.src ? reinterpret_cast<const uint16_t *>(pc.src)[i] : 0;
        reinterpret_cast<uint16_t *>(pc.dst)[i] = e;
      } else {
        uint32_t e = pc.src ? reinterpret_cast<const uint32_t *>(pc.src)[i] : 0;
        reinterpret_cast<uint32_t *>(pc.dst)[i] = e;
      }
    }
  } else {
    for (uint64_t i = beg + threadIdx.x; i < end; i += kGradThreads) {
      if (ESZ == 2) {
        uint16_t v = pc.src ? reinterpret_cast<const uint16_t *>(pc.src)[i] : 0;
        reinterpret_cast<uint16_t *>(pc.dst)[i] = v;
      } else {
        uint32_t v = pc.src ? reinterpret_cast<const uint32_t *>(pc.src)[i] : 0;
        reinterpret_cast<uint32_t *>(pc.dst)[i] = v;
      }
    }
  }
}

static uint32_t blocks_for(uint64_t numel) {
  return (uint32_t)((numel + kPieceElems - 1) / kPieceElems);
}

template <int ESZ>
static hipError_t launch_pieces(PieceTable &t, hipStream_t st) {
  uint32_t nb = 0;
  for (int i = 0; i < t.npiece; ++i) {
    t.p[i].block0 = nb;
    nb += blocks_for(t.p[i].numel);
  }
  if (nb == 0) return hipSuccess;
  hipLaunchKernelGGL((copy_pieces_kernel<ESZ>), dim3(nb), dim3(kGradThreads),
                     0, st, t);
  return hipGetLastError();
}

// Segments are validated (inside the group, non-overlapping) by the caller.
hipError_t launch_pack(const fg_segment *segs, int32_t nseg, uint16_t *group,
                       uint64_t group_numel, hipStream_t st) {
  int order[FG_MAX_SEGMENTS];
  for (int i = 0; i < nseg; ++i) order[i] = i;
  for (int i = 1; i < nseg; ++i)  // insertion sort by offset
    for (int j = i; j > 0 && segs[order[j - 1]].offset > segs[order[j]].offset;
         --j) {
      int tmp = order[j];
      order[j] = order[j - 1];
      order[j - 1] = tmp;
    }
  PieceTable t;
  t.npiece = 0;
  const uint64_t gbase = (uint64_t)group;
  uint64_t cur = 0;
  for (int ii = 0; ii < nseg; ++ii) {
    const fg_segment &s = segs[order[ii]];
    if (s.offset > cur)
      t.p[t.npiece++] = Piece{0, gbase + cur * 2, (uint32_t)(s.offset - cur), 0};
    if (s.numel)
      t.p[t.npiece++] = Piece{s.ptr, gbase + s.offset * 2, (uint32_t)s.numel, 0};
    cur = s.offset + s.numel;
  }
  if (group_numel > cur)
    t.p[t.npiece++] = Piece{0, gbase + cur * 2, (uint32_t)(group_numel - cur), 0};
  return launch_pieces<2>(t, st);
}

hipError_t launch_unpack(const float *group, const fg_segment *segs,
                         int32_t nseg, hipStream_t st) {
  PieceTable t;
  t.npiece = 0;
  const uint64_t gbase = (uint64_t)group;
  for (int i = 0; i < nseg; ++i)
    if (segs[i].numel)
      t.p[t.npiece++] =
          Piece{gbase + segs[i].offset * 4, segs[i].ptr, (uint32_t)segs[i].numel,
                0};
  return launch_pieces<4>(t, st);
}

// ---------------------------------------------------------------------------
// out[j] = fp32(value(in[j]) * inv_scale) and flag |= any non-finite.
// The fp16 -> fp32 conversion is exact and the fp32 multiply rounds the exact
// product once (nearest-even), which is the definition of the result.
__device__ __forceinline__ bool nonfinite16(uint32_t h) {
  return (h & 0x7C00u) == 0x7C00u;
}

// Vectors of 8 fp16 values: each thread issues its kUnscaleVecs 16-byte
// loads before converting and storing.
constexpr int kUnscaleVecs = FG_GRAD_VECS;

__global__ __launch_bounds__(kGradThreads) void unscale_vec_kernel(
    const uint16_t *in, uint64_t nvec, float inv, float *out, int32_t *flag) {
  const uint64_t base = (uint64_t)blockIdx.x * (kGradThreads * kUnscaleVecs);
  u32x4 w[kUnscaleVecs];
#pragma unroll
  for (int j = 0; j < kUnscaleVecs; ++j) {
    const uint64_t v = base + (uint64_t)j * kGradThreads + threadIdx.x;
    w[j] = u32x4{0, 0, 0, 0};
    if (v < nvec) w[j] = ld_stream(reinterpret_cast<const u32x4 *>(in + v * 8));
  }
  bool bad = false;
#pragma unroll
  for (int j = 0; j < kUnscaleVecs; ++j) {
    const uint64_t v = base + (uint64_t)j * kGradThreads + threadIdx.x;
    f32x4 o0, o1;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t lo = w[j][e] & 0xFFFFu, hi = w[j][e] >> 16;
      bad |= nonfinite16(lo) | nonfinite16(hi);
      const float a = h_to_f32((uint16_t)lo) * inv;
      const float b = h_to_f32((uint16_t)hi) * inv;
      if (e < 2) {
        o0[2 * e] = a;
        o0[2 * e + 1] = b;
      } else {
        o1[2 * e - 4] = a;
        o1[2 * e - 3] = b;
      }
    }
    if (v < nvec) {
      st_stream(reinterpret_cast<f32x4 *>(out + v * 8), o0);
      st_stream(reinterpret_cast<f32x4 *>(out + v * 8 + 4), o1);
    }
  }
  // zero words past the end convert to finite values: bad is exact
  flag_nonfinite(flag, bad);
}

__global__ __launch_bounds__(kGradThreads) void unscale_scalar_kernel(
    const uint16_t *in, uint64_t beg, uint64_t end, float inv, float *out,
    int32_t *flag) {
  bool bad = false;
  const uint64_t stride = (uint64_t)gridDim.x * kGradThreads;
  for (uint64_t i = beg + (uint64_t)blockIdx.x * kGradThreads + threadIdx.x;
       i < end; i += stride) {
    uint16_t h = in[i];
    bad |= nonfinite16(h);
    out[i] = h_to_f32(h) * inv;
  }
  if (__ballot(bad) != 0 && (threadIdx.x & 63) == __builtin_ctzll(__ballot(bad)))
    *flag = 1;
}

hipError_t launch_unscale(const uint16_t *group, uint64_t numel,
                          float inv_scale, float *out, int32_t *flag,
                          hipStream_t st) {
  const bool vec = (((uint64_t)group % 16) == 0) && (((uint64_t)out % 16) == 0);
  uint64_t nvec = vec ? numel / 8 : 0;
  if (nvec) {
    const uint64_t per = (uint64_t)kGradThreads * kUnscaleVecs;
    const uint64_t blocks = (nvec + per - 1) / per;  // < 2^26 for numel < 2^31
    hipLaunchKernelGGL(unscale_vec_kernel, dim3((unsigned)blocks),
                       dim3(kGradThreads), 0, st, group, nvec, inv_scale, out,
                       flag);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  uint64_t beg = nvec * 8;
  if (beg < numel) {
    uint64_t n = numel - beg;
    uint64_t blocks = (n + kGradThreads - 1) / kGradThreads;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(unscale_scalar_kernel, dim3((unsigned)blocks),
                       dim3(kGradThreads), 0, st, group, beg, numel, inv_scale,
                       out, flag);
    return hipGetLastError();
  }
  return hipSuccess;
}

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kGradThreads) void flags_clear_kernel(int32_t *f,
                                                                   int32_t n) {
  const int32_t i = blockIdx.x * kGradThreads + threadIdx.x;
  if (i < n) f[i] = 0;
}

hipError_t launch_flags_clear(int32_t *flags, int32_t n, hipStream_t st) {
  hipLaunchKernelGGL(flags_clear_kernel,
                     dim3((unsigned)((n + kGradThreads - 1) / kGradThreads)),
                     dim3(kGradThreads), 0, st, flags, n);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kGradThreads) void head_grad_kernel(
    const uint16_t *y, const float *t, uint64_t numel, double scale,
    uint16_t *dy) {
  const uint64_t stride = (uint64_t)gridDim.x * kGradThreads;
  for (uint64_t i = (uint64_t)blockIdx.x * kGradThreads + threadIdx.x;
       i < numel; i += stride) {
    double d = ((double)h_to_f32(y[i]) - (double)t[i]) * scale;
    dy[i] = f64_to_h(d);
  }
}

hipError_t launch_head_grad(const uint16_t *y, const float *t, uint64_t numel,
                            double scale, uint16_t *dy, hipStream_t st) {
  uint64_t blocks = (numel + kGradThreads - 1) / kGradThreads;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(head_grad_kernel, dim3((unsigned)blocks),
                     dim3(kGradThreads), 0, st, y, t, numel, scale, dy);
  return hipGetLastError();
}

__global__ __launch_bounds__(kGradThreads) void relu_backward_kernel(
    const uint16_t *dy, const uint16_t *act, uint64_t numel, uint16_t *out) {
  const uint64_t stride = (uint64_t)gridDim.x * kGradThreads;
  for (uint64_t i = (uint64_t)blockIdx.x * kGradThreads + threadIdx.x;
       i < numel; i += stride)
    out[i] = h_to_f32(act[i]) > 0.f ? dy[i] : (uint16_t)0;
}

hipError_t launch_relu_backward(const uint16_t *dy, const uint16_t *act,
                                uint64_t numel, uint16_t *out,
                                hipStream_t st) {
  uint64_t blocks = (numel + kGradThreads - 1) / kGradThreads;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(relu_backward_kernel, dim3((unsigned)blocks),
                     dim3(kGradThreads), 0, st, dy, act, numel, out);
  return hipGetLastError();
}

}  // namespace fg
