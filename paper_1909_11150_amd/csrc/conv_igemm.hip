// Implicit-GEMM fp16 convolutions on fp16 MFMA (fp32 accumulate) for gfx950.
//
// Data convolutions (forward, input gradient, transposed forward) are one
// kernel: GEMM rows are output channels, columns are output positions of one
// phase, and the reduction runs over (tap, input channel). The input image is
// gathered straight from NHWC memory (zero outside the image); nothing is
// materialised. Strided input gradients and transposed convolutions are split
// into output phases so that no multiply touches an inserted zero.
//
// The kernel gradient is a second kernel: rows are (tap, input channel),
// columns output channels, reduction over all output positions, split across
// workgroups with fp32 partials summed afterwards in a fixed order.
//
// Both kernels stage 64-deep reduction slices of each operand in LDS (double
// buffered, one barrier per slice) in a layout where every MFMA operand is a
// single 16-byte read. Operands whose reduction dimension is strided in
// memory are transposed in registers on their way to LDS.
#include "common.h"
#include "internal.h"

namespace fg {

constexpr int BK = 64;        // reduction slice per LDS stage
constexpr int LDK = BK + 8;   // LDS row pitch in halves (16-byte skew)
constexpr int NT = 256;       // threads per workgroup (4 waves, 2 x 2)

// ---------------------------------------------------------------------------
// MFMA core: each wave owns a (BM/2) x (BN/2) block of the tile.
template <int BM, int BN>
struct Core {
  static constexpr int WM = BM / 2, WN = BN / 2;
  static constexpr int FM = WM / 32, FN = WN / 32;
  f32x16 acc[FM][FN];

  __device__ void zero() {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
  }

  __device__ void step(const uint16_t *sA, const uint16_t *sB, int wm0,
                       int wn0, int lane) {
    const int r = lane & 31, kh = (lane >> 5) * 8;
#pragma unroll
    for (int ks = 0; ks < BK; ks += 16) {
      u32x4 a[FM], b[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        a[i] = *reinterpret_cast<const u32x4 *>(
            sA + (wm0 + i * 32 + r) * LDK + ks + kh);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        b[j] = *reinterpret_cast<const u32x4 *>(
            sB + (wn0 + j * 32 + r) * LDK + ks + kh);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma32(a[i], b[j], acc[i][j]);
    }
  }
};

// Transpose 4 rows of 8 halves (reduction index = row) into 8 columns of 4
// halves and store column j at dst + j*LDK (8 bytes each).
__device__ __forceinline__ void store_t4x8(uint16_t *dst, const u32x4 q[4]) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    u32x2 lo, hi;
    lo[0] = pack_lo(q[0][e], q[1][e]);
    lo[1] = pack_lo(q[2][e], q[3][e]);
    hi[0] = pack_hi(q[0][e], q[1][e]);
    hi[1] = pack_hi(q[2][e], q[3][e]);
    *reinterpret_cast<u32x2 *>(dst + (2 * e) * LDK) = lo;
    *reinterpret_cast<u32x2 *>(dst + (2 * e + 1) * LDK) = hi;
  }
}

__device__ __forceinline__ u32x4 ldg16(const uint16_t *p) {
  return *reinterpret_cast<const u32x4 *>(p);
}

// ---------------------------------------------------------------------------
// Data convolution kernel.
//   WK    weights are k-major (forward: reduction contiguous per output
//         channel) or mn-major (input gradient / transposed: output channel
//         contiguous), the latter transposed in registers.
//   FAST  reduction channels are a multiple of BK, so a slice is one tap.
template <int BM, int BN, bool WK, bool FAST>
__global__ __launch_bounds__(NT) void data_conv_kernel(DataConvArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][BN * LDK];

  const Phase P = a.ph[blockIdx.z];
  const int npix = a.n * P.mh * P.mw;
  const int n0 = blockIdx.x * BN;
  const int m0 = blockIdx.y * BM;
  if (n0 >= npix) return;
  const int ntap = P.nr * P.ns;
  const int ktot = ntap * a.cr;
  const int nk = (ktot + BK - 1) / BK;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * (BM / 2), wn0 = (wave & 1) * (BN / 2);

  // --- B (activation gather) loader state: BN/32 columns per thread.
  constexpr int BCOL = BN / 32;
  const int bc8 = tid & 7;
  int bimg[BCOL], bh[BCOL], bw[BCOL];
#pragma unroll
  for (int i = 0; i < BCOL; ++i) {
    int col = n0 + (tid >> 3) + 32 * i;
    if (col < npix) {
      int b = col % P.mw, t = col / P.mw;
      int aa = t % P.mh, nn = t / P.mh;
      bimg[i] = nn;
      bh[i] = aa * a.istr;
      bw[i] = b * a.istr;
    } else {
      bimg[i] = -1;
      bh[i] = 0;
      bw[i] = 0;
    }
  }

  // --- A (weight) loader: k-major uses BM/32 rows per thread; mn-major uses
  // units of 4 reduction rows x 8 output channels.
  constexpr int AROW = BM / 32;
  constexpr int AUNITS = (BK / 4) * (BM / 8);
  constexpr int AUPT = (AUNITS + NT - 1) / NT;

  u32x4 ra[WK ? AROW : 4 * AUPT];
  u32x4 rb[BCOL];

  auto tap_of = [&](int kk, int &dh, int &dw, int &woff, int &cr) {
    int t = kk / a.cr;
    cr = kk - t * a.cr;
    int i = t / P.ns, j = t - (t / P.ns) * P.ns;
    dh = P.dh0 + P.dstep * i;
    dw = P.dw0 + P.dstep * j;
    woff = (P.r0 + P.rstep * i) * a.s + (P.s0 + P.rstep * j);
  };

  auto load = [&](int kt) {
    const int k0 = kt * BK;
    // B: activations
    {
      int kk = k0 + bc8 * 8;
      int dh, dw, woff, cr;
      bool kv = kk < ktot;
      if (FAST) {
        tap_of(k0, dh, dw, woff, cr);
        cr += bc8 * 8;
      } else {
        tap_of(kv ? kk : 0, dh, dw, woff, cr);
      }
#pragma unroll
      for (int i = 0; i < BCOL; ++i) {
        int hh = bh[i] + dh, ww = bw[i] + dw;
        bool v = kv && bimg[i] >= 0 && hh >= 0 && hh < a.hi && ww >= 0 &&
                 ww < a.wi;
        if (v)
          rb[i] = ldg16(a.act +
                        ((size_t)((bimg[i] * a.hi + hh) * a.wi + ww)) * a.cr +
                        cr);
        else
          rb[i] = u32x4{0, 0, 0, 0};
      }
    }
    // A: weights
    if (WK) {
      int kk = k0 + bc8 * 8;
      int dh, dw, woff, cr;
      bool kv = kk < ktot;
      tap_of(kv ? kk : 0, dh, dw, woff, cr);
#pragma unroll
      for (int i = 0; i < AROW; ++i) {
        int row = m0 + (tid >> 3) + 32 * i;
        if (kv && row < a.co)
          ra[i] = ldg16(a.wgt + (size_t)row * a.ldw + (size_t)woff * a.cr + cr);
        else
          ra[i] = u32x4{0, 0, 0, 0};
      }
    } else {
#pragma unroll
      for (int u = 0; u < AUPT; ++u) {
        int unit = tid + u * NT;
        int cg = unit % (BM / 8), kq = unit / (BM / 8);
        int kk = k0 + kq * 4;
        int row = m0 + cg * 8;
        bool v = unit < AUNITS && kk < ktot && row < a.co;
        int dh, dw, woff, cr;
        tap_of(v ? kk : 0, dh, dw, woff, cr);
        const uint16_t *src =
            a.wgt + (size_t)cr * a.w_red + (size_t)woff * a.w_tap + row;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          // 4 consecutive reduction indices stay inside one tap (cr % 8 == 0)
          if (v)
            ra[4 * u + e] = ldg16(src + (size_t)e * a.w_red);
          else
            ra[4 * u + e] = u32x4{0, 0, 0, 0};
        }
      }
    }
  };

  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < BCOL; ++i)
      *reinterpret_cast<u32x4 *>(&sB[buf][((tid >> 3) + 32 * i) * LDK +
                                           bc8 * 8]) = rb[i];
    if (WK) {
#pragma unroll
      for (int i = 0; i < AROW; ++i)
        *reinterpret_cast<u32x4 *>(&sA[buf][((tid >> 3) + 32 * i) * LDK +
                                             bc8 * 8]) = ra[i];
    } else {
#pragma unroll
      for (int u = 0; u < AUPT; ++u) {
        int unit = tid + u * NT;
        if (unit < AUNITS) {
          int cg = unit % (BM / 8), kq = unit / (BM / 8);
          store_t4x8(&sA[buf][(cg * 8) * LDK + kq * 4], &ra[4 * u]);
        }
      }
    }
  };

  Core<BM, BN> core;
  core.zero();
  load(0);
  store(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) load(kt + 1);
    core.step(sA[cur], sB[cur], wm0, wn0, lane);
    if (kt + 1 < nk) store(cur ^ 1);
    __syncthreads();
  }

  // --- epilogue: lane holds 4 consecutive output channels of one position.
  constexpr int FM = Core<BM, BN>::FM, FN = Core<BM, BN>::FN;
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    int col = n0 + wn0 + j * 32 + (lane & 31);
    if (col >= npix) continue;
    int b = col % P.mw, t = col / P.mw;
    int aa = t % P.mh, nn = t / P.mh;
    size_t obase = ((size_t)(nn * a.ho + aa * a.ostr + P.ooh) * a.wo +
                    b * a.ostr + P.oow) *
                   a.co;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        int co = m0 + wm0 + i * 32 + 8 * g + 4 * (lane >> 5);
        if (co >= a.co) continue;
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = core.acc[i][j][4 * g + e];
        if (a.epi == FG_EPI_RELU) {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = v[e] > 0.f ? v[e] : 0.f;
        } else if (a.epi == FG_EPI_GATE) {
          u32x2 gw = *reinterpret_cast<const u32x2 *>(a.gate + obase + co);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            uint16_t gb = (uint16_t)(gw[e >> 1] >> (16 * (e & 1)));
            v[e] = h_to_f32(gb) > 0.f ? v[e] : 0.f;
          }
        }
        u32x2 o;
        o[0] = (uint32_t)f32_to_h(v[0]) | ((uint32_t)f32_to_h(v[1]) << 16);
        o[1] = (uint32_t)f32_to_h(v[2]) | ((uint32_t)f32_to_h(v[3]) << 16);
        *reinterpret_cast<u32x2 *>(a.out + obase + co) = o;
      }
  }
}

// ---------------------------------------------------------------------------
// Kernel-gradient kernel: rows rho = (tap, c) of the x patch, columns k.
template <int BM, int BN>
__global__ __launch_bounds__(NT) void wgrad_kernel(WgradArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][BM * LDK];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][BN * LDK];

  const int rsc = a.r * a.s * a.c;
  const int m0 = blockIdx.x * BM;  // rho
  const int n0 = blockIdx.y * BN;  // k
  const int split = blockIdx.z;
  const int mbeg = split * a.mchunk;
  const int mend = min(a.mtot, mbeg + a.mchunk);
  const int nk = (mend - mbeg + BK - 1) / BK;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * (BM / 2), wn0 = (wave & 1) * (BN / 2);
  const int pq = a.p * a.q;

  constexpr int AUNITS = (BK / 4) * (BM / 8);
  constexpr int AUPT = (AUNITS + NT - 1) / NT;
  constexpr int BUNITS = (BK / 4) * (BN / 8);
  constexpr int BUPT = (BUNITS + NT - 1) / NT;
  u32x4 ra[4 * AUPT], rb[4 * BUPT];

  auto load = [&](int kt) {
    const int k0 = mbeg + kt * BK;
#pragma unroll
    for (int u = 0; u < AUPT; ++u) {
      int unit = tid + u * NT;
      int rg = unit % (BM / 8), mq = unit / (BM / 8);
      int rho = m0 + rg * 8;
      bool uv = unit < AUNITS && rho < rsc;
      int t = rho / a.c, c = rho - (rho / a.c) * a.c;
      int r = t / a.s, s = t - (t / a.s) * a.s;
      int m = k0 + mq * 4;
      int nn = m / pq, rem = m - (m / pq) * pq;
      int p = rem / a.q, q = rem - (rem / a.q) * a.q;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        int hh = p * a.sh - a.ph + r, ww = q * a.sw - a.pw + s;
        bool v = uv && (m + e) < mend && hh >= 0 && hh < a.h && ww >= 0 &&
                 ww < a.w;
        if (v)
          ra[4 * u + e] =
              ldg16(a.x + ((size_t)((nn * a.h + hh) * a.w + ww)) * a.c + c);
        else
          ra[4 * u + e] = u32x4{0, 0, 0, 0};
        // next reduction row: advance (n, p, q)
        if (++q == a.q) {
          q = 0;
          if (++p == a.p) {
            p = 0;
            ++nn;
          }
        }
      }
    }
#pragma unroll
    for (int u = 0; u < BUPT; ++u) {
      int unit = tid + u * NT;
      int kg = unit % (BN / 8), mq = unit / (BN / 8);
      int k = n0 + kg * 8;
      int m = k0 + mq * 4;
      bool uv = unit < BUNITS && k < a.k;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (uv && (m + e) < mend)
          rb[4 * u + e] = ldg16(a.dy + (size_t)(m + e) * a.k + k);
        else
          rb[4 * u + e] = u32x4{0, 0, 0, 0};
      }
    }
  };

  auto store = [&](int buf) {
#pragma unroll
    for (int u = 0; u < AUPT; ++u) {
      int unit = tid + u * NT;
      if (unit < AUNITS) {
        int rg = unit % (BM / 8), mq = unit / (BM / 8);
        store_t4x8(&sA[buf][(rg * 8) * LDK + mq * 4], &ra[4 * u]);
      }
    }
#pragma unroll
    for (int u = 0; u < BUPT; ++u) {
      int unit = tid + u * NT;
      if (unit < BUNITS) {
        int kg = unit % (BN / 8), mq = unit / (BN / 8);
        store_t4x8(&sB[buf][(kg * 8) * LDK + mq * 4], &rb[4 * u]);
      }
    }
  };

  Core<BM, BN> core;
  core.zero();
  if (nk > 0) {
    load(0);
    store(0);
  }
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) load(kt + 1);
    core.step(sA[cur], sB[cur], wm0, wn0, lane);
    if (kt + 1 < nk) store(cur ^ 1);
    __syncthreads();
  }

  constexpr int FM = Core<BM, BN>::FM, FN = Core<BM, BN>::FN;
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    int k = n0 + wn0 + j * 32 + (lane & 31);
    if (k >= a.k) continue;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        int rho = m0 + wm0 + i * 32 + 8 * g + 4 * (lane >> 5);
        if (rho >= rsc) continue;
        if (a.nsplit == 1) {
          u32x2 o;
          o[0] = (uint32_t)f32_to_h(core.acc[i][j][4 * g]) |
                 ((uint32_t)f32_to_h(core.acc[i][j][4 * g + 1]) << 16);
          o[1] = (uint32_t)f32_to_h(core.acc[i][j][4 * g + 2]) |
                 ((uint32_t)f32_to_h(core.acc[i][j][4 * g + 3]) << 16);
          *reinterpret_cast<u32x2 *>(a.dw + (size_t)k * rsc + rho) = o;
        } else {
          f32x4 o;
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = core.acc[i][j][4 * g + e];
          *reinterpret_cast<f32x4 *>(
              a.part + ((size_t)split * a.k + k) * rsc + rho) = o;
        }
      }
  }
}

// Sum nsplit fp32 partial arrays of len elements in split order, round to
// fp16. len is a multiple of 4.
__global__ __launch_bounds__(256) void split_reduce_kernel(const float *part,
                                                           int nsplit,
                                                           int64_t len,
                                                           uint16_t *out) {
  int64_t i4 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i4 >= len) return;
  f32x4 s = *reinterpret_cast<const f32x4 *>(part + i4);
  for (int k = 1; k < nsplit; ++k) {
    f32x4 v = *reinterpret_cast<const f32x4 *>(part + (size_t)k * len + i4);
#pragma unroll
    for (int e = 0; e < 4; ++e) s[e] += v[e];
  }
  u32x2 o;
  o[0] = (uint32_t)f32_to_h(s[0]) | ((uint32_t)f32_to_h(s[1]) << 16);
  o[1] = (uint32_t)f32_to_h(s[2]) | ((uint32_t)f32_to_h(s[3]) << 16);
  *reinterpret_cast<u32x2 *>(out + i4) = o;
}

// ---------------------------------------------------------------------------
// Single-output-channel 1x1 convolution (the network head): bandwidth-bound,
// so no MFMA. L lanes (a power of two) cooperate on one position.
__global__ __launch_bounds__(256) void head_fwd_kernel(
    const uint16_t *x, const uint16_t *w, uint16_t *y, int64_t npix, int c,
    int L, int logL, int epi, const uint16_t *gate) {
  const int lane = threadIdx.x & 63;
  const int sub = lane & (L - 1);
  const int per_wave = 64 / L;
  const int64_t wave_id = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  const int nchunk = c / 8;
  for (int64_t base = wave_id * per_wave; base < npix;
       base += nwaves * per_wave) {
    int64_t pix = base + (lane >> logL);
    float acc = 0.f;
    if (pix < npix) {
      for (int ch = sub; ch < nchunk; ch += L) {
        u32x4 xv = ldg16(x + pix * c + ch * 8);
        u32x4 wv = ldg16(w + ch * 8);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc += h_to_f32((uint16_t)xv[e]) * h_to_f32((uint16_t)wv[e]);
          acc += h_to_f32((uint16_t)(xv[e] >> 16)) *
                 h_to_f32((uint16_t)(wv[e] >> 16));
        }
      }
    }
    for (int o = 1; o < L; o <<= 1) acc += __shfl_xor(acc, o, 64);
    if (pix < npix && sub == 0) {
      float v = acc;
      if (epi == FG_EPI_RELU) v = v > 0.f ? v : 0.f;
      if (epi == FG_EPI_GATE) v = h_to_f32(gate[pix]) > 0.f ? v : 0.f;
      y[pix] = f32_to_h(v);
    }
  }
}

// dx[m][c] = epi(dy[m] * w[c]); one thread per 8 channels.
__global__ __launch_bounds__(256) void head_bwd_data_kernel(
    const uint16_t *dy, const uint16_t *w, uint16_t *dx, int64_t npix, int c,
    int epi, const uint16_t *gate) {
  const int nchunk = c / 8;
  int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= npix * nchunk) return;
  int64_t pix = idx / nchunk;
  int ch = (int)(idx - pix * nchunk);
  float d = h_to_f32(dy[pix]);
  u32x4 wv = ldg16(w + ch * 8);
  u32x4 gv = u32x4{0, 0, 0, 0};
  if (epi == FG_EPI_GATE) gv = ldg16(gate + pix * c + ch * 8);
  u32x4 o;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    float v0 = d * h_to_f32((uint16_t)wv[e]);
    float v1 = d * h_to_f32((uint16_t)(wv[e] >> 16));
    if (epi == FG_EPI_RELU) {
      v0 = v0 > 0.f ? v0 : 0.f;
      v1 = v1 > 0.f ? v1 : 0.f;
    } else if (epi == FG_EPI_GATE) {
      v0 = h_to_f32((uint16_t)gv[e]) > 0.f ? v0 : 0.f;
      v1 = h_to_f32((uint16_t)(gv[e] >> 16)) > 0.f ? v1 : 0.f;
    }
    o[e] = (uint32_t)f32_to_h(v0) | ((uint32_t)f32_to_h(v1) << 16);
  }
  *reinterpret_cast<u32x4 *>(dx + pix * c + ch * 8) = o;
}

// Partial kernel gradient of the head: block b sums positions
// [b*chunk, (b+1)*chunk) for all c channels into part[b][c] (fixed order).
constexpr int kHeadWgradThreads = 256;
__global__ __launch_bounds__(kHeadWgradThreads) void head_wgrad_kernel(
    const uint16_t *x, const uint16_t *dy, int64_t npix, int c, int64_t chunk,
    float *part) {
  __shared__ float red[kHeadWgradThreads * 8];
  const int nchunk = c / 8;
  const int rows = kHeadWgradThreads / nchunk;  // positions in flight
  const int ch = threadIdx.x % nchunk, row = threadIdx.x / nchunk;
  float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  int64_t beg = (int64_t)blockIdx.x * chunk;
  int64_t end = beg + chunk < npix ? beg + chunk : npix;
  if (row < rows) {
    for (int64_t pix = beg + row; pix < end; pix += rows) {
      float d = h_to_f32(dy[pix]);
      u32x4 xv = ldg16(x + pix * c + ch * 8);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[2 * e] += d * h_to_f32((uint16_t)xv[e]);
        acc[2 * e + 1] += d * h_to_f32((uint16_t)(xv[e] >> 16));
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) red[threadIdx.x * 8 + e] = acc[e];
  __syncthreads();
  if (threadIdx.x < nchunk) {
    float s[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) s[e] = 0.f;
    for (int rr = 0; rr < rows; ++rr)
#pragma unroll
      for (int e = 0; e < 8; ++e) s[e] += red[(rr * nchunk + ch) * 8 + e];
#pragma unroll
    for (int e = 0; e < 8; ++e) part[(size_t)blockIdx.x * c + ch * 8 + e] = s[e];
  }
}

// ---------------------------------------------------------------------------
// Host launchers.
template <int BM, int BN, bool WK, bool FAST>
static hipError_t launch_dc(const DataConvArgs &a, hipStream_t st) {
  int maxpix = 0;
  for (int i = 0; i < a.nphase; ++i)
    maxpix = max(maxpix, a.n * a.ph[i].mh * a.ph[i].mw);
  dim3 grid((maxpix + BN - 1) / BN, (a.co + BM - 1) / BM, a.nphase);
  hipLaunchKernelGGL((data_conv_kernel<BM, BN, WK, FAST>), grid, dim3(NT), 0,
                     st, a);
  return hipGetLastError();
}

hipError_t launch_data_conv(const DataConvArgs &a, bool w_kmajor,
                            hipStream_t st) {
  const bool fast = (a.cr % BK) == 0;
  if (w_kmajor)
    return fast ? launch_dc<128, 128, true, true>(a, st)
                : launch_dc<128, 128, true, false>(a, st);
  return fast ? launch_dc<128, 128, false, true>(a, st)
              : launch_dc<128, 128, false, false>(a, st);
}

const char *data_conv_kernel_name(int32_t cr, bool w_kmajor) {
  const bool fast = (cr % BK) == 0;
  if (w_kmajor)
    return fast ? "data_conv_kernel<128, 128, true, true>"
                : "data_conv_kernel<128, 128, true, false>";
  return fast ? "data_conv_kernel<128, 128, false, true>"
              : "data_conv_kernel<128, 128, false, false>";
}

const char *wgrad_kernel_name() { return "wgrad_kernel<128, 128>"; }

WgradPlan plan_wgrad(const fg_conv_desc &d, int32_t p, int32_t q) {
  WgradPlan pl;
  const int64_t rsc = (int64_t)d.r * d.s * d.c;
  const int64_t tiles = ((rsc + 127) / 128) * ((d.k + 127) / 128);
  const int64_t mtot = (int64_t)d.n * p * q;
  int64_t want = (512 + tiles - 1) / tiles;             // ~2 waves of CUs
  int64_t maxs = (mtot + 4 * BK - 1) / (4 * BK);         // >= 4 slices each
  int64_t ns = want < maxs ? want : maxs;
  if (ns < 1) ns = 1;
  int64_t chunk = (mtot + ns - 1) / ns;
  chunk = (chunk + BK - 1) / BK * BK;
  ns = (mtot + chunk - 1) / chunk;
  pl.nsplit = (int32_t)ns;
  pl.mchunk = (int32_t)chunk;
  pl.ws_bytes = ns > 1 ? (size_t)ns * d.k * rsc * sizeof(float) : 0;
  return pl;
}

hipError_t launch_wgrad(const WgradArgs &a, hipStream_t st) {
  const int rsc = a.r * a.s * a.c;
  dim3 grid((rsc + 127) / 128, (a.k + 127) / 128, a.nsplit);
  hipLaunchKernelGGL((wgrad_kernel<128, 128>), grid, dim3(NT), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.nsplit == 1) return e;
  const int64_t len = (int64_t)a.k * rsc;
  dim3 g2((unsigned)((len / 4 + 255) / 256));
  hipLaunchKernelGGL(split_reduce_kernel, g2, dim3(256), 0, st, a.part,
                     a.nsplit, len, a.dw);
  return hipGetLastError();
}

static int pow2_at_least(int v) {
  int p = 1;
  while (p < v) p <<= 1;
  return p;
}

hipError_t launch_head_fwd(const uint16_t *x, const uint16_t *w, uint16_t *y,
                           int64_t npix, int32_t c, int32_t epi,
                           const uint16_t *gate, hipStream_t st) {
  int L = pow2_at_least(c / 8);
  if (L > 64) L = 64;
  int logL = 0;
  while ((1 << logL) < L) ++logL;
  int64_t waves = (npix * L + 63) / 64;
  int64_t blocks = (waves + 3) / 4;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(head_fwd_kernel, dim3((unsigned)blocks), dim3(256), 0, st,
                     x, w, y, npix, c, L, logL, epi, gate);
  return hipGetLastError();
}

hipError_t launch_head_bwd_data(const uint16_t *dy, const uint16_t *w,
                                uint16_t *dx, int64_t npix, int32_t c,
                                int32_t epi, const uint16_t *gate,
                                hipStream_t st) {
  int64_t n = npix * (c / 8);
  hipLaunchKernelGGL(head_bwd_data_kernel, dim3((unsigned)((n + 255) / 256)),
                     dim3(256), 0, st, dy, w, dx, npix, c, epi, gate);
  return hipGetLastError();
}

static int64_t head_wgrad_blocks(int64_t npix) {
  int64_t b = (npix + 1023) / 1024;
  return b < 1 ? 1 : (b > 1024 ? 1024 : b);
}

size_t head_wgrad_ws_bytes(const fg_conv_desc &d) {
  int64_t npix = (int64_t)d.n * d.h * d.w;
  return (size_t)head_wgrad_blocks(npix) * d.c * sizeof(float);
}

hipError_t launch_head_wgrad(const uint16_t *x, const uint16_t *dy,
                             uint16_t *dw, int64_t npix, int32_t c, float *ws,
                             hipStream_t st) {
  int64_t nb = head_wgrad_blocks(npix);
  int64_t chunk = (npix + nb - 1) / nb;
  hipLaunchKernelGGL(head_wgrad_kernel, dim3((unsigned)nb),
                     dim3(kHeadWgradThreads), 0, st, x, dy, npix, c, chunk,
                     ws);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(split_reduce_kernel, dim3((unsigned)((c / 4 + 255) / 256)),
                     dim3(256), 0, st, ws, (int)nb, (int64_t)c, dw);
  return hipGetLastError();
}

}  // namespace fg
