// Implicit-GEMM fp16 convolutions on fp16 MFMA (fp32 accumulate) for gfx950.
//
// Data convolutions (forward, input gradient, transposed forward) are one
// kernel: GEMM rows are output channels, columns are output positions of one
// phase, and the reduction runs over (tap, input channel). The input image is
// gathered straight from NHWC memory (zero outside the image); nothing is
// materialised. Strided input gradients and transposed convolutions are split
// into output phases so that no multiply touches an inserted zero. Shapes
// that give too few output tiles to fill the GPU split the reduction across
// workgroups; fp32 partials are then summed in split order by a second kernel
// that also applies the epilogue.
//
// The kernel gradient is a second kernel: rows are (tap, input channel),
// columns output channels, reduction over all output positions, split across
// workgroups with fp32 partials summed afterwards in a fixed order.
//
// Both kernels stage 64-deep reduction slices of each operand in LDS (double
// buffered, one barrier per slice). LDS rows are 128 bytes with the eight
// 16-byte chunks of a row permuted by an XOR of row bits, so the 16-byte MFMA
// operand reads of 8 consecutive rows hit distinct banks. Operands whose
// reduction dimension is strided in memory are transposed in registers on
// their way to LDS. Each of the 4 waves owns a (BM/2) x (BN/2) block of the
// tile and issues v_mfma_f32_32x32x16_f16 over it.
#include "common.h"
#include "internal.h"

namespace fg {

constexpr int BK = 64;        // reduction slice per LDS stage (halves)

// Tile configuration: BM x BN output tile, WGM x WGN waves, each owning a
// (BM/WGM) x (BN/WGN) block of 32x32 MFMA fragments.
template <int BM_, int BN_, int WGM_, int WGN_>
struct Cfg {
  static constexpr int BM = BM_, BN = BN_, WGM = WGM_, WGN = WGN_;
  static constexpr int NT = 64 * WGM * WGN;
  static constexpr int WM = BM / WGM, WN = BN / WGN;
  static constexpr int FM = WM / 32, FN = WN / 32;
};
// 256x256 tile, 8 waves (two per SIMD) of 128x64: one wave's MFMAs overlap
// the other's address, load and LDS instructions.
using BigCfg = Cfg<256, 256, 2, 4>;
// 128x128 tile, 4 waves of 64x64; two workgroups fit on a CU.
using SmallCfg = Cfg<128, 128, 2, 2>;

// Offset (in halves) of 16-byte chunk `chunk` (0..7) of LDS row `row`.
__device__ __forceinline__ int lds_idx(int row, int chunk) {
  return row * BK + ((chunk ^ ((row ^ (row >> 3)) & 7)) << 3);
}

// ---------------------------------------------------------------------------
template <class C>
struct Core {
  static constexpr int FM = C::FM, FN = C::FN;
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
    const int r = lane & 31, kh = lane >> 5;
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      u32x4 a[FM], b[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        a[i] = *reinterpret_cast<const u32x4 *>(
            sA + lds_idx(wm0 + i * 32 + r, 2 * ks + kh));
#pragma unroll
      for (int j = 0; j < FN; ++j)
        b[j] = *reinterpret_cast<const u32x4 *>(
            sB + lds_idx(wn0 + j * 32 + r, 2 * ks + kh));
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = mfma32(a[i], b[j], acc[i][j]);
    }
  }
};

// Transpose 4 rows of 8 halves (row = reduction index) into 8 LDS rows
// row0..row0+7 at 4-half unit kq (8 bytes each).
__device__ __forceinline__ void store_t4x8(uint16_t *s, int row0, int kq,
                                           const u32x4 q[4]) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    u32x2 lo, hi;
    lo[0] = pack_lo(q[0][e], q[1][e]);
    lo[1] = pack_lo(q[2][e], q[3][e]);
    hi[0] = pack_hi(q[0][e], q[1][e]);
    hi[1] = pack_hi(q[2][e], q[3][e]);
    const int r0 = row0 + 2 * e, r1 = r0 + 1;
    *reinterpret_cast<u32x2 *>(s + lds_idx(r0, kq >> 1) + (kq & 1) * 4) = lo;
    *reinterpret_cast<u32x2 *>(s + lds_idx(r1, kq >> 1) + (kq & 1) * 4) = hi;
  }
}

__device__ __forceinline__ u32x4 ldg16(const uint16_t *p) {
  return *reinterpret_cast<const u32x4 *>(p);
}

__device__ __forceinline__ u32x2 to_h4(float a, float b, float c, float d) {
  u32x2 o;
  o[0] = (uint32_t)f32_to_h(a) | ((uint32_t)f32_to_h(b) << 16);
  o[1] = (uint32_t)f32_to_h(c) | ((uint32_t)f32_to_h(d) << 16);
  return o;
}

// Apply the epilogue to 4 consecutive channels; gate and out point at them
// (out is read for FG_EPI_ACC only).
__device__ __forceinline__ void epilogue4(float v[4], int epi, const uint16_t *gate,
                                          const uint16_t *out) {
  if (epi == FG_EPI_RELU) {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = v[e] > 0.f ? v[e] : 0.f;
  } else if (epi == FG_EPI_GATE) {
    u32x2 gw = *reinterpret_cast<const u32x2 *>(gate);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      uint16_t gb = (uint16_t)(gw[e >> 1] >> (16 * (e & 1)));
      v[e] = h_to_f32(gb) > 0.f ? v[e] : 0.f;
    }
  } else if (epi == FG_EPI_ACC) {
    u32x2 ow = *reinterpret_cast<const u32x2 *>(out);
#pragma unroll
    for (int e = 0; e < 4; ++e)
      v[e] += h_to_f32((uint16_t)(ow[e >> 1] >> (16 * (e & 1))));
  }
}

// ---------------------------------------------------------------------------
// Data convolution kernel.
//   WK    weights are k-major (forward: reduction contiguous per output
//         channel) or mn-major (input gradient / transposed: output channel
//         contiguous), the latter transposed in registers.
//   FAST  reduction channels are a multiple of BK, so a slice is one tap.
//   SPLIT the reduction is split across workgroups: write fp32 partials
//         (a.nsplit > 1) instead of the fp16 output.
// blockIdx.z = phase * nsplit + split.
template <class C, bool WK, bool FAST, bool SPLIT>
__global__ __launch_bounds__(C::NT) void data_conv_kernel(DataConvArgs a) {
  constexpr int BM = C::BM, BN = C::BN, NT = C::NT;
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][BM * BK];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][BN * BK];

  const int phase = blockIdx.z / a.nsplit, split = blockIdx.z % a.nsplit;
  const Phase P = a.ph[phase];
  const int npix = a.n * P.mh * P.mw;
  const int n0 = blockIdx.x * BN;
  const int m0 = blockIdx.y * BM;
  if (n0 >= npix) return;
  const int ntap = P.nr * P.ns;
  const int ktot = ntap * a.cr;
  const int nk = (ktot + BK - 1) / BK;
  const int kchunk = (nk + a.nsplit - 1) / a.nsplit;
  const int kbeg = min(nk, split * kchunk), kend = min(nk, kbeg + kchunk);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave / C::WGN) * C::WM, wn0 = (wave % C::WGN) * C::WN;

  // --- B (activation gather) loader state: 8 threads per column (one
  // 16-byte chunk each), NT/8 columns per pass, BCOL passes.
  constexpr int RPP = NT / 8;  // rows per pass
  constexpr int BCOL = BN / RPP;
  const int bc8 = tid & 7;
  int bbase[BCOL], bh[BCOL], bw[BCOL];
#pragma unroll
  for (int i = 0; i < BCOL; ++i) {
    int col = n0 + (tid >> 3) + RPP * i;
    if (col < npix) {
      int b = col % P.mw, t = col / P.mw;
      int aa = t % P.mh, nn = t / P.mh;
      bh[i] = aa * a.istr;
      bw[i] = b * a.istr;
      bbase[i] = ((nn * a.hi + bh[i]) * a.wi + bw[i]) * a.ldi;
    } else {
      bh[i] = -(1 << 29);  // fails every bounds check
      bw[i] = 0;
      bbase[i] = 0;
    }
  }

  constexpr int AROW = BM / RPP;
  constexpr int AUNITS = (BK / 4) * (BM / 8);
  constexpr int AUPT = (AUNITS + NT - 1) / NT;
  u32x4 ra[WK ? AROW : 4 * AUPT];
  u32x4 rb[BCOL];

  // tap t -> input offset (dh, dw) and kernel element offset woff = r*S + s
  auto tap_geom = [&](int t, int &dh, int &dw, int &woff) {
    int i = t / P.ns, j = t - (t / P.ns) * P.ns;
    dh = P.dh0 + P.dstep * i;
    dw = P.dw0 + P.dstep * j;
    woff = (P.r0 + P.rstep * i) * a.s + (P.s0 + P.rstep * j);
  };

  auto load = [&](int kt) {
    const int k0 = kt * BK;
    int ft = 0, fcr = 0, fdh = 0, fdw = 0, fwoff = 0;
    if (FAST) {  // the whole slice lies in one tap
      ft = k0 / a.cr;
      fcr = k0 - ft * a.cr;
      tap_geom(ft, fdh, fdw, fwoff);
    }
    // B: activations
    {
      int kk = k0 + bc8 * 8, dh, dw, woff, cr;
      bool kv = kk < ktot;
      if (FAST) {
        dh = fdh; dw = fdw; cr = fcr + bc8 * 8;
      } else {
        int t = kv ? kk / a.cr : 0;
        cr = kv ? kk - t * a.cr : 0;
        tap_geom(t, dh, dw, woff);
      }
      const int delta = (dh * a.wi + dw) * a.ldi + cr;
#pragma unroll
      for (int i = 0; i < BCOL; ++i) {
        int hh = bh[i] + dh, ww = bw[i] + dw;
        bool v = kv && hh >= 0 && hh < a.hi && ww >= 0 && ww < a.wi;
        rb[i] = v ? ldg16(a.act + (size_t)(bbase[i] + delta)) : u32x4{0, 0, 0, 0};
      }
    }
    // A: weights
    if (WK) {
      int kk = k0 + bc8 * 8, dh, dw, woff, cr;
      bool kv = kk < ktot;
      if (FAST) {
        woff = fwoff; cr = fcr + bc8 * 8;
      } else {
        int t = kv ? kk / a.cr : 0;
        cr = kv ? kk - t * a.cr : 0;
        tap_geom(t, dh, dw, woff);
      }
      const uint16_t *src = a.wgt + (size_t)woff * a.cr + cr;
#pragma unroll
      for (int i = 0; i < AROW; ++i) {
        int row = m0 + (tid >> 3) + RPP * i;
        ra[i] = (kv && row < a.co) ? ldg16(src + (size_t)row * a.ldw)
                                   : u32x4{0, 0, 0, 0};
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
        if (FAST) {
          woff = fwoff; cr = fcr + kq * 4;
        } else {
          int t = v ? kk / a.cr : 0;
          cr = v ? kk - t * a.cr : 0;
          tap_geom(t, dh, dw, woff);
        }
        // 4 consecutive reduction indices stay inside one tap (cr % 8 == 0)
        const uint16_t *src =
            a.wgt + (size_t)cr * a.w_red + (size_t)woff * a.w_tap + row;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          ra[4 * u + e] = v ? ldg16(src + (size_t)e * a.w_red) : u32x4{0, 0, 0, 0};
      }
    }
  };

  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < BCOL; ++i)
      *reinterpret_cast<u32x4 *>(&sB[buf][lds_idx((tid >> 3) + RPP * i, bc8)]) =
          rb[i];
    if (WK) {
#pragma unroll
      for (int i = 0; i < AROW; ++i)
        *reinterpret_cast<u32x4 *>(
            &sA[buf][lds_idx((tid >> 3) + RPP * i, bc8)]) = ra[i];
    } else {
#pragma unroll
      for (int u = 0; u < AUPT; ++u) {
        int unit = tid + u * NT;
        if (unit < AUNITS) {
          int cg = unit % (BM / 8), kq = unit / (BM / 8);
          store_t4x8(sA[buf], cg * 8, kq, &ra[4 * u]);
        }
      }
    }
  };

  Core<C> core;
  core.zero();
  if (kbeg < kend) {
    load(kbeg);
    store(0);
  }
  __syncthreads();
  for (int kt = kbeg; kt < kend; ++kt) {
    const int cur = (kt - kbeg) & 1;
    if (kt + 1 < kend) load(kt + 1);
    core.step(sA[cur], sB[cur], wm0, wn0, lane);
    if (kt + 1 < kend) store(cur ^ 1);
    __syncthreads();
  }

  // --- epilogue: lane holds 4 consecutive output channels of one position.
  constexpr int FM = C::FM, FN = C::FN;
  const size_t out_total = (size_t)a.n * a.ho * a.wo * a.co;
#pragma unroll
  for (int j = 0; j < FN; ++j) {
    int col = n0 + wn0 + j * 32 + (lane & 31);
    if (col >= npix) continue;
    int b = col % P.mw, t = col / P.mw;
    int aa = t % P.mh, nn = t / P.mh;
    // split partials are dense; the output has its own pixel stride
    size_t obase = ((size_t)(nn * a.ho + aa * a.ostr + P.ooh) * a.wo +
                    b * a.ostr + P.oow) *
                   (SPLIT ? a.co : a.ldo);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        int co = m0 + wm0 + i * 32 + 8 * g + 4 * (lane >> 5);
        if (co >= a.co) continue;
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = core.acc[i][j][4 * g + e];
        if (SPLIT) {
          f32x4 o = {v[0], v[1], v[2], v[3]};
          *reinterpret_cast<f32x4 *>(a.part + split * out_total + obase + co) = o;
        } else {
          epilogue4(v, a.epi, a.gate + obase + co, a.out + obase + co);
          *reinterpret_cast<u32x2 *>(a.out + obase + co) =
              to_h4(v[0], v[1], v[2], v[3]);
        }
      }
  }
}

// Sum nsplit fp32 partial arrays of len elements (dense, co channels per
// pixel) in split order, apply the epilogue, round to fp16 into out (and
// read gate) at pixel stride ldo. len and co are multiples of 4.
__global__ __launch_bounds__(256) void split_epilogue_kernel(
    const float *part, int nsplit, int64_t len, int co, int ldo, int epi,
    const uint16_t *gate, uint16_t *out) {
  int64_t i4 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i4 >= len) return;
  f32x4 s = *reinterpret_cast<const f32x4 *>(part + i4);
  for (int k = 1; k < nsplit; ++k) {
    f32x4 v = *reinterpret_cast<const f32x4 *>(part + (size_t)k * len + i4);
#pragma unroll
    for (int e = 0; e < 4; ++e) s[e] += v[e];
  }
  const int64_t pix = i4 / co;
  const int64_t o = pix * ldo + (i4 - pix * co);
  float v[4] = {s[0], s[1], s[2], s[3]};
  epilogue4(v, epi, gate + o, out + o);
  *reinterpret_cast<u32x2 *>(out + o) = to_h4(v[0], v[1], v[2], v[3]);
}

// ---------------------------------------------------------------------------
// Kernel-gradient kernel: rows rho = (tap, c) of the x patch, columns k.
template <class C, bool SPLIT>
__global__ __launch_bounds__(C::NT) void wgrad_kernel(WgradArgs a) {
  constexpr int BM = C::BM, BN = C::BN, NT = C::NT;
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][BM * BK];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][BN * BK];

  const int rsc = a.r * a.s * a.c;
  const int m0 = blockIdx.x * BM;  // rho
  const int n0 = blockIdx.y * BN;  // k
  const int split = blockIdx.z;
  const int mbeg = split * a.mchunk;
  const int mend = min(a.mtot, mbeg + a.mchunk);
  const int nk = mend > mbeg ? (mend - mbeg + BK - 1) / BK : 0;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave / C::WGN) * C::WM, wn0 = (wave % C::WGN) * C::WN;
  const int pq = a.p * a.q;

  constexpr int AUNITS = (BK / 4) * (BM / 8);
  constexpr int AUPT = (AUNITS + NT - 1) / NT;
  constexpr int BUNITS = (BK / 4) * (BN / 8);
  constexpr int BUPT = (BUNITS + NT - 1) / NT;
  u32x4 ra[4 * AUPT], rb[4 * BUPT];

  // per A unit: the tap and channel of its 8 rows are fixed for the block
  int ar[AUPT], as_[AUPT], ac[AUPT];
  bool arv[AUPT];
#pragma unroll
  for (int u = 0; u < AUPT; ++u) {
    int unit = tid + u * NT;
    int rho = m0 + (unit % (BM / 8)) * 8;
    arv[u] = unit < AUNITS && rho < rsc;
    int t = rho / a.c;
    ac[u] = rho - t * a.c;
    ar[u] = t / a.s;
    as_[u] = t - ar[u] * a.s;
  }

  auto load = [&](int kt) {
    const int k0 = mbeg + kt * BK;
#pragma unroll
    for (int u = 0; u < AUPT; ++u) {
      int unit = tid + u * NT;
      int mq = unit / (BM / 8);
      int m = k0 + mq * 4;
      int nn = m / pq, rem = m - nn * pq;
      int p = rem / a.q, q = rem - p * a.q;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        int hh = p * a.sh - a.ph + ar[u], ww = q * a.sw - a.pw + as_[u];
        bool v = arv[u] && (m + e) < mend && hh >= 0 && hh < a.h && ww >= 0 &&
                 ww < a.w;
        ra[4 * u + e] =
            v ? ldg16(a.x + ((size_t)((nn * a.h + hh) * a.w + ww)) * a.ldx + ac[u])
              : u32x4{0, 0, 0, 0};
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
      const uint16_t *src = a.dy + (size_t)m * a.k + k;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        rb[4 * u + e] = (uv && (m + e) < mend) ? ldg16(src + (size_t)e * a.k)
                                               : u32x4{0, 0, 0, 0};
    }
  };

  auto store = [&](int buf) {
#pragma unroll
    for (int u = 0; u < AUPT; ++u) {
      int unit = tid + u * NT;
      if (unit < AUNITS)
        store_t4x8(sA[buf], (unit % (BM / 8)) * 8, unit / (BM / 8), &ra[4 * u]);
    }
#pragma unroll
    for (int u = 0; u < BUPT; ++u) {
      int unit = tid + u * NT;
      if (unit < BUNITS)
        store_t4x8(sB[buf], (unit % (BN / 8)) * 8, unit / (BN / 8), &rb[4 * u]);
    }
  };

  Core<C> core;
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

  constexpr int FM = C::FM, FN = C::FN;
  bool bad = false;
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
        const f32x16 &c = core.acc[i][j];
        if (!SPLIT) {
          const u32x2 h = to_h4(c[4 * g], c[4 * g + 1], c[4 * g + 2], c[4 * g + 3]);
          bad |= nonfinite_h2(h[0]) | nonfinite_h2(h[1]);
          *reinterpret_cast<u32x2 *>(a.dw + (size_t)k * rsc + rho) = h;
        } else {
          f32x4 o = {c[4 * g], c[4 * g + 1], c[4 * g + 2], c[4 * g + 3]};
          *reinterpret_cast<f32x4 *>(
              a.part + ((size_t)split * a.k + k) * rsc + rho) = o;
        }
      }
  }
  if (!SPLIT && a.flag) flag_nonfinite(a.flag, bad);
}

// Sum nsplit fp32 partial arrays of len elements in split order, round to
// fp16. len is a multiple of 4. flag (or null): set to 1 if a result is
// +-inf or NaN.
__global__ __launch_bounds__(256) void split_reduce_kernel(const float *part,
                                                           int nsplit,
                                                           int64_t len,
                                                           uint16_t *out,
                                                           int32_t *flag) {
  int64_t i4 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  bool bad = false;
  if (i4 < len) {
    f32x4 s = *reinterpret_cast<const f32x4 *>(part + i4);
    for (int k = 1; k < nsplit; ++k) {
      f32x4 v = *reinterpret_cast<const f32x4 *>(part + (size_t)k * len + i4);
#pragma unroll
      for (int e = 0; e < 4; ++e) s[e] += v[e];
    }
    const u32x2 h = to_h4(s[0], s[1], s[2], s[3]);
    bad = nonfinite_h2(h[0]) | nonfinite_h2(h[1]);
    *reinterpret_cast<u32x2 *>(out + i4) = h;
  }
  if (flag) flag_nonfinite(flag, bad);
}

// Same sum when the partials are many and short (nsplit large, len small):
// one workgroup per 4 outputs; thread t adds splits t, t+256, ... in order,
// then a fixed-shape tree in LDS combines the 256 thread sums.
__global__ __launch_bounds__(256) void split_reduce_wide_kernel(
    const float *part, int nsplit, int64_t len, uint16_t *out, int32_t *flag) {
  __shared__ f32x4 red[256];
  const int64_t i4 = (int64_t)blockIdx.x * 4;
  f32x4 s = {0.f, 0.f, 0.f, 0.f};
  for (int k = threadIdx.x; k < nsplit; k += 256) {
    f32x4 v = *reinterpret_cast<const f32x4 *>(part + (size_t)k * len + i4);
#pragma unroll
    for (int e = 0; e < 4; ++e) s[e] += v[e];
  }
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) {
      f32x4 a = red[threadIdx.x], b = red[threadIdx.x + w];
#pragma unroll
      for (int e = 0; e < 4; ++e) a[e] += b[e];
      red[threadIdx.x] = a;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    f32x4 t = red[0];
    const u32x2 h = to_h4(t[0], t[1], t[2], t[3]);
    *reinterpret_cast<u32x2 *>(out + i4) = h;
    if (flag && (nonfinite_h2(h[0]) | nonfinite_h2(h[1]))) *flag = 1;
  }
}

// Same sum for a moderate number of longer partials (more than
// kMaxSerialSplit splits): each workgroup covers 64 outputs as 16 groups of
// 4, with 16 lanes per group; lane j adds splits j, j + 16, ... in order,
// then a fixed-shape tree combines the 16 lane sums. (The serial sum of
// split_reduce_kernel would wait on its many loads one by one.)
constexpr int kMaxSerialSplit = 16;
__global__ __launch_bounds__(256) void split_reduce_multi_kernel(
    const float *part, int nsplit, int64_t len, uint16_t *out, int32_t *flag) {
  __shared__ f32x4 red[16][16];  // [lane][group]
  const int grp = threadIdx.x & 15, lane = threadIdx.x >> 4;
  const int64_t i4 = ((int64_t)blockIdx.x * 16 + grp) * 4;
  f32x4 s = {0.f, 0.f, 0.f, 0.f};
  if (i4 < len)
    for (int k = lane; k < nsplit; k += 16) {
      const f32x4 v = *reinterpret_cast<const f32x4 *>(part + (size_t)k * len + i4);
#pragma unroll
      for (int e = 0; e < 4; ++e) s[e] += v[e];
    }
  red[lane][grp] = s;
  __syncthreads();
  for (int w = 8; w > 0; w >>= 1) {
    if (lane < w) {
      f32x4 a = red[lane][grp], b = red[lane + w][grp];
#pragma unroll
      for (int e = 0; e < 4; ++e) a[e] += b[e];
      red[lane][grp] = a;
    }
    __syncthreads();
  }
  bool bad = false;
  if (lane == 0 && i4 < len) {
    const f32x4 t = red[0][grp];
    const u32x2 h = to_h4(t[0], t[1], t[2], t[3]);
    bad = nonfinite_h2(h[0]) | nonfinite_h2(h[1]);
    *reinterpret_cast<u32x2 *>(out + i4) = h;
  }
  if (flag) flag_nonfinite(flag, bad);
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
    // four positions per iteration, their loads issued together
    int64_t pix = beg + row;
    for (; pix + 3 * rows < end; pix += 4 * rows) {
      float d[4];
      u32x4 xv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        d[u] = h_to_f32(dy[pix + u * rows]);
        xv[u] = ldg16(x + (pix + u * rows) * c + ch * 8);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[2 * e] += d[u] * h_to_f32((uint16_t)xv[u][e]);
          acc[2 * e + 1] += d[u] * h_to_f32((uint16_t)(xv[u][e] >> 16));
        }
    }
    for (; pix < end; pix += rows) {
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
// Host side: tile selection and launchers.
namespace {

int64_t data_tiles(const DataConvArgs &a, int bm, int bn) {
  int64_t t = 0;
  for (int i = 0; i < a.nphase; ++i) {
    int64_t np = (int64_t)a.n * a.ph[i].mh * a.ph[i].mw;
    t += ((np + bn - 1) / bn) * ((a.co + bm - 1) / bm);
  }
  return t;
}

int64_t data_nk_max(const DataConvArgs &a) {
  int64_t nk = 0;
  for (int i = 0; i < a.nphase; ++i) {
    int64_t kt = (int64_t)a.ph[i].nr * a.ph[i].ns * a.cr;
    nk = std::max<int64_t>(nk, (kt + BK - 1) / BK);
  }
  return nk;
}

constexpr int64_t kCUs = 256;
// flop/s of one 128x128 workgroup of the LDS-DMA kernel, in the units of
// the 256x256 rate below: alone on its CU (a launch of at most one
// workgroup per CU), and with a second one sharing the CU. Timed on the
// network's 16x16 and 32x32 layers at forced splits: a CU holding one
// workgroup runs 1.25x as fast as one holding two (0.39 against 0.97 us
// per workgroup stage), so splits that double the workgroups to fill the
// second slot lose.
constexpr double kRateSmallDmaAlone = 2.1e12, kRateSmallDmaPaired = 0.85e12;
// The register-staged 128x128 kernel, alone or paired.
constexpr double kRateSmallRegs = 1.3e12;

}  // namespace

// Split/tile choice by an estimate of the run time: resident workgroup
// slots per GPU (one 256x256 workgroup or two 128x128 ones per CU), the
// per-workgroup MFMA rate each reaches (measured on MI355X; for 128x128
// tiles it depends on whether the launch fits one workgroup per CU), waves of
// workgroups with a fixed cost per wave (prologue and tile store, which one
// workgroup per CU cannot overlap with its MFMA work), and the fp32
// partials a split writes and re-reads.
struct TileChoice {
  bool big;
  int32_t nsplit;
};
struct TileCost {
  double rate_big, rate_small;  // flop/s of one 256x256 / 128x128 workgroup
  double partial_bw;            // B/s for fp32 partial traffic (8 B/element)
  double split_const;           // s, the reduction launch of a split
  double wave_const;            // s per wave of workgroups
  double rate_small_alone;      // a 128x128 workgroup with its CU to itself
};
// Data convolutions: rates chosen by timing the network's layers.
static TileCost data_cost(bool dma_small) {
  return dma_small ? TileCost{3.0e12, kRateSmallDmaPaired, 6.0e12, 4e-6, 0.0,
                              kRateSmallDmaAlone}
                   : TileCost{3.0e12, kRateSmallRegs, 6.0e12, 4e-6, 0.0, kRateSmallRegs};
}
// Kernel gradient: a least-squares fit of this model to the DMA kernel's
// times on the network's twelve kernel-gradient shapes at 1-8 splits
// (per 256x256x32 stage 0.66 us, 4.2 us per wave, partials at 4.05 TB/s,
// 6.3 us per split launch; mean error 9%). The 128x128 rate is the
// register-staged kernel's, which only shapes too small for 256x256 tiles
// take.
constexpr TileCost kWgradCost{6.35e12, 1.3e12, 4.05e12, 6.3e-6, 4.2e-6, 1.3e12};

TileChoice choose_tiles(int64_t tiles_big, int64_t tiles_small, int64_t nk,
                        int64_t out_elems, bool allow_big, const TileCost &cost,
                        int max_split = 16) {
  TileChoice best{false, 1};
  double best_t = 1e30;
  for (int big = 0; big < 2; ++big) {
    if (big && !allow_big) continue;
    const int64_t tiles = big ? tiles_big : tiles_small;
    const int64_t slots = big ? kCUs : 2 * kCUs;
    const int t = big ? 256 : 128;
    for (int ns = 1; ns <= max_split; ++ns) {
      if (ns > 1 && (nk + ns - 1) / ns < 4) break;  // >= 4 slices per split
      const double rate = big                 ? cost.rate_big
                          : tiles * ns <= kCUs ? cost.rate_small_alone
                                               : cost.rate_small;
      const int64_t waves = (tiles * ns + slots - 1) / slots;
      const int64_t nk_split = (nk + ns - 1) / ns;
      const double t_block = 2.0 * t * t * BK * (double)nk_split / rate;
      double tt = waves * (t_block + cost.wave_const);
      if (ns > 1) tt += ns * (double)out_elems * 8.0 / cost.partial_bw + cost.split_const;
      if (tt < best_t * 0.98) {  // prefer fewer splits on near ties
        best_t = tt;
        best = TileChoice{big != 0, ns};
      }
    }
  }
  return best;
}

DataPlan plan_data_conv(const DataConvArgs &a) {
  DataPlan pl;
  const int64_t out = (int64_t)a.n * a.ho * a.wo * a.co;
  const TileChoice c = choose_tiles(data_tiles(a, 256, 256),
                                    data_tiles(a, 128, 128), data_nk_max(a), out,
                                    a.co >= 256, data_cost(data_dma_ok(a)));
  pl.big = c.big;
  pl.nsplit = c.nsplit;
  pl.ws_bytes = pl.nsplit > 1 ? (size_t)pl.nsplit * out * sizeof(float) : 0;
  return pl;
}

template <class C, bool WK, bool FAST>
static hipError_t launch_dc(const DataConvArgs &a, hipStream_t st) {
  int maxpix = 0;
  for (int i = 0; i < a.nphase; ++i)
    maxpix = std::max(maxpix, a.n * a.ph[i].mh * a.ph[i].mw);
  dim3 grid((maxpix + C::BN - 1) / C::BN, (a.co + C::BM - 1) / C::BM,
            a.nphase * a.nsplit);
  if (a.nsplit > 1)
    hipLaunchKernelGGL((data_conv_kernel<C, WK, FAST, true>), grid, dim3(C::NT),
                       0, st, a);
  else
    hipLaunchKernelGGL((data_conv_kernel<C, WK, FAST, false>), grid,
                       dim3(C::NT), 0, st, a);
  return hipGetLastError();
}

template <class C>
static hipError_t launch_dc_tile(const DataConvArgs &a, bool w_kmajor,
                                 hipStream_t st) {
  const bool fast = (a.cr % BK) == 0;
  if (w_kmajor)
    return fast ? launch_dc<C, true, true>(a, st)
                : launch_dc<C, true, false>(a, st);
  return fast ? launch_dc<C, false, true>(a, st)
              : launch_dc<C, false, false>(a, st);
}

hipError_t launch_data_conv(const DataConvArgs &a0, bool w_kmajor,
                            hipStream_t st) {
  DataConvArgs a = a0;
  const DataPlan pl = plan_data_conv(a);
  a.nsplit = pl.nsplit;
  hipError_t e = prof_begin(st);
  if (e != hipSuccess) return e;
  e = !pl.big ? (data_dma_ok(a) ? launch_data_conv_dma_small(a, w_kmajor, st)
                                : launch_dc_tile<SmallCfg>(a, w_kmajor, st))
      : data_halo_ok(a) ? launch_data_conv_halo(a, w_kmajor, st)
      : data_dma_ok(a)  ? launch_data_conv_dma(a, w_kmajor, st)
                        : launch_dc_tile<BigCfg>(a, w_kmajor, st);
  if (e == hipSuccess) e = prof_end(st);
  if (e != hipSuccess || a.nsplit == 1) return e;
  const int64_t len = (int64_t)a.n * a.ho * a.wo * a.co;
  hipLaunchKernelGGL(split_epilogue_kernel,
                     dim3((unsigned)((len / 4 + 255) / 256)), dim3(256), 0, st,
                     a.part, a.nsplit, len, a.co, a.ldo, a.epi, a.gate, a.out);
  return hipGetLastError();
}

const char *data_conv_kernel_name(const DataConvArgs &a, bool w_kmajor) {
  // [big][w_kmajor][fast][split], as a kernel trace prints them
  static const char *names[2][2][2][2] = {
      {{{"data_conv_kernel<Cfg<128, 128, 2, 2>, false, false, false>",
         "data_conv_kernel<Cfg<128, 128, 2, 2>, false, false, true>"},
        {"data_conv_kernel<Cfg<128, 128, 2, 2>, false, true, false>",
         "data_conv_kernel<Cfg<128, 128, 2, 2>, false, true, true>"}},
       {{"data_conv_kernel<Cfg<128, 128, 2, 2>, true, false, false>",
         "data_conv_kernel<Cfg<128, 128, 2, 2>, true, false, true>"},
        {"data_conv_kernel<Cfg<128, 128, 2, 2>, true, true, false>",
         "data_conv_kernel<Cfg<128, 128, 2, 2>, true, true, true>"}}},
      {{{"data_conv_kernel<Cfg<256, 256, 2, 4>, false, false, false>",
         "data_conv_kernel<Cfg<256, 256, 2, 4>, false, false, true>"},
        {"data_conv_kernel<Cfg<256, 256, 2, 4>, false, true, false>",
         "data_conv_kernel<Cfg<256, 256, 2, 4>, false, true, true>"}},
       {{"data_conv_kernel<Cfg<256, 256, 2, 4>, true, false, false>",
         "data_conv_kernel<Cfg<256, 256, 2, 4>, true, false, true>"},
        {"data_conv_kernel<Cfg<256, 256, 2, 4>, true, true, false>",
         "data_conv_kernel<Cfg<256, 256, 2, 4>, true, true, true>"}}}};
  const DataPlan pl = plan_data_conv(a);
  if (pl.big && data_halo_ok(a)) {
    static const char *hn[2][2] = {
        {"data_conv_halo_kernel<false, false>", "data_conv_halo_kernel<false, true>"},
        {"data_conv_halo_kernel<true, false>", "data_conv_halo_kernel<true, true>"}};
    return hn[w_kmajor][pl.nsplit > 1];
  }
  if (!pl.big && data_dma_ok(a)) {
    static const char *sn[2][2] = {
        {"data_conv_dma_kernel<128, false, false>", "data_conv_dma_kernel<128, false, true>"},
        {"data_conv_dma_kernel<128, true, false>", "data_conv_dma_kernel<128, true, true>"}};
    return sn[w_kmajor][pl.nsplit > 1];
  }
  if (pl.big && data_dma_ok(a)) {
    static const char *dn[2][2] = {
        {"data_conv_dma_kernel<false, false>", "data_conv_dma_kernel<false, true>"},
        {"data_conv_dma_kernel<true, false>", "data_conv_dma_kernel<true, true>"}};
    return dn[w_kmajor][pl.nsplit > 1];
  }
  return names[pl.big][w_kmajor][(a.cr % BK) == 0][pl.nsplit > 1];
}

// max_ws_bytes bounds the fp32 partials of a split (and so the split count).
// A kernel gradient whose R*S*C or K is below 256 (so no 256 x 256 tile)
// with a long reduction needs many splits to fill the GPU: a 1x1 layer of
// 128 x 64 has a single 128 x 128 tile. Such shapes may split up to
// kMaxWgradSplit ways (at least 4 stages each); the others keep the cap of
// 16, under which the network's layers were fitted and timed.
constexpr int kMaxWgradSplit = 256;

static TileChoice wgrad_choice(const fg_conv_desc &d, int32_t p, int32_t q,
                               size_t max_ws_bytes) {
  const int64_t rsc = (int64_t)d.r * d.s * d.c;
  const int64_t mtot = (int64_t)d.n * p * q;
  const int64_t tb = ((rsc + 255) / 256) * ((d.k + 255) / 256);
  const int64_t ts = ((rsc + 127) / 128) * ((d.k + 127) / 128);
  const size_t per_split = (size_t)d.k * rsc * sizeof(float);
  const size_t cap = max_ws_bytes / per_split;
  const bool allow_big = rsc >= 256 && d.k >= 256;
  const int limit = allow_big ? 16 : kMaxWgradSplit;
  const int max_split = cap >= (size_t)limit ? limit : (cap < 2 ? 1 : (int)cap);
  return choose_tiles(tb, ts, (mtot + BK - 1) / BK, (int64_t)d.k * rsc, allow_big,
                      kWgradCost, max_split);
}

const char *wgrad_kernel_name(const fg_conv_desc &d) {
  int32_t p = (d.h + 2 * d.pad_h - d.r) / d.stride_h + 1;
  int32_t q = (d.w + 2 * d.pad_w - d.s) / d.stride_w + 1;
  const WgradPlan pl = plan_wgrad(d, p, q);
  WgradArgs wa;
  wa.n = d.n; wa.h = d.h; wa.w = d.w; wa.c = d.c; wa.k = d.k;
  wa.ldx = d.x_ld ? d.x_ld : d.c;
  wa.mtot = d.n * p * q;
  if (pl.big && wgrad_dma_ok(wa))
    return pl.nsplit > 1 ? "wgrad_dma_kernel<true>" : "wgrad_dma_kernel<false>";
  static const char *names[2][2] = {
      {"wgrad_kernel<Cfg<128, 128, 2, 2>, false>",
       "wgrad_kernel<Cfg<128, 128, 2, 2>, true>"},
      {"wgrad_kernel<Cfg<256, 256, 2, 4>, false>",
       "wgrad_kernel<Cfg<256, 256, 2, 4>, true>"}};
  return names[pl.big][pl.nsplit > 1];
}

WgradPlan plan_wgrad(const fg_conv_desc &d, int32_t p, int32_t q,
                     size_t max_ws_bytes) {
  WgradPlan pl;
  const TileChoice c = wgrad_choice(d, p, q, max_ws_bytes);
  const int64_t rsc = (int64_t)d.r * d.s * d.c;
  const int64_t mtot = (int64_t)d.n * p * q;
  int64_t ns = c.nsplit;
  int64_t chunk = (mtot + ns - 1) / ns;
  chunk = (chunk + BK - 1) / BK * BK;
  ns = (mtot + chunk - 1) / chunk;
  pl.big = c.big;
  pl.nsplit = (int32_t)ns;
  pl.mchunk = (int32_t)chunk;
  pl.ws_bytes = ns > 1 ? (size_t)ns * d.k * rsc * sizeof(float) : 0;
  return pl;
}

hipError_t launch_wgrad(const WgradArgs &a, bool big, hipStream_t st) {
  const int rsc = a.r * a.s * a.c;
  const bool split = a.nsplit > 1;
  hipError_t e = prof_begin(st);
  if (e != hipSuccess) return e;
  if (big && wgrad_dma_ok(a)) {
    e = launch_wgrad_dma(a, st);
  } else if (big) {
    dim3 grid((rsc + 255) / 256, (a.k + 255) / 256, a.nsplit);
    if (split)
      hipLaunchKernelGGL((wgrad_kernel<BigCfg, true>), grid, dim3(BigCfg::NT), 0,
                         st, a);
    else
      hipLaunchKernelGGL((wgrad_kernel<BigCfg, false>), grid, dim3(BigCfg::NT), 0,
                         st, a);
    e = hipGetLastError();
  } else {
    dim3 grid((rsc + 127) / 128, (a.k + 127) / 128, a.nsplit);
    if (split)
      hipLaunchKernelGGL((wgrad_kernel<SmallCfg, true>), grid, dim3(SmallCfg::NT),
                         0, st, a);
    else
      hipLaunchKernelGGL((wgrad_kernel<SmallCfg, false>), grid,
                         dim3(SmallCfg::NT), 0, st, a);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = prof_end(st);
  if (e != hipSuccess || !split) return e;
  const int64_t len = (int64_t)a.k * rsc;
  if (a.nsplit > kMaxSerialSplit) {
    hipLaunchKernelGGL(split_reduce_multi_kernel, dim3((unsigned)((len + 63) / 64)),
                       dim3(256), 0, st, a.part, a.nsplit, len, a.dw, a.flag);
    return hipGetLastError();
  }
  dim3 g2((unsigned)((len / 4 + 255) / 256));
  hipLaunchKernelGGL(split_reduce_kernel, g2, dim3(256), 0, st, a.part,
                     a.nsplit, len, a.dw, a.flag);
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
  hipError_t e = prof_begin(st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(head_fwd_kernel, dim3((unsigned)blocks), dim3(256), 0, st,
                     x, w, y, npix, c, L, logL, epi, gate);
  e = hipGetLastError();
  return e == hipSuccess ? prof_end(st) : e;
}

hipError_t launch_head_bwd_data(const uint16_t *dy, const uint16_t *w,
                                uint16_t *dx, int64_t npix, int32_t c,
                                int32_t epi, const uint16_t *gate,
                                hipStream_t st) {
  int64_t n = npix * (c / 8);
  hipError_t e = prof_begin(st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(head_bwd_data_kernel, dim3((unsigned)((n + 255) / 256)),
                     dim3(256), 0, st, dy, w, dx, npix, c, epi, gate);
  e = hipGetLastError();
  return e == hipSuccess ? prof_end(st) : e;
}

static int64_t head_wgrad_blocks(int64_t npix) {
  // about 256 positions per workgroup, four workgroups per CU on the
  // full-size head
  int64_t b = (npix + 255) / 256;
  return b < 1 ? 1 : (b > 2048 ? 2048 : b);
}

size_t head_wgrad_ws_bytes(const fg_conv_desc &d) {
  int64_t npix = (int64_t)d.n * d.h * d.w;
  return (size_t)head_wgrad_blocks(npix) * d.c * sizeof(float);
}

hipError_t launch_head_wgrad(const uint16_t *x, const uint16_t *dy,
                             uint16_t *dw, int64_t npix, int32_t c, float *ws,
                             int32_t *flag, hipStream_t st) {
  int64_t nb = head_wgrad_blocks(npix);
  int64_t chunk = (npix + nb - 1) / nb;
  hipError_t e = prof_begin(st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(head_wgrad_kernel, dim3((unsigned)nb),
                     dim3(kHeadWgradThreads), 0, st, x, dy, npix, c, chunk,
                     ws);
  e = hipGetLastError();
  if (e == hipSuccess) e = prof_end(st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(split_reduce_wide_kernel, dim3((unsigned)(c / 4)),
                     dim3(256), 0, st, ws, (int)nb, (int64_t)c, dw, flag);
  return hipGetLastError();
}

}  // namespace fg
