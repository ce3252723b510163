// Implicit-GEMM convolutions fed by LDS DMA (gfx950 buffer_load ... lds).
//
// Same GEMM formulation as the register-staged kernels in conv_igemm.hip
// (data convolutions: rows = output channels, columns = output positions of
// one phase; kernel gradient: rows = (tap, input channel), columns = output
// channels), for 256 x 256 tiles with 8 waves of 128 x 64. Operands go from
// global memory straight into LDS: no register staging, no LDS store
// instructions, and a ring of four 32-deep reduction stages (128 KiB), so
// each stage's loads are issued three stages before they are consumed.
// Padding and ragged tails cost nothing: an out-of-range buffer offset
// returns zeros.
//
// Two LDS tile layouts:
//   k-major  (row = GEMM row/column, 32 reduction halves = 64 bytes per row;
//            16-byte chunk c stored at c ^ g(row)); MFMA operands are single
//            16-byte reads, conflict-free for 8 or 16 consecutive rows.
//   mn-major (row = reduction index, 256 halves = 512 bytes per row; 32-byte
//            block b stored at b ^ s(row)); MFMA operands are two transposing
//            8-byte reads (ds_read_b64_tr_b16), each 64-lane read touching
//            every bank pair at most twice.
// The mn-major layout lets operands whose reduction index is strided in
// memory (input-gradient and transposed-conv weights, both kernel-gradient
// operands) be copied row by row as they lie in memory.
#include "common.h"
#include "internal.h"

namespace fg {
namespace dma {

constexpr int BK = 32;        // reduction per stage
constexpr int NS = 4;         // stages in the ring
constexpr int TM = 256, TN = 256;
constexpr int NT = 512;       // 8 waves: 2 (rows) x 4 (columns)
constexpr int WM = 128, WN = 64;
constexpr int FM = WM / 32, FN = WN / 32;
constexpr int TILE_BYTES = TM * BK * 2;  // 16 KiB per operand per stage
constexpr unsigned kOOB = 0x80000000u;   // beyond any tensor: loads zero
constexpr int kRsrcFlags = 0x00020000;   // raw buffer, 32-bit data format

typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s;
typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ int kmaj_off(int row, int c) {  // bytes
  return row * 64 + ((c ^ (((row >> 1) ^ (row >> 3)) & 3)) << 4);
}
__device__ __forceinline__ int mn_swz(int k) {
  return (k & 3) | (((k >> 3) & 1) << 2);
}
__device__ __forceinline__ int mnmaj_off(int k, int n) {  // bytes, n % 4 == 0
  return k * 512 + ((2 * n) ^ (mn_swz(k) << 5));
}

// Workgroup barrier without a memory fence. __syncthreads() would add a
// release fence, which waits for every outstanding LDS-DMA load (vmcnt(0))
// and so drains the ring; ordering is established instead by each wave's
// explicit vmcnt wait on its own loads before it arrives here. The empty asm
// statements keep the compiler from moving LDS accesses across the barrier.
__device__ __forceinline__ void barrier_nofence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// s_waitcnt with only vmcnt constrained (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vm() {
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | (((N >> 4) & 3) << 14));
}

__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t rs, uint8_t *lds,
                                      unsigned voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void *)lds, 16, voff, 0, 0, 0);
}

// MFMA operand of a 32-row block starting at `base` for reduction step ks.
template <bool KMAJOR>
__device__ __forceinline__ u32x4 frag(const uint8_t *tile, int base, int ks,
                                      int lane) {
  if (KMAJOR) {
    return *reinterpret_cast<const u32x4 *>(
        tile + kmaj_off(base + (lane & 31), 2 * ks + (lane >> 5)));
  } else {
    const int g = lane >> 4, m = lane & 15;
    const int k = 8 * (g >> 1) + (m >> 2) + 16 * ks;
    const int n = base + 16 * (g & 1) + 4 * (m & 3);
    v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_v4s *)(tile + mnmaj_off(k, n)));
    v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_v4s *)(tile + mnmaj_off(k + 4, n)));
    u32x2 a = __builtin_bit_cast(u32x2, lo), b = __builtin_bit_cast(u32x2, hi);
    return u32x4{a[0], a[1], b[0], b[1]};
  }
}

template <bool AK, bool BKM>
__device__ __forceinline__ void mma_stage(f32x16 (&acc)[FM][FN],
                                          const uint8_t *ta, const uint8_t *tb,
                                          int wm0, int wn0, int lane) {
#pragma unroll
  for (int ks = 0; ks < BK / 16; ++ks) {
    u32x4 a[FM], b[FN];
#pragma unroll
    for (int i = 0; i < FM; ++i) a[i] = frag<AK>(ta, wm0 + 32 * i, ks, lane);
#pragma unroll
    for (int j = 0; j < FN; ++j) b[j] = frag<BKM>(tb, wn0 + 32 * j, ks, lane);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) acc[i][j] = mfma32(a[i], b[j], acc[i][j]);
  }
}

// Position of this lane's two DMA slots in a k-major tile (rows) and in an
// mn-major tile (reduction rows, column offsets), per wave instruction jj.
struct KmSlot {
  int row[2], coff[2];  // tile row, reduction offset (halves) of the chunk
};
struct MnSlot {
  int krow[2], ncol[2];  // reduction row within the stage, tile column
};

__device__ __forceinline__ KmSlot km_slots(int wave, int lane) {
  KmSlot s;
#pragma unroll
  for (int jj = 0; jj < 2; ++jj) {
    int row = 16 * (2 * wave + jj) + (lane >> 2);
    int pc = lane & 3;
    s.row[jj] = row;
    s.coff[jj] = 8 * (pc ^ (((row >> 1) ^ (row >> 3)) & 3));
  }
  return s;
}

__device__ __forceinline__ MnSlot mn_slots(int wave, int lane) {
  MnSlot s;
#pragma unroll
  for (int jj = 0; jj < 2; ++jj) {
    int k = 2 * (2 * wave + jj) + (lane >> 5);
    int p = lane & 31;
    s.krow[jj] = k;
    s.ncol[jj] = ((p >> 1) ^ mn_swz(k)) * 16 + (p & 1) * 8;
  }
  return s;
}

// LDS destination of wave instruction jj of a stage (wave-uniform).
__device__ __forceinline__ int km_dst(int wave, int jj) {
  return 16 * (2 * wave + jj) * 64;
}
__device__ __forceinline__ int mn_dst(int wave, int jj) {
  return 2 * (2 * wave + jj) * 512;
}

__device__ __forceinline__ u32x2 to_h4(float a, float b, float c, float d) {
  u32x2 o;
  o[0] = (uint32_t)f32_to_h(a) | ((uint32_t)f32_to_h(b) << 16);
  o[1] = (uint32_t)f32_to_h(c) | ((uint32_t)f32_to_h(d) << 16);
  return o;
}

__device__ __forceinline__ void epilogue4(float v[4], int epi,
                                          const uint16_t *gate) {
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
  }
}

// The ring: stage s of operand X lives in its own LDS array so that the
// compiler can tell the stages apart when it places waits.
struct Ring {
  uint8_t *a[NS];
  uint8_t *b[NS];
};

// Runs the pipelined main loop over stages [0, nst): issue(st, slot) issues
// this wave's 4 DMA loads of stage st into ring slot `slot`.
template <bool AK, bool BKM, class Issue>
__device__ __forceinline__ void pipeline(f32x16 (&acc)[FM][FN], const Ring &R,
                                         int nst, int wm0, int wn0, int lane,
                                         Issue &&issue) {
#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    if (s < nst) issue(s, s);
  for (int it0 = 0; it0 < nst; it0 += NS) {
#pragma unroll
    for (int u = 0; u < NS; ++u) {
      const int it = it0 + u;
      if (it < nst) {
        // own loads of stage `it` done: only later stages may remain
        const int after = min(NS - 2, nst - 1 - it);
        if (after >= 2) wait_vm<8>();
        else if (after == 1) wait_vm<4>();
        else wait_vm<0>();
        barrier_nofence();  // every wave's stage `it` landed; slot of it-1 free
        if (it + NS - 1 < nst) issue(it + NS - 1, (u + NS - 1) % NS);
        mma_stage<AK, BKM>(acc, R.a[u], R.b[u], wm0, wn0, lane);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Data convolution (forward / input gradient / transposed forward).
// Requires reduction channels cr % 32 == 0 (a stage lies in one tap).
template <bool WK, bool SPLIT>
__global__ __launch_bounds__(NT) void data_conv_dma_kernel(DataConvArgs a) {
  __shared__ __attribute__((aligned(1024))) uint8_t sA0[TILE_BYTES], sA1[TILE_BYTES],
      sA2[TILE_BYTES], sA3[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sB0[TILE_BYTES], sB1[TILE_BYTES],
      sB2[TILE_BYTES], sB3[TILE_BYTES];
  const Ring R{{sA0, sA1, sA2, sA3}, {sB0, sB1, sB2, sB3}};

  const int phase = blockIdx.z / a.nsplit, split = blockIdx.z % a.nsplit;
  const Phase P = a.ph[phase];
  const int npix = a.n * P.mh * P.mw;
  const int n0 = blockIdx.x * TN;
  const int m0 = blockIdx.y * TM;
  if (n0 >= npix) return;
  const int ktot = P.nr * P.ns * a.cr;
  const int nk = ktot / BK;
  const int kchunk = (nk + a.nsplit - 1) / a.nsplit;
  const int kbeg = min(nk, split * kchunk), kend = min(nk, kbeg + kchunk);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 2) * WM, wn0 = (wave & 3) * WN;

  const __amdgpu_buffer_rsrc_t rs_act = __builtin_amdgcn_make_buffer_rsrc(
      (void *)a.act, 0, (int)((size_t)a.n * a.hi * a.wi * a.cr * 2), kRsrcFlags);
  const __amdgpu_buffer_rsrc_t rs_w = __builtin_amdgcn_make_buffer_rsrc(
      (void *)a.wgt, 0, a.wbytes, kRsrcFlags);

  // B: this lane's two output positions and chunk offsets
  const KmSlot bs = km_slots(wave, lane);
  int bh[2], bw[2], bbase[2];
#pragma unroll
  for (int jj = 0; jj < 2; ++jj) {
    int col = n0 + bs.row[jj];
    if (col < npix) {
      int b = col % P.mw, t = col / P.mw;
      int aa = t % P.mh, nn = t / P.mh;
      bh[jj] = aa * a.istr;
      bw[jj] = b * a.istr;
      bbase[jj] = ((nn * a.hi + bh[jj]) * a.wi + bw[jj]) * a.cr + bs.coff[jj];
    } else {
      bh[jj] = -(1 << 29);
      bw[jj] = 0;
      bbase[jj] = 0;
    }
  }
  const KmSlot as_k = km_slots(wave, lane);
  const MnSlot as_m = mn_slots(wave, lane);

  auto issue = [&](int st, int slot) {
    const int k0 = (kbeg + st) * BK;
    const int t = k0 / a.cr, cr0 = k0 - t * a.cr;
    const int ti = t / P.ns, tj = t - ti * P.ns;
    const int dh = P.dh0 + P.dstep * ti, dw = P.dw0 + P.dstep * tj;
    const int woff = (P.r0 + P.rstep * ti) * a.s + (P.s0 + P.rstep * tj);
    const int delta = (dh * a.wi + dw) * a.cr + cr0;
    uint8_t *ta = R.a[slot], *tb = R.b[slot];
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      int hh = bh[jj] + dh, ww = bw[jj] + dw;
      bool v = hh >= 0 && hh < a.hi && ww >= 0 && ww < a.wi;
      unsigned off = v ? (unsigned)(bbase[jj] + delta) * 2u : kOOB;
      dma16(rs_act, tb + km_dst(wave, jj), off);
    }
    if (WK) {
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        int co = m0 + as_k.row[jj];
        unsigned off =
            co < a.co ? (unsigned)(co * a.ldw + woff * a.cr + cr0 + as_k.coff[jj]) * 2u
                      : kOOB;
        dma16(rs_w, ta + km_dst(wave, jj), off);
      }
    } else {
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        int kred = cr0 + as_m.krow[jj];
        int co = m0 + as_m.ncol[jj];
        unsigned off =
            co < a.co ? (unsigned)(kred * a.w_red + woff * a.w_tap + co) * 2u : kOOB;
        dma16(rs_w, ta + mn_dst(wave, jj), off);
      }
    }
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  pipeline<WK, true>(acc, R, kend - kbeg, wm0, wn0, lane, issue);

  const size_t out_total = (size_t)a.n * a.ho * a.wo * a.co;
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
        for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * g + e];
        if (SPLIT) {
          f32x4 o = {v[0], v[1], v[2], v[3]};
          *reinterpret_cast<f32x4 *>(a.part + split * out_total + obase + co) = o;
        } else {
          epilogue4(v, a.epi, a.gate + obase + co);
          *reinterpret_cast<u32x2 *>(a.out + obase + co) =
              to_h4(v[0], v[1], v[2], v[3]);
        }
      }
  }
}

// ---------------------------------------------------------------------------
// Kernel gradient: rows rho = (tap, c) of one tap (c % 256 == 0 tiles),
// columns k (K % 256 == 0), reduction over output positions m.
template <bool SPLIT>
__global__ __launch_bounds__(NT) void wgrad_dma_kernel(WgradArgs a) {
  __shared__ __attribute__((aligned(1024))) uint8_t sA0[TILE_BYTES], sA1[TILE_BYTES],
      sA2[TILE_BYTES], sA3[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) uint8_t sB0[TILE_BYTES], sB1[TILE_BYTES],
      sB2[TILE_BYTES], sB3[TILE_BYTES];
  const Ring R{{sA0, sA1, sA2, sA3}, {sB0, sB1, sB2, sB3}};

  const int rsc = a.r * a.s * a.c;
  const int m0 = blockIdx.x * TM;  // rho
  const int n0 = blockIdx.y * TN;  // k
  const int split = blockIdx.z;
  const int mbeg = split * a.mchunk;
  const int mend = min(a.mtot, mbeg + a.mchunk);
  const int nst = mend > mbeg ? (mend - mbeg + BK - 1) / BK : 0;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 2) * WM, wn0 = (wave & 3) * WN;

  const int tap = m0 / a.c, c0 = m0 - tap * a.c;
  const int tr = tap / a.s, ts = tap - tr * a.s;

  const __amdgpu_buffer_rsrc_t rs_x = __builtin_amdgcn_make_buffer_rsrc(
      (void *)a.x, 0, (int)((size_t)a.n * a.h * a.w * a.c * 2), kRsrcFlags);
  const __amdgpu_buffer_rsrc_t rs_dy = __builtin_amdgcn_make_buffer_rsrc(
      (void *)a.dy, 0, (int)((size_t)a.mtot * a.k * 2), kRsrcFlags);

  // this lane's two reduction rows per stage: m = mbeg + 32*st + krow
  const MnSlot sl = mn_slots(wave, lane);
  int qn[2], qp[2], qq[2];  // (n, p, q) of the row at the current stage
#pragma unroll
  for (int jj = 0; jj < 2; ++jj) {
    int m = mbeg + sl.krow[jj];
    qn[jj] = m / (a.p * a.q);
    int rem = m - qn[jj] * a.p * a.q;
    qp[jj] = rem / a.q;
    qq[jj] = rem - qp[jj] * a.q;
  }
  int next_st = 0;  // stage the (n, p, q) above belong to

  auto issue = [&](int st, int slot) {
    // advance the row decode to stage st (stages are issued in order)
    while (next_st < st) {
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        qq[jj] += BK;
        while (qq[jj] >= a.q) {
          qq[jj] -= a.q;
          if (++qp[jj] == a.p) {
            qp[jj] = 0;
            ++qn[jj];
          }
        }
      }
      ++next_st;
    }
    uint8_t *ta = R.a[slot], *tb = R.b[slot];
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
      const int m = mbeg + st * BK + sl.krow[jj];
      const bool mv = m < mend;
      const int hh = qp[jj] * a.sh - a.ph + tr, ww = qq[jj] * a.sw - a.pw + ts;
      const bool v = mv && hh >= 0 && hh < a.h && ww >= 0 && ww < a.w;
      unsigned ox = v ? (unsigned)((((qn[jj] * a.h + hh) * a.w + ww) * a.c) + c0 +
                                   sl.ncol[jj]) * 2u
                      : kOOB;
      dma16(rs_x, ta + mn_dst(wave, jj), ox);
      unsigned od = mv ? (unsigned)(m * a.k + n0 + sl.ncol[jj]) * 2u : kOOB;
      dma16(rs_dy, tb + mn_dst(wave, jj), od);
    }
  };

  f32x16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  pipeline<false, false>(acc, R, nst, wm0, wn0, lane, issue);

#pragma unroll
  for (int j = 0; j < FN; ++j) {
    int k = n0 + wn0 + j * 32 + (lane & 31);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        int rho = m0 + wm0 + i * 32 + 8 * g + 4 * (lane >> 5);
        const f32x16 &c = acc[i][j];
        if (!SPLIT) {
          *reinterpret_cast<u32x2 *>(a.dw + (size_t)k * rsc + rho) =
              to_h4(c[4 * g], c[4 * g + 1], c[4 * g + 2], c[4 * g + 3]);
        } else {
          f32x4 o = {c[4 * g], c[4 * g + 1], c[4 * g + 2], c[4 * g + 3]};
          *reinterpret_cast<f32x4 *>(
              a.part + ((size_t)split * a.k + k) * rsc + rho) = o;
        }
      }
  }
}

}  // namespace dma

// ---------------------------------------------------------------------------
bool data_dma_ok(const DataConvArgs &a) {
  return a.cr % dma::BK == 0 &&
         (size_t)a.n * a.hi * a.wi * a.cr * 2 < 0x7FFFFFFFull &&
         (size_t)a.wbytes < 0x7FFFFFFFull;
}

bool wgrad_dma_ok(const WgradArgs &a) {
  return a.c % dma::TM == 0 && a.k % dma::TN == 0 &&
         (size_t)a.n * a.h * a.w * a.c * 2 < 0x7FFFFFFFull &&
         (size_t)a.mtot * a.k * 2 < 0x7FFFFFFFull;
}

hipError_t launch_data_conv_dma(const DataConvArgs &a, bool w_kmajor,
                                hipStream_t st) {
  int maxpix = 0;
  for (int i = 0; i < a.nphase; ++i)
    maxpix = std::max(maxpix, a.n * a.ph[i].mh * a.ph[i].mw);
  dim3 grid((maxpix + dma::TN - 1) / dma::TN, (a.co + dma::TM - 1) / dma::TM,
            a.nphase * a.nsplit);
  const bool split = a.nsplit > 1;
  if (w_kmajor) {
    if (split)
      hipLaunchKernelGGL((dma::data_conv_dma_kernel<true, true>), grid,
                         dim3(dma::NT), 0, st, a);
    else
      hipLaunchKernelGGL((dma::data_conv_dma_kernel<true, false>), grid,
                         dim3(dma::NT), 0, st, a);
  } else {
    if (split)
      hipLaunchKernelGGL((dma::data_conv_dma_kernel<false, true>), grid,
                         dim3(dma::NT), 0, st, a);
    else
      hipLaunchKernelGGL((dma::data_conv_dma_kernel<false, false>), grid,
                         dim3(dma::NT), 0, st, a);
  }
  return hipGetLastError();
}

hipError_t launch_wgrad_dma(const WgradArgs &a, hipStream_t st) {
  const int rsc = a.r * a.s * a.c;
  dim3 grid(rsc / dma::TM, a.k / dma::TN, a.nsplit);
  if (a.nsplit > 1)
    hipLaunchKernelGGL((dma::wgrad_dma_kernel<true>), grid, dim3(dma::NT), 0, st,
                       a);
  else
    hipLaunchKernelGGL((dma::wgrad_dma_kernel<false>), grid, dim3(dma::NT), 0, st,
                       a);
  return hipGetLastError();
}

}  // namespace fg
