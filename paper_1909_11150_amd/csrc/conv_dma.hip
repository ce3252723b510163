// Implicit-GEMM convolutions fed by LDS DMA (gfx950 buffer_load ... lds).
//
// Same GEMM formulation as the register-staged kernels in conv_igemm.hip
// (data convolutions: rows = output channels, columns = output positions of
// one phase; kernel gradient: rows = (tap, input channel), columns = output
// channels), for 256 x 256 tiles. Operands go from global memory straight
// into LDS: no register staging and no LDS store instructions. A ring of NS
// reduction stages, each BK deep, holds 128 KiB, so a stage's loads are
// issued NS - 1 stages before they are consumed. Padding and ragged tails
// cost nothing: an out-of-range buffer offset returns zeros. The tile is
// split among WGM x WGN waves; stage depth, ring length and wave grid are
// template parameters (the configurations in use are named below).
//
// Two LDS tile layouts:
//   k-major  (row = GEMM row/column, BK reduction halves per row; 16-byte
//            chunk c stored at c ^ g(row)); MFMA operands are single 16-byte
//            reads of 32 consecutive rows.
//   mn-major (row = reduction index, 256 halves = 512 bytes per row; 64-byte
//            block b stored at b ^ (row & 3), or for the halo kernel's
//            weights 32-byte blocks as described at mn_xor); MFMA operands
//            are two transposing 8-byte reads (ds_read_b64_tr_b16).
// The permutations are chosen by measurement on gfx950, whose LDS has 64
// banks of 4 bytes: g(row) = (row >> 2) & 3 reads 32 consecutive 64-byte rows
// at full rate from any starting row (the previous ((row >> 1) ^ (row >> 3))
// & 3 ran at half rate), and the mn-major xor of (row & 3) * 64 bytes serves
// each half-wave of a transposing read without conflicts (xor of 32-byte
// blocks: two-way conflicts).
// The mn-major layout lets operands whose reduction index is strided in
// memory (input-gradient and transposed-conv weights, both kernel-gradient
// operands) be copied row by row as they lie in memory.
#include <algorithm>
#include <type_traits>

#include "common.h"
#include "internal.h"

namespace fg {
namespace dma {

constexpr int TM = 256, TN = 256;       // output tile of the large kernels
constexpr unsigned kOOB = 0x80000000u;   // beyond any tensor: loads zero

// Pipeline configuration: T x T output tile, BK-deep reduction stages, NS of
// them in the LDS ring, WGM x WGN waves each owning (T/WGM) x (T/WGN).
template <int BK_, int NS_, int WGM_, int WGN_, int T_ = 256>
struct K {
  static constexpr int BK = BK_, NS = NS_, WGM = WGM_, WGN = WGN_, T = T_;
  static constexpr int NW = WGM * WGN, NT = 64 * NW;
  static constexpr int WM = T / WGM, WN = T / WGN;
  static constexpr int FM = WM / 32, FN = WN / 32;
  static constexpr int KS = BK / 16;                 // MFMA steps per stage
  static constexpr int TILE_BYTES = T * BK * 2;      // per operand per stage
  static constexpr int NI = TILE_BYTES / 1024;       // DMA instrs per operand
  static constexpr int PW = NI / NW;                 // ... per wave
  static constexpr int CPR = BK / 8;                 // 16-byte chunks per row
  static constexpr int RB = 2 * T;                   // mn-major row bytes
  static constexpr int RPI = 1024 / RB;              // mn-major rows per DMA
  // waves per SIMD the kernel must fit (small tiles run two per CU)
  static constexpr int WPE = T == 128 ? 2 * NW / 4 : (NW + 3) / 4;
  static_assert(NI % NW == 0, "DMA instructions must divide among waves");
};
// The configurations the library runs, chosen by timing the network's layers:
// data convolutions take 32-deep stages in a 5-stage ring (160 KiB) with 8
// waves of 128 x 64; the kernel gradient 32-deep stages in a 4-stage ring
// (128 KiB) with 8 waves of 128 x 64.
#ifndef FG_DMA_DATA_CFG
#define FG_DMA_DATA_CFG 32, 5, 2, 4
#endif
#ifndef FG_DMA_WGRAD_CFG
#define FG_DMA_WGRAD_CFG 32, 4, 2, 4
#endif
using DataRun = K<FG_DMA_DATA_CFG>;
using WgradRun = K<FG_DMA_WGRAD_CFG>;
#ifndef FG_DMA_HALO_NS
#define FG_DMA_HALO_NS 3
#endif
using HaloRun = K<32, FG_DMA_HALO_NS, 2, 4>;  // weights ring; the rest is patches
// 128 x 128 tiles for layers with few output positions: 4 waves of 64 x 64,
// 80 KiB of ring, two workgroups per CU
using SmallRun = K<32, 5, 2, 2, 128>;
constexpr int kRsrcFlags = 0x00020000;   // raw buffer, 32-bit data format

typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s;
typedef __attribute__((address_space(3))) void lds_void;

// k-major: 16-byte chunk c of tile row `row` (bytes). 64-byte rows (BK 32)
// permute the 4 chunks by g(row); 128-byte rows (BK 64) the 8 chunks.
// mn-major: byte xor of reduction row k, below 256 so that rows of 256 bytes
// take it too. MX = 1: 64-byte blocks permuted by k & 3 (conflict-free
// transposing reads); MX = 0: 32-byte blocks permuted by (k & 3) | bit 3 of k
// (two-way conflicts), kept for the halo kernel's weights, whose register
// allocation spills into its main loop with the other permutation.
template <int BK>
__device__ __forceinline__ int kmaj_swz(int row) {
  return BK == 32 ? ((row >> 2) & 3) : ((row ^ (row >> 3)) & 7);
}
template <int BK>
__device__ __forceinline__ int kmaj_off(int row, int c) {
  return row * (2 * BK) + ((c ^ kmaj_swz<BK>(row)) << 4);
}
template <int MX>
__device__ __forceinline__ int mn_xor(int k) {
  return MX ? (k & 3) << 6 : ((k & 3) | (((k >> 3) & 1) << 2)) << 5;
}
template <int RB, int MX = 1>
__device__ __forceinline__ int mnmaj_off(int k, int n) {  // bytes, n % 4 == 0
  return k * RB + ((2 * n) ^ mn_xor<MX>(k));
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

// Tile order across the chip. Workgroups are handed to the 8 XCDs (each with
// its own L2) round-robin by launch index L; tile v = (L % 8) * per + L / 8
// gives each XCD a contiguous run of the tile sequence, in which neighbours
// share operands (the output channels of one column tile, the halo rows of
// adjacent column tiles, one reduction chunk), so they are fetched into that
// XCD's L2 once. The grid is 8 * per one-dimensional; indices past the tile
// count exit.
// With `linear`, tile v = L instead: launch order is tile order, for launches
// whose tiles differ in cost and are listed costliest first.
struct TileMap {
  int32_t n0, n1, n2;  // tile counts, fastest first
  int32_t per;         // ceil(n0 * n1 * n2 / 8)
  int32_t linear;
  __device__ __forceinline__ bool decode(int L, int &i0, int &i1, int &i2) const {
    const int v = linear ? L : (L & 7) * per + (L >> 3);
    if (v >= n0 * n1 * n2) return false;
    i0 = v % n0;
    const int r = v / n0;
    i1 = r % n1;
    i2 = r / n1;
    return true;
  }
};

// Unsigned division by a divisor fixed per launch, as a multiply-high and two
// shifts (Granlund and Montgomery, "Division by invariant integers using
// multiplication", 1994): exact for every 32-bit dividend.
struct FastDiv {
  uint32_t magic;
  int32_t s1, s2;
  __device__ __forceinline__ unsigned div(unsigned n) const {
    const unsigned t = __umulhi(magic, n);
    return (t + ((n - t) >> s1)) >> s2;
  }
};
struct WgradDiv {
  FastDiv pq, q;  // by p * q and by q
};

// MFMA operand of a 32-row block starting at `base` for reduction step ks.
template <int BK, bool KMAJOR, int RB = 512, int MX = 1>
__device__ __forceinline__ u32x4 frag(const uint8_t *tile, int base, int ks,
                                      int lane) {
  if (KMAJOR) {
    return *reinterpret_cast<const u32x4 *>(
        tile + kmaj_off<BK>(base + (lane & 31), 2 * ks + (lane >> 5)));
  } else {
    const int g = lane >> 4, m = lane & 15;
    const int k = 8 * (g >> 1) + (m >> 2) + 16 * ks;
    const int n = base + 16 * (g & 1) + 4 * (m & 3);
    v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_v4s *)(tile + mnmaj_off<RB, MX>(k, n)));
    v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_v4s *)(tile + mnmaj_off<RB, MX>(k + 4, n)));
    u32x2 a = __builtin_bit_cast(u32x2, lo), b = __builtin_bit_cast(u32x2, hi);
    return u32x4{a[0], a[1], b[0], b[1]};
  }
}

// Fragments of one 16-deep reduction step for this wave.
template <class C>
struct Frags {
  u32x4 a[C::FM], b[C::FN];
};

template <class C, bool AK, bool BKM>
__device__ __forceinline__ void load_frags(Frags<C> &f, const uint8_t *ta,
                                           const uint8_t *tb, int ks, int wm0,
                                           int wn0, int lane) {
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
    f.a[i] = frag<C::BK, AK, C::RB>(ta, wm0 + 32 * i, ks, lane);
#pragma unroll
  for (int j = 0; j < C::FN; ++j)
    f.b[j] = frag<C::BK, BKM, C::RB>(tb, wn0 + 32 * j, ks, lane);
}

template <class C>
__device__ __forceinline__ void mma(f32x16 (&acc)[C::FM][C::FN],
                                    const Frags<C> &f) {
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j) acc[i][j] = mfma32(f.a[i], f.b[j], acc[i][j]);
}

// s_waitcnt with only lgkmcnt (LDS) constrained to 0.
__device__ __forceinline__ void wait_lds() {
  __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));
}

// Position of this lane's DMA slots (one per wave instruction jj) in a
// k-major tile (row, reduction offset of the chunk) and in an mn-major tile
// (reduction row within the stage, tile column). Each instruction fills 1 KiB
// of LDS: 512/BK k-major rows or 1024/RB mn-major rows.
template <class C>
struct KmSlot {
  int row[C::PW], coff[C::PW];
};
template <class C>
struct MnSlot {
  int krow[C::PW], ncol[C::PW];
};

template <class C>
__device__ __forceinline__ KmSlot<C> km_slots(int wave, int lane) {
  KmSlot<C> s;
#pragma unroll
  for (int jj = 0; jj < C::PW; ++jj) {
    int row = (512 / C::BK) * (C::PW * wave + jj) + lane / C::CPR;
    int pc = lane % C::CPR;
    s.row[jj] = row;
    s.coff[jj] = 8 * (pc ^ kmaj_swz<C::BK>(row));
  }
  return s;
}

template <class C, int MX = 1>
__device__ __forceinline__ MnSlot<C> mn_slots(int wave, int lane) {
  MnSlot<C> s;
#pragma unroll
  for (int jj = 0; jj < C::PW; ++jj) {
    constexpr int CPM = C::RB / 16;  // 16-byte chunks per mn-major row
    int k = C::RPI * (C::PW * wave + jj) + lane / CPM;
    int p = lane % CPM;
    s.krow[jj] = k;
    s.ncol[jj] = ((16 * p) ^ mn_xor<MX>(k)) / 2;
  }
  return s;
}

// LDS destination (bytes, wave-uniform) of wave instruction jj of a stage.
template <class C>
__device__ __forceinline__ int dma_dst(int wave, int jj) {
  return 1024 * (C::PW * wave + jj);
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

// fp16(a + b) for 8 packed pairs (fp32 sum of two fp16 values, one rounding
// to fp16; the sum of two fp16 values is exact in fp32 unless it is far
// below the larger's last bit, where the rounding is the same)
__device__ __forceinline__ u32x4 add_h8(const u32x4 &a, const u32x4 &b) {
  u32x4 o;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float lo = h_to_f32((uint16_t)(a[w] & 0xFFFFu)) + h_to_f32((uint16_t)(b[w] & 0xFFFFu));
    const float hi = h_to_f32((uint16_t)(a[w] >> 16)) + h_to_f32((uint16_t)(b[w] >> 16));
    o[w] = (uint32_t)f32_to_h(lo) | ((uint32_t)f32_to_h(hi) << 16);
  }
  return o;
}

// The ring: stage s of operand X lives in its own LDS array so that the
// compiler can tell the stages apart when it places waits. Unused slots of a
// ring shorter than five stages are token-sized.
struct Ring {
  uint8_t *a[5];
  uint8_t *b[5];
};
#define FG_DMA_RING(C, R)                                                     \
  constexpr int T0_ = C::TILE_BYTES, T2_ = C::NS > 2 ? T0_ : 16,              \
                T3_ = C::NS > 3 ? T0_ : 16, T4_ = C::NS > 4 ? T0_ : 16;       \
  __shared__ __attribute__((aligned(1024))) uint8_t sA0[T0_], sA1[T0_],       \
      sA2[T2_], sA3[T3_], sA4[T4_];                                           \
  __shared__ __attribute__((aligned(1024))) uint8_t sB0[T0_], sB1[T0_],       \
      sB2[T2_], sB3[T3_], sB4[T4_];                                           \
  Ring R;                                                                     \
  R.a[0] = sA0, R.a[1] = sA1, R.a[2] = sA2, R.a[3] = sA3, R.a[4] = sA4;        \
  R.b[0] = sB0, R.b[1] = sB1, R.b[2] = sB2, R.b[3] = sB3, R.b[4] = sB4

// Wait until at most n stages of this wave's DMA loads remain outstanding
// (n <= 3; each stage is 2 * PW load instructions).
template <class C>
__device__ __forceinline__ void wait_stages(int n) {
  constexpr int PS = 2 * C::PW;
  static_assert(3 * PS < 64, "vmcnt range");
  if (n >= 3) wait_vm<3 * PS>();
  else if (n == 2) wait_vm<2 * PS>();
  else if (n == 1) wait_vm<PS>();
  else wait_vm<0>();
}

// Instruction-scheduling hints (LLVM AMDGPU IGroupLP): within the current
// scheduling region, place the MFMAs one by one and put `per` LDS reads
// after each of the first ones, so the reads of the next step issue among
// the MFMAs of this one instead of in a block.
template <int NMF, int NRD>
__device__ __forceinline__ void sched_mfma_reads() {
  constexpr int per = (NRD + NMF - 1) / NMF;
#pragma unroll
  for (int i = 0; i < NMF; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
    if (i * per < NRD) __builtin_amdgcn_sched_group_barrier(0x100, per, 0);  // DS read
  }
}
// After the barrier: reads first (they gate the next step), then the DMA
// loads of the refilled slot with their address arithmetic.
template <int NMF, int NRD, int NVM>
__device__ __forceinline__ void sched_mfma_reads_dma() {
  constexpr int per = (NRD + NMF / 2 - 1) / (NMF / 2);
#pragma unroll
  for (int i = 0; i < NMF / 2; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if (i * per < NRD) __builtin_amdgcn_sched_group_barrier(0x100, per, 0);
  }
  constexpr int pv = (NVM + NMF / 2 - 1) / (NMF / 2);
#pragma unroll
  for (int i = 0; i < NMF / 2; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if (i * pv < NVM) {
      __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);  // VALU
      __builtin_amdgcn_sched_group_barrier(0x020, pv, 0);  // VMEM read
    }
  }
}

// One stage (ring slot U) of the main loop. With `next`, the stage has a
// successor: the barrier that publishes it is crossed before the last step
// and the successor's first fragments are read into f[0]. `full` asserts
// that NS - 2 stages after the successor have been issued and that stage
// it + NS exists.
template <class C, bool AK, bool BKM, int U, class Issue>
__device__ __forceinline__ void stage(f32x16 (&acc)[C::FM][C::FN],
                                      Frags<C> (&f)[2], const Ring &R, int it,
                                      int nst, bool next, bool full, int wm0,
                                      int wn0, int lane, Issue &issue) {
  constexpr int NS = C::NS, KS = C::KS;
  constexpr int NMF = C::FM * C::FN;
  constexpr int NRD = C::FM * (AK ? 1 : 2) + C::FN * (BKM ? 1 : 2);
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    if (ks + 1 < KS)
      load_frags<C, AK, BKM>(f[(ks + 1) & 1], R.a[U], R.b[U], ks + 1, wm0, wn0,
                             lane);
    mma<C>(acc, f[ks & 1]);
    if (ks + 1 < KS) sched_mfma_reads<NMF, NRD>();
    __builtin_amdgcn_s_setprio(0);
    if (ks == KS - 2 && next) {
      // own DMA of stage it+1 done: later stages may remain in flight
      wait_stages<C>(full ? NS - 2 : min(NS - 2, nst - 2 - it));
      wait_lds();  // this wave's reads of slot U are complete
      barrier_nofence();
      // Past the barrier a wave has memory work to start (the refill DMA,
      // the next stage's first fragments) before its next MFMAs: raise its
      // issue priority over the other wave on its SIMD until those MFMAs
      // are issued, so the loads go out early. The priority drops back to 0
      // after every MFMA block. (Measured: 1-4% per layer.)
      __builtin_amdgcn_s_setprio(2);
      if (full || it + NS < nst) issue(it + NS, U);
      load_frags<C, AK, BKM>(f[0], R.a[(U + 1) % NS], R.b[(U + 1) % NS], 0, wm0,
                             wn0, lane);
    }
  }
  if (next) sched_mfma_reads_dma<NMF, NRD, 2 * C::PW>();
}

template <class C, bool AK, bool BKM, int U, class Issue>
__device__ __forceinline__ void group(f32x16 (&acc)[C::FM][C::FN],
                                      Frags<C> (&f)[2], const Ring &R, int it0,
                                      int nst, bool tail, int wm0, int wn0,
                                      int lane, Issue &issue) {
  if constexpr (U < C::NS) {
    const int it = it0 + U;
    if (!tail) {
      stage<C, AK, BKM, U>(acc, f, R, it, nst, true, true, wm0, wn0, lane, issue);
    } else if (it < nst) {
      stage<C, AK, BKM, U>(acc, f, R, it, nst, it + 1 < nst, false, wm0, wn0,
                           lane, issue);
    }
    group<C, AK, BKM, U + 1>(acc, f, R, it0, nst, tail, wm0, wn0, lane, issue);
  }
}

// Runs the pipelined main loop over stages [0, nst): issue(st, slot) issues
// this wave's DMA loads of stage st into ring slot `slot`; stages are issued
// strictly in order. Full groups of NS stages run in a loop whose body has no
// data-dependent control flow around the MFMAs (so the compiler's own LDS
// waits stay exact and its scheduling regions span whole steps); the last
// groups run with per-stage checks.
template <class C, bool AK, bool BKM, class Issue>
__device__ __forceinline__ void pipeline(f32x16 (&acc)[C::FM][C::FN],
                                         const Ring &R, int nst, int wm0,
                                         int wn0, int lane, Issue &&issue) {
  constexpr int NS = C::NS, KS = C::KS;
  static_assert(NS >= 2 && NS <= 5 && KS >= 2 && KS % 2 == 0, "pipeline shape");
  if (nst <= 0) return;
#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    if (s < nst) issue(s, s);
  wait_stages<C>(min(NS - 2, nst - 1));  // publish stage 0
  barrier_nofence();
  if (NS - 1 < nst) issue(NS - 1, NS - 1);
  Frags<C> f[2];
  load_frags<C, AK, BKM>(f[0], R.a[0], R.b[0], 0, wm0, wn0, lane);
  // In a full group every stage has a successor, NS - 2 stages issued after
  // it, and a stage NS ahead to issue, so its waits and issues need no
  // checks: it0 + 2 NS - 1 < nst.
  int it0 = 0;
  for (; it0 + 2 * NS - 1 < nst; it0 += NS)
    group<C, AK, BKM, 0>(acc, f, R, it0, nst, false, wm0, wn0, lane, issue);
  for (; it0 < nst; it0 += NS)
    group<C, AK, BKM, 0>(acc, f, R, it0, nst, true, wm0, wn0, lane, issue);
}

template <class C>
__device__ __forceinline__ void zero(f32x16 (&acc)[C::FM][C::FN]) {
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
}

// ---------------------------------------------------------------------------
// Output tile store of the data convolutions. The accumulator layout gives
// each lane 4 consecutive channels of one output position per register
// group, so storing it directly would scatter 8-byte pieces over 32
// positions per instruction. Instead each wave stages its 128-channel x
// 64-position block in LDS (the ring is free once the last stage is read),
// position-major with 16-byte chunks permuted by the position, and reads it
// back so that 16 lanes cover one position's 256 contiguous bytes: stores
// (and, for the gate epilogue, the gate loads) are whole 128-byte lines.
// fp32 partials (SPLIT) go in two passes of 64 channels.
// `buf` is this wave's 16 KiB of staging LDS and `pos` its 64-entry table;
// the caller guarantees that no wave still reads, and no DMA still writes,
// the LDS they alias (the store begins with a workgroup barrier).
template <class C, bool SPLIT>
__device__ __forceinline__ void store_tile(f32x16 (&acc)[C::FM][C::FN],
                                           uint8_t *buf, int32_t *pos,
                                           const DataConvArgs &a,
                                           const Phase &P, int npix, int n0,
                                           int m0, int wm0, int wn0, int lane,
                                           int split) {
  static_assert(C::WM == 128 && C::WN == 64, "store_tile expects 128 x 64 waves");
  __syncthreads();
  if (lane < 32) {
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
      const int col = n0 + wn0 + j * 32 + lane;
      int32_t ob = -1;
      if (col < npix) {
        const int b = col % P.mw, t = col / P.mw;
        const int aa = t % P.mh, nn = t / P.mh;
        // split partials are dense; the output has its own pixel stride
        ob = ((nn * a.ho + aa * a.ostr + P.ooh) * a.wo + b * a.ostr + P.oow) *
             (SPLIT ? a.co : a.ldo);
      }
      pos[j * 32 + lane] = ob;
    }
  }
  const size_t out_total = (size_t)a.n * a.ho * a.wo * a.co;
  const int cw = m0 + wm0;  // first channel of this wave's block
  constexpr int PASSES = SPLIT ? 2 : 1;
#pragma unroll
  for (int pass = 0; pass < PASSES; ++pass) {
    // acc -> LDS: position p = j*32 + lane%32, 4 channels per register group
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
      const int p = j * 32 + (lane & 31);
      uint8_t *row = buf + p * 256;
#pragma unroll
      for (int ii = 0; ii < C::FM / PASSES; ++ii) {
        const int i = pass * (C::FM / PASSES) + ii;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * g + e];
          if (SPLIT) {
            const int chunk = 8 * ii + 2 * g + (lane >> 5);
            *reinterpret_cast<f32x4 *>(row + ((chunk ^ (p & 15)) << 4)) =
                f32x4{v[0], v[1], v[2], v[3]};
          } else {
            if (a.epi == FG_EPI_RELU) {
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] = v[e] > 0.f ? v[e] : 0.f;
            }
            const int chunk = 4 * i + g;
            *reinterpret_cast<u32x2 *>(row + ((chunk ^ (p & 15)) << 4) +
                                       8 * (lane >> 5)) =
                to_h4(v[0], v[1], v[2], v[3]);
          }
        }
      }
    }
    wait_lds();
    __builtin_amdgcn_wave_barrier();
    // LDS -> global: 16 lanes per position, 16-byte chunk q of its row.
    // All reads (and gate loads) are issued before any use, so their
    // latencies overlap; gate loads of absent positions read element 0.
    const int q = lane & 15;
    const int ch = SPLIT ? pass * 64 + 4 * q : 8 * q;  // channel within block
    const bool chok = cw + ch < a.co;
    u32x4 d[16];
    int32_t ob[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const int p = 4 * k + (lane >> 4);
      d[k] = *reinterpret_cast<const u32x4 *>(buf + p * 256 + ((q ^ (p & 15)) << 4));
      ob[k] = chok ? pos[p] : -1;
    }
    if (!SPLIT && a.epi == FG_EPI_GATE) {
      u32x4 gw[16];
#pragma unroll
      for (int k = 0; k < 16; ++k)
        gw[k] = *reinterpret_cast<const u32x4 *>(a.gate + (ob[k] < 0 ? 0 : ob[k] + cw + ch));
#pragma unroll
      for (int k = 0; k < 16; ++k)
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const uint32_t lo = h_to_f32((uint16_t)(gw[k][w] & 0xFFFFu)) > 0.f
                                  ? 0x0000FFFFu : 0u;
          const uint32_t hi = h_to_f32((uint16_t)(gw[k][w] >> 16)) > 0.f
                                  ? 0xFFFF0000u : 0u;
          d[k][w] &= lo | hi;
        }
    }
    if (!SPLIT && a.epi == FG_EPI_ACC) {  // add what the output holds
      u32x4 ow[16];
#pragma unroll
      for (int k = 0; k < 16; ++k)
        ow[k] = *reinterpret_cast<const u32x4 *>(a.out + (ob[k] < 0 ? 0 : ob[k] + cw + ch));
#pragma unroll
      for (int k = 0; k < 16; ++k) d[k] = add_h8(d[k], ow[k]);
    }
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      if (ob[k] < 0) continue;
      if (SPLIT)
        *reinterpret_cast<u32x4 *>(a.part + (size_t)split * out_total + ob[k] + cw +
                                   ch) = d[k];
      else
        *reinterpret_cast<u32x4 *>(a.out + ob[k] + cw + ch) = d[k];
    }
    if (pass + 1 < PASSES) {
      wait_lds();
      __builtin_amdgcn_wave_barrier();
    }
  }
}

// Direct store of the accumulators (small tiles, whose ring has no room to
// stage a wave's block): 8-byte pieces of 4 channels per lane.
template <class C, bool SPLIT>
__device__ __forceinline__ void store_direct(f32x16 (&acc)[C::FM][C::FN],
                                             const DataConvArgs &a, const Phase &P,
                                             int npix, int n0, int m0, int wm0,
                                             int wn0, int lane, int split) {
  const size_t out_total = (size_t)a.n * a.ho * a.wo * a.co;
#pragma unroll
  for (int j = 0; j < C::FN; ++j) {
    const int col = n0 + wn0 + j * 32 + (lane & 31);
    if (col >= npix) continue;
    const int b = col % P.mw, t = col / P.mw;
    const int aa = t % P.mh, nn = t / P.mh;
    const size_t obase =
        ((size_t)(nn * a.ho + aa * a.ostr + P.ooh) * a.wo + b * a.ostr + P.oow) *
        (SPLIT ? a.co : a.ldo);
#pragma unroll
    for (int i = 0; i < C::FM; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int co = m0 + wm0 + i * 32 + 8 * g + 4 * (lane >> 5);
        if (co >= a.co) continue;
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * g + e];
        if (SPLIT) {
          *reinterpret_cast<f32x4 *>(a.part + split * out_total + obase + co) =
              f32x4{v[0], v[1], v[2], v[3]};
        } else {
          epilogue4(v, a.epi, a.gate + obase + co, a.out + obase + co);
          *reinterpret_cast<u32x2 *>(a.out + obase + co) =
              to_h4(v[0], v[1], v[2], v[3]);
        }
      }
  }
}

// ---------------------------------------------------------------------------
// Data convolution (forward / input gradient / transposed forward).
// Requires reduction channels cr % BK == 0 (a stage lies in one tap).
template <class C, bool WK, bool SPLIT>
__global__ __launch_bounds__(C::NT, C::WPE) void data_conv_dma_kernel(DataConvArgs a,
                                                              TileMap tm) {
  FG_DMA_RING(C, R);
  constexpr int PW = C::PW;

  int tz, ty, tx;  // phase x split, output-channel tile, position tile
  if (tm.linear ? !tm.decode(blockIdx.x, tx, ty, tz)
                : !tm.decode(blockIdx.x, tz, ty, tx))
    return;
  const int phase = tz / a.nsplit, split = tz % a.nsplit;
  const Phase P = a.ph[phase];
  const int npix = a.n * P.mh * P.mw;
  const int n0 = tx * C::T;
  const int m0 = ty * C::T;
  if (n0 >= npix) return;
  const int ktot = P.nr * P.ns * a.cr;
  const int nk = ktot / C::BK;
  const int kchunk = (nk + a.nsplit - 1) / a.nsplit;
  const int kbeg = min(nk, split * kchunk), kend = min(nk, kbeg + kchunk);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm0 = (wave / C::WGN) * C::WM, wn0 = (wave % C::WGN) * C::WN;

  const __amdgpu_buffer_rsrc_t rs_act = __builtin_amdgcn_make_buffer_rsrc(
      (void *)a.act, 0, (int)act_span_bytes(a), kRsrcFlags);
  const __amdgpu_buffer_rsrc_t rs_w = __builtin_amdgcn_make_buffer_rsrc(
      (void *)a.wgt, 0, a.wbytes, kRsrcFlags);

  // B: this lane's output positions (image row/column of tap (0, 0) of the
  // phase) and element offsets
  const KmSlot<C> bs = km_slots<C>(wave, lane);
  int bh[PW], bw[PW], bbase[PW];
#pragma unroll
  for (int jj = 0; jj < PW; ++jj) {
    int col = n0 + bs.row[jj];
    if (col < npix) {
      int b = col % P.mw, t = col / P.mw;
      int aa = t % P.mh, nn = t / P.mh;
      bh[jj] = aa * a.istr;
      bw[jj] = b * a.istr;
      bbase[jj] = ((nn * a.hi + bh[jj]) * a.wi + bw[jj]) * a.ldi + bs.coff[jj];
    } else {
      bh[jj] = -(1 << 29);  // never inside the image
      bw[jj] = 0;
      bbase[jj] = 0;
    }
  }
  // A: this lane's weight offsets without the stage part, and whether its
  // output channel exists
  int wbase[PW];
  bool wok[PW];
#pragma unroll
  for (int jj = 0; jj < PW; ++jj) {
    if (WK) {
      const KmSlot<C> as = km_slots<C>(wave, lane);
      const int co = m0 + as.row[jj];
      wok[jj] = co < a.co;
      wbase[jj] = co * a.ldw + as.coff[jj];
    } else {
      const MnSlot<C> as = mn_slots<C>(wave, lane);
      const int co = m0 + as.ncol[jj];
      wok[jj] = co < a.co;
      wbase[jj] = as.krow[jj] * a.w_red + co;
    }
  }

  // Stage decode (uniform), advanced by one stage per issue() call: the
  // pipeline issues stages strictly in order. Stage st covers reduction
  // offsets [k0, k0 + BK) of tap t = k0 / cr, t = ti * ns + tj.
  int cr0, ti, tj;
  {
    const int k0 = kbeg * C::BK, t = k0 / a.cr;
    cr0 = k0 - t * a.cr;
    ti = t / P.ns;
    tj = t - ti * P.ns;
  }
  auto issue = [&](int, int slot) __attribute__((always_inline)) {
    const int dh = P.dh0 + P.dstep * ti, dw = P.dw0 + P.dstep * tj;
    const int woff = (P.r0 + P.rstep * ti) * a.s + (P.s0 + P.rstep * tj);
    const int delta = (dh * a.wi + dw) * a.ldi + cr0;
    const int wst = WK ? woff * a.cr + cr0 : cr0 * a.w_red + woff * a.w_tap;
    uint8_t *ta = R.a[slot], *tb = R.b[slot];
#pragma unroll
    for (int jj = 0; jj < PW; ++jj) {
      const bool v = (unsigned)(bh[jj] + dh) < (unsigned)a.hi &&
                     (unsigned)(bw[jj] + dw) < (unsigned)a.wi;
      const unsigned o = (unsigned)(bbase[jj] + delta) * 2u;
      dma16(rs_act, tb + dma_dst<C>(wave, jj), v ? o : kOOB);
    }
#pragma unroll
    for (int jj = 0; jj < PW; ++jj) {
      const unsigned o = (unsigned)(wbase[jj] + wst) * 2u;
      dma16(rs_w, ta + dma_dst<C>(wave, jj), wok[jj] ? o : kOOB);
    }
    // next stage, without branches (keeps the scheduling region whole)
    cr0 += C::BK;
    const bool wrap = cr0 == a.cr;
    cr0 = wrap ? 0 : cr0;
    tj += wrap;
    const bool wrap2 = tj == P.ns;
    tj = wrap2 ? 0 : tj;
    ti += wrap2;
  };

  f32x16 acc[C::FM][C::FN];
  zero<C>(acc);
  pipeline<C, WK, true>(acc, R, kend - kbeg, wm0, wn0, lane, issue);

  if constexpr (C::WM == 128 && C::WN == 64) {
    // staging: ring array `wave` (a-side arrays first, constant indices
    // only) and the position tables in the next one
    static_assert(2 * C::NS >= C::NW + 1 && C::TILE_BYTES >= 16384,
                  "the store needs one 16 KiB ring array per wave plus one");
    uint8_t *sbuf = R.a[0];
#pragma unroll
    for (int k = 1; k < C::NW; ++k)
      if (wave == k) sbuf = k < C::NS ? R.a[k] : R.b[k - C::NS];
    int32_t *spos = reinterpret_cast<int32_t *>(R.b[C::NW - C::NS]) + 64 * wave;
    store_tile<C, SPLIT>(acc, sbuf, spos, a, P, npix, n0, m0, wm0, wn0, lane, split);
  } else {
    store_direct<C, SPLIT>(acc, a, P, npix, n0, m0, wm0, wn0, lane, split);
  }
}

// ---------------------------------------------------------------------------
// Data convolution with input reuse ("halo" tiles): stride-1 3x3 convolutions
// (forward, and input gradient, which is one phase whose taps walk the input
// backward) whose 256-position
// tile is a block of whole output rows of one image. Instead of gathering the
// activation operand once per tap (9 times), the tile's input window, with a
// one-pixel halo, is loaded into LDS once per 32-channel chunk as a "patch"
// of (rows + 2) x (width + 2) positions; the 9 taps read shifted views of it.
// The reduction runs channel chunk by chunk, taps inside: stage s = 9 c + t.
// Weights take a 3-stage ring of 32-deep stages; the patch two slots, the
// next chunk's patch being loaded during the current chunk. Every stage
// issues the same number of loads (stages and patches past the end load
// nothing, through the out-of-range offset), so all waits are constants. The
// next chunk's patch is loaded a block per stage, spread over the chunk.
constexpr int kHaloTaps = 9;

// f(integral_constant<int, U>) for U = B .. E-1, unrolled at compile time.
template <int B, int E, class F>
__device__ __forceinline__ void unroll(F &f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    unroll<B + 1, E>(f);
  }
}
constexpr int kPatchRows = 768;                  // capacity, rows of 64 bytes
constexpr int kPatchBytes = kPatchRows * 64;

template <class C>
__device__ __forceinline__ u32x4 frag_row(const uint8_t *tile, int row, int ks,
                                          int lane) {
  return *reinterpret_cast<const u32x4 *>(
      tile + kmaj_off<32>(row, 2 * ks + (lane >> 5)));
}

// Loads in flight after stage s+1's loads, at the barrier inside stage s
// (position u of the unrolled group). The barrier of stage b issues weight
// stage b + NS and then, when its tap t(b) < NPW, this wave's patch block
// t(b) of the next chunk; stage s+1's weights were issued at the barrier of
// stage s+1-NS. (Stages before the first have taps 9-NS+1 .. 8 >= NPW, so
// the prologue needs no stand-ins.)
template <class C, int NPW>
__device__ __forceinline__ constexpr int halo_flight(int u) {
  int f = (C::NS - 2) * C::PW;
  for (int b = 1; b <= C::NS - 1; ++b)
    f += ((u - b) % kHaloTaps + kHaloTaps) % kHaloTaps < NPW ? 1 : 0;
  return f;
}

template <class C, bool WK, bool SPLIT>
__global__ __launch_bounds__(C::NT) void data_conv_halo_kernel(DataConvArgs a,
                                                               TileMap tm) {
  static_assert(C::BK == 32 && (C::NS == 3 || C::NS == 4) && C::KS == 2,
                "halo pipeline shape");
  static_assert(C::WM == 128 && C::WN == 64 && C::NW == 8, "halo wave layout");
  constexpr int NS = C::NS, PW = C::PW;
  constexpr int NPW = kPatchRows / 16 / C::NW;  // patch loads per wave
  // stages per unrolled group: whole pairs of chunks (both patch slots) and
  // whole turns of the weight ring
  constexpr int UNR = NS == 3 ? 2 * kHaloTaps : 4 * kHaloTaps;
  constexpr int TA3 = NS > 3 ? C::TILE_BYTES : 16;
  __shared__ __attribute__((aligned(1024))) uint8_t sA0[C::TILE_BYTES],
      sA1[C::TILE_BYTES], sA2[C::TILE_BYTES], sA3[TA3];
  __shared__ __attribute__((aligned(1024))) uint8_t sP0[kPatchBytes],
      sP1[kPatchBytes];
  uint8_t *ringA[4];
  ringA[0] = sA0, ringA[1] = sA1, ringA[2] = sA2, ringA[3] = sA3;
  uint8_t *patch[2];
  patch[0] = sP0, patch[1] = sP1;

  int split, ty, tx;  // reduction split, output-channel tile, position tile
  if (!tm.decode(blockIdx.x, split, ty, tx)) return;
  const Phase P = a.ph[0];
  const int n0 = tx * TN, m0 = ty * TM;
  const int nchunk = a.cr / 32;
  const int cps = (nchunk + a.nsplit - 1) / a.nsplit;
  const int cbeg = min(nchunk, split * cps), cend = min(nchunk, cbeg + cps);
  const int nst = kHaloTaps * (cend - cbeg);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm0 = (wave / C::WGN) * C::WM, wn0 = (wave % C::WGN) * C::WN;

  const __amdgpu_buffer_rsrc_t rs_act = __builtin_amdgcn_make_buffer_rsrc(
      (void *)a.act, 0, (int)act_span_bytes(a), kRsrcFlags);
  const __amdgpu_buffer_rsrc_t rs_w = __builtin_amdgcn_make_buffer_rsrc(
      (void *)a.wgt, 0, a.wbytes, kRsrcFlags);

  // tile geometry: rows [aa0, aa0 + 256 / mw) of image img
  const int mw = P.mw, pwid = mw + 2;
  const int img = n0 / (P.mh * mw), aa0 = (n0 / mw) % P.mh;
  const int prows = (TN / mw + 2) * pwid;
  // window origin: the taps walk the input forward (dstep 1, forward pass)
  // or backward (dstep -1, input gradient)
  const int dsg = P.dstep, back = dsg < 0 ? 2 : 0;
  const int h0 = aa0 + P.dh0 - back, w0 = P.dw0 - back;
  // patch loads of this lane: row r, 16-byte chunk (lane & 3) ^ g(r); byte
  // offset of channel 0 of its input position, or -1 outside the image
  int pbase[NPW];
#pragma unroll
  for (int jj = 0; jj < NPW; ++jj) {
    const int r = 16 * (NPW * wave + jj) + (lane >> 2);
    const int h = h0 + r / pwid, w = w0 + r % pwid;
    const bool v = r < prows && (unsigned)h < (unsigned)a.hi &&
                   (unsigned)w < (unsigned)a.wi;
    pbase[jj] = v ? (((img * a.hi + h) * a.wi + w) * a.ldi +
                     8 * ((lane & 3) ^ kmaj_swz<32>(r))) * 2
                  : -1;
  }
  // B fragment rows (patch row of tap (0, 0)) of this lane's positions
  int brow[C::FN];
#pragma unroll
  for (int j = 0; j < C::FN; ++j) {
    const int i = wn0 + 32 * j + (lane & 31);
    brow[j] = (i / mw) * pwid + i % mw;
  }
  // A: weight offsets without the stage part
  int wbase[PW];
  bool wok[PW];
#pragma unroll
  for (int jj = 0; jj < PW; ++jj) {
    if (WK) {
      const KmSlot<C> as = km_slots<C>(wave, lane);
      const int co = m0 + as.row[jj];
      wok[jj] = co < a.co;
      wbase[jj] = co * a.ldw + as.coff[jj];
    } else {
      const MnSlot<C> as = mn_slots<C, 0>(wave, lane);
      const int co = m0 + as.ncol[jj];
      wok[jj] = co < a.co;
      wbase[jj] = as.krow[jj] * a.w_red + co;
    }
  }
  // weight stage decode, advanced by one stage per issue (in order)
  int ic = cbeg, it_ = 0;
  auto issue_w = [&](int slot) __attribute__((always_inline)) {
    const int ti = it_ / 3, tj = it_ - 3 * ti;
    const int woff = (P.r0 + P.rstep * ti) * a.s + (P.s0 + P.rstep * tj);
    const int cr0 = 32 * ic;
    const int wst = WK ? woff * a.cr + cr0 : cr0 * a.w_red + woff * a.w_tap;
    const bool live = ic < cend;
#pragma unroll
    for (int jj = 0; jj < PW; ++jj) {
      const unsigned o = (unsigned)(wbase[jj] + wst) * 2u;
      dma16(rs_w, ringA[slot] + dma_dst<C>(wave, jj), live && wok[jj] ? o : kOOB);
    }
    const bool wrap = ++it_ == kHaloTaps;
    it_ = wrap ? 0 : it_;
    ic += wrap;
  };
  // block jj of this wave's share of chunk c's patch
  auto issue_pb = [&](int pslot, int c, int jj) __attribute__((always_inline)) {
    const unsigned o = (unsigned)(pbase[jj] + 64 * c);
    dma16(rs_act, patch[pslot] + 1024 * (NPW * wave + jj),
          c < cend && pbase[jj] >= 0 ? o : kOOB);
  };

  f32x16 acc[C::FM][C::FN];
  zero<C>(acc);
  Frags<C> f[2];
  auto load = [&](Frags<C> &fr, int slot, int pslot, int t, int ks) __attribute__((always_inline)) {
    const int toff = back * (pwid + 1) + dsg * ((t / 3) * pwid + t % 3);
#pragma unroll
    for (int i = 0; i < C::FM; ++i)
      fr.a[i] = frag<32, WK, 512, 0>(ringA[slot], wm0 + 32 * i, ks, lane);
#pragma unroll
    for (int j = 0; j < C::FN; ++j)
      fr.b[j] = frag_row<C>(patch[pslot], brow[j] + toff, ks, lane);
  };
  constexpr int NMF = C::FM * C::FN;
  constexpr int NRD = C::FM * (WK ? 1 : 2) + C::FN;

  // One stage at position U of the unrolled pair of chunks: A slot U % 3,
  // patch slot U / 9, tap U % 9.
  auto stage = [&](auto Uc, int it) __attribute__((always_inline)) {
    constexpr int U = decltype(Uc)::value;
    constexpr int T = U % kHaloTaps, SLOT = U % NS, PS = (U / kHaloTaps) & 1;
    constexpr int U1 = (U + 1) % UNR;
    // The patch row of a fragment depends on the tap; keep the compiler
    // from precomputing all taps' addresses across the unrolled stages.
#pragma unroll
    for (int j = 0; j < C::FN; ++j) asm volatile("" : "+v"(brow[j]));
    load(f[1], SLOT, PS, T, 1);
    mma<C>(acc, f[0]);
    sched_mfma_reads<NMF, NRD>();
    __builtin_amdgcn_s_setprio(0);
    wait_vm<halo_flight<C, NPW>(U)>();
    wait_lds();
    barrier_nofence();
    __builtin_amdgcn_s_setprio(2);  // as in stage(): loads first past the barrier
    issue_w(SLOT);  // stage it + NS
    // the next chunk's patch, one block per stage over its first NPW taps
    // (its slot's previous chunk is done: every wave is past this barrier)
    if (T < NPW) issue_pb(PS ^ 1, cbeg + it / kHaloTaps + 1, T);
    load(f[0], U1 % NS, (U1 / kHaloTaps) & 1, U1 % kHaloTaps, 0);
    mma<C>(acc, f[1]);
    sched_mfma_reads_dma<NMF, NRD, (T < NPW ? PW + 1 : PW)>();
    __builtin_amdgcn_s_setprio(0);
  };

  static_assert(NPW <= kHaloTaps - (NS - 1), "patch blocks fit the taps");
  // prologue: patch of the first chunk, weight stages 0 .. NS-2; publish
  // stage 0; weight stage NS-1
#pragma unroll
  for (int jj = 0; jj < NPW; ++jj) issue_pb(0, cbeg, jj);
#pragma unroll
  for (int st = 0; st < NS - 1; ++st) issue_w(st);
  wait_vm<(NS - 2) * PW>();
  barrier_nofence();
  issue_w(NS - 1);
  load(f[0], 0, 0, 0, 0);
  int it0 = 0;
  auto step = [&](auto Uc) __attribute__((always_inline)) { stage(Uc, it0 + decltype(Uc)::value); };
  for (; it0 + UNR <= nst; it0 += UNR) unroll<0, UNR>(step);
  // the rest, a whole number of chunks, as a prefix of a group
  constexpr int G9 = kHaloTaps;
  if (it0 + G9 <= nst) unroll<0, G9>(step);
  if constexpr (UNR > 2 * G9) {
    if (it0 + 2 * G9 <= nst) unroll<G9, 2 * G9>(step);
    if (it0 + 3 * G9 <= nst) unroll<2 * G9, 3 * G9>(step);
  }
  wait_vm<0>();  // loads issued past the end have landed

  // staging for the store: A slots, then 16 KiB pieces of the patch slots;
  // position tables after them
  uint8_t *sbuf = sA0;
  if (wave == 1) sbuf = sA1;
  if (wave == 2) sbuf = sA2;
  if (wave >= 3 && wave < 6) sbuf = sP0 + 16384 * (wave - 3);  // (sA3 unused)
  if (wave >= 6) sbuf = sP1 + 16384 * (wave - 6);
  int32_t *spos = reinterpret_cast<int32_t *>(sP1 + 32768) + 64 * wave;
  const int npix = a.n * P.mh * P.mw;
  store_tile<C, SPLIT>(acc, sbuf, spos, a, P, npix, n0, m0, wm0, wn0, lane, split);
}

// ---------------------------------------------------------------------------
// Output tile store of the kernel gradient: rows rho (contiguous in memory
// for a fixed output channel k), columns k. As for the data convolutions, a
// wave's block is staged in LDS k-major, 64 rows of rho at a time (128-byte
// rows: 64 fp16 or, per pass, 32 fp32 values; 16-byte chunks permuted by the
// row), and read back so that 8 lanes write one row's contiguous 128 bytes.
// Waves 64 rows high stage 8 KiB (two per 16 KiB ring array), waves 128 rows
// high two halves of 8 KiB in a ring array of their own.
template <class C, bool SPLIT>
__device__ __forceinline__ void store_tile_w(f32x16 (&acc)[C::FM][C::FN],
                                             const Ring &R, const WgradArgs &a,
                                             int rsc, int rho0, int k0, int lane,
                                             int wave, int split) {
  static_assert((C::WM == 64 || C::WM == 128) && C::WN == 64,
                "store_tile_w expects waves 64 wide and 64 or 128 high");
  constexpr int HM = C::WM / 64;   // 64-row halves of the wave's block
  constexpr int WPA = 2 / HM;      // waves per 16 KiB ring array
  // the ring arrays 0..NW/WPA-1 (a[0..NS-1], then b[0..]) must exist and be
  // 16 KiB each
  static_assert(C::TILE_BYTES == 16384 && C::NW / WPA <= 2 * C::NS,
                "store_tile_w stages in 16 KiB ring arrays");
  __syncthreads();  // every wave is done reading the ring
  uint8_t *buf = R.a[0];
#pragma unroll
  for (int k = 1; k < C::NW / WPA; ++k)
    if (wave / WPA == k) buf = k < C::NS ? R.a[k] : R.b[k - C::NS];
  if (HM == 1) buf += (wave & 1) * 8192;
  constexpr int PASSES = SPLIT ? 2 : 1;
  bool bad = false;  // an fp16 result is +-inf or NaN
#pragma unroll
  for (int h = 0; h < HM; ++h) {
    uint8_t *hb = buf + h * 8192;
#pragma unroll
    for (int pass = 0; pass < PASSES; ++pass) {
#pragma unroll
      for (int j = 0; j < C::FN; ++j) {
        const int kr = j * 32 + (lane & 31);  // row within the block
        uint8_t *row = hb + kr * 128;
        const int sw = (kr >> 1) & 7;
#pragma unroll
        for (int ii = 0; ii < 2 / PASSES; ++ii) {
          const int il = pass * (2 / PASSES) + ii;  // fragment within the half
          const f32x16 &c = acc[2 * h + il][j];
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            if (SPLIT) {
              const int chunk = 2 * g + (lane >> 5);
              *reinterpret_cast<f32x4 *>(row + ((chunk ^ sw) << 4)) =
                  f32x4{c[4 * g], c[4 * g + 1], c[4 * g + 2], c[4 * g + 3]};
            } else {
              const int chunk = 4 * il + g;
              *reinterpret_cast<u32x2 *>(row + ((chunk ^ sw) << 4) + 8 * (lane >> 5)) =
                  to_h4(c[4 * g], c[4 * g + 1], c[4 * g + 2], c[4 * g + 3]);
            }
          }
        }
      }
      wait_lds();
      __builtin_amdgcn_wave_barrier();
      // 8 lanes per row, 16-byte chunk q
      const int q = lane & 7;
      u32x4 d[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int kr = 8 * t + (lane >> 3);
        d[t] = *reinterpret_cast<const u32x4 *>(hb + kr * 128 +
                                                ((q ^ ((kr >> 1) & 7)) << 4));
      }
      const int rho = rho0 + 64 * h;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int k = k0 + 8 * t + (lane >> 3);
        if (SPLIT) {
          *reinterpret_cast<u32x4 *>(a.part + ((size_t)split * a.k + k) * rsc + rho +
                                     pass * 32 + 4 * q) = d[t];
        } else {
#pragma unroll
          for (int w = 0; w < 4; ++w) bad |= nonfinite_h2(d[t][w]);
          *reinterpret_cast<u32x4 *>(a.dw + (size_t)k * rsc + rho + 8 * q) = d[t];
        }
      }
      if (pass + 1 < PASSES || h + 1 < HM) {
        wait_lds();
        __builtin_amdgcn_wave_barrier();
      }
    }
  }
  if (!SPLIT && a.flag) flag_nonfinite(a.flag, bad);
}

// ---------------------------------------------------------------------------
// Kernel gradient: rows rho = (tap, c) of one tap (c % 256 == 0 tiles),
// columns k (K % 256 == 0), reduction over output positions m.
template <class C, bool SPLIT>
__global__ __launch_bounds__(C::NT) void wgrad_dma_kernel(WgradArgs a, WgradDiv fd,
                                                          TileMap tm) {
  FG_DMA_RING(C, R);
  constexpr int PW = C::PW;

  const int rsc = a.r * a.s * a.c;
  int tx, ty, split;  // rho tile, k tile, reduction split
  if (!tm.decode(blockIdx.x, tx, ty, split)) return;
  const int m0 = tx * C::T;  // rho
  const int n0 = ty * C::T;  // k
  const int mbeg = split * a.mchunk;
  const int mend = min(a.mtot, mbeg + a.mchunk);
  const int nst = mend > mbeg ? (mend - mbeg + C::BK - 1) / C::BK : 0;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm0 = (wave / C::WGN) * C::WM, wn0 = (wave % C::WGN) * C::WN;

  const int tap = m0 / a.c, c0 = m0 - tap * a.c;
  const int tr = tap / a.s, ts = tap - tr * a.s;

  const __amdgpu_buffer_rsrc_t rs_x = __builtin_amdgcn_make_buffer_rsrc(
      (void *)a.x, 0, (int)x_span_bytes(a), kRsrcFlags);
  const __amdgpu_buffer_rsrc_t rs_dy = __builtin_amdgcn_make_buffer_rsrc(
      (void *)a.dy, 0, (int)((size_t)a.mtot * a.k * 2), kRsrcFlags);

  // This lane's reduction row m = mbeg + BK * st + krow is decoded into
  // (n, p, q) once, with multiply-shift division; each stage then advances
  // it by BK rows with adds and at most one carry into p and one into n
  // (BK = dq + Q * (dp + P * dn) with dq < Q, dp < P), tracking the input
  // position (hh, ww) and the byte offsets of both operands directly.
  // Integer multiplies run at a quarter of the VALU rate: a division per
  // stage cost more VALU time than the stage's MFMAs leave free.
  const MnSlot<C> sl = mn_slots<C>(wave, lane);
  const int h0 = tr - a.ph, w0 = ts - a.pw;
  const int pixb = a.ldx * 2, rowb = a.w * pixb, imgb = a.h * rowb;
  int hh[PW], ww[PW], ox[PW], od[PW];
#pragma unroll
  for (int jj = 0; jj < PW; ++jj) {
    const int m = mbeg + sl.krow[jj];
    const unsigned nn = fd.pq.div((unsigned)m);
    const unsigned rem = (unsigned)m - nn * (unsigned)(a.p * a.q);
    const unsigned pp = fd.q.div(rem);
    const int qq = (int)(rem - pp * (unsigned)a.q);
    hh[jj] = (int)pp * a.sh + h0;
    ww[jj] = qq * a.sw + w0;
    ox[jj] = (int)nn * imgb + hh[jj] * rowb + ww[jj] * pixb + (c0 + sl.ncol[jj]) * 2;
    od[jj] = (m * a.k + n0 + sl.ncol[jj]) * 2;
  }
  const int dq = C::BK % a.q, dpt = C::BK / a.q, dp = dpt % a.p, dn = dpt / a.p;
  const int inc_w = dq * a.sw, inc_h = dp * a.sh;
  const int inc_o = inc_w * pixb + inc_h * rowb + dn * imgb;
  const int wlim = a.q * a.sw + w0, hlim = a.p * a.sh + h0;
  const int wrap_o = a.sh * rowb - a.q * a.sw * pixb;  // q wraps into p
  const int hwrap_o = imgb - a.p * a.sh * rowb;         // p wraps into n
  const int inc_d = C::BK * a.k * 2;
  const int mleft = mend - mbeg;

  auto issue = [&](int st, int slot) __attribute__((always_inline)) {
    uint8_t *ta = R.a[slot], *tb = R.b[slot];
#pragma unroll
    for (int jj = 0; jj < PW; ++jj) {
      // row krow = RPI (PW wave + jj) + lane / (RB / 16) of stage st exists
      const bool mv = (int)(lane / (C::RB / 16)) <
                      mleft - C::BK * st - C::RPI * (C::PW * wave + jj);
      const bool v = mv && (unsigned)hh[jj] < (unsigned)a.h &&
                     (unsigned)ww[jj] < (unsigned)a.w;
      dma16(rs_x, ta + dma_dst<C>(wave, jj), v ? (unsigned)ox[jj] : kOOB);
      dma16(rs_dy, tb + dma_dst<C>(wave, jj), mv ? (unsigned)od[jj] : kOOB);
      od[jj] += inc_d;
      ww[jj] += inc_w;
      hh[jj] += inc_h;
      ox[jj] += inc_o;
      if (ww[jj] >= wlim) {
        ww[jj] -= a.q * a.sw;
        hh[jj] += a.sh;
        ox[jj] += wrap_o;
      }
      if (hh[jj] >= hlim) {
        hh[jj] -= a.p * a.sh;
        ox[jj] += hwrap_o;
      }
    }
  };

  f32x16 acc[C::FM][C::FN];
  zero<C>(acc);
  pipeline<C, false, false>(acc, R, nst, wm0, wn0, lane, issue);
  if constexpr ((C::WM == 64 || C::WM == 128) && C::WN == 64) {
    store_tile_w<C, SPLIT>(acc, R, a, rsc, m0 + wm0, n0 + wn0, lane, wave, split);
  } else {
    // direct: each lane writes 4 consecutive rho of one output channel k
    bool bad = false;
#pragma unroll
    for (int j = 0; j < C::FN; ++j) {
      const int k = n0 + wn0 + j * 32 + (lane & 31);
#pragma unroll
      for (int i = 0; i < C::FM; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int rho = m0 + wm0 + i * 32 + 8 * g + 4 * (lane >> 5);
          const f32x16 &c = acc[i][j];
          if (!SPLIT) {
            const u32x2 hv = to_h4(c[4 * g], c[4 * g + 1], c[4 * g + 2], c[4 * g + 3]);
            bad |= nonfinite_h2(hv[0]) | nonfinite_h2(hv[1]);
            *reinterpret_cast<u32x2 *>(a.dw + (size_t)k * rsc + rho) = hv;
          } else {
            *reinterpret_cast<f32x4 *>(a.part + ((size_t)split * a.k + k) * rsc +
                                       rho) =
                f32x4{c[4 * g], c[4 * g + 1], c[4 * g + 2], c[4 * g + 3]};
          }
        }
    }
    if (!SPLIT && a.flag) flag_nonfinite(a.flag, bad);
  }
}

}  // namespace dma

// ---------------------------------------------------------------------------
bool data_dma_ok(const DataConvArgs &a) {
  return a.cr % dma::DataRun::BK == 0 &&
         act_span_bytes(a) < 0x7FFFFFFFull &&
         (size_t)a.wbytes < 0x7FFFFFFFull;
}

bool wgrad_dma_ok(const WgradArgs &a) {
  return a.c % dma::TM == 0 && a.k % dma::TN == 0 &&
         x_span_bytes(a) < 0x7FFFFFFFull &&
         (size_t)a.mtot * a.k * 2 < 0x7FFFFFFFull;
}

bool data_halo_ok(const DataConvArgs &a) {
  if (a.nphase != 1 || a.istr != 1 || a.cr % 32 != 0) return false;
  const Phase &P = a.ph[0];
  if ((P.dstep != 1 && P.dstep != -1) || P.nr != 3 || P.ns != 3 || P.mw <= 0 ||
      dma::TN % P.mw != 0)
    return false;
  const int rt = dma::TN / P.mw;  // output rows per tile
  if (P.mh % rt != 0 || (rt + 2) * (P.mw + 2) > dma::kPatchRows) return false;
  return act_span_bytes(a) < 0x7FFFFFFFull &&
         (size_t)a.wbytes < 0x7FFFFFFFull;
}

hipError_t launch_data_conv_halo(const DataConvArgs &a, bool w_kmajor,
                                 hipStream_t st) {
  const int npix = a.n * a.ph[0].mh * a.ph[0].mw;
  dma::TileMap tm{a.nsplit, (a.co + dma::TM - 1) / dma::TM,
                  (npix + dma::TN - 1) / dma::TN, 0, 0};
  tm.per = (tm.n0 * tm.n1 * tm.n2 + 7) / 8;
  dim3 grid(8 * tm.per), block(dma::HaloRun::NT);
  const bool split = a.nsplit > 1;
  if (w_kmajor) {
    if (split)
      hipLaunchKernelGGL((dma::data_conv_halo_kernel<dma::HaloRun, true, true>),
                         grid, block, 0, st, a, tm);
    else
      hipLaunchKernelGGL((dma::data_conv_halo_kernel<dma::HaloRun, true, false>),
                         grid, block, 0, st, a, tm);
  } else {
    if (split)
      hipLaunchKernelGGL((dma::data_conv_halo_kernel<dma::HaloRun, false, true>),
                         grid, block, 0, st, a, tm);
    else
      hipLaunchKernelGGL((dma::data_conv_halo_kernel<dma::HaloRun, false, false>),
                         grid, block, 0, st, a, tm);
  }
  return hipGetLastError();
}

template <class C>
static hipError_t launch_dma_cfg(const DataConvArgs &a0, bool w_kmajor,
                                 hipStream_t st) {
  DataConvArgs a = a0;
  int maxpix = 0;
  bool uneven = false;
  for (int i = 0; i < a.nphase; ++i) {
    maxpix = std::max(maxpix, a.n * a.ph[i].mh * a.ph[i].mw);
    uneven |= a.ph[i].nr * a.ph[i].ns != a.ph[0].nr * a.ph[0].ns;
  }
  const int tco = (a.co + C::T - 1) / C::T, tpix = (maxpix + C::T - 1) / C::T;
  dma::TileMap tm;
  if (uneven) {
    // phases with different tap counts (strided input gradients): costliest
    // phase first, in launch order, so the cheap tiles fill the tail
    std::stable_sort(a.ph, a.ph + a.nphase, [](const Phase &x, const Phase &y) {
      return x.nr * x.ns > y.nr * y.ns;
    });
    tm = dma::TileMap{tpix, tco, a.nphase * a.nsplit, 0, 1};
  } else {
    // phases and splits fastest, so every XCD gets an even share of each
    // and the phases of one position tile share input
    tm = dma::TileMap{a.nphase * a.nsplit, tco, tpix, 0, 0};
  }
  tm.per = (tm.n0 * tm.n1 * tm.n2 + 7) / 8;
  dim3 grid(8 * tm.per), block(C::NT);
  const bool split = a.nsplit > 1;
  if (w_kmajor) {
    if (split)
      hipLaunchKernelGGL((dma::data_conv_dma_kernel<C, true, true>), grid, block, 0,
                         st, a, tm);
    else
      hipLaunchKernelGGL((dma::data_conv_dma_kernel<C, true, false>), grid, block, 0,
                         st, a, tm);
  } else {
    if (split)
      hipLaunchKernelGGL((dma::data_conv_dma_kernel<C, false, true>), grid, block, 0,
                         st, a, tm);
    else
      hipLaunchKernelGGL((dma::data_conv_dma_kernel<C, false, false>), grid, block,
                         0, st, a, tm);
  }
  return hipGetLastError();
}

hipError_t launch_data_conv_dma(const DataConvArgs &a, bool w_kmajor,
                                hipStream_t st) {
  return launch_dma_cfg<dma::DataRun>(a, w_kmajor, st);
}

hipError_t launch_data_conv_dma_small(const DataConvArgs &a, bool w_kmajor,
                                      hipStream_t st) {
  return launch_dma_cfg<dma::SmallRun>(a, w_kmajor, st);
}

static dma::FastDiv make_fastdiv(uint32_t d) {
  int l = 0;
  while ((1ull << l) < d) ++l;
  const uint64_t m = ((1ull << 32) * ((1ull << l) - d)) / d + 1;
  return {(uint32_t)m, l ? 1 : 0, l ? l - 1 : 0};
}

hipError_t launch_wgrad_dma(const WgradArgs &a, hipStream_t st) {
  const int rsc = a.r * a.s * a.c;
  const dma::WgradDiv fd{make_fastdiv((uint32_t)(a.p * a.q)), make_fastdiv((uint32_t)a.q)};
  dma::TileMap tm{rsc / dma::TM, a.k / dma::TN, a.nsplit, 0, 0};
  tm.per = (tm.n0 * tm.n1 * tm.n2 + 7) / 8;
  dim3 grid(8 * tm.per);
  if (a.nsplit > 1)
    hipLaunchKernelGGL((dma::wgrad_dma_kernel<dma::WgradRun, true>), grid, dim3(dma::WgradRun::NT), 0, st,
                       a, fd, tm);
  else
    hipLaunchKernelGGL((dma::wgrad_dma_kernel<dma::WgradRun, false>), grid, dim3(dma::WgradRun::NT), 0, st,
                       a, fd, tm);
  return hipGetLastError();
}

}  // namespace fg
