// Grouped SwiGLU expert FFN (Section 2.1: MLP^j read as SwiGLU) on gfx950.
//
// Two passes per call:
//   gate/up:  H[i, n] = SiLU(X_i . Wg[n]) * (X_i . Wu[n])   (rows gathered
//             through group_rows; a tile owns matching gate and up columns so
//             the SwiGLU runs in the epilogue; H is stored in the element type)
//   down:     Y[row_i] = H[i] . Wd^T                        (rows scattered
//             through group_rows)
// bf16 runs on MFMA (v_mfma_f32_16x16x32_bf16 or _32x32x16_bf16, fp32
// accumulation) with both operand tiles staged through a ring of LDS slots
// by direct global->LDS copies; few-row passes stream the weights straight
// into registers.  The launcher picks the tile variant per pass from the
// shape.  fp32 runs on the vector ALUs.
//
// Groups have ragged row counts known only on the device.  Every workgroup
// rebuilds the per-group m-tile prefix from group_offsets in LDS, then walks
// the tile space (group, n-tile, m-tile; m fastest) in a loop.  The tile
// space is cut into eight contiguous ranges, one per XCD (workgroups are
// dispatched round-robin over the XCDs), so tiles sharing a weight panel or
// a row panel run under one L2.

#include <stdlib.h>

#include <type_traits>

#include "common.hpp"
#include "internal.hpp"

namespace fs {
namespace {

constexpr int kMaxGroups = 512;
constexpr int kXcd = 8;
enum { MODE_GATEUP = 0, MODE_DOWN = 1 };

// SiLU(g) * u for the bf16 epilogues, whose result is rounded to bf16: the
// hardware exponential and reciprocal (about 1 ulp each in fp32) replace the
// IEEE division, which costs ten instructions per element.
__device__ __forceinline__ float swiglu_bf16_epi(float g, float u) {
  return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u;
}

// Group offsets and the exclusive prefix of m-tiles per group, in LDS.
template <int NT, int BM>
__device__ void sched_setup(const int32_t* __restrict__ goff, int G, int64_t m_total,
                            int* s_goff, int* s_tpre, int* s_wtot) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // Offsets are clamped to [0, m_total]: rows past the host bound are never
  // read or written, so a short bound cannot overrun the H workspace.
  for (int g = tid; g <= G; g += NT) {
    int v = goff ? goff[g] : (g == 0 ? 0 : (int)m_total);
    s_goff[g] = v < 0 ? 0 : (v > (int)m_total ? (int)m_total : v);
  }
  __syncthreads();
  constexpr int IPT = (kMaxGroups + 1 + NT - 1) / NT;
  int cnt[IPT];
  int local = 0;
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    const int g = tid * IPT + i;
    const int c = (g < G && s_goff[g + 1] > s_goff[g]) ? (s_goff[g + 1] - s_goff[g] + BM - 1) / BM : 0;
    cnt[i] = c;
    local += c;
  }
  int incl = local;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int v = __shfl_up(incl, o, FS_WAVE);
    if (lane >= o) incl += v;
  }
  if (lane == 63) s_wtot[wave] = incl;
  __syncthreads();
  int pre = 0;
  for (int w = 0; w < wave; ++w) pre += s_wtot[w];
  int run = pre + incl - local;
#pragma unroll
  for (int i = 0; i < IPT; ++i) {
    const int g = tid * IPT + i;
    if (g <= G) s_tpre[g] = run;
    run += cnt[i];
  }
  __syncthreads();
}

// Largest g in [0, G) with nn * tpre[g] <= L.
__device__ __forceinline__ int find_group(const int* s_tpre, int G, int nn, int64_t L) {
  int lo = 0, hi = G - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if ((int64_t)nn * s_tpre[mid] <= L)
      lo = mid;
    else
      hi = mid - 1;
  }
  return lo;
}

// find_group for a workgroup's items, which come in increasing order: the
// answer is at least lo (the previous item's group), and most often lo or
// lo + 1, so two LDS reads usually settle it before any binary search.
__device__ __forceinline__ int find_group_from(const int* s_tpre, int G, int nn, int64_t L, int lo) {
  if (lo + 1 < G && (int64_t)nn * s_tpre[lo + 1] <= L) {
    ++lo;
    if (lo + 1 < G && (int64_t)nn * s_tpre[lo + 1] <= L) {
      int hi = G - 1;
      ++lo;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if ((int64_t)nn * s_tpre[mid] <= L)
          lo = mid;
        else
          hi = mid - 1;
      }
    }
  }
  return lo;
}

// ---------------------------------------------------------------- bf16 MFMA
template <int MODE, int BM, int BN, int BK, int WAVES_M, int WAVES_N>
__global__ __launch_bounds__(64 * WAVES_M * WAVES_N) void gemm_bf16_kernel(
    const bf16_t* __restrict__ A, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ goff, int G, int64_t m_total, const bf16_t* __restrict__ B, int K,
    int NOUT, bf16_t* __restrict__ C, int ldc) {
  constexpr int NT = 64 * WAVES_M * WAVES_N;
  constexpr int WTM = BM / WAVES_M, WTN = BN / WAVES_N;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int LDK = BK + 8;  // LDS row stride in bf16: 16-byte skew per row
  constexpr int CPR = BK / 8;  // 16-byte chunks per tile row
  constexpr int ACH = BM * CPR / NT, BCH = BN * CPR / NT;
  constexpr int NCOL = (MODE == MODE_GATEUP) ? BN / 2 : BN;
  constexpr int STAGE = (BM + BN) * LDK;
  static_assert(BM * CPR % NT == 0 && BN * CPR % NT == 0, "tile loads must divide evenly");
  static_assert(MODE != MODE_GATEUP || TN % 2 == 0, "gate/up tiles come in pairs");

  __shared__ int s_goff[kMaxGroups + 1];
  __shared__ int s_tpre[kMaxGroups + 1];
  __shared__ int s_wtot[NT / 64];
  __shared__ __align__(16) bf16_t lds[2 * STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WAVES_N, wn = wave % WAVES_N;
  sched_setup<NT, BM>(goff, G, m_total, s_goff, s_tpre, s_wtot);

  const int nn = NOUT / NCOL;
  const int64_t total = (int64_t)nn * s_tpre[G];
  const int64_t per_xcd = (total + kXcd - 1) / kXcd;
  const int64_t xcd_base = (int64_t)(blockIdx.x % kXcd) * per_xcd;
  const int64_t stride = gridDim.x / kXcd;
  const int KT = K / BK;
  const size_t bstride = (size_t)((MODE == MODE_GATEUP) ? 2 * NOUT : NOUT) * K;

  for (int64_t j = blockIdx.x / kXcd; j < per_xcd; j += stride) {
    const int64_t L = xcd_base + j;
    if (L >= total) break;
    const int g = find_group(s_tpre, G, nn, L);
    const int Tg = s_tpre[g + 1] - s_tpre[g];
    const int64_t local = L - (int64_t)nn * s_tpre[g];
    const int nt = (int)(local / Tg), mt = (int)(local % Tg);
    const int row_base = s_goff[g], rows_g = s_goff[g + 1] - row_base;
    const int m0 = mt * BM, n0 = nt * NCOL;
    const bf16_t* Bg = B + (size_t)g * bstride;

    const bf16_t* pa[ACH];
    bool va[ACH];
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int c = tid + i * NT;
      const int r = c / CPR, kc = (c % CPR) * 8;
      const int m = m0 + r;
      va[i] = m < rows_g;
      const int grow = row_base + (va[i] ? m : 0);
      const int64_t src = (MODE == MODE_GATEUP && rows) ? (int64_t)rows[grow] : (int64_t)grow;
      pa[i] = A + src * K + kc;
    }
    const bf16_t* pb[BCH];
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int c = tid + i * NT;
      const int r = c / CPR, kc = (c % CPR) * 8;
      int wrow;
      if (MODE == MODE_GATEUP)
        wrow = (r < BN / 2) ? n0 + r : NOUT + n0 + (r - BN / 2);
      else
        wrow = n0 + r;
      pb[i] = Bg + (size_t)wrow * K + kc;
    }

    floatx16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int jn = 0; jn < TN; ++jn)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][jn][v] = 0.f;

    uint4 ra[ACH], rb[BCH];
    auto gload = [&](int k0) {
#pragma unroll
      for (int i = 0; i < ACH; ++i) ra[i] = va[i] ? ld16(pa[i] + k0) : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int i = 0; i < BCH; ++i) rb[i] = ld16(pb[i] + k0);
    };
    auto lstore = [&](int buf) {
      bf16_t* As = lds + buf * STAGE;
      bf16_t* Bs = As + BM * LDK;
#pragma unroll
      for (int i = 0; i < ACH; ++i) {
        const int c = tid + i * NT;
        st16(As + (c / CPR) * LDK + (c % CPR) * 8, ra[i]);
      }
#pragma unroll
      for (int i = 0; i < BCH; ++i) {
        const int c = tid + i * NT;
        st16(Bs + (c / CPR) * LDK + (c % CPR) * 8, rb[i]);
      }
    };

    gload(0);
    for (int kt = 0; kt < KT; ++kt) {
      lstore(kt & 1);
      __syncthreads();
      if (kt + 1 < KT) gload((kt + 1) * BK);
      const bf16_t* As = lds + (kt & 1) * STAGE;
      const bf16_t* Bs = As + BM * LDK;
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        const int kofs = ks * 16 + (lane >> 5) * 8;
        bf16x8 af[TM], bfr[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int r = wm * WTM + i * 32 + (lane & 31);
          af[i] = *reinterpret_cast<const bf16x8*>(As + r * LDK + kofs);
        }
#pragma unroll
        for (int jn = 0; jn < TN; ++jn) {
          int br;
          if (MODE == MODE_GATEUP)
            br = (jn < TN / 2) ? wn * (WTN / 2) + jn * 32
                               : BN / 2 + wn * (WTN / 2) + (jn - TN / 2) * 32;
          else
            br = wn * WTN + jn * 32;
          bfr[jn] = *reinterpret_cast<const bf16x8*>(Bs + (br + (lane & 31)) * LDK + kofs);
        }
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int jn = 0; jn < TN; ++jn)
            acc[i][jn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[jn], acc[i][jn], 0,
                                                                 0, 0);
      }
    }

    // Epilogue.  Accumulator element v of lane l holds row
    // 8*(v/4) + 4*(l/32) + v%4 and column l%32 of its 32x32 tile.
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int m = m0 + wm * WTM + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
        if (m >= rows_g) continue;
        const int grow = row_base + m;
        if (MODE == MODE_GATEUP) {
#pragma unroll
          for (int jn = 0; jn < TN / 2; ++jn) {
            const float gt = acc[i][jn][v], up = acc[i][jn + TN / 2][v];
            const float h = swiglu_bf16_epi(gt, up);
            const int col = n0 + wn * (WTN / 2) + jn * 32 + (lane & 31);
            C[(size_t)grow * ldc + col] = f2bf(h);
          }
        } else {
          const int64_t orow = rows ? (int64_t)rows[grow] : (int64_t)grow;
#pragma unroll
          for (int jn = 0; jn < TN; ++jn) {
            const int col = n0 + wn * WTN + jn * 32 + (lane & 31);
            C[orow * ldc + col] = f2bf(acc[i][jn][v]);
          }
        }
      }
    }
    __syncthreads();  // LDS stages are reused by the next tile
  }
}

// ---------------------------------------------------------------- bf16 MFMA, DMA ring
// BM x BN x 64 tiles, four waves (2 x 2), each wave BM/2 x BN/2 through
// v_mfma_f32_32x32x16_bf16.  Operand tiles stream into an LDS ring of
// STAGES slots with direct global->LDS 16-byte loads (no staging
// registers), STAGES-1 K blocks ahead of the MFMAs.  A 64-element K row is
// 8 chunks of 16 bytes; chunk c of row r sits at position c ^ ((r / 2) % 8):
// the LDS serves a ds_read_b128 sixteen lanes at a time over 64 banks, and
// sixteen consecutive rows then cover all 64 banks once.  Rows past the end of a group load a valid row of the
// group instead (a DMA cannot write zeros); their results are never stored.
// The epilogue stages the output tile through LDS so that global stores are
// whole 16-byte row chunks.

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glb_void_t;

// One direct global->LDS load of 16 bytes per lane: lane l's bytes land at
// LDS address lds + 16 * l, where lds is the wave's destination as a
// wave-uniform 32-bit LDS address (kept in SGPRs by the caller, so a copy
// needs no address-space conversion or lane broadcast).  Issued as inline
// assembly so that the compiler does not add a conservative wait for every
// outstanding DMA before each LDS read; the kernels order them themselves
// with explicit vmcnt waits and barriers.  M0 carries the LDS address and has
// no other user in these kernels.
__device__ __forceinline__ void dma16_at(const void* g, unsigned lds) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
               :
               : "s"(lds), "v"(g)
               : "memory");
}

// The same with the global address split into a wave-uniform 64-bit base
// (SGPRs) and a 32-bit per-lane byte offset: the weight rows of a wave's DMAs
// share one base, so they hold two VGPRs of offsets instead of a 64-bit
// pointer per DMA.
__device__ __forceinline__ void dma16_sb(const void* base, unsigned off, unsigned lds) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
               :
               : "s"(lds), "v"(off), "s"(base)
               : "memory");
}

// A pointer made wave-uniform (held in SGPRs): lane 0's value.
template <typename T>
__device__ __forceinline__ T* uniform_ptr(T* p) {
  const uint64_t v = (uint64_t)(uintptr_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return (T*)(uintptr_t)(((uint64_t)hi << 32) | lo);
}

// A 16-byte load marked non-temporal (the streaming hint), for the expert
// weights that the fragment-ordered decode passes read exactly once.
// DeepSeek-V3-shaped decode, routed gate/up 266 -> 239 us (6.43 TB/s, 0.80
// of HBM), down 142 -> 140 us, step 0.531 -> 0.508 ms (same-box A/B).  The
// 64-row shared expert's weight-streaming kernels were slower with it
// (gate/up 28 -> 30 us, down 17 -> 18 us) and keep ordinary loads.
template <typename V>
__device__ __forceinline__ V ld_stream(const void* p) {
  typedef int v4i __attribute__((ext_vector_type(4)));
  static_assert(sizeof(V) == 16, "16-byte loads");
  const v4i v = __builtin_nontemporal_load(reinterpret_cast<const v4i*>(p));
  return __builtin_bit_cast(V, v);
}

// LDS address of a __shared__ location as a wave-uniform 32-bit value.
__device__ __forceinline__ unsigned lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane((unsigned)(uintptr_t)(const lds_void_t*)p);
}

// s_waitcnt with only vmcnt constrained (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

__device__ __forceinline__ void barrier_nofence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// ---------------------------------------------------------------- bf16 MFMA, interleaved
// Same tiles, ring and swizzle as above, with the memory work hidden under
// the MFMAs by a rolling pipeline over 16-wide K steps.  Each step first
// issues the LDS reads of the next step's fragments (double-buffered
// registers), then its own MFMAs; the DMAs of the block two ahead are spread
// over the first steps of a block, one after each of the first MFMAs.  The
// block's last step starts with the only barrier of the block, once the
// next block has landed.  A wave issues memory instructions in the shadow of
// an executing MFMA, so with one wave per SIMD the MFMA pipe stays busy.
// The grid is persistent (one workgroup per CU).
//
// F8: the same kernel on FP8 E4M3 operands with BK = 128 elements, so a
// staged row is still 128 bytes and the ring, swizzle and DMAs are
// unchanged.  A K step is one v_mfma_scale_f32_32x32x64_f8f6f4 per tile
// (unit scales): lane l supplies row l % 32 and the 32 bytes
// [32 (l / 32), 32 (l / 32) + 32) of the step's 64, read as two 16-byte
// chunks (any split works as long as A and B use the same one).  A block has
// two steps of half as many, twice as long MFMAs, so the MFMA time per block
// equals bf16's for twice the K.  The epilogue multiplies each accumulator by
// its row's scale sA (indexed like the A rows) and its column's scale sB
// (per group: 2 NOUT gate/up columns or NOUT down columns).
//
// Split K (SPL; the other instantiations carry none of it): every tile is
// cut into `splits` K slices of `kps`
// blocks (the last may be shorter, none empty); a work item is one slice of
// one tile, the slices of a tile adjacent in the XCD's range.  An item writes
// its fp32 partial (scales applied) to P[slice][row][col], columns as in
// stream_reduce_kernel (gate/up: gate 0..NOUT-1, up NOUT..2 NOUT-1), which
// then adds the slices in order and applies SwiGLU or the scatter.  Passes
// whose tiles cannot fill the CUs use it.
//
// Across tiles (XT: 128-row tiles without split K whose epilogue staging
// fits one ring slot): the ring's slot numbering runs on from tile
// to tile, and the last STAGES - 1 blocks of a tile issue the DMAs of the
// next tile's first STAGES - 1 blocks, so they land during the epilogue and
// the next tile starts without a load latency.  The epilogue stages through
// the slot of the tile's last block, the one slot no DMA is writing.  The
// next tile's gathered A rows are read with scalar loads, which the vector
// memory counter the ring's waits rely on does not see.  Vector memory
// operations complete in issue order, so the epilogue's stores, issued after
// the next tile's first DMAs, only make later waits a little stricter.
//
// The epilogue goes through LDS in passes of IPP 32-row accumulator rows per
// wave, every wave converting in every pass (gate/up: SiLU(g) * u), then all
// threads store whole 16-byte chunks of the staged rows.
//
// Waves: a WGM x WGN grid, each wave BM / WGM x BN / WGN.  Four waves (2 x 2)
// hold one per SIMD; eight hold two per SIMD, whose instruction streams
// interleave: with one wave per SIMD the wave waits to issue 44% of its
// cycles (SQ_WAIT_INST_ANY, Llama-4-Scout-shaped routed gate/up) while the
// MFMA pipe is busy 55%.  The 128 x 256 tile runs 2 x 4 waves of 64 x 64
// (routed gate/up 1493 -> 1432 us Scout-shaped, 377 -> 362 us
// DeepSeek-V2-Lite-shaped; DeepSeek-V3-shaped down 1073 -> 997 us; alone
// on the GPU).
//
// M16 (bf16): 16 x 16 fragments on v_mfma_f32_16x16x32_bf16 (lane l: row
// l % 16, k 8 (l / 16) .. + 7 of a 32-wide step; accumulator element v of
// lane l: row 4 (l / 16) + v, column l % 16), two K steps per 64-wide
// block, the same bytes per MFMA cycle from LDS.  The smaller MFMA runs at
// a higher clock under the part's power limit: with eight waves of 64 x 64
// on the 128 x 256 tile, Llama-4-Scout-shaped block step 4.34 -> 4.16 ms
// (routed gate/up 1458 -> 1415 us, dense shared gate/up 1266 -> 1210 us),
// DeepSeek-V3-shaped prefill 3.92 -> 3.83 ms, DeepSeek-V2-Lite-shaped
// 0.925 -> 0.893 ms (same-box A/B).  (With four waves of 64 x 128 it had
// been slower on every pass.)

__device__ __forceinline__ void wait_lgkm0() {
  // lgkmcnt(0), vmcnt and expcnt unconstrained
  __builtin_amdgcn_s_waitcnt((0xF) | (0x3 << 14) | (0x7 << 4) | (0x0 << 8));
}

typedef int int32x8 __attribute__((ext_vector_type(8)));

template <int MODE, int BM, int BN, int BK, int STAGES, int OCC, bool F8 = false, bool SPL = false,
          int WGM = 2, int WGN = 2, bool M16 = false>
__global__ __launch_bounds__(64 * WGM * WGN, OCC) void gemm_bf16_il_kernel(
    const typename std::conditional<F8, uint8_t, bf16_t>::type* __restrict__ A,
    const int32_t* __restrict__ rows, const int32_t* __restrict__ goff, int G, int64_t m_total,
    const typename std::conditional<F8, uint8_t, bf16_t>::type* __restrict__ B, int K, int NOUT,
    bf16_t* __restrict__ C, int ldc, const float* __restrict__ sA, const float* __restrict__ sB,
    int splits, int kps, float* __restrict__ P) {
  using TE = typename std::conditional<F8, uint8_t, bf16_t>::type;
  using FragT = typename std::conditional<F8, int32x8, bf16x8>::type;
  constexpr int NT = 64 * WGM * WGN;               // WGM x WGN waves
  constexpr int WTM = BM / WGM, WTN = BN / WGN;
  static_assert(!(F8 && M16), "16 x 16 fragments for bf16 only");
  constexpr int FR = M16 ? 16 : 32;                // fragment rows
  constexpr int TM = WTM / FR, TN = WTN / FR;      // fragments per wave tile
  constexpr int TU = WTM / 32;                     // 32-row accumulator units
  constexpr int BPU = 32 / FR;                     // fragments per unit
  constexpr int AV = M16 ? 4 : 16;                 // accumulator elements
  using AccT = typename std::conditional<M16, floatx4, floatx16>::type;
  constexpr int ES = F8 ? 1 : 2;                   // element bytes
  constexpr int CE = 16 / ES;                      // elements per 16-byte chunk
  constexpr int ROWB = BK * ES;
  constexpr int CPR = ROWB / 16;
  constexpr int RPB = 1024 / ROWB;
  constexpr int SWD = 16 / CPR;
  constexpr int STAGE = (BM + BN) * ROWB;
  constexpr int A_LD = BM / RPB / (WGN * WGM), B_LD = BN / RPB / (WGN * WGM);
  constexpr int NLD = A_LD + B_LD;
  constexpr int NCOL = (MODE == MODE_GATEUP) ? BN / 2 : BN;
  constexpr int SST = NCOL + 8;                    // staged row, bf16 elements
  constexpr int KS = ROWB / (F8 || M16 ? 64 : 32); // K steps per block
  constexpr int NF = TM + TN;                      // fragments per K step
  constexpr int MPS = TM * TN;                     // MFMAs per K step
  // read r of the next step goes out after MFMA read_slot(r) of this one
  // (with fewer MFMAs than fragments per step, as for one 32-row block per
  // wave, the first reads all go out after MFMA 0)
  auto read_slot = [](int r) { return std::max(0, ((r + 1) * MPS) / NF - 1); };
  // The DMAs of block kt + STAGES - 1 go out during block kt: spread over its
  // steps 0..KS-2 with three or more slots, all in step 0 with two (they must
  // land before the block's last step).
  constexpr int DSTEPS = (STAGES == 2) ? 1 : KS - 1;
  constexpr int DPS = (NLD + DSTEPS - 1) / DSTEPS;  // DMAs per step
  constexpr int DPQ = (DPS + MPS - 1) / MPS;        // DMAs after one MFMA
  static_assert(STAGES >= 2 && STAGES <= 6, "ring of two to six slots");
  static_assert(NLD * (STAGES - 2) < 64, "vmcnt range");
  static_assert(KS >= 2, "at least two K steps per block");
  static_assert(DPQ <= 2, "two DMAs per MFMA at most");
  static_assert(!F8 || BK == 128, "FP8 rows are 128 elements");
  static_assert(A_LD >= 1 && B_LD >= 1 && BM % (WGN * WGM * RPB) == 0 && BN % (WGN * WGM * RPB) == 0,
                "tile");
  // Cross-tile candidates: 128-row tiles without split K (256-row tiles
  // already use every register).  Their staging must fit one slot, the
  // others' the whole ring.  IPP: accumulator rows (of 32) per wave and
  // epilogue pass; SROWS: staged rows per pass.
  constexpr bool XTC = !SPL && BM == 128 && WGM == 2;
  constexpr int SCAP = XTC ? STAGE : STAGES * STAGE;
  constexpr int IPP = (TU % 4 == 0 && WGM * 128 * SST * 2 <= SCAP)  ? 4
                      : (TU % 2 == 0 && WGM * 64 * SST * 2 <= SCAP) ? 2
                                                                    : 1;
  constexpr int SROWS = WGM * 32 * IPP;
  constexpr bool XT = XTC && SROWS * SST * 2 <= STAGE;
  static_assert(SROWS * SST * 2 <= STAGES * STAGE, "epilogue pass must fit in the ring");
  static_assert((SROWS * NCOL / 8) % NT == 0, "whole store rounds");
  static_assert(MODE != MODE_GATEUP || TN % 2 == 0, "gate/up tiles come in pairs");

  __shared__ int s_goff[kMaxGroups + 1];
  __shared__ int s_tpre[kMaxGroups + 1];
  __shared__ int s_wtot[NT / 64];
  __shared__ float s_sa[F8 ? BM : 1];              // F8: the tile's row scales
  __shared__ __align__(1024) unsigned char ring[STAGES * STAGE];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  sched_setup<NT, BM>(goff, G, m_total, s_goff, s_tpre, s_wtot);

  const int nn = NOUT / NCOL;
  const int nspl = SPL ? splits : 1;
  const int64_t total = (int64_t)nn * s_tpre[G] * nspl;
  const int64_t per_xcd = (total + kXcd - 1) / kXcd;
  const int64_t xcd_base = (int64_t)(blockIdx.x % kXcd) * per_xcd;
  const int64_t stride = gridDim.x / kXcd;
  const int KT_all = K / BK;
  const int kpsv = SPL ? kps : KT_all;
  const size_t bstride = (size_t)((MODE == MODE_GATEUP) ? 2 * NOUT : NOUT) * K;
  const int drow = lane / CPR, dpos = lane % CPR;
  auto dchunk = [&](int block) { return dpos ^ (((block * RPB + drow) / SWD) % CPR); };

  // fragment byte offsets inside a slot, per K step (tile-independent)
  int aoff[TM], boff[TN], asw[TM], bsw[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int r = wm * WTM + i * FR + (lane & (FR - 1));
    aoff[i] = r * ROWB;
    asw[i] = (r / SWD) % CPR;
  }
#pragma unroll
  for (int jn = 0; jn < TN; ++jn) {
    int r;
    if (MODE == MODE_GATEUP)
      r = (jn < TN / 2) ? wn * (WTN / 2) + jn * FR : BN / 2 + wn * (WTN / 2) + (jn - TN / 2) * FR;
    else
      r = wn * WTN + jn * FR;
    r += lane & (FR - 1);
    boff[jn] = BM * ROWB + r * ROWB;
    bsw[jn] = (r / SWD) % CPR;
  }

  // A work item: its tile, its K range and the DMA sources of its rows.
  struct Item {
    int g, m0, n0, row_base, rows_g, ksl, kbase, KT;
  };
  const int wave_s = XT ? __builtin_amdgcn_readfirstlane(wave) : wave;
  int ghint = 0;   // group of the previous item: a lower bound for the next
  // B DMA i of a wave (block wave * B_LD + i of the tile's B rows) reads
  // base + i RPB K + the lane's offset; the chunk swizzle repeats every two
  // blocks, so two lane offsets serve all of them
  static_assert((2 * (RPB / SWD)) % CPR == 0, "B swizzle period of two blocks");
  unsigned bdl[2];
#pragma unroll
  for (int j = 0; j < 2; ++j)
    bdl[j] = (unsigned)((drow * K + dchunk(wave * B_LD + j) * CE) * ES);
  auto decode = [&](int64_t L, Item& it, const TE* (&sp)[A_LD], const TE*& bsp) {
    const int64_t Lt = SPL ? L / nspl : L;
    it.ksl = SPL ? (int)(L - Lt * nspl) : 0;
    it.kbase = it.ksl * kpsv;
    it.KT = (KT_all - it.kbase < kpsv) ? KT_all - it.kbase : kpsv;
    // (wave-uniform values; XT makes them scalar for the row-index loads)
    auto uni = [](int v) { return XT ? __builtin_amdgcn_readfirstlane(v) : v; };
    it.g = uni(find_group_from(s_tpre, G, nn, Lt, ghint));
    ghint = it.g;
    const int Tg = s_tpre[it.g + 1] - s_tpre[it.g];
    const int local = (int)(Lt - (int64_t)nn * s_tpre[it.g]);   // < nn * Tg
    const int ntile = local / Tg;
    it.n0 = uni(ntile * NCOL);
    it.m0 = uni((local - ntile * Tg) * BM);
    it.row_base = uni(s_goff[it.g]);
    it.rows_g = uni(s_goff[it.g + 1]) - it.row_base;
    const TE* Bg = B + (size_t)it.g * bstride;
#pragma unroll
    for (int i = 0; i < A_LD; ++i) {
      const int blk = wave_s * A_LD + i;
      int64_t sr;
      if (XT && MODE == MODE_GATEUP && rows) {
        // the block's RPB row indices with wave-uniform (scalar) loads; a
        // lane takes the one of its row
        int v = 0;
#pragma unroll
        for (int r = 0; r < RPB; ++r) {
          int m = it.m0 + blk * RPB + r;
          if (m >= it.rows_g) m = it.rows_g - 1;
          const int x = rows[it.row_base + m];
          v = drow == r ? x : v;
        }
        sr = v;
      } else {
        int m = it.m0 + blk * RPB + drow;
        if (m >= it.rows_g) m = it.rows_g - 1;
        const int grow = it.row_base + m;
        sr = (MODE == MODE_GATEUP && rows) ? (int64_t)rows[grow] : (int64_t)grow;
      }
      sp[i] = A + sr * K + (size_t)it.kbase * BK + dchunk(blk) * CE;
    }
    // the wave's B rows lie in one half (gate or up) of the tile's B rows
    const int r0 = wave * B_LD * RPB;
    const int wrow0 = (MODE == MODE_GATEUP && r0 >= BN / 2) ? NOUT + it.n0 + (r0 - BN / 2) : it.n0 + r0;
    bsp = uniform_ptr(Bg + (size_t)wrow0 * K + (size_t)it.kbase * BK);
  };

  // wave-uniform LDS destinations: ring base + slot + this wave's blocks
  const unsigned ring_lds = lds_addr(ring);
  const unsigned wave_u = __builtin_amdgcn_readfirstlane(wave);
  auto dst_of = [&](int i) {
    return i < A_LD ? (wave_u * A_LD + i) * 1024u
                    : (unsigned)(BM * ROWB) + (wave_u * B_LD + (i - A_LD)) * 1024u;
  };
  const bool xt_ok = XT && KT_all >= STAGES - 1;
  int sb = 0;            // ring slot of the current item's block 0
  bool primed = false;   // its first STAGES - 1 blocks are already in flight
  static_assert(MODE != MODE_GATEUP || (BN / 2) % (B_LD * RPB) == 0, "a wave's B rows in one half");
  const TE* src[A_LD];
  const TE* srcN[A_LD];
  const TE* bsrc = nullptr;    // wave-uniform B row base of the current item
  const TE* bsrcN = nullptr;   // and of the next
  Item itN;              // the next item, decoded during this one's last blocks

  for (int64_t j = blockIdx.x / kXcd; j < per_xcd; j += stride) {
    const int64_t L = xcd_base + j;
    if (L >= total) break;
    Item it;
    if (XT && primed) {
      it = itN;
#pragma unroll
      for (int i = 0; i < A_LD; ++i) src[i] = srcN[i];
      bsrc = bsrcN;
    } else {
      decode(L, it, src, bsrc);
    }
    const int KT = it.KT, m0 = it.m0, n0 = it.n0, row_base = it.row_base, rows_g = it.rows_g;
    const int g = it.g, ksl = it.ksl;
    const int64_t jnext = j + stride;
    const bool has_next = xt_ok && jnext < per_xcd && xcd_base + jnext < total;

    auto slot_of = [&](int b) { return (unsigned)((sb + b) % STAGES); };
    // DMA i of block b: b < KT from this item, b >= KT block b - KT of the next
    auto dma_cur = [&](int i, int b) {
      const unsigned lds = ring_lds + slot_of(b) * (unsigned)STAGE + dst_of(i);
      if (i < A_LD)
        dma16_at(src[i] + b * BK, lds);
      else
        dma16_sb(bsrc + (size_t)b * BK + (size_t)(i - A_LD) * RPB * K, bdl[(i - A_LD) & 1], lds);
    };
    auto dma_nxt = [&](int i, int b) {
      const unsigned lds = ring_lds + slot_of(b) * (unsigned)STAGE + dst_of(i);
      if (i < A_LD)
        dma16_at(srcN[i] + (b - KT) * BK, lds);
      else
        dma16_sb(bsrcN + (size_t)(b - KT) * BK + (size_t)(i - A_LD) * RPB * K, bdl[(i - A_LD) & 1], lds);
    };

    AccT acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int jn = 0; jn < TN; ++jn)
#pragma unroll
        for (int v = 0; v < AV; ++v) acc[i][jn][v] = 0.f;

    FragT Fa[NF], Fb[NF];
    // fragment r of a step in the order its MFMAs use them: A0, B0..B(TN-1),
    // A1..A(TM-1); read r is issued after MFMA read_slot(r) of the step before
    auto read_one = [&](FragT (&F)[NF], int kt, int ks, int r) {
      const unsigned char* slot = ring + slot_of(kt) * STAGE;
      const int f = r == 0 ? 0 : (r <= TN ? TM + r - 1 : r - TN);
      if constexpr (F8) {
        const int c = ks * 4 + 2 * (lane >> 5);
        const int base = f < TM ? aoff[f] : boff[f - TM];
        const int sw = f < TM ? asw[f] : bsw[f - TM];
        const int4 lo = *reinterpret_cast<const int4*>(slot + base + ((c ^ sw) << 4));
        const int4 hi = *reinterpret_cast<const int4*>(slot + base + (((c + 1) ^ sw) << 4));
        F[f] = int32x8{lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
      } else {
        const int c = M16 ? ks * 4 + (lane >> 4) : ks * 2 + (lane >> 5);
        const int off = f < TM ? aoff[f] + ((c ^ asw[f]) << 4) : boff[f - TM] + ((c ^ bsw[f - TM]) << 4);
        F[f] = *reinterpret_cast<const bf16x8*>(slot + off);
      }
    };
    auto read_step = [&](FragT (&F)[NF], int kt, int ks) {
#pragma unroll
      for (int r = 0; r < NF; ++r) read_one(F, kt, ks, r);
    };
    // One K step: the MFMAs of this step, with the reads of the next step's
    // fragments spread between them (in the order the next step uses them)
    // and up to DPS DMAs of block kt + STAGES - 1 after the first MFMAs.  A
    // block's last step waits for the next block after its first MFMA, so the
    // MFMA pipe is busy while the waves meet.  PF (compile time) says where
    // block kt + STAGES - 1 comes from: 1 this item (the main loop, no
    // per-DMA branch), 2 the next item if there is one, else nowhere (the
    // last STAGES - 1 blocks; a wave-uniform branch).
    auto step = [&](FragT (&Fc)[NF], FragT (&Fn)[NF], int kt, int ks, auto PF) {
      constexpr int pf = decltype(PF)::value;
      const bool more = ks < KS - 1 || kt + 1 < KT;
      const int rkt = ks < KS - 1 ? kt : kt + 1, rks = ks < KS - 1 ? ks + 1 : 0;
#pragma unroll
      for (int q = 0; q < MPS; ++q) {
        const int i = q / TN, jn = q % TN;
        if constexpr (F8)
          acc[i][jn] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(Fc[i], Fc[TM + jn], acc[i][jn],
                                                                       0, 0, 0, 127, 0, 127);
        else if constexpr (M16)
          acc[i][jn] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(Fc[i], Fc[TM + jn], acc[i][jn], 0, 0, 0);
        else
          acc[i][jn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(Fc[i], Fc[TM + jn], acc[i][jn], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
        if (q == 0 && ks == KS - 1 && kt + 1 < KT) {
          // block kt+1 has landed once at most the DMAs issued after it
          // (blocks kt+2 .. kt+STAGES-1, of this item or the next) remain;
          // with nothing prefetched, fewer were issued and the wait is complete
          wait_lgkm0();
          if (pf == 1 || has_next)
            wait_vmcnt<(STAGES - 2) * NLD>();
          else
            wait_vmcnt<0>();
          barrier_nofence();
          __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int r = 0; r < NF; ++r)
          if (q == read_slot(r) && more) read_one(Fn, rkt, rks, r);
        if (ks < DSTEPS) {
#pragma unroll
          for (int u = 0; u < DPQ; ++u) {
            const int dl = q * DPQ + u;
            const int d = ks * DPS + dl;
            if (dl < DPS && d < NLD) {
              if constexpr (pf == 1) dma_cur(d, kt + STAGES - 1);
              if constexpr (pf == 2)
                if (has_next) dma_nxt(d, kt + STAGES - 1);
            }
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    };

    // prologue: blocks 0 .. STAGES-2 in flight (issued here, or by the last
    // blocks of the item before), then block 0's first fragments
    if (!primed) {
#pragma unroll
      for (int i = 0; i < NLD; ++i) dma_cur(i, 0);
      if (KT >= STAGES - 1) {
#pragma unroll
        for (int b = 1; b < STAGES - 1; ++b)
#pragma unroll
          for (int i = 0; i < NLD; ++i) dma_cur(i, b);
        wait_vmcnt<(STAGES - 2) * NLD>();
      } else {
        for (int b = 1; b < KT; ++b)
#pragma unroll
          for (int i = 0; i < NLD; ++i) dma_cur(i, b);
        wait_vmcnt<0>();
      }
    } else {
      // DMAs issued after block 0's: blocks 1 .. STAGES-2, then the
      // previous epilogue's stores
      wait_vmcnt<(STAGES - 2) * NLD>();
    }
    barrier_nofence();
    read_step(Fa, 0, 0);
    auto run_block = [&](int kt, auto PF) {
#pragma unroll
      for (int ks = 0; ks < KS; ks += 2) {
        step(Fa, Fb, kt, ks, PF);
        step(Fb, Fa, kt, ks + 1, PF);
      }
    };
    const int kt_pf = KT - (STAGES - 1);   // blocks that prefetch from this item
    for (int kt = 0; kt < kt_pf; ++kt) run_block(kt, std::integral_constant<int, 1>{});
    if (has_next) decode(xcd_base + jnext, itN, srcN, bsrcN);
    for (int kt = kt_pf < 0 ? 0 : kt_pf; kt < KT; ++kt)
      run_block(kt, std::integral_constant<int, 2>{});

    // Epilogue; F8 applies the row and column scales.
    float sbg[F8 ? TN : 1];
    if constexpr (F8) {
      for (int r = tid; r < BM; r += NT) {
        int m = m0 + r;
        if (m >= rows_g) m = rows_g - 1;
        const int grow = row_base + m;
        const int64_t sr = (MODE == MODE_GATEUP && rows) ? (int64_t)rows[grow] : (int64_t)grow;
        s_sa[r] = sA[sr];
      }
      const float* sBg = sB + (size_t)g * ((MODE == MODE_GATEUP) ? 2 * NOUT : NOUT);
#pragma unroll
      for (int jn = 0; jn < TN; ++jn) {
        int col;
        if (MODE == MODE_GATEUP)
          col = (jn < TN / 2) ? n0 + wn * (WTN / 2) + jn * 32
                              : NOUT + n0 + wn * (WTN / 2) + (jn - TN / 2) * 32;
        else
          col = n0 + wn * WTN + jn * 32;
        sbg[jn] = sBg[col + (lane & 31)];
      }
    }
    if constexpr (SPL) {
      // split K: this slice's fp32 partial, straight from the accumulators
      // (32 consecutive columns per row and accumulator element)
      if constexpr (F8) __syncthreads();   // s_sa
      const int W = (MODE == MODE_GATEUP) ? 2 * NOUT : NOUT;
      float* Ps = P + (size_t)ksl * m_total * W;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int v = 0; v < AV; ++v) {
          const int r = wm * WTM + i * FR +
                        (M16 ? 4 * (lane >> 4) + v : 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3));
          if (m0 + r >= rows_g) continue;
          const float sa = F8 ? s_sa[r] : 1.f;
          float* prow = Ps + (size_t)(row_base + m0 + r) * W;
#pragma unroll
          for (int jn = 0; jn < TN; ++jn) {
            int col;
            if (MODE == MODE_GATEUP)
              col = (jn < TN / 2) ? n0 + wn * (WTN / 2) + jn * FR
                                  : NOUT + n0 + wn * (WTN / 2) + (jn - TN / 2) * FR;
            else
              col = n0 + wn * WTN + jn * FR;
            float y = acc[i][jn][v];
            if constexpr (F8) y = y * sa * sbg[jn];
            prow[col + (lane & (FR - 1))] = y;
          }
        }
      // the next tile's prologue refills ring slots that slower waves may
      // still be reading in their last steps (and F8 rewrites s_sa)
      __syncthreads();
      continue;
    }
    // staged rows: wave row wm's accumulator rows [p IPP, (p + 1) IPP) at
    // staged rows [wm IPP 32, (wm + 1) IPP 32)
    bf16_t* Cs = reinterpret_cast<bf16_t*>(ring + (XT ? slot_of(KT - 1) * STAGE : 0));
#pragma unroll
    for (int p = 0; p < TU / IPP; ++p) {
      __syncthreads();
#pragma unroll
      for (int ii = 0; ii < IPP; ++ii) {
#pragma unroll
        for (int sb = 0; sb < BPU; ++sb) {
          const int i = (p * IPP + ii) * BPU + sb;
#pragma unroll
          for (int v = 0; v < AV; ++v) {
            const int rr = M16 ? sb * 16 + 4 * (lane >> 4) + v
                               : 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
            const int r = wm * WTM + (p * IPP + ii) * 32 + rr;   // tile row
            const int sr = wm * (IPP * 32) + ii * 32 + rr;      // staged row
            const float sa = F8 ? s_sa[r] : 1.f;
            if (MODE == MODE_GATEUP) {
#pragma unroll
              for (int jn = 0; jn < TN / 2; ++jn) {
                float gt = acc[i][jn][v], up = acc[i][jn + TN / 2][v];
                if constexpr (F8) {
                  gt = gt * sa * sbg[jn];
                  up = up * sa * sbg[jn + TN / 2];
                }
                const int col = wn * (WTN / 2) + jn * FR + (lane & (FR - 1));
                Cs[sr * SST + col] = f2bf(swiglu_bf16_epi(gt, up));
              }
            } else {
#pragma unroll
              for (int jn = 0; jn < TN; ++jn) {
                const int col = wn * WTN + jn * FR + (lane & (FR - 1));
                float y = acc[i][jn][v];
                if constexpr (F8) y = y * sa * sbg[jn];
                Cs[sr * SST + col] = f2bf(y);
              }
            }
          }
        }
      }
      __syncthreads();
      constexpr int CPRC = NCOL / 8;   // 16-byte chunks per staged row
#pragma unroll 4
      for (int c = tid; c < SROWS * CPRC; c += NT) {
        const int sr = c / CPRC, ch = c % CPRC;
        const int r = (sr / (IPP * 32)) * WTM + p * IPP * 32 + sr % (IPP * 32);
        const int m = m0 + r;
        if (m < rows_g) {
          const int grow = row_base + m;
          const int64_t orow = (MODE == MODE_DOWN && rows) ? (int64_t)rows[grow] : (int64_t)grow;
          st16(C + orow * ldc + n0 + ch * 8, *reinterpret_cast<const uint4*>(Cs + sr * SST + ch * 8));
        }
      }
    }
    __syncthreads();
    if constexpr (XT) {
      sb = (sb + KT) % STAGES;
      primed = has_next;
    }
  }
}

// ---------------------------------------------------------------- bf16 MFMA, fragment-ordered weights
// Expert weights stored in MFMA fragment order (one 1 KB block per 32 rows x
// 16 k: lane l's 16 bytes are row l % 32, k 8 (l / 32) .. + 7, the B operand
// of v_mfma_f32_32x32x16_bf16) stream from HBM straight into registers: a
// load instruction reads 1 KB contiguously and a wave reads one 32-row
// group's whole K range in address order, so the weights never pass
// through LDS.  Only the activation rows (64 per tile, gathered) are staged,
// by direct global->LDS DMAs in a three-slot ring.  For groups of few rows
// (decode), where the pass streams every active expert's weights once and is
// bound by HBM.
//
// Tile: 64 rows x (gate/up: 128 H columns, wave w the gate group and the up
// group of columns 32 w .. 32 w + 31; down: 256 output columns, wave w two
// 32-column groups).  Weight blocks of 64 k go two blocks ahead of the
// MFMAs (three register slots of 32 VGPRs), activation blocks two ahead.
// The persistent grid walks (group, n-tile, m-tile; m fastest) in eight
// contiguous XCD ranges, as the LDS-ring kernels do: m-tiles of one weight
// panel run together under one L2.
//
// F8: E4M3 codes on v_mfma_scale_f32_32x32x64_f8f6f4 (unit block scales).
// A fragment is 32 rows x 64 k (2 KB), lane l's 32 bytes being row l % 32,
// k 32 (l / 32) .. + 31 of the step (the lane split of the LDS-ring FP8
// kernel, so the MFMAs see the same operands); stored as two 1 KB halves,
// half h holding bytes 16 h .. 16 h + 15 of every lane's 32, so each load
// still reads 1 KB contiguously.  A block is 128 k (a staged activation row
// is still 128 bytes) in two steps; a block's weight bytes, loads and MFMA
// time equal bf16's.  The epilogue applies the row scales of the
// activations and the column scales of the weights, as the LDS-ring kernel
// does.
constexpr int kFoBM = 64;

// One 32-row weight group: 32 rows x K of 1- or 2-byte elements.
template <typename TE>
__device__ __forceinline__ const TE* fo_group(const TE* Wg, int K, int grp) {
  return Wg + (size_t)grp * 32 * K;
}

template <int MODE, bool F8 = false>
__global__ __launch_bounds__(256) void gemm_bf16_fo_kernel(
    const typename std::conditional<F8, uint8_t, bf16_t>::type* __restrict__ A,
    const int32_t* __restrict__ rows, const int32_t* __restrict__ goff, int G, int64_t m_total,
    const typename std::conditional<F8, uint8_t, bf16_t>::type* __restrict__ Bfo, int K, int NOUT,
    bf16_t* __restrict__ C, int ldc, const float* __restrict__ sA, const float* __restrict__ sB) {
  using TE = typename std::conditional<F8, uint8_t, bf16_t>::type;
  using FragT = typename std::conditional<F8, int32x8, bf16x8>::type;
  constexpr int BM = kFoBM, NT = 256, TM = BM / 32, NST = 3;
  constexpr int KB = F8 ? 128 : 64;                  // K elements per block (128 bytes)
  constexpr int KS = F8 ? 2 : 4;                     // MFMA steps per block
  constexpr int CE = F8 ? 16 : 8;                    // elements per 16 bytes
  constexpr int ROWB = 128, ASTAGE = BM * ROWB;
  constexpr int ALD = BM * ROWB / 1024 / 4;          // 1 KB DMAs per wave per block
  constexpr int NB = 8;                              // 1 KB weight loads per wave per block
  constexpr int LPS = F8 ? 4 : 3;                    // weight loads issued per step
  constexpr int WAITN = ALD + (NB < LPS * (KS - 1) ? NB : LPS * (KS - 1));
  constexpr int NCOL = (MODE == MODE_GATEUP) ? 128 : 256;
  __shared__ int s_goff[kMaxGroups + 1];
  __shared__ int s_tpre[kMaxGroups + 1];
  __shared__ int s_wtot[NT / 64];
  __shared__ __align__(1024) unsigned char ring[NST * ASTAGE];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  sched_setup<NT, BM>(goff, G, m_total, s_goff, s_tpre, s_wtot);

  const int nn = NOUT / NCOL;
  const int64_t total = (int64_t)nn * s_tpre[G];
  // as many workgroups as give every one the same number of tiles (within
  // one per XCD range): the tile count is known only here, and a part-full
  // last round streams no faster than a full one
  const int64_t rounds = (total + gridDim.x - 1) / gridDim.x;
  int64_t eff = rounds > 0 ? (total + rounds - 1) / rounds : (int64_t)gridDim.x;
  eff = (eff + kXcd - 1) / kXcd * kXcd;
  if (eff > (int64_t)gridDim.x) eff = gridDim.x;
  if ((int64_t)blockIdx.x >= eff) return;   // a whole workgroup, before any barrier below
  const int64_t per_xcd = (total + kXcd - 1) / kXcd;
  const int64_t xcd_base = (int64_t)(blockIdx.x % kXcd) * per_xcd;
  const int64_t stride = eff / kXcd;
  const int KT = K / KB;
  const size_t bstride = (size_t)((MODE == MODE_GATEUP) ? 2 * NOUT : NOUT) * K;
  const int drow = lane / 8, dpos = lane % 8;
  const unsigned ring_lds = lds_addr(ring);
  const unsigned wave_u = __builtin_amdgcn_readfirstlane(wave);
  int aoff[TM], asw[TM];
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int r = i * 32 + (lane & 31);
    aoff[i] = r * ROWB;
    asw[i] = (r >> 1) & 7;
  }
  int ghint = 0;

  for (int64_t j = blockIdx.x / kXcd; j < per_xcd; j += stride) {
    const int64_t L = xcd_base + j;
    if (L >= total) break;
    const int g = find_group_from(s_tpre, G, nn, L, ghint);
    ghint = g;
    const int Tg = s_tpre[g + 1] - s_tpre[g];
    const int local = (int)(L - (int64_t)nn * s_tpre[g]);
    const int nt = local / Tg;
    const int m0 = (local - nt * Tg) * BM, n0 = nt * NCOL;
    const int row_base = s_goff[g], rows_g = s_goff[g + 1] - row_base;
    const TE* Bg = Bfo + (size_t)g * bstride;
    // activation rows of this wave's DMAs (rows past the group's end load
    // its last row; their results are not stored)
    const TE* asrc[ALD];
#pragma unroll
    for (int i = 0; i < ALD; ++i) {
      const int r = (wave * ALD + i) * 8 + drow;
      int m = m0 + r;
      if (m >= rows_g) m = rows_g - 1;
      const int grow = row_base + m;
      const int64_t sr = (MODE == MODE_GATEUP && rows) ? (int64_t)rows[grow] : (int64_t)grow;
      asrc[i] = A + sr * K + ((dpos ^ ((r >> 1) & 7)) * CE);
    }
    // this wave's two 32-row weight groups
    const TE* bsrc[2];
    if (MODE == MODE_GATEUP) {
      bsrc[0] = fo_group(Bg, K, n0 / 32 + wave) + lane * CE;
      bsrc[1] = fo_group(Bg, K, (NOUT + n0) / 32 + wave) + lane * CE;
    } else {
      bsrc[0] = fo_group(Bg, K, n0 / 32 + 2 * wave) + lane * CE;
      bsrc[1] = fo_group(Bg, K, n0 / 32 + 2 * wave + 1) + lane * CE;
    }
    auto dA = [&](int kt, int i) __attribute__((always_inline)) {
      dma16_at(asrc[i] + (size_t)kt * KB,
               ring_lds + (unsigned)((kt % NST) * ASTAGE) + (wave_u * ALD + i) * 1024u);
    };
    floatx16 acc[TM][2];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][t][v] = 0.f;
    // weight load q of a block: group q & 1; bf16 step q >> 1; F8 step
    // q >> 2, half (q >> 1) & 1 (1 KB pieces of the group, in address order)
    int4 Bf[3][NB];
    FragT Fa[2][TM];
    auto gB = [&](int slot, int kt, int q) __attribute__((always_inline)) {
      const size_t piece = F8 ? ((size_t)kt * KS + (q >> 2)) * 2 + ((q >> 1) & 1)
                              : (size_t)kt * KS + (q >> 1);
      // (FP8 down passes keep ordinary loads: 86.6 -> 90.8 us with the hint)
      const TE* p = bsrc[q & 1] + piece * (1024 / sizeof(TE));
      if constexpr (F8 && MODE == MODE_DOWN)
        Bf[slot][q] = *reinterpret_cast<const int4*>(p);
      else
        Bf[slot][q] = ld_stream<int4>(p);
    };
    auto bfrag = [&](int slot, int ks, int t) __attribute__((always_inline)) {
      if constexpr (F8) {
        const int4 lo = Bf[slot][(ks << 2) | t], hi = Bf[slot][(ks << 2) | 2 | t];
        return int32x8{lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
      } else {
        return __builtin_bit_cast(bf16x8, Bf[slot][2 * ks + t]);
      }
    };
    auto rA = [&](int buf, int kt, int ks, int i) __attribute__((always_inline)) {
      const unsigned char* sl = ring + (kt % NST) * ASTAGE;
      if constexpr (F8) {
        const int c = ks * 4 + 2 * (lane >> 5);
        const int4 lo = *reinterpret_cast<const int4*>(sl + aoff[i] + ((c ^ asw[i]) << 4));
        const int4 hi = *reinterpret_cast<const int4*>(sl + aoff[i] + (((c + 1) ^ asw[i]) << 4));
        Fa[buf][i] = int32x8{lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
      } else {
        const int c = ks * 2 + (lane >> 5);
        Fa[buf][i] = *reinterpret_cast<const bf16x8*>(sl + aoff[i] + ((c ^ asw[i]) << 4));
      }
    };
    // prologue: activation blocks 0 and 1, weight blocks 0 and 1
#pragma unroll
    for (int i = 0; i < ALD; ++i) dA(0, i);
#pragma unroll
    for (int q = 0; q < NB; ++q) gB(0, 0, q);
    if (KT > 1) {
#pragma unroll
      for (int i = 0; i < ALD; ++i) dA(1, i);
#pragma unroll
      for (int q = 0; q < NB; ++q) gB(1, 1, q);
    }
    wait_vmcnt<0>();
    barrier_nofence();
#pragma unroll
    for (int i = 0; i < TM; ++i) rA(0, 0, 0, i);
    // block kt: weights from slot kt % 3; issues the DMAs of activation block
    // kt + 2 (step 0) and the loads of weight block kt + 2 (LPS per step,
    // after the step's last MFMAs).  The last step waits for activation
    // block kt + 1: after its DMAs, only the WAITN loads of block kt + 2
    // issued before the wait may still be in flight.
    auto block = [&](int kt, auto SLOT, auto N1, auto N2) __attribute__((always_inline)) {
      constexpr int sl = decltype(SLOT)::value;
      constexpr int s2 = (sl + 2) % 3;
      const bool n1 = bool(N1), n2 = bool(N2);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int cb = ks & 1;
#pragma unroll
        for (int q = 0; q < TM * 2; ++q) {
          const int i = q >> 1, t = q & 1;
          if constexpr (F8)
            acc[i][t] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                Fa[cb][i], bfrag(sl, ks, t), acc[i][t], 0, 0, 0, 127, 0, 127);
          else
            acc[i][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(Fa[cb][i], bfrag(sl, ks, t),
                                                                acc[i][t], 0, 0, 0);
          __builtin_amdgcn_sched_barrier(0);
          if (ks == KS - 1 && q == 0 && n1) {
            wait_lgkm0();
            if (n2)
              wait_vmcnt<WAITN>();
            else
              wait_vmcnt<0>();
            barrier_nofence();
            __builtin_amdgcn_sched_barrier(0);
          }
          if (q < TM) {
            if (ks < KS - 1)
              rA(cb ^ 1, kt, ks + 1, q);
            else if (n1)
              rA(cb ^ 1, kt + 1, 0, q);
          }
          if (ks == 0 && n2 && q < ALD) dA(kt + 2, q);
          if (ks * LPS < NB && n2) {
            // weight loads LPS ks .. LPS ks + LPS - 1 of block kt + 2, after
            // the step's last MFMAs
            const int qq = LPS * ks + (q - (TM * 2 - LPS));
            if (q >= TM * 2 - LPS && qq < NB) gB(s2, kt + 2, qq);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    };
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    using T = std::true_type;
    int kt = 0;
    for (; kt + 5 <= KT; kt += 3) {
      block(kt, I0{}, T{}, T{});
      block(kt + 1, I1{}, T{}, T{});
      block(kt + 2, I2{}, T{}, T{});
    }
    // the last one to four blocks
    block(kt, I0{}, kt + 1 < KT, kt + 2 < KT);
    if (kt + 1 < KT) block(kt + 1, I1{}, kt + 2 < KT, kt + 3 < KT);
    if (kt + 2 < KT) block(kt + 2, I2{}, kt + 3 < KT, false);
    if (kt + 3 < KT) block(kt + 3, I0{}, false, false);

    // epilogue: accumulator element v of lane l is row 8 (v / 4) + 4 (l / 32)
    // + v % 4, column l % 32 of its 32 x 32 block; 32 lanes store 64
    // contiguous bytes of a row.  F8: y = acc * row scale * column scale.
    float sbc[2] = {1.f, 1.f};
    if constexpr (F8) {
      const float* sBg = sB + (size_t)g * ((MODE == MODE_GATEUP) ? 2 * NOUT : NOUT);
      if (MODE == MODE_GATEUP) {
        sbc[0] = sBg[n0 + 32 * wave + (lane & 31)];
        sbc[1] = sBg[NOUT + n0 + 32 * wave + (lane & 31)];
      } else {
        sbc[0] = sBg[n0 + 64 * wave + (lane & 31)];
        sbc[1] = sBg[n0 + 64 * wave + 32 + (lane & 31)];
      }
    }
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int m = m0 + i * 32 + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
        if (m < rows_g) {
          const int grow = row_base + m;
          float y0 = acc[i][0][v], y1 = acc[i][1][v];
          if constexpr (F8) {
            const float sa =
                sA[(MODE == MODE_GATEUP && rows) ? (int64_t)rows[grow] : (int64_t)grow];
            y0 = y0 * sa * sbc[0];
            y1 = y1 * sa * sbc[1];
          }
          if (MODE == MODE_GATEUP) {
            C[(int64_t)grow * ldc + n0 + 32 * wave + (lane & 31)] = f2bf(swiglu_bf16_epi(y0, y1));
          } else {
            const int64_t orow = rows ? (int64_t)rows[grow] : (int64_t)grow;
            C[orow * ldc + n0 + 64 * wave + (lane & 31)] = f2bf(y0);
            C[orow * ldc + n0 + 64 * wave + 32 + (lane & 31)] = f2bf(y1);
          }
        }
      }
    // the next item's prologue refills ring slots slower waves may still read
    __syncthreads();
  }
}

// Fragment order of row-major [rows, cols] matrices (rows % 32 == 0,
// cols % 16 == 0): one thread per 16-byte piece of the destination.
__global__ __launch_bounds__(256) void fragment_order_kernel(const bf16_t* __restrict__ src,
                                                             int64_t n_mats, int rows, int cols,
                                                             bf16_t* __restrict__ dst) {
  const int64_t per = (int64_t)rows * cols / 8;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n_mats * per) return;
  const int64_t mat = i / per, r = i % per;
  const int lane = (int)(r % 64);
  const int64_t chunk = r / 64;
  const int ks = (int)(chunk % (cols / 16));
  const int64_t ng = chunk / (cols / 16);
  const int64_t row = ng * 32 + lane % 32;
  const int col = ks * 16 + (lane / 32) * 8;
  reinterpret_cast<uint4*>(dst)[i] =
      *reinterpret_cast<const uint4*>(src + (mat * rows + row) * cols + col);
}

// FP8 fragment order of row-major [rows, cols] E4M3 code matrices (rows % 32
// == 0, cols % 64 == 0): [rows / 32][cols / 64][2][64][16 bytes], half h of
// lane l holding row l % 32, bytes 32 (l / 32) + 16 h .. + 15 of its 64-byte
// step.  One thread per 16-byte piece of the destination.
__global__ __launch_bounds__(256) void fragment_order_fp8_kernel(const uint8_t* __restrict__ src,
                                                                 int64_t n_mats, int rows,
                                                                 int cols,
                                                                 uint8_t* __restrict__ dst) {
  const int64_t per = (int64_t)rows * cols / 16;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n_mats * per) return;
  const int64_t mat = i / per, r = i % per;
  const int lane = (int)(r % 64), half = (int)((r / 64) % 2);
  const int64_t frag = r / 128;
  const int ks = (int)(frag % (cols / 64));
  const int64_t ng = frag / (cols / 64);
  const int64_t row = ng * 32 + lane % 32;
  const int col = ks * 64 + (lane / 32) * 32 + 16 * half;
  reinterpret_cast<uint4*>(dst)[i] =
      *reinterpret_cast<const uint4*>(src + (mat * rows + row) * cols + col);
}

// ---------------------------------------------------------------- bf16 MFMA, weight streaming
// For groups of few rows (decode), where the GEMM reads each weight once and
// is bound by HBM: one wave per workgroup owns 64 weight rows of one group
// (gate/up: 32 gate rows and the matching 32 up rows; down: 64 output
// columns) over one slice of K, for 16 * MF activation rows at a time.
// Operand fragments go straight from global memory into the registers of
// v_mfma_f32_16x16x32_bf16 (lane l holds row l % 16, K elements
// 8 * (l / 16) .. + 7 of a 32-wide step), so one load instruction reads 16
// rows x 64 contiguous bytes: whole 64-byte L2 requests, nothing re-read.
// The next 64-wide K block is always in flight.  Many small workgroups keep
// many loads in flight per CU.  With one K slice the SwiGLU / scatter
// epilogue runs here; with several, each slice stores fp32 partials
// P[slice][row][col] and stream_reduce_kernel sums them in slice order.
constexpr int kStreamWrows = 64;       // weight rows per workgroup
constexpr int kStreamMaxRows = 4096;   // larger batches use the LDS-ring kernels
// workgroups aimed for: about two waves per CU keep enough loads in flight,
// while every extra K slice adds fp32 partials of all the pass's rows
// (decode shared expert: 2048 -> 512 took gate/up 44 -> 29 us, down 33 ->
// 22 us)
constexpr int kStreamWgs = 512;
constexpr size_t kStreamPartialCap = size_t(64) << 20;
typedef float floatx4 __attribute__((ext_vector_type(4)));

template <int MODE, int MF>
__global__ __launch_bounds__(64, 2) void gemm_bf16_stream_kernel(
    const bf16_t* __restrict__ A, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ goff, int G, int64_t m_total, const bf16_t* __restrict__ B, int K,
    int NOUT, bf16_t* __restrict__ C, int ldc, float* __restrict__ P, int splits, int kb_per_split) {
  constexpr int NCOL = MODE == MODE_GATEUP ? kStreamWrows / 2 : kStreamWrows;
  constexpr int NF = kStreamWrows / 16;   // 16-row weight fragments
  constexpr int BMR = 16 * MF;            // activation rows per pass
  const int lane = threadIdx.x;
  const int n_tiles = NOUT / NCOL;
  int64_t w = blockIdx.x;
  const int sp = (int)(w % splits);
  w /= splits;
  const int nt = (int)(w % n_tiles);
  const int g = (int)(w / n_tiles);
  if (g >= G) return;
  auto clampo = [&](int v) { return v < 0 ? 0 : (v > (int)m_total ? (int)m_total : v); };
  const int row_base = clampo(goff ? goff[g] : 0);
  const int rows_g = clampo(goff ? goff[g + 1] : (int)m_total) - row_base;
  const int KT = K / 64;
  const int kb0 = sp * kb_per_split;
  const int kb1 = min(KT, kb0 + kb_per_split);
  if (rows_g <= 0 || kb0 >= kb1) return;

  const size_t bstride = (size_t)(MODE == MODE_GATEUP ? 2 * NOUT : NOUT) * K;
  const bf16_t* Bg = B + (size_t)g * bstride;
  const int q = lane >> 4, l16 = lane & 15;
  // weight fragment f: gate/up f < 2 are gate rows, f >= 2 the matching up rows
  const bf16_t* pb[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    const int wrow = MODE == MODE_GATEUP ? (f / 2) * NOUT + nt * NCOL + (f % 2) * 16 + l16
                                         : nt * NCOL + f * 16 + l16;
    pb[f] = Bg + (size_t)wrow * K + 8 * q;
  }
  for (int m0 = 0; m0 < rows_g; m0 += BMR) {
    const bf16_t* pa[MF];
#pragma unroll
    for (int i = 0; i < MF; ++i) {
      int m = m0 + i * 16 + l16;
      if (m >= rows_g) m = rows_g - 1;   // padding rows read a valid row, never stored
      const int grow = row_base + m;
      const int64_t src = (MODE == MODE_GATEUP && rows) ? (int64_t)rows[grow] : (int64_t)grow;
      pa[i] = A + src * K + 8 * q;
    }
    floatx4 acc[MF][NF];
#pragma unroll
    for (int i = 0; i < MF; ++i)
#pragma unroll
      for (int f = 0; f < NF; ++f)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[i][f][v] = 0.f;
    bf16x8 fa0[MF][2], fb0[NF][2], fa1[MF][2], fb1[NF][2];
    auto load = [&](bf16x8 (&fa)[MF][2], bf16x8 (&fb)[NF][2], int kb) {
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
#pragma unroll
        for (int f = 0; f < NF; ++f)
          fb[f][s2] = *reinterpret_cast<const bf16x8*>(pb[f] + (size_t)kb * 64 + s2 * 32);
#pragma unroll
        for (int i = 0; i < MF; ++i)
          fa[i][s2] = *reinterpret_cast<const bf16x8*>(pa[i] + (size_t)kb * 64 + s2 * 32);
      }
    };
    auto mma = [&](bf16x8 (&fa)[MF][2], bf16x8 (&fb)[NF][2]) {
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
        for (int i = 0; i < MF; ++i)
#pragma unroll
          for (int f = 0; f < NF; ++f)
            acc[i][f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[i][s2], fb[f][s2], acc[i][f], 0, 0, 0);
    };
    load(fa0, fb0, kb0);
    int kb = kb0;
    for (; kb + 2 <= kb1; kb += 2) {
      load(fa1, fb1, kb + 1);
      mma(fa0, fb0);
      if (kb + 2 < kb1) load(fa0, fb0, kb + 2);
      mma(fa1, fb1);
    }
    if (kb < kb1) mma(fa0, fb0);

    // element v of lane l: row 4 * (l / 16) + v, column l % 16 of its 16 x 16 tile
#pragma unroll
    for (int i = 0; i < MF; ++i) {
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int m = m0 + i * 16 + 4 * q + v;
        if (m >= rows_g) continue;
        const int grow = row_base + m;
        if (splits > 1) {
          float* pr = P + ((size_t)sp * m_total + grow) * (MODE == MODE_GATEUP ? 2 * NOUT : NOUT);
#pragma unroll
          for (int f = 0; f < NF; ++f) {
            const int col = MODE == MODE_GATEUP ? (f / 2) * NOUT + nt * NCOL + (f % 2) * 16 + l16
                                                : nt * NCOL + f * 16 + l16;
            pr[col] = acc[i][f][v];
          }
        } else if (MODE == MODE_GATEUP) {
#pragma unroll
          for (int f = 0; f < 2; ++f)
            C[(size_t)grow * ldc + nt * NCOL + f * 16 + l16] =
                f2bf(swiglu_bf16_epi(acc[i][f][v], acc[i][f + 2][v]));
        } else {
          const int64_t orow = rows ? (int64_t)rows[grow] : (int64_t)grow;
#pragma unroll
          for (int f = 0; f < NF; ++f) C[orow * ldc + nt * NCOL + f * 16 + l16] = f2bf(acc[i][f][v]);
        }
      }
    }
  }
}

// Sum of the split-K partials in slice order, then the pass's epilogue:
// gate/up H[r, c] = SiLU(sum gate) * (sum up); down out[row(r), c] = sum.
// One thread per output element of the rows that exist (goff[G]).
template <int MODE>
__global__ __launch_bounds__(256) void stream_reduce_kernel(
    const float* __restrict__ P, const int32_t* __restrict__ rows, const int32_t* __restrict__ goff,
    int G, int64_t m_total, int NOUT, int splits, bf16_t* __restrict__ C, int ldc) {
  int64_t m_rows = goff ? goff[G] : m_total;
  m_rows = m_rows < 0 ? 0 : (m_rows > m_total ? m_total : m_rows);
  const int W = MODE == MODE_GATEUP ? 2 * NOUT : NOUT;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < m_rows * NOUT;
       e += (int64_t)gridDim.x * 256) {
    const int64_t r = e / NOUT;
    const int c = (int)(e % NOUT);
    float a = 0.f, b = 0.f;
    for (int s = 0; s < splits; ++s) {
      const float* pr = P + ((size_t)s * m_total + r) * W;
      a += pr[c];
      if (MODE == MODE_GATEUP) b += pr[NOUT + c];
    }
    if (MODE == MODE_GATEUP) {
      C[r * ldc + c] = f2bf(swiglu_bf16_epi(a, b));
    } else {
      const int64_t orow = rows ? (int64_t)rows[r] : r;
      C[orow * ldc + c] = f2bf(a);
    }
  }
}

// ---------------------------------------------------------------- fp32 VALU
// 64 x 64 tiles, 256 threads, 4 rows x 4 columns per thread.  For gate/up a
// tile holds 32 gate and the matching 32 up columns; a thread owns 2 H
// columns (their gate and up values).
// ---------------------------------------------------------------- bf16 MFMA, skinny down pass
// The down pass of one group of at most 64 rows (a decode batch's shared
// expert): workgroup w owns 32 output columns over the whole K, so d / 32
// workgroups fill the CUs without a K split across workgroups and no fp32
// partials go through memory.  Its four waves take a quarter of K each on
// v_mfma_f32_16x16x32_bf16 (the 64 H rows as four 16-row A blocks, the 32
// weight rows as two B blocks; operand lane l: row l % 16, k 8 (l / 16) ..
// + 7 of a 32-wide step), loading both operands straight into a four-step
// register ring (weights from HBM, H from L2), and add their partial tiles
// in LDS in wave order.  Accumulator element v of lane l: row 4 (l / 16) +
// v, column l % 16.  K % 512 == 0: whole four-step rounds per wave.
// (Measured on the DeepSeek-V3-shaped decode shared expert: down 22 ->
// 17 us against the split-K streaming kernel; the same scheme for gate/up,
// 8 H columns per workgroup, was slower, 28 -> 41 us: each workgroup
// re-reads all 64 activation rows for only 16 weight rows.)
__global__ __launch_bounds__(256) void gemm_bf16_skinny_down_kernel(
    const bf16_t* __restrict__ H, const int32_t* __restrict__ rows,
    const int32_t* __restrict__ goff, int64_t m_total, const bf16_t* __restrict__ B, int K,
    int NOUT, bf16_t* __restrict__ C, int ldc) {
  constexpr int NB = 2;                              // 16-row weight fragments
  constexpr int NW = 16 * NB;                        // weight rows (output columns) per workgroup
  constexpr int D = 4;                               // register ring depth (steps)
  __shared__ float part[4][64][NW + 1];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, q = lane >> 4;
  auto clampo = [&](int v) { return v < 0 ? 0 : (v > (int)m_total ? (int)m_total : v); };
  const int row_base = clampo(goff ? goff[0] : 0);
  const int rows_g = clampo(goff ? goff[1] : (int)m_total) - row_base;
  if (rows_g <= 0) return;   // the same for the whole workgroup
  const int c0 = blockIdx.x * NW;   // first output column

  const bf16_t* pb[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) pb[j] = B + (size_t)(c0 + j * 16 + l16) * K + 8 * q;
  const bf16_t* pa[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = min(i * 16 + l16, rows_g - 1);   // padding rows read a valid row, never stored
    pa[i] = H + (int64_t)(row_base + m) * K + 8 * q;
  }
  const int kbeg = wave * (K / 4), nsteps = K / 4 / 32;   // a multiple of D
  floatx4 acc[4][NB];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) acc[i][j][v] = 0.f;
  bf16x8 ra[D][4], rb[D][NB];
  auto load = [&](int slot, int st) {
    const int k = kbeg + st * 32;
#pragma unroll
    for (int j = 0; j < NB; ++j) rb[slot][j] = *reinterpret_cast<const bf16x8*>(pb[j] + k);
#pragma unroll
    for (int i = 0; i < 4; ++i) ra[slot][i] = *reinterpret_cast<const bf16x8*>(pa[i] + k);
  };
  auto mma = [&](int slot) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ra[slot][i], rb[slot][j], acc[i][j], 0, 0, 0);
  };
  // every round but the last refills each slot right after its MFMAs
  // (unconditionally, so that each wait is for the one slot's loads only)
#pragma unroll
  for (int u = 0; u < D; ++u) load(u, u);
  for (int s0 = 0; s0 + D < nsteps; s0 += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      mma(u);
      load(u, s0 + D + u);
    }
  }
#pragma unroll
  for (int u = 0; u < D; ++u) mma(u);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) part[wave][i * 16 + 4 * q + v][j * 16 + l16] = acc[i][j][v];
  __syncthreads();
  // the four quarters' sum in wave order, scattered to the rows' slots
  for (int e = tid; e < 64 * NW; e += 256) {
    const int r = e / NW, c = e % NW;
    if (r >= rows_g) continue;
    const float y = ((part[0][r][c] + part[1][r][c]) + part[2][r][c]) + part[3][r][c];
    const int grow = row_base + r;
    const int64_t orow = rows ? (int64_t)rows[grow] : (int64_t)grow;
    C[orow * ldc + c0 + c] = f2bf(y);
  }
}

template <int MODE>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A,
                                                       const int32_t* __restrict__ rows,
                                                       const int32_t* __restrict__ goff, int G,
                                                       int64_t m_total,
                                                       const float* __restrict__ B, int K,
                                                       int NOUT, float* __restrict__ C,
                                                       int ldc) {
  constexpr int BM = 64, BN = 64, BK = 16, NT = 256;
  constexpr int NCOL = (MODE == MODE_GATEUP) ? BN / 2 : BN;
  __shared__ int s_goff[kMaxGroups + 1];
  __shared__ int s_tpre[kMaxGroups + 1];
  __shared__ int s_wtot[NT / 64];
  __shared__ __align__(16) float As[BK][BM + 4];
  __shared__ __align__(16) float Bs[BK][BN + 4];

  const int tid = threadIdx.x;
  const int tm = tid % 16, tn = tid / 16;
  sched_setup<NT, BM>(goff, G, m_total, s_goff, s_tpre, s_wtot);
  const int nn = NOUT / NCOL;
  const int64_t total = (int64_t)nn * s_tpre[G];
  const int64_t per_xcd = (total + kXcd - 1) / kXcd;
  const int64_t xcd_base = (int64_t)(blockIdx.x % kXcd) * per_xcd;
  const int64_t stride = gridDim.x / kXcd;
  const size_t bstride = (size_t)((MODE == MODE_GATEUP) ? 2 * NOUT : NOUT) * K;

  for (int64_t j = blockIdx.x / kXcd; j < per_xcd; j += stride) {
    const int64_t L = xcd_base + j;
    if (L >= total) break;
    const int g = find_group(s_tpre, G, nn, L);
    const int Tg = s_tpre[g + 1] - s_tpre[g];
    const int64_t local = L - (int64_t)nn * s_tpre[g];
    const int nt = (int)(local / Tg), mt = (int)(local % Tg);
    const int row_base = s_goff[g], rows_g = s_goff[g + 1] - row_base;
    const int m0 = mt * BM, n0 = nt * NCOL;
    const float* Bg = B + (size_t)g * bstride;

    // one 16-byte chunk of A and of B per thread per K step
    const int lr = tid / 4, lk = (tid % 4) * 4;
    const bool va = m0 + lr < rows_g;
    const int grow_l = row_base + (va ? m0 + lr : 0);
    const int64_t src = (MODE == MODE_GATEUP && rows) ? (int64_t)rows[grow_l] : (int64_t)grow_l;
    const float* pa = A + src * K + lk;
    int wrow;
    if (MODE == MODE_GATEUP)
      wrow = (lr < BN / 2) ? n0 + lr : NOUT + n0 + (lr - BN / 2);
    else
      wrow = n0 + lr;
    const float* pb = Bg + (size_t)wrow * K + lk;

    float acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[i][c] = 0.f;

    float4 ra = va ? *reinterpret_cast<const float4*>(pa) : make_float4(0, 0, 0, 0);
    float4 rb = *reinterpret_cast<const float4*>(pb);
    for (int k0 = 0; k0 < K; k0 += BK) {
      __syncthreads();
      As[lk + 0][lr] = ra.x;
      As[lk + 1][lr] = ra.y;
      As[lk + 2][lr] = ra.z;
      As[lk + 3][lr] = ra.w;
      Bs[lk + 0][lr] = rb.x;
      Bs[lk + 1][lr] = rb.y;
      Bs[lk + 2][lr] = rb.z;
      Bs[lk + 3][lr] = rb.w;
      __syncthreads();
      if (k0 + BK < K) {
        ra = va ? *reinterpret_cast<const float4*>(pa + k0 + BK) : make_float4(0, 0, 0, 0);
        rb = *reinterpret_cast<const float4*>(pb + k0 + BK);
      }
#pragma unroll
      for (int kk = 0; kk < BK; ++kk) {
        const float4 av = *reinterpret_cast<const float4*>(&As[kk][tm * 4]);
        float bv[4];
        if (MODE == MODE_GATEUP) {
          bv[0] = Bs[kk][tn * 2];
          bv[1] = Bs[kk][tn * 2 + 1];
          bv[2] = Bs[kk][BN / 2 + tn * 2];
          bv[3] = Bs[kk][BN / 2 + tn * 2 + 1];
        } else {
          const float4 b4 = *reinterpret_cast<const float4*>(&Bs[kk][tn * 4]);
          bv[0] = b4.x;
          bv[1] = b4.y;
          bv[2] = b4.z;
          bv[3] = b4.w;
        }
        const float a4[4] = {av.x, av.y, av.z, av.w};
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int c = 0; c < 4; ++c) acc[i][c] = fmaf(a4[i], bv[c], acc[i][c]);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + tm * 4 + i;
      if (m >= rows_g) continue;
      const int grow = row_base + m;
      if (MODE == MODE_GATEUP) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const float gt = acc[i][c], up = acc[i][c + 2];
          C[(size_t)grow * ldc + n0 + tn * 2 + c] = gt / (1.0f + expf(-gt)) * up;
        }
      } else {
        const int64_t orow = rows ? (int64_t)rows[grow] : (int64_t)grow;
#pragma unroll
        for (int c = 0; c < 4; ++c) C[orow * ldc + n0 + tn * 4 + c] = acc[i][c];
      }
    }
  }
}

constexpr int kBM = 128, kBN = 128, kBK = 64;

int64_t grid_for(int64_t max_rows, int G, int BM, int nn) {
  int64_t upper = (cdiv64(max_rows, BM) + G) * nn;
  upper = ((upper + kXcd - 1) / kXcd) * kXcd;
  if (upper < kXcd) upper = kXcd;
  const int64_t cap = (int64_t)kXcd * 65536;
  return upper > cap ? cap : upper;
}

int num_cus() {
  static const int cus = [] {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    return n;
  }();
  return cus;
}

// Tile variant of the LDS-ring GEMMs, per pass: the interleaved 128 x 256
// x 64 ring with eight waves (5) for every shape, except down passes whose
// output width is a multiple of 128 but not of 256 (10: 128 x 128 tiles).
// Measured against it and dropped (block steps, same box):
// - a register-staged 256 x 256 kernel on dense gate/up (Llama-4-Scout-shaped
//   shared expert 1317 -> 1232 us for the ring);
// - 256-row tiles on routed passes, whose half-empty tail tiles waste MFMA
//   work;
// - 256 x 256 tiles (eight waves of 128 x 64, two 64 KB slots, 16 x 16 x 32
//   MFMAs) on dense passes.  Alone they are faster on the DeepSeek-V3-shaped
//   shared expert (gate/up 195 -> 184 us, down 119 -> 111 us), but their
//   workgroups hold a whole CU's registers, and in the block, where the
//   shared passes run beside the Dispatch stand-in copy, the copy's cost
//   moves to whichever pass it overlaps: gate/up alone on them, 380 -> 230
//   us, shared down 133 -> 399 us, step 3.78 -> 3.93 ms.  Llama-4-Scout-shaped
//   shared gate/up (eight rounds of tiles) 1215 -> 1402 us;
// - two K groups of four waves on the 128 x 256 tile (each wave 64 x 128
//   over every other 32-wide K step, partial sums added in LDS): a quarter
//   fewer LDS fragment reads, yet Llama-4-Scout-shaped routed gate/up 1390
//   -> 1408 us, DeepSeek-V3-shaped down 977 -> 1050 us.
// nout: output columns of the pass (F for gate/up, d for down).
int tile_choice(bool down, int nout) {
  if (down && nout % 256 != 0) return 10;   // the only down variant for such widths
  return 5;
}

// occ workgroups per compute unit (capped by the tile count, a multiple of 8).
int64_t persistent_grid(int64_t max_rows, int G, int BM, int nn, int occ) {
  const int cus = num_cus();
  const int64_t upper = grid_for(max_rows, G, BM, nn);
  int64_t g = ((int64_t)cus * occ + kXcd - 1) / kXcd * kXcd;
  return g < upper ? g : upper;
}

// One bf16 GEMM pass with the LDS-ring variant v.  NCOL output columns per
// tile: BN / 2 for gate/up (a tile holds matching gate and up rows), BN for
// down.
// K split of an interleaved-ring pass: `splits` slices of `kps` K blocks
// with fp32 partials in P (splits == 1: no split).
struct KSplit {
  int splits = 1;
  int kps = 0;
  float* P = nullptr;
};

template <int MODE, int BM, int BN, int BK, int ST, int OCC, int WGM = 2, int WGN = 2,
          bool M16 = false>
void run_il(const bf16_t* A, const int32_t* rows, const int32_t* goff, int G, int64_t m_total,
            const bf16_t* B, int K, int NOUT, bf16_t* C, int ldc, hipStream_t s,
            const KSplit& sp = KSplit{}) {
  constexpr int NCOL = MODE == MODE_GATEUP ? BN / 2 : BN;
  const int64_t g = persistent_grid(m_total, G, BM, NOUT / NCOL * sp.splits, OCC);
  // (split K: the 128 x 256 ring only)
  if constexpr (BM == 128 && BN == 256) {
    if (sp.splits > 1) {
      launch_k(gemm_bf16_il_kernel<MODE, BM, BN, BK, ST, OCC, false, true, WGM, WGN, M16>, (unsigned)g,
               64 * WGM * WGN, 0, s, A, rows, goff, G, m_total, B, K, NOUT, C, ldc, nullptr, nullptr,
               sp.splits, sp.kps, sp.P);
      return;
    }
  }
  launch_k(gemm_bf16_il_kernel<MODE, BM, BN, BK, ST, OCC, false, false, WGM, WGN, M16>, (unsigned)g,
           64 * WGM * WGN, 0, s, A, rows, goff, G, m_total, B, K, NOUT, C, ldc, nullptr, nullptr, 1,
           K / BK, nullptr);
}
template <int MODE, int BM, int BN, int ST, int WGM = 2, int WGN = 2>
void run_il_f8(const uint8_t* A, const int32_t* rows, const int32_t* goff, int G, int64_t m_total,
               const uint8_t* B, int K, int NOUT, bf16_t* C, int ldc, const float* sA,
               const float* sB, hipStream_t s, const KSplit& sp) {
  constexpr int NCOL = MODE == MODE_GATEUP ? BN / 2 : BN;
  const int64_t g = persistent_grid(m_total, G, BM, NOUT / NCOL * sp.splits, 1);
  if (sp.splits > 1)
    launch_k(gemm_bf16_il_kernel<MODE, BM, BN, 128, ST, 1, true, true, WGM, WGN>, (unsigned)g,
             64 * WGM * WGN, 0, s, A, rows, goff, G, m_total, B, K, NOUT, C, ldc, sA, sB, sp.splits,
             sp.kps, sp.P);
  else
    launch_k(gemm_bf16_il_kernel<MODE, BM, BN, 128, ST, 1, true, false, WGM, WGN>, (unsigned)g,
             64 * WGM * WGN, 0, s, A, rows, goff, G, m_total, B, K, NOUT, C, ldc, sA, sB, 1, K / 128,
             nullptr);
}
// Variant 5 has BN = 256 and BK = 64: it needs NOUT % 128 == 0 for
// gate/up, NOUT % 256 == 0 for down and K % 64 == 0.  Variant 10 (down
// only) has 128 x 128 tiles for NOUT % 128 == 0.  (A K split applies to
// variant 5 only.)
template <int MODE>
void gemm_pass(int v, const bf16_t* A, const int32_t* rows, const int32_t* goff, int G,
               int64_t m_total, const bf16_t* B, int K, int NOUT, bf16_t* C, int ldc,
               hipStream_t s, const KSplit& sp = KSplit{}) {
#define FS_ARGS A, rows, goff, G, m_total, B, K, NOUT, C, ldc, s
  switch (v) {
    case 10:
      // 128 x 128 tiles, four waves of 64 x 64, four 32 KB slots
      if constexpr (MODE == MODE_DOWN) run_il<MODE, 128, 128, 64, 4, 1>(FS_ARGS);
      break;
    default: run_il<MODE, 128, 256, 64, 3, 1, 2, 4, true>(FS_ARGS, sp); break;   // 5
  }
#undef FS_ARGS
}

}  // namespace

// fp32 partials of the weight-streaming passes (shared by both passes): up
// to 32 K slices of max_rows x max(2F, d), at most kStreamPartialCap.  It
// grows with max_rows, so a workspace sized for a bound serves any smaller
// bound.
size_t stream_partial_bytes(int dtype, int64_t max_rows, int ffn, int d) {
  if (dtype != 1) return 0;
  const size_t want = (size_t)32 * max_rows * std::max(2 * ffn, d) * 4;
  return std::min(want, kStreamPartialCap);
}

// K slices of one weight-streaming pass: enough workgroups (groups x 64-row
// weight tiles x slices) to fill the chip, at least two K blocks per slice,
// and partials that fit the buffer above.
int stream_splits(int64_t max_rows, int G, int nw, int K, size_t partial_bytes) {
  const int64_t tiles = (int64_t)G * (nw / kStreamWrows);
  int64_t s = cdiv64(kStreamWgs, tiles);
  const int64_t by_k = (K / 64) / 2;
  if (s > by_k) s = by_k;
  const int64_t by_mem = (int64_t)(partial_bytes / ((size_t)(max_rows > 0 ? max_rows : 1) * nw * 4));
  if (s > by_mem) s = by_mem;
  return s < 1 ? 1 : (int)s;
}

// The streaming kernel takes a pass when its groups average at most 64 rows
// and the LDS-ring kernel's 128 x 256 tiles would not give every CU one.
bool use_stream(int dtype, int64_t max_rows, int G, int ffn, int d) {
  if (dtype != 1 || max_rows > kStreamMaxRows || max_rows > (int64_t)64 * G || ffn % 64 != 0 ||
      d % 64 != 0)
    return false;
  const int64_t ring_tiles =
      (int64_t)G * std::max<int64_t>(1, cdiv64(max_rows, (int64_t)128 * G)) * std::max(1, ffn / 128);
  return ring_tiles < 256;
}

// One FP8 GEMM pass on 128 x 256 tiles, eight waves of 64 x 64 (as bf16:
// routed gate/up of the DeepSeek-V3-shaped prefill 1000 -> 955 us, down
// 660 -> 616 us against four waves of 64 x 128).  Measured on the routed
// and dense expert shapes, 256-row FP8 tiles lose everywhere (the routed
// down pass of the 32-expert 7168-wide prefill: 817 against 760 us).
template <int MODE>
void gemm_pass_f8(const uint8_t* A, const int32_t* rows, const int32_t* goff, int G,
                  int64_t m_total, const uint8_t* B, int K, int NOUT, bf16_t* C, int ldc,
                  const float* sA, const float* sB, hipStream_t s, const KSplit& sp) {
  run_il_f8<MODE, 128, 256, 3, 2, 4>(A, rows, goff, G, m_total, B, K, NOUT, C, ldc, sA, sB, s, sp);
}

// K slices for an interleaved-ring pass with fewer tiles (BM rows x 128
// gate/up or 256 down columns, estimated from the row bound) than CUs, so
// that most CUs would idle: enough slices for about eight rounds of work
// items, at most 8, at least 4 K blocks each, partials [slices, max_rows, W]
// within pbytes.  A pass with at least one tile per CU is not split: there
// the fp32 partials and the reduction cost more than the balance gains
// (weight-streaming decode passes slow down by a sixth when split).
int ring_splits(bool gateup, int BM, int64_t max_rows, int G, int KT, int NOUT, size_t pbytes) {
  const int NCOL = gateup ? 128 : 256;
  const int64_t tiles =
      (int64_t)G * std::max<int64_t>(1, cdiv64(max_rows, (int64_t)BM * G)) * (NOUT / NCOL);
  const int64_t want = (int64_t)8 * num_cus();
  int64_t sl = tiles >= num_cus() ? 1 : std::min<int64_t>(8, cdiv64(want, tiles));
  sl = std::min<int64_t>(sl, KT / 4);
  const size_t per = (size_t)std::max<int64_t>(max_rows, 1) * (gateup ? 2 * NOUT : NOUT) * 4;
  while (sl > 1 && (size_t)sl * per > pbytes) --sl;
  return sl < 2 ? 1 : (int)sl;
}

KSplit make_split(int sl, int KT, float* P) {
  KSplit sp;
  if (sl > 1 && P) {
    sp.kps = (int)cdiv64(KT, sl);
    sp.splits = (int)cdiv64(KT, sp.kps);    // no empty slice
    sp.P = sp.splits > 1 ? P : nullptr;
    if (sp.splits < 2) sp.splits = 1;
  }
  return sp;
}

// The slices' sum, in slice order, then SwiGLU into H (gate/up) or the rows
// scattered through `rows` (down).
template <int MODE>
void reduce_split(const KSplit& sp, const int32_t* rows, const int32_t* goff, int G,
                  int64_t m_total, int NOUT, bf16_t* C, int ldc, hipStream_t s) {
  if (sp.splits < 2) return;
  launch_k(stream_reduce_kernel<MODE>, (unsigned)std::min<int64_t>(cdiv64(m_total * NOUT, 256), 8192),
           256, 0, s, (const float*)sp.P, rows, goff, G, m_total, NOUT, sp.splits, C, ldc);
}

// fp32 partials of the split interleaved-ring passes: up to 8 slices of
// max_rows x max(2F, d), at most kStreamPartialCap.
size_t split_partial_bytes(int64_t max_rows, int ffn, int d) {
  const size_t want = (size_t)8 * max_rows * std::max(2 * ffn, d) * 4;
  return std::min(want, kStreamPartialCap);
}

size_t ffn_fp8_ws_bytes(int64_t max_rows, int ffn, int d) {
  const size_t h = (size_t)max_rows * ffn;
  return (h * 2 + 255) / 256 * 256 + (h + 255) / 256 * 256 + ((size_t)max_rows * 4 + 255) / 256 * 256 +
         (split_partial_bytes(max_rows, ffn, d) + 255) / 256 * 256;
}

hipError_t launch_grouped_ffn_fp8(int G, int ffn, int d, const uint8_t* x, const float* x_scale,
                                  const int32_t* rows_in, const int32_t* rows_out,
                                  const int32_t* goff, int64_t max_rows, const uint8_t* w_gate_up,
                                  const float* s_gate_up, const uint8_t* w_down,
                                  const float* s_down, void* out, void* ws, hipStream_t s,
                                  int prof_gate_up) {
  if (max_rows <= 0) return hipSuccess;
  const bool profile = prof_gate_up >= 0;
  const size_t h = (size_t)max_rows * ffn;
  bf16_t* H = reinterpret_cast<bf16_t*>(ws);
  uint8_t* Hq = reinterpret_cast<uint8_t*>(ws) + (h * 2 + 255) / 256 * 256;
  float* Hs = reinterpret_cast<float*>(Hq + (h + 255) / 256 * 256);
  float* P = reinterpret_cast<float*>(reinterpret_cast<char*>(Hs) +
                                      ((size_t)max_rows * 4 + 255) / 256 * 256);
  const size_t pbytes = split_partial_bytes(max_rows, ffn, d);
  bf16_t* Y = static_cast<bf16_t*>(out);
  if (profile) prof_begin(prof_gate_up, s);
  {
    const KSplit sp =
        make_split(ring_splits(true, 128, max_rows, G, d / 128, ffn, pbytes), d / 128, P);
    gemm_pass_f8<MODE_GATEUP>(x, rows_in, goff, G, max_rows, w_gate_up, d, ffn, H, ffn,
                              x_scale, s_gate_up, s, sp);
    reduce_split<MODE_GATEUP>(sp, rows_in, goff, G, max_rows, ffn, H, ffn, s);
  }
  if (profile) prof_end(prof_gate_up, s);
  if (profile) prof_begin(prof_gate_up + 1, s);
  hipError_t e = launch_quantize_fp8(1, H, max_rows, ffn, goff ? goff + G : nullptr, Hq, Hs, s);
  if (e != hipSuccess) return e;
  {
    const KSplit sp = make_split(ring_splits(false, 128, max_rows, G, ffn / 128, d, pbytes),
                                 ffn / 128, P);
    gemm_pass_f8<MODE_DOWN>(Hq, rows_out, goff, G, max_rows, w_down, ffn, d, Y, d, Hs, s_down,
                            s, sp);
    reduce_split<MODE_DOWN>(sp, rows_out, goff, G, max_rows, d, Y, d, s);
  }
  if (profile) prof_end(prof_gate_up + 1, s);
  return hipGetLastError();
}

size_t ffn_ws_bytes(int dtype, int64_t max_rows, int ffn, int d) {
  const size_t h = (size_t)max_rows * ffn * (dtype == 0 ? 4 : 2);
  return (h + 255) / 256 * 256 + (stream_partial_bytes(dtype, max_rows, ffn, d) + 255) / 256 * 256;
}

hipError_t launch_grouped_ffn(int dtype, int G, int ffn, int d, const void* in,
                              const int32_t* rows_in, const int32_t* rows_out,
                              const int32_t* goff, int64_t max_rows,
                              const void* w_gate_up, const void* w_down, void* out, void* ws,
                              hipStream_t s, int prof_gate_up) {
  const bool profile = prof_gate_up >= 0;
  const int pg = prof_gate_up, pd = prof_gate_up + 1;
  if (max_rows <= 0) return hipSuccess;
  if (use_stream(dtype, max_rows, G, ffn, d)) {
    bf16_t* H = reinterpret_cast<bf16_t*>(ws);
    float* P = reinterpret_cast<float*>(reinterpret_cast<char*>(ws) +
                                        ((size_t)max_rows * ffn * 2 + 255) / 256 * 256);
    const size_t pbytes = stream_partial_bytes(dtype, max_rows, ffn, d);
    // 64 activation rows per pass when the groups average more than 32
    const bool wide = max_rows > (int64_t)32 * G;
    // gate/up: 32 H columns per workgroup; down: 64 output columns
    {
      const int kt = d / 64, sp = stream_splits(max_rows, G, 2 * ffn, d, pbytes);
      const int kps = (int)cdiv64(kt, sp), spe = (int)cdiv64(kt, kps);
      if (profile) prof_begin(pg, s);
      const unsigned grid = (unsigned)((int64_t)G * (ffn / 32) * spe);
      if (wide)
        launch_k(gemm_bf16_stream_kernel<MODE_GATEUP, 4>, grid, 64, 0, s,
            (const bf16_t*)in, rows_in, goff, G, max_rows, (const bf16_t*)w_gate_up, d, ffn, H, ffn,
            P, spe, kps);
      else
        launch_k(gemm_bf16_stream_kernel<MODE_GATEUP, 2>, grid, 64, 0, s,
            (const bf16_t*)in, rows_in, goff, G, max_rows, (const bf16_t*)w_gate_up, d, ffn, H, ffn,
            P, spe, kps);
      if (spe > 1)
        launch_k(stream_reduce_kernel<MODE_GATEUP>,
                 (unsigned)std::min<int64_t>(cdiv64(max_rows * ffn, 256), 8192), 256, 0, s, P,
                 rows_in, goff, G, max_rows, ffn, spe, H, ffn);
      if (profile) prof_end(pg, s);
    }
    // one group of at most 64 rows: the skinny down pass where K allows it
    if (G == 1 && max_rows <= 64 && ffn % 512 == 0 && d % 32 == 0) {
      if (profile) prof_begin(pd, s);
      launch_k(gemm_bf16_skinny_down_kernel, (unsigned)(d / 32), 256, 0, s, H, rows_out, goff,
               max_rows, (const bf16_t*)w_down, ffn, d, (bf16_t*)out, d);
      if (profile) prof_end(pd, s);
    } else {
      const int kt = ffn / 64, sp = stream_splits(max_rows, G, d, ffn, pbytes);
      const int kps = (int)cdiv64(kt, sp), spe = (int)cdiv64(kt, kps);
      if (profile) prof_begin(pd, s);
      const unsigned grid = (unsigned)((int64_t)G * (d / 64) * spe);
      if (wide)
        launch_k(gemm_bf16_stream_kernel<MODE_DOWN, 4>, grid, 64, 0, s, H, rows_out, goff, G,
                 max_rows, (const bf16_t*)w_down, ffn, d, (bf16_t*)out, d, P, spe, kps);
      else
        launch_k(gemm_bf16_stream_kernel<MODE_DOWN, 2>, grid, 64, 0, s, H, rows_out, goff, G,
                 max_rows, (const bf16_t*)w_down, ffn, d, (bf16_t*)out, d, P, spe, kps);
      if (spe > 1)
        launch_k(stream_reduce_kernel<MODE_DOWN>,
                 (unsigned)std::min<int64_t>(cdiv64(max_rows * d, 256), 8192), 256, 0, s, P,
                 rows_out, goff, G, max_rows, d, spe, (bf16_t*)out, d);
      if (profile) prof_end(pd, s);
    }
  } else if (dtype == 1 && ffn % 128 == 0 && d % 256 == 0) {
    bf16_t* H = reinterpret_cast<bf16_t*>(ws);
    float* P = reinterpret_cast<float*>(reinterpret_cast<char*>(ws) +
                                        ((size_t)max_rows * ffn * 2 + 255) / 256 * 256);
    const size_t pbytes = stream_partial_bytes(dtype, max_rows, ffn, d);
    auto split_of = [&](int v, bool gateup, int K, int NOUT) {
      if (v != 5) return KSplit{};
      return make_split(ring_splits(gateup, 128, max_rows, G, K / 64, NOUT, pbytes), K / 64, P);
    };
    if (profile) prof_begin(pg, s);
    {
      const int v = tile_choice(false, ffn);
      const KSplit sp = split_of(v, true, d, ffn);
      gemm_pass<MODE_GATEUP>(v, (const bf16_t*)in, rows_in, goff, G, max_rows,
                             (const bf16_t*)w_gate_up, d, ffn, H, ffn, s, sp);
      reduce_split<MODE_GATEUP>(sp, rows_in, goff, G, max_rows, ffn, H, ffn, s);
    }
    if (profile) prof_end(pg, s);
    if (profile) prof_begin(pd, s);
    {
      const int v = tile_choice(true, d);
      const KSplit sp = split_of(v, false, ffn, d);
      gemm_pass<MODE_DOWN>(v, H, rows_out, goff, G, max_rows, (const bf16_t*)w_down, ffn, d,
                           (bf16_t*)out, d, s, sp);
      reduce_split<MODE_DOWN>(sp, rows_out, goff, G, max_rows, d, (bf16_t*)out, d, s);
    }
    if (profile) prof_end(pd, s);
  } else if (dtype == 1) {
    bf16_t* H = reinterpret_cast<bf16_t*>(ws);
    const int64_t g1 = grid_for(max_rows, G, kBM, ffn / (kBN / 2));
    if (profile) prof_begin(pg, s);
    launch_k(gemm_bf16_kernel<MODE_GATEUP, kBM, kBN, kBK, 2, 2>, (unsigned)g1, 256, 0, s,
        (const bf16_t*)in, rows_in, goff, G, max_rows, (const bf16_t*)w_gate_up, d, ffn, H, ffn);
    if (profile) prof_end(pg, s);
    const int64_t g2 = grid_for(max_rows, G, kBM, d / kBN);
    if (profile) prof_begin(pd, s);
    launch_k(gemm_bf16_kernel<MODE_DOWN, kBM, kBN, kBK, 2, 2>, (unsigned)g2, 256, 0, s,
        H, rows_out, goff, G, max_rows, (const bf16_t*)w_down, ffn, d, (bf16_t*)out, d);
    if (profile) prof_end(pd, s);
  } else {
    float* H = reinterpret_cast<float*>(ws);
    const int64_t g1 = grid_for(max_rows, G, 64, ffn / 32);
    if (profile) prof_begin(pg, s);
    launch_k(gemm_f32_kernel<MODE_GATEUP>, (unsigned)g1, 256, 0, s,
        (const float*)in, rows_in, goff, G, max_rows, (const float*)w_gate_up, d, ffn, H, ffn);
    if (profile) prof_end(pg, s);
    const int64_t g2 = grid_for(max_rows, G, 64, d / 64);
    if (profile) prof_begin(pd, s);
    launch_k(gemm_f32_kernel<MODE_DOWN>, (unsigned)g2, 256, 0, s,
        H, rows_out, goff, G, max_rows, (const float*)w_down, ffn, d, (float*)out, d);
    if (profile) prof_end(pd, s);
  }
  return hipGetLastError();
}

hipError_t launch_fragment_order(const void* src, int64_t n_mats, int rows, int cols, void* dst,
                                 hipStream_t s) {
  const int64_t n = n_mats * rows * (int64_t)cols / 8;
  if (n == 0) return hipSuccess;
  launch_k(fragment_order_kernel, (unsigned)cdiv64(n, 256), 256, 0, s, (const bf16_t*)src, n_mats,
           rows, cols, (bf16_t*)dst);
  return hipGetLastError();
}

hipError_t launch_grouped_ffn_fo(int G, int ffn, int d, const void* in, const int32_t* rows_in,
                                 const int32_t* rows_out, const int32_t* goff, int64_t max_rows,
                                 const void* w_gate_up_fo, const void* w_down_fo, void* out,
                                 void* ws, hipStream_t s, int prof_gate_up) {
  if (max_rows <= 0) return hipSuccess;
  const bool profile = prof_gate_up >= 0;
  bf16_t* H = reinterpret_cast<bf16_t*>(ws);
  // one workgroup per CU at most (streaming from HBM gains nothing from a
  // second: measured on 26 experts x 4096 x 7168, 208 workgroups stream at
  // 5.9 TB/s, 416 at 5.4)
  auto grid = [&](int ncol, int nout) {
    int64_t g = grid_for(max_rows, G, kFoBM, nout / ncol);
    const int64_t cap = (int64_t)num_cus() / kXcd * kXcd;
    return (unsigned)(g < cap ? g : cap);
  };
  if (profile) prof_begin(prof_gate_up, s);
  launch_k(gemm_bf16_fo_kernel<MODE_GATEUP>, grid(128, ffn), 256, 0, s, (const bf16_t*)in,
           rows_in, goff, G, max_rows, (const bf16_t*)w_gate_up_fo, d, ffn, H, ffn,
           (const float*)nullptr, (const float*)nullptr);
  if (profile) prof_end(prof_gate_up, s);
  if (profile) prof_begin(prof_gate_up + 1, s);
  launch_k(gemm_bf16_fo_kernel<MODE_DOWN>, grid(256, d), 256, 0, s, (const bf16_t*)H, rows_out,
           goff, G, max_rows, (const bf16_t*)w_down_fo, ffn, d, (bf16_t*)out, d,
           (const float*)nullptr, (const float*)nullptr);
  if (profile) prof_end(prof_gate_up + 1, s);
  return hipGetLastError();
}

hipError_t launch_fragment_order_fp8(const uint8_t* src, int64_t n_mats, int rows, int cols,
                                     uint8_t* dst, hipStream_t s) {
  const int64_t n = n_mats * rows * (int64_t)cols / 16;
  if (n == 0) return hipSuccess;
  launch_k(fragment_order_fp8_kernel, (unsigned)cdiv64(n, 256), 256, 0, s, src, n_mats, rows, cols,
           dst);
  return hipGetLastError();
}

hipError_t launch_grouped_ffn_fo_fp8(int G, int ffn, int d, const uint8_t* x, const float* x_scale,
                                     const int32_t* rows_in, const int32_t* rows_out,
                                     const int32_t* goff, int64_t max_rows,
                                     const uint8_t* w_gate_up_fo, const float* s_gate_up,
                                     const uint8_t* w_down_fo, const float* s_down, void* out,
                                     void* ws, hipStream_t s, int prof_gate_up) {
  if (max_rows <= 0) return hipSuccess;
  const bool profile = prof_gate_up >= 0;
  // the workspace of launch_grouped_ffn_fp8: H, then its codes and scales
  const size_t h = (size_t)max_rows * ffn;
  bf16_t* H = reinterpret_cast<bf16_t*>(ws);
  uint8_t* Hq = reinterpret_cast<uint8_t*>(ws) + (h * 2 + 255) / 256 * 256;
  float* Hs = reinterpret_cast<float*>(Hq + (h + 255) / 256 * 256);
  auto grid = [&](int ncol, int nout) {
    int64_t g = grid_for(max_rows, G, kFoBM, nout / ncol);
    const int64_t cap = (int64_t)num_cus() / kXcd * kXcd;
    return (unsigned)(g < cap ? g : cap);
  };
  if (profile) prof_begin(prof_gate_up, s);
  launch_k(gemm_bf16_fo_kernel<MODE_GATEUP, true>, grid(128, ffn), 256, 0, s, x, rows_in, goff, G,
           max_rows, w_gate_up_fo, d, ffn, H, ffn, x_scale, s_gate_up);
  if (profile) prof_end(prof_gate_up, s);
  if (profile) prof_begin(prof_gate_up + 1, s);
  hipError_t e = launch_quantize_fp8(1, H, max_rows, ffn, goff ? goff + G : nullptr, Hq, Hs, s);
  if (e != hipSuccess) return e;
  launch_k(gemm_bf16_fo_kernel<MODE_DOWN, true>, grid(256, d), 256, 0, s, (const uint8_t*)Hq,
           rows_out, goff, G, max_rows, w_down_fo, ffn, d, (bf16_t*)out, d, (const float*)Hs,
           s_down);
  if (profile) prof_end(prof_gate_up + 1, s);
  return hipGetLastError();
}

hipError_t launch_dense_linear(int dtype, int m, int n, int kdim, const void* a, const void* w,
                               void* out, hipStream_t s) {
  if (m <= 0) return hipSuccess;
  if (dtype == 1 && n % 128 == 0) {
    // the LDS-ring kernels as one group of m rows (128 x 128 tiles when n is
    // not a multiple of 256)
    gemm_pass<MODE_DOWN>(tile_choice(true, n), (const bf16_t*)a, nullptr, nullptr, 1,
                         m, (const bf16_t*)w, kdim, n, (bf16_t*)out, n, s);
  } else if (dtype == 1) {
    const int64_t g = grid_for(m, 1, kBM, n / kBN);
    launch_k(gemm_bf16_kernel<MODE_DOWN, kBM, kBN, kBK, 2, 2>, (unsigned)g, 256, 0, s,
        (const bf16_t*)a, nullptr, nullptr, 1, m, (const bf16_t*)w, kdim, n, (bf16_t*)out, n);
  } else {
    const int64_t g = grid_for(m, 1, 64, n / 64);
    launch_k(gemm_f32_kernel<MODE_DOWN>, (unsigned)g, 256, 0, s,
        (const float*)a, nullptr, nullptr, 1, m, (const float*)w, kdim, n, (float*)out, n);
  }
  return hipGetLastError();
}

}  // namespace fs
