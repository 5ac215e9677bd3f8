// Router scoring and top-k selection (Section 2.1: G(A) = s(A W_R^T)).
//
// Logits run on the vector ALUs in fp32 with a fixed reduction order: the
// hidden dimension is cut into 256-element slices; inside a slice the
// products are added one at a time in ascending order starting from zero;
// slice sums are added one at a time in ascending slice order starting from
// zero.  bf16 products are exact in fp32, so a fused multiply-add rounds
// like a rounded product followed by a rounded add; fp32 inputs use a
// rounded product then a rounded add (this file is compiled without
// floating-point contraction).  The order does not depend on the launch
// shape, so routing decisions are reproducible bit for bit.
//
// Top-k runs one wavefront per token: keys, optional group limit (group
// score = sum of the two largest keys, keep the best topk_groups groups,
// ties to the lower group), k rounds of a wave arg-max (ties to the lower
// expert), then gate weights.

#include <float.h>
#include <limits.h>

#include "common.hpp"
#include "internal.hpp"

namespace fs {
namespace {

constexpr int kBK = 32;  // hidden elements staged per step (divides the slice)
constexpr int kRouterSmallN = 128;  // token counts that take the 16-token tiles

template <typename T>
__device__ __forceinline__ float prod_acc(float acc, float a, float b);
template <>
__device__ __forceinline__ float prod_acc<bf16_t>(float acc, float a, float b) {
  return __builtin_fmaf(a, b, acc);
}
template <>
__device__ __forceinline__ float prod_acc<float>(float acc, float a, float b) {
  float p = a * b;
  return acc + p;
}

// Each workgroup computes a BT x BE tile of logits; each thread TT tokens x 4
// experts.  split != 0: the workgroup handles the single slice blockIdx.z
// and writes its slice sum to out[slice][N][E]; otherwise it runs every
// slice in order and writes the final logits to out[N][E].
template <typename T, int BT, int BE, int TT>
__global__ __launch_bounds__(256) void router_logits_kernel(const T* __restrict__ x,
                                                            const T* __restrict__ w, int N, int d,
                                                            int E, int split,
                                                            float* __restrict__ out) {
  constexpr int TE = 4;
  constexpr int NTG = BT / TT;
  static_assert(NTG * (BE / TE) == 256, "tile must map onto 256 threads");
  constexpr int V = 16 / sizeof(T);
  constexpr int CPR = kBK / V;                       // 16-B chunks per tile row per step
  constexpr int XCH = (BT * CPR + 255) / 256;        // x chunks per thread
  constexpr int WCH = (BE * CPR + 255) / 256;        // w chunks per thread
  __shared__ float xs[kBK][BT + 4];
  __shared__ float ws[kBK][BE + 4];

  const int tid = threadIdx.x;
  const int tg = tid % NTG, eg = tid / NTG;
  const int t0 = blockIdx.x * BT, e0 = blockIdx.y * BE;
  const int S = (d + kRouterSlice - 1) / kRouterSlice;
  const int s_begin = split ? (int)blockIdx.z : 0;
  const int s_end = split ? s_begin + 1 : S;

  // steps of this workgroup: every BK block of slices [s_begin, s_end)
  const int k_begin = s_begin * kRouterSlice;
  const int k_end = min(d, s_end * kRouterSlice);
  const int n_steps = (k_end - k_begin) / kBK;

  Vec16<T> rx[XCH], rw[WCH];
  auto load = [&](int kb) {
#pragma unroll
    for (int i = 0; i < XCH; ++i) {
      int c = tid + i * 256;
      int row = c / CPR, col = (c % CPR) * V;
      int t = t0 + row;
      rx[i].raw = make_uint4(0, 0, 0, 0);
      if (c < BT * CPR && t < N) rx[i].raw = ld16(x + (size_t)t * d + kb + col);
    }
#pragma unroll
    for (int i = 0; i < WCH; ++i) {
      int c = tid + i * 256;
      int row = c / CPR, col = (c % CPR) * V;
      int e = e0 + row;
      rw[i].raw = make_uint4(0, 0, 0, 0);
      if (c < BE * CPR && e < E) rw[i].raw = ld16(w + (size_t)e * d + kb + col);
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int i = 0; i < XCH; ++i) {
      int c = tid + i * 256;
      if (c < BT * CPR) {
        int row = c / CPR, col = (c % CPR) * V;
#pragma unroll
        for (int v = 0; v < V; ++v) xs[col + v][row] = rx[i].get(v);
      }
    }
#pragma unroll
    for (int i = 0; i < WCH; ++i) {
      int c = tid + i * 256;
      if (c < BE * CPR) {
        int row = c / CPR, col = (c % CPR) * V;
#pragma unroll
        for (int v = 0; v < V; ++v) ws[col + v][row] = rw[i].get(v);
      }
    }
  };

  float tot[TT][TE], part[TT][TE];
#pragma unroll
  for (int i = 0; i < TT; ++i)
#pragma unroll
    for (int j = 0; j < TE; ++j) tot[i][j] = part[i][j] = 0.f;

  if (n_steps > 0) load(k_begin);
  for (int st = 0; st < n_steps; ++st) {
    const int kb = k_begin + st * kBK;
    __syncthreads();
    store();
    __syncthreads();
    if (st + 1 < n_steps) load(kb + kBK);
#pragma unroll
    for (int kk = 0; kk < kBK; ++kk) {
      float xa[TT];
      if constexpr (TT == 4) {
        const float4 xv = *reinterpret_cast<const float4*>(&xs[kk][tg * TT]);
        xa[0] = xv.x, xa[1] = xv.y, xa[2] = xv.z, xa[3] = xv.w;
      } else {
#pragma unroll
        for (int i = 0; i < TT; ++i) xa[i] = xs[kk][tg * TT + i];
      }
      const float4 wv = *reinterpret_cast<const float4*>(&ws[kk][eg * TE]);
      const float wa[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
      for (int i = 0; i < TT; ++i)
#pragma unroll
        for (int j = 0; j < TE; ++j) part[i][j] = prod_acc<T>(part[i][j], xa[i], wa[j]);
    }
    // end of a slice: fold its sum in (or emit it)
    const int kn = kb + kBK;
    if (kn % kRouterSlice == 0 || kn == k_end) {
      const int slice = kb / kRouterSlice;
#pragma unroll
      for (int i = 0; i < TT; ++i) {
        const int t = t0 + tg * TT + i;
#pragma unroll
        for (int j = 0; j < TE; ++j) {
          const int e = e0 + eg * TE + j;
          if (split) {
            if (t < N && e < E) out[((size_t)slice * N + t) * E + e] = part[i][j];
          } else {
            tot[i][j] = tot[i][j] + part[i][j];
          }
          part[i][j] = 0.f;
        }
      }
    }
  }
  if (!split) {
#pragma unroll
    for (int i = 0; i < TT; ++i) {
      const int t = t0 + tg * TT + i;
#pragma unroll
      for (int j = 0; j < TE; ++j) {
        const int e = e0 + eg * TE + j;
        if (t < N && e < E) out[(size_t)t * E + e] = tot[i][j];
      }
    }
  }
}

// bf16 logits on the fp32 matrix cores.  v_mfma_f32_32x32x1_2b_f32 adds, for
// each of two 32 x 32 blocks, one product per output: d = c + a * b.  A
// bf16 product is exact in fp32, so a chain of these over ascending k is the
// same sequence of rounded adds as the vector kernel's fused multiply-adds,
// and the logits are identical bit for bit (checked on the device against
// a sequential fp32 sum); the matrix cores run fp32 at twice the rate of
// unpacked vector FMAs.  Lane layout: for block b, lanes [32b, 32b+32) give
// the rows (A) and the columns (B); accumulator element v of lane l is block
// v / 16, row 8 ((v % 16) / 4) + 4 (l / 32) + v % 4, column l % 32.
//
// A workgroup of four waves computes (32 WT) tokens x (64 WE) experts, each
// wave 32 tokens x 64 experts: A lane l holds token l % 32 of its rows (the
// same token in both halves), B lane l expert l of its columns.  The token
// and expert rows of a 64-wide K chunk are staged in LDS (128-byte rows,
// 16-byte chunk c of row r at position c ^ ((r / 2) % 8), so the 32 or 64
// rows one read touches fall in different banks) by coalesced loads one
// chunk ahead in registers, double-buffered with one barrier per chunk; a
// lane then reads its eight k of a step as one 16-byte LDS read.  (One
// buffer and two barriers per chunk measured no faster: registers, not
// LDS, bound its residency.)
typedef float floatx32 __attribute__((ext_vector_type(32)));

template <int WT, int WE, bool SPLIT>
__global__ __launch_bounds__(256) void router_mfma_kernel(const bf16_t* __restrict__ x,
                                                          const bf16_t* __restrict__ w, int N,
                                                          int d, int E, float* __restrict__ out) {
  constexpr bool split = SPLIT;
  static_assert(WT * WE == 4, "four waves");
  constexpr int BT = 32 * WT, BE = 64 * WE, ROWS = BT + BE;
  constexpr int LPT = ROWS * 8 / 256;                  // 16-byte loads per thread per chunk
  static_assert(ROWS * 8 % 256 == 0, "whole load rounds");
  __shared__ __align__(16) unsigned char sm[2][ROWS * 128];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wt = wave % WT, we = wave / WT;
  const int t0 = blockIdx.x * BT, e0 = blockIdx.y * BE;
  const int S = (d + kRouterSlice - 1) / kRouterSlice;
  const int s_begin = split ? (int)blockIdx.z : 0;
  const int s_end = split ? s_begin + 1 : S;
  const int k_begin = s_begin * kRouterSlice;
  const int k_end = min(d, s_end * kRouterSlice);
  const int nch = (k_end - k_begin) / 64;            // d % 128 == 0: whole chunks

  // staged loads: chunk q = tid + 256 i is row q / 8, 16-byte piece q % 8;
  // rows past N / E read the last valid row (their outputs are not stored)
  const bf16_t* src[LPT];
  int dst[LPT];
#pragma unroll
  for (int i = 0; i < LPT; ++i) {
    const int q = tid + 256 * i, row = q / 8, pc = q % 8;
    const bf16_t* base = row < BT ? x + (size_t)min(t0 + row, N - 1) * d
                                  : w + (size_t)min(e0 + row - BT, E - 1) * d;
    src[i] = base + k_begin + pc * 8;
    dst[i] = row * 128 + ((pc ^ ((row >> 1) & 7)) << 4);
  }
  uint4 stg[LPT];
  auto gload = [&](int c) {
#pragma unroll
    for (int i = 0; i < LPT; ++i) stg[i] = ld16(src[i] + 64 * c);
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < LPT; ++i) st16(sm[buf] + dst[i], stg[i]);
  };
  const int ra = wt * 32 + (lane & 31), rb = BT + we * 64 + lane;
  const int offa = ra * 128, swa = (ra >> 1) & 7, offb = rb * 128, swb = (rb >> 1) & 7;

  floatx32 part, tot;
#pragma unroll
  for (int v = 0; v < 32; ++v) part[v] = tot[v] = 0.f;
  auto store_out = [&](float* o, const floatx32& val) {
#pragma unroll
    for (int v = 0; v < 32; ++v) {
      const int j = v & 15;
      const int t = t0 + wt * 32 + 8 * (j >> 2) + 4 * (lane >> 5) + (j & 3);
      const int e = e0 + we * 64 + 32 * (v >> 4) + (lane & 31);
      if (t < N && e < E) o[(size_t)t * E + e] = val[v];
    }
  };

  if (nch > 0) {
    gload(0);
    lstore(0);
  }
  __syncthreads();
  for (int c = 0; c < nch; ++c) {
    if (c + 1 < nch) gload(c + 1);
    const unsigned char* sb = sm[c & 1];
    // eight k per step; the next step's operands are read during this one
    // (the scheduling barriers keep the compiler from hoisting every step's
    // reads and conversions, which would take registers from occupancy)
    uint4 ua = *reinterpret_cast<const uint4*>(sb + offa + (swa << 4));
    uint4 ub = *reinterpret_cast<const uint4*>(sb + offb + (swb << 4));
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      uint4 na = ua, nb = ub;
      if (ks < 7) {
        na = *reinterpret_cast<const uint4*>(sb + offa + (((ks + 1) ^ swa) << 4));
        nb = *reinterpret_cast<const uint4*>(sb + offb + (((ks + 1) ^ swb) << 4));
      }
      const uint32_t av[4] = {ua.x, ua.y, ua.z, ua.w}, bv[4] = {ub.x, ub.y, ub.z, ub.w};
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        part = __builtin_amdgcn_mfma_f32_32x32x1f32(__uint_as_float(av[h] << 16),
                                                    __uint_as_float(bv[h] << 16), part, 0, 0, 0);
        part = __builtin_amdgcn_mfma_f32_32x32x1f32(__uint_as_float(av[h] & 0xFFFF0000u),
                                                    __uint_as_float(bv[h] & 0xFFFF0000u), part,
                                                    0, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
      ua = na;
      ub = nb;
    }
    // end of a slice: fold its sum in (or emit it)
    const int kn = k_begin + 64 * (c + 1);
    if (kn % kRouterSlice == 0 || kn == k_end) {
      if constexpr (SPLIT) {
        store_out(out + (size_t)((kn - 1) / kRouterSlice) * N * E, part);
      } else {
#pragma unroll
        for (int v = 0; v < 32; ++v) tot[v] = tot[v] + part[v];
      }
#pragma unroll
      for (int v = 0; v < 32; ++v) part[v] = 0.f;
    }
    if (c + 1 < nch) lstore((c + 1) & 1);
    __syncthreads();
  }
  if constexpr (!SPLIT) store_out(out, tot);
}

// Routers of at most 16 experts on v_mfma_f32_16x16x1_4b_f32: four
// 16 x 16 blocks, each adding one product per output (d = c + a * b), so a
// chain over ascending k is the same sequence of rounded adds as above (bit
// for bit, checked on the device).  Lane layout: for block b, lanes
// [16b, 16b+16) give the rows (A) and the columns (B); accumulator element
// v of lane l is block v / 4, row 4 (l / 16) + v % 4, column l % 16.  A lane
// l holds token l of its wave's 64 (block b: tokens 16b .. 16b+15) and B
// lane l expert l % 16 (the same 16 experts in every block), so one
// instruction covers 64 tokens x 16 experts with no padding column.  A
// workgroup of four waves computes 256 tokens; swizzle and slice order are
// those of router_mfma_kernel, with one LDS staging buffer (the next chunk
// waits in registers), so that four workgroups fit a CU.
template <bool SPLIT>
__global__ __launch_bounds__(256) void router_mfma16_kernel(const bf16_t* __restrict__ x,
                                                            const bf16_t* __restrict__ w, int N,
                                                            int d, int E, float* __restrict__ out) {
  constexpr int BT = 256, BE = 16, ROWS = BT + BE;
  constexpr int PIECES = ROWS * 8;                     // 16-byte pieces per chunk
  constexpr int LPT = (PIECES + 255) / 256;            // loads per thread (the last partial)
  __shared__ __align__(16) unsigned char sm[ROWS * 128];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int t0 = blockIdx.x * BT;
  const int S = (d + kRouterSlice - 1) / kRouterSlice;
  const int s_begin = SPLIT ? (int)blockIdx.z : 0;
  const int s_end = SPLIT ? s_begin + 1 : S;
  const int k_begin = s_begin * kRouterSlice;
  const int k_end = min(d, s_end * kRouterSlice);
  const int nch = (k_end - k_begin) / 64;            // d % 128 == 0: whole chunks

  // staged loads: piece q = tid + 256 i is row q / 8, 16-byte piece q % 8;
  // token rows past N and expert rows past E read the last valid row
  const bf16_t* src[LPT];
  int dst[LPT];
  bool live[LPT];
#pragma unroll
  for (int i = 0; i < LPT; ++i) {
    const int q = tid + 256 * i, row = min(q / 8, ROWS - 1), pc = q % 8;
    live[i] = q < PIECES;
    const bf16_t* base = row < BT ? x + (size_t)min(t0 + row, N - 1) * d
                                  : w + (size_t)min(row - BT, E - 1) * d;
    src[i] = base + k_begin + pc * 8;
    dst[i] = row * 128 + ((pc ^ ((row >> 1) & 7)) << 4);
  }
  uint4 stg[LPT];
  auto gload = [&](int c) {
#pragma unroll
    for (int i = 0; i < LPT; ++i)
      if (live[i]) stg[i] = ld16(src[i] + 64 * c);
  };
  auto lstore = [&]() {
#pragma unroll
    for (int i = 0; i < LPT; ++i)
      if (live[i]) st16(sm + dst[i], stg[i]);
  };
  const int ra = wave * 64 + lane, rb = BT + (lane & 15);
  const int offa = ra * 128, swa = (ra >> 1) & 7, offb = rb * 128, swb = (rb >> 1) & 7;

  floatx16 part, tot;
#pragma unroll
  for (int v = 0; v < 16; ++v) part[v] = tot[v] = 0.f;
  auto store_out = [&](float* o, const floatx16& val) {
    const int e = lane & 15;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int t = t0 + wave * 64 + 16 * (v >> 2) + 4 * (lane >> 4) + (v & 3);
      if (t < N && e < E) o[(size_t)t * E + e] = val[v];
    }
  };

  if (nch > 0) {
    gload(0);
    lstore();
  }
  __syncthreads();
  for (int c = 0; c < nch; ++c) {
    if (c + 1 < nch) gload(c + 1);
    const unsigned char* sb = sm;
    uint4 ua = *reinterpret_cast<const uint4*>(sb + offa + (swa << 4));
    uint4 ub = *reinterpret_cast<const uint4*>(sb + offb + (swb << 4));
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      uint4 na = ua, nb = ub;
      if (ks < 7) {
        na = *reinterpret_cast<const uint4*>(sb + offa + (((ks + 1) ^ swa) << 4));
        nb = *reinterpret_cast<const uint4*>(sb + offb + (((ks + 1) ^ swb) << 4));
      }
      const uint32_t av[4] = {ua.x, ua.y, ua.z, ua.w}, bv[4] = {ub.x, ub.y, ub.z, ub.w};
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        part = __builtin_amdgcn_mfma_f32_16x16x1f32(__uint_as_float(av[h] << 16),
                                                    __uint_as_float(bv[h] << 16), part, 0, 0, 0);
        part = __builtin_amdgcn_mfma_f32_16x16x1f32(__uint_as_float(av[h] & 0xFFFF0000u),
                                                    __uint_as_float(bv[h] & 0xFFFF0000u), part,
                                                    0, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
      ua = na;
      ub = nb;
    }
    // end of a slice: fold its sum in (or emit it)
    const int kn = k_begin + 64 * (c + 1);
    if (kn % kRouterSlice == 0 || kn == k_end) {
      if constexpr (SPLIT) {
        store_out(out + (size_t)((kn - 1) / kRouterSlice) * N * E, part);
      } else {
#pragma unroll
        for (int v = 0; v < 16; ++v) tot[v] = tot[v] + part[v];
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) part[v] = 0.f;
    }
    // one staging buffer (34 KB, for more resident workgroups): every wave
    // has read it before the next chunk overwrites it
    __syncthreads();
    if (c + 1 < nch) lstore();
    __syncthreads();
  }
  if constexpr (!SPLIT) store_out(out, tot);
}

// The matrix-core kernels serve bf16 routers with more tokens than the
// decode-sized tiles of the vector kernel take (hidden sizes are multiples
// of 128, so slices hold whole 64-element chunks): router_mfma16_kernel up
// to 16 experts, router_mfma_kernel above.  At 64 tokens the 32-token tiles
// give too few workgroups (DeepSeek-V3-shaped decode: 19 us against 13 us on
// the vector kernel's 16-token tiles).
bool use_mfma_router(int dtype, int N, int E) { return dtype == 1 && N > kRouterSmallN; }

__device__ __forceinline__ float sigmoidf_(float z) { return 1.0f / (1.0f + expf(-z)); }

// One wavefront per token, four tokens per workgroup.  EPL experts per lane:
// lane l holds experts l, l+64, l+128, ...
template <int EPL>
__global__ __launch_bounds__(256) void topk_kernel(const float* __restrict__ src, int n_partials,
                                                   int N, int E, const float* __restrict__ bias,
                                                   int score, int k, int G, int TG, int norm,
                                                   float scale, float* __restrict__ logits_out,
                                                   int32_t* __restrict__ ids,
                                                   float* __restrict__ wout) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= N) return;  // uniform per wavefront
  const float NEG = -INFINITY;

  float z[EPL], key[EPL];
  if (n_partials == 0) {
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const int e = lane + 64 * j;
      z[j] = e < E ? src[(size_t)t * E + e] : NEG;
    }
  } else {
    // slice sums, each expert's in ascending slice order starting from zero;
    // the loads of eight slices for all EPL experts go out together
#pragma unroll
    for (int j = 0; j < EPL; ++j) z[j] = 0.f;
    int s = 0;
    for (; s + 8 <= n_partials; s += 8) {
      float p[8][EPL];
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < EPL; ++j) {
          // lanes past the last expert load the last one's and take 0
          const int e = lane + 64 * j, ec = e < E ? e : E - 1;
          const float v = src[((size_t)(s + i) * N + t) * E + ec];
          p[i][j] = e < E ? v : 0.f;
        }
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < EPL; ++j) z[j] = z[j] + p[i][j];
    }
    for (; s < n_partials; ++s)
#pragma unroll
      for (int j = 0; j < EPL; ++j) {
        const int e = lane + 64 * j, ec = e < E ? e : E - 1;
        const float v = src[((size_t)s * N + t) * E + ec];
        z[j] = z[j] + (e < E ? v : 0.f);
      }
#pragma unroll
    for (int j = 0; j < EPL; ++j)
      if (lane + 64 * j >= E) z[j] = NEG;
  }
  if (logits_out) {
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const int e = lane + 64 * j;
      if (e < E) logits_out[(size_t)t * E + e] = z[j];
    }
  }

  float zmax = NEG, sumexp = 0.f;
  if (score == 0) {
#pragma unroll
    for (int j = 0; j < EPL; ++j) zmax = fmaxf(zmax, z[j]);
    zmax = wave_max(zmax);
#pragma unroll
    for (int j = 0; j < EPL; ++j)
      if (lane + 64 * j < E) sumexp += expf(z[j] - zmax);
    sumexp = wave_sum(sumexp);
  }
#pragma unroll
  for (int j = 0; j < EPL; ++j) {
    const int e = lane + 64 * j;
    float kv = NEG;
    if (e < E) kv = (score == 0) ? z[j] : sigmoidf_(z[j]) + (bias ? bias[e] : 0.f);
    key[j] = kv;
  }

  if (G > 1) {
    const int gsz = E / G;
    // group of each of this lane's experts (E for lanes past the last)
    int grp[EPL];
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const int e = lane + 64 * j;
      grp[j] = e < E ? e / gsz : G;
    }
    float gscore = NEG;
    for (int g = 0; g < G; ++g) {
      float m1 = NEG;
      int i1 = INT_MAX;
#pragma unroll
      for (int j = 0; j < EPL; ++j) {
        // (selects, not branches: see argmax_pick)
        const int e = lane + 64 * j;
        const bool take = (grp[j] == g) & ((key[j] > m1) | ((key[j] == m1) & (e < i1)));
        m1 = take ? key[j] : m1;
        i1 = take ? e : i1;
      }
      wave_argmax(m1, i1);
      float sc = m1;
      if (gsz >= 2) {
        float m2 = NEG;
#pragma unroll
        for (int j = 0; j < EPL; ++j) {
          const int e = lane + 64 * j;
          m2 = ((grp[j] == g) & (e != i1)) ? fmaxf(m2, key[j]) : m2;
        }
        m2 = wave_max(m2);
        sc = m1 + m2;
      }
      gscore = lane == g ? sc : gscore;
    }
    uint64_t keep = 0;
    float gk = (lane < G) ? gscore : NEG;
    const int gi = (lane < G) ? lane : INT_MAX;
    for (int r = 0; r < TG; ++r) {
      float bk = gk;
      int bi = gi;
      wave_argmax(bk, bi);
      if (bi < 64) keep |= 1ull << bi;
      gk = lane == bi ? NEG : gk;
    }
#pragma unroll
    for (int j = 0; j < EPL; ++j)
      key[j] = ((grp[j] < G) & !((keep >> grp[j]) & 1ull)) ? NEG : key[j];
  }

  int my_id = 0;
  float my_w = 0.f;
  for (int r = 0; r < k; ++r) {
    float bk = NEG;
    int bi = INT_MAX;
#pragma unroll
    for (int j = 0; j < EPL; ++j) {
      const bool take = key[j] > bk;
      bk = take ? key[j] : bk;
      bi = take ? lane + 64 * j : bi;
    }
    wave_argmax(bk, bi);
    float zb = NEG;
#pragma unroll
    for (int j = 0; j < EPL; ++j) zb = lane + 64 * j == bi ? z[j] : zb;
    zb = lane_f(zb, bi & 63);
    const float base = (score == 0) ? expf(zb - zmax) / sumexp : sigmoidf_(zb);
    my_id = lane == r ? bi : my_id;
    my_w = lane == r ? base : my_w;
#pragma unroll
    for (int j = 0; j < EPL; ++j) key[j] = lane + 64 * j == bi ? NEG : key[j];
  }
  float wsum = 0.f;
  for (int r = 0; r < k; ++r) wsum += lane_f(my_w, r);
  if (lane < k) {
    float wv = norm ? my_w / wsum : my_w;
    ids[(size_t)t * k + lane] = my_id;
    wout[(size_t)t * k + lane] = wv * scale;
  }
}

template <typename T>
hipError_t launch_logits_t(const T* x, const T* w, int N, int d, int E, bool split, float* out,
                           hipStream_t s) {
  const int S = router_slices(d);
  if (E <= 16) {
    dim3 grid((N + 255) / 256, (E + 15) / 16, split ? S : 1);
    launch_k(router_logits_kernel<T, 256, 16, 4>, grid, 256, 0, s, x, w, N, d, E, split ? 1 : 0, out);
  } else if (N <= kRouterSmallN) {
    // few tokens (decode): 16-token tiles, one token per thread, for more
    // workgroups
    dim3 grid((N + 15) / 16, (E + 63) / 64, split ? S : 1);
    launch_k(router_logits_kernel<T, 16, 64, 1>, grid, 256, 0, s, x, w, N, d, E, split ? 1 : 0, out);
  } else {
    dim3 grid((N + 63) / 64, (E + 63) / 64, split ? S : 1);
    launch_k(router_logits_kernel<T, 64, 64, 4>, grid, 256, 0, s, x, w, N, d, E, split ? 1 : 0, out);
  }
  return hipGetLastError();
}

}  // namespace

int router_slices(int d) { return (d + kRouterSlice - 1) / kRouterSlice; }

// Split the hidden dimension over workgroups (one 256-slice each, summed in
// order by top-k) when the output tiles alone would not fill the chip: 512
// tiles for the vector kernel and the 16-expert matrix-core one, 4096 waves
// of 32 x 64 for the wider matrix-core one.
bool router_split(int dtype, int N, int d, int E) {
  if (router_slices(d) <= 1) return false;
  if (use_mfma_router(dtype, N, E) && E <= 16) return cdiv64(N, 256) < 512;
  if (use_mfma_router(dtype, N, E)) return cdiv64(N, 32) * cdiv64(E, 64) < 4096;
  const int64_t BT = E <= 16 ? 256 : (N <= kRouterSmallN ? 16 : 64), BE = E <= 16 ? 16 : 64;
  const int64_t tiles = cdiv64(N, BT) * cdiv64(E, BE);
  return tiles < 512;
}

size_t router_ws_bytes(int dtype, int N, int d, int E) {
  size_t b = (size_t)N * E * sizeof(float);  // logits when the caller keeps none
  if (router_split(dtype, N, d, E)) b += (size_t)router_slices(d) * N * E * sizeof(float);
  return b;
}

hipError_t launch_router_logits(int dtype, const void* x, const void* w, int N, int d, int E,
                                bool split, float* out, hipStream_t s) {
  if (dtype == 0)
    return launch_logits_t<float>((const float*)x, (const float*)w, N, d, E, split, out, s);
  if (use_mfma_router(dtype, N, E) && E <= 16) {
    const dim3 g((N + 255) / 256, 1, split ? router_slices(d) : 1);
    if (split)
      launch_k(router_mfma16_kernel<true>, g, 256, 0, s, (const bf16_t*)x, (const bf16_t*)w, N, d,
               E, out);
    else
      launch_k(router_mfma16_kernel<false>, g, 256, 0, s, (const bf16_t*)x, (const bf16_t*)w, N, d,
               E, out);
    return hipGetLastError();
  }
  if (use_mfma_router(dtype, N, E)) {
    // workgroup tile: 64 tokens x 128 experts, or 128 x 64 where 64-wide
    // expert tiles pad less (measured on 4096 tokens over 256 experts:
    // 64 x 128 192 us, 32 x 256 198 us; over 160 experts, d 5120: 128 x 64
    // 96 us against 122 us for 64 x 128, which pads 160 to 256)
    const int z = split ? router_slices(d) : 1;
#define FS_ROUTER_MFMA(WT, WE)                                                               \
  do {                                                                                       \
    const dim3 g((N + 32 * WT - 1) / (32 * WT), (E + 64 * WE - 1) / (64 * WE), z);           \
    if (split)                                                                               \
      launch_k(router_mfma_kernel<WT, WE, true>, g, 256, 0, s, (const bf16_t*)x,            \
               (const bf16_t*)w, N, d, E, out);                                              \
    else                                                                                     \
      launch_k(router_mfma_kernel<WT, WE, false>, g, 256, 0, s, (const bf16_t*)x,           \
               (const bf16_t*)w, N, d, E, out);                                              \
  } while (0)
    if (E > 64 && cdiv64(E, 128) * 128 <= cdiv64(E, 64) * 64)
      FS_ROUTER_MFMA(2, 2);
    else
      FS_ROUTER_MFMA(4, 1);
#undef FS_ROUTER_MFMA
    return hipGetLastError();
  }
  return launch_logits_t<bf16_t>((const bf16_t*)x, (const bf16_t*)w, N, d, E, split, out, s);
}

hipError_t launch_topk(const float* src, int n_partials, int N, int E, const float* bias,
                       int score, int k, int G, int TG, int norm, float scale,
                       float* logits_out, int32_t* ids, float* w, hipStream_t s) {
  dim3 grid((N + 3) / 4);
#define FS_TOPK(EPL)                                                                       \
  launch_k(topk_kernel<EPL>, grid, 256, 0, s, src, n_partials, N, E, bias, score, k, G, TG, norm, \
                                        scale, logits_out, ids, w)
  if (E <= 64)
    FS_TOPK(1);
  else if (E <= 128)
    FS_TOPK(2);
  else if (E <= 256)
    FS_TOPK(4);
  else
    FS_TOPK(8);
#undef FS_TOPK
  return hipGetLastError();
}

}  // namespace fs
