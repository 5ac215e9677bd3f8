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

bool router_split(int N, int d, int E) {
  const int64_t BT = E <= 16 ? 256 : (N <= kRouterSmallN ? 16 : 64), BE = E <= 16 ? 16 : 64;
  const int64_t tiles = cdiv64(N, BT) * cdiv64(E, BE);
  return router_slices(d) > 1 && tiles < 512;
}

size_t router_ws_bytes(int N, int d, int E) {
  size_t b = (size_t)N * E * sizeof(float);  // logits when the caller keeps none
  if (router_split(N, d, E)) b += (size_t)router_slices(d) * N * E * sizeof(float);
  return b;
}

hipError_t launch_router_logits(int dtype, const void* x, const void* w, int N, int d, int E,
                                bool split, float* out, hipStream_t s) {
  if (dtype == 0)
    return launch_logits_t<float>((const float*)x, (const float*)w, N, d, E, split, out, s);
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
