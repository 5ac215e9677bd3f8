// Combine + unpack with the deferred FarSkip residual add, and the plain
// residual add (Section 2.1 Combine; Section 3, Eq. 7).
//
// Combine is a gather: token t reads its k expert-output rows through
// slot_to_row, so no atomics are needed and the fp32 sum runs in slot order
// j = 0..k-1.  All adds run in fp32 and round once at the store.
//
// The partial Combine of the replicated-activation variant is the same
// gather restricted to the plan rows [lo, hi) of this rank's experts, read
// from y at row - lo; other slots contribute nothing.

#include "common.hpp"
#include "internal.hpp"

namespace fs {
namespace {

// Each lane handles one 16-byte chunk of one token row; waves are laid out
// (token, 64-chunk block) so that short batches still fill the machine.
// KC > 0 fixes k at compile time: the k row indices and weights, then the k
// row chunks and the residual chunk are all requested before the first add,
// so a lane has k + 1 loads in flight; KC = 0 handles any k with a loop.
template <typename T, bool LOCAL, int KC>
__global__ __launch_bounds__(256) void combine_kernel(const T* __restrict__ y,
                                                      const int32_t* __restrict__ slot_to_row,
                                                      const float* __restrict__ topk_w,
                                                      const T* __restrict__ shared_out,
                                                      T* __restrict__ routed_out,
                                                      T* __restrict__ residual,
                                                      const int32_t* __restrict__ row_range,
                                                      int N, int k, int d) {
  constexpr int V = 16 / sizeof(T);
  const int nch = d / V;
  const int nb = (nch + 63) / 64;
  const int64_t wave = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int t = (int)(wave / nb);
  const int c = (int)(wave % nb) * 64 + (threadIdx.x & 63);
  if (t >= N || c >= nch) return;
  const size_t off = (size_t)t * d + (size_t)c * V;
  float acc[V];
#pragma unroll
  for (int i = 0; i < V; ++i) acc[i] = 0.f;
  int lo = 0, hi = 0;
  if (LOCAL) {
    lo = row_range[0];
    hi = row_range[1];
  }
  if constexpr (KC > 0) {
    int rw[KC];
    float wj[KC];
#pragma unroll
    for (int j = 0; j < KC; ++j) {
      rw[j] = slot_to_row[(size_t)t * KC + j];
      wj[j] = topk_w[(size_t)t * KC + j];
      if (rw[j] >= 0 && LOCAL) rw[j] = (rw[j] < lo || rw[j] >= hi) ? -1 : rw[j] - lo;
    }
    Vec16<T> v[KC];
#pragma unroll
    for (int j = 0; j < KC; ++j)
      if (rw[j] >= 0) v[j].raw = ld16(y + (size_t)rw[j] * d + (size_t)c * V);
    Vec16<T> rv;
    if (residual) rv.raw = ld16(residual + off);
#pragma unroll
    for (int j = 0; j < KC; ++j)
      if (rw[j] >= 0) {
#pragma unroll
        for (int i = 0; i < V; ++i) acc[i] = fmaf(wj[j], v[j].get(i), acc[i]);
      }
    if (shared_out) {
      Vec16<T> sv;
      sv.raw = ld16(shared_out + off);
#pragma unroll
      for (int i = 0; i < V; ++i) acc[i] += sv.get(i);
    }
    if (routed_out) {
      Vec16<T> o;
#pragma unroll
      for (int i = 0; i < V; ++i) o.set(i, acc[i]);
      st16(routed_out + off, o.raw);
    }
    if (residual) {
      Vec16<T> o;
#pragma unroll
      for (int i = 0; i < V; ++i) o.set(i, rv.get(i) + acc[i]);
      st16(residual + off, o.raw);
    }
    return;
  }
  for (int j = 0; j < k; ++j) {
    int row = slot_to_row[(size_t)t * k + j];
    if (row < 0) continue;
    if (LOCAL) {
      if (row < lo || row >= hi) continue;
      row -= lo;
    }
    const float wj = topk_w[(size_t)t * k + j];
    Vec16<T> v;
    v.raw = ld16(y + (size_t)row * d + (size_t)c * V);
#pragma unroll
    for (int i = 0; i < V; ++i) acc[i] = fmaf(wj, v.get(i), acc[i]);
  }
  if (shared_out) {
    Vec16<T> v;
    v.raw = ld16(shared_out + off);
#pragma unroll
    for (int i = 0; i < V; ++i) acc[i] += v.get(i);
  }
  if (routed_out) {
    Vec16<T> o;
#pragma unroll
    for (int i = 0; i < V; ++i) o.set(i, acc[i]);
    st16(routed_out + off, o.raw);
  }
  if (residual) {
    Vec16<T> rv, o;
    rv.raw = ld16(residual + off);
#pragma unroll
    for (int i = 0; i < V; ++i) o.set(i, rv.get(i) + acc[i]);
    st16(residual + off, o.raw);
  }
}

// out = a + b (+ c), elementwise in fp32, 16-byte vectors, grid-stride.
template <typename T>
__global__ __launch_bounds__(256) void residual_kernel(T* out, const T* a, const T* b,
                                                       const T* c, int64_t n_vec) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n_vec;
       i += (int64_t)gridDim.x * blockDim.x) {
    Vec16<T> va, vb, vc, o;
    va.raw = ld16(a + i * Vec16<T>::N);
    if (b) vb.raw = ld16(b + i * Vec16<T>::N);
    if (c) vc.raw = ld16(c + i * Vec16<T>::N);
#pragma unroll
    for (int v = 0; v < Vec16<T>::N; ++v) {
      float s = va.get(v);
      if (b) s += vb.get(v);
      if (c) s += vc.get(v);
      o.set(v, s);
    }
    st16(out + i * Vec16<T>::N, o.raw);
  }
}

}  // namespace

hipError_t launch_combine(int dtype, const void* y_ret, const int32_t* slot_to_row,
                          const float* topk_w, const void* shared_out, void* routed_out,
                          void* residual, const int32_t* row_range, int N, int k, int d,
                          hipStream_t s) {
  const int64_t nb = ((int64_t)d / (dtype == 0 ? 4 : 8) + 63) / 64;
  dim3 grid((unsigned)((N * nb + 3) / 4));
#define FS_COMBINE_K(T, L, KC)                                                              \
  launch_k(combine_kernel<T, L, KC>, grid, 256, 0, s, (const T*)y_ret, slot_to_row, topk_w,      \
                                                (const T*)shared_out, (T*)routed_out,      \
                                                (T*)residual, row_range, N, k, d)
#define FS_COMBINE(T, L)                    \
  do {                                      \
    switch (k) {                            \
      case 1: FS_COMBINE_K(T, L, 1); break; \
      case 2: FS_COMBINE_K(T, L, 2); break; \
      case 4: FS_COMBINE_K(T, L, 4); break; \
      case 6: FS_COMBINE_K(T, L, 6); break; \
      case 8: FS_COMBINE_K(T, L, 8); break; \
      default: FS_COMBINE_K(T, L, 0); break; \
    }                                       \
  } while (0)
  if (dtype == 0) {
    if (row_range) FS_COMBINE(float, true);
    else FS_COMBINE(float, false);
  } else {
    if (row_range) FS_COMBINE(bf16_t, true);
    else FS_COMBINE(bf16_t, false);
  }
#undef FS_COMBINE
#undef FS_COMBINE_K
  return hipGetLastError();
}

hipError_t launch_residual(int dtype, void* out, const void* a, const void* b, const void* c,
                           int64_t n_elems, hipStream_t s) {
  const int V = dtype == 0 ? 4 : 8;
  const int64_t n_vec = n_elems / V;
  int64_t blocks = (n_vec + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  if (dtype == 0)
    launch_k(residual_kernel<float>, (int)blocks, 256, 0, s, (float*)out, (const float*)a,
                                                       (const float*)b, (const float*)c, n_vec);
  else
    launch_k(residual_kernel<bf16_t>, (int)blocks, 256, 0, s, (bf16_t*)out, (const bf16_t*)a,
                                                        (const bf16_t*)b, (const bf16_t*)c,
                                                        n_vec);
  return hipGetLastError();
}

}  // namespace fs
