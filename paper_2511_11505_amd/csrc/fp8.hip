// Row-wise FP8 (OCP E4M3) quantisation for the FP8 experts.
//
// A row x (activations: one token or expert row; weights: one output
// channel) is stored as codes and one fp32 scale: amax = max |x_i|;
// scale = amax / 448 and inv = 448 / amax, each a correctly rounded fp32
// division; v_i = x_i * inv (one fp32 rounding) clamped to [-448, 448];
// code_i = v_i rounded to E4M3 to nearest, ties to even
// (v_cvt_pk_fp8_f32, which gives NaN above 464 unless clamped first).  An
// all-zero row gets scale 1 and zero codes.  The row then stands for
// dec(code_i) * scale.
//
// Rows may be gathered (output row i from source row gather[i]) and
// bounded by a device row count.  bf16 rows of up to 8192 elements, at
// least 1024 rows: one wave per row (four per workgroup, grid-stride) holds
// the row in registers, takes amax with the wave reduction and converts
// from registers.  Other shapes and fp32: one workgroup per row, a pass for
// amax over 16-byte vectors, a block reduction, and a pass that converts and
// stores 8 or 4 codes per thread.  The amax is exact in any order, so both
// give the same codes.

#include "common.hpp"
#include "internal.hpp"

namespace fs {
namespace {

constexpr float kE4M3Max = 448.f;

__device__ __forceinline__ float block_max(float v, float* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float m = red[0];
#pragma unroll
  for (int w = 1; w < 4; ++w) m = fmaxf(m, red[w]);
  __syncthreads();   // red is reused by the next row
  return m;
}

__device__ __forceinline__ float clamp_e4m3(float v) {
  return fminf(fmaxf(v, -kE4M3Max), kE4M3Max);
}

template <typename T>
__global__ __launch_bounds__(256) void quantize_fp8_kernel(const T* __restrict__ src, int64_t rows,
                                                           int cols,
                                                           const int32_t* __restrict__ row_count,
                                                           const int32_t* __restrict__ gather,
                                                           uint8_t* __restrict__ codes,
                                                           float* __restrict__ scales) {
  __shared__ float red[4];
  constexpr int V = 16 / sizeof(T);
  int64_t n = rows;
  if (row_count) {
    const int64_t c = *row_count;
    n = c < 0 ? 0 : (c < rows ? c : rows);
  }
  const int nv = cols / V;
  for (int64_t r = blockIdx.x; r < n; r += gridDim.x) {
    const T* row = src + (gather ? (int64_t)gather[r] : r) * cols;
    float m = 0.f;
    for (int i = threadIdx.x; i < nv; i += 256) {
      Vec16<T> v;
      v.raw = ld16(row + (size_t)i * V);
#pragma unroll
      for (int j = 0; j < V; ++j) m = fmaxf(m, fabsf(v.get(j)));
    }
    m = block_max(m, red);
    const float scale = m > 0.f ? __fdiv_rn(m, kE4M3Max) : 1.f;
    const float inv = m > 0.f ? __fdiv_rn(kE4M3Max, m) : 0.f;
    if (threadIdx.x == 0) scales[r] = scale;
    uint8_t* out = codes + r * cols;
    for (int i = threadIdx.x; i < nv; i += 256) {
      Vec16<T> v;
      v.raw = ld16(row + (size_t)i * V);
      float q[V];
#pragma unroll
      for (int j = 0; j < V; ++j) q[j] = clamp_e4m3(__fmul_rn(v.get(j), inv));
      int w0 = 0;
      w0 = __builtin_amdgcn_cvt_pk_fp8_f32(q[0], q[1], w0, false);
      w0 = __builtin_amdgcn_cvt_pk_fp8_f32(q[2], q[3], w0, true);
      if constexpr (V == 8) {
        int w1 = 0;
        w1 = __builtin_amdgcn_cvt_pk_fp8_f32(q[4], q[5], w1, false);
        w1 = __builtin_amdgcn_cvt_pk_fp8_f32(q[6], q[7], w1, true);
        *reinterpret_cast<uint2*>(out + (size_t)i * 8) = make_uint2((uint32_t)w0, (uint32_t)w1);
      } else {
        *reinterpret_cast<uint32_t*>(out + (size_t)i * 4) = (uint32_t)w0;
      }
    }
  }
}

// One wave per row, the row's 16-byte vectors in registers (lane l holds
// vectors l, l + 64, ...; VPL per lane at most).
template <int VPL>
__global__ __launch_bounds__(256) void quantize_fp8_wave_kernel(const bf16_t* __restrict__ src,
                                                                int64_t rows, int cols,
                                                                const int32_t* __restrict__ row_count,
                                                                const int32_t* __restrict__ gather,
                                                                uint8_t* __restrict__ codes,
                                                                float* __restrict__ scales) {
  constexpr int V = 8;
  const int lane = threadIdx.x & 63;
  int64_t n = rows;
  if (row_count) {
    const int64_t c = *row_count;
    n = c < 0 ? 0 : (c < rows ? c : rows);
  }
  const int nv = cols / V;
  for (int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); r < n; r += (int64_t)gridDim.x * 4) {
    const bf16_t* row = src + (gather ? (int64_t)gather[r] : r) * cols;
    Vec16<bf16_t> v[VPL];
    float m = 0.f;
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
      const int i = lane + 64 * j;
      if (i < nv) {
        v[j].raw = ld16(row + (size_t)i * V);
#pragma unroll
        for (int e = 0; e < V; ++e) m = fmaxf(m, fabsf(v[j].get(e)));
      }
    }
    m = wave_max(m);
    const float scale = m > 0.f ? __fdiv_rn(m, kE4M3Max) : 1.f;
    const float inv = m > 0.f ? __fdiv_rn(kE4M3Max, m) : 0.f;
    if (lane == 0) scales[r] = scale;
    uint8_t* out = codes + r * cols;
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
      const int i = lane + 64 * j;
      if (i < nv) {
        float q[V];
#pragma unroll
        for (int e = 0; e < V; ++e) q[e] = clamp_e4m3(__fmul_rn(v[j].get(e), inv));
        int w0 = 0, w1 = 0;
        w0 = __builtin_amdgcn_cvt_pk_fp8_f32(q[0], q[1], w0, false);
        w0 = __builtin_amdgcn_cvt_pk_fp8_f32(q[2], q[3], w0, true);
        w1 = __builtin_amdgcn_cvt_pk_fp8_f32(q[4], q[5], w1, false);
        w1 = __builtin_amdgcn_cvt_pk_fp8_f32(q[6], q[7], w1, true);
        *reinterpret_cast<uint2*>(out + (size_t)i * 8) = make_uint2((uint32_t)w0, (uint32_t)w1);
      }
    }
  }
}

}  // namespace

hipError_t launch_quantize_fp8(int dtype, const void* src, int64_t rows, int cols,
                               const int32_t* row_count, uint8_t* codes, float* scales,
                               hipStream_t s, const int32_t* gather) {
  if (rows <= 0) return hipSuccess;
  // (a wave per row needs many rows to fill the GPU: with fewer than 1024,
  // as in decode, four waves per row load more in parallel)
  if (dtype != 0 && cols <= 64 * 8 * 16 && rows >= 1024) {
    const unsigned g4 = (unsigned)((rows + 3) / 4 < 65536 ? (rows + 3) / 4 : 65536);
    if (cols <= 64 * 8 * 4)
      launch_k(quantize_fp8_wave_kernel<4>, g4, 256, 0, s, (const bf16_t*)src, rows, cols,
               row_count, gather, codes, scales);
    else
      launch_k(quantize_fp8_wave_kernel<16>, g4, 256, 0, s, (const bf16_t*)src, rows, cols,
               row_count, gather, codes, scales);
    return hipGetLastError();
  }
  const unsigned grid = (unsigned)(rows < 65536 ? rows : 65536);
  if (dtype == 0)
    launch_k(quantize_fp8_kernel<float>, grid, 256, 0, s, (const float*)src, rows, cols, row_count,
                                                    gather, codes, scales);
  else
    launch_k(quantize_fp8_kernel<bf16_t>, grid, 256, 0, s,
        (const bf16_t*)src, rows, cols, row_count,
                                                     gather, codes, scales);
  return hipGetLastError();
}

}  // namespace fs
