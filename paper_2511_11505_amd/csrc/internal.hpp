// Launchers behind the C ABI.  Each enqueues kernels on `s` and returns the
// first HIP error; arguments were validated by the caller.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace fs {

constexpr int kRouterSlice = 256;  // router reduction-order slice length

// Per-kernel event timing (implemented in api.cpp).
void prof_begin(int kernel, hipStream_t s);
void prof_end(int kernel, hipStream_t s);
// Events a kernel launched now on s records from its dispatch packet (both
// null when no timing window is open on s).
void prof_kernel_events(hipStream_t s, hipEvent_t* start, hipEvent_t* stop);

// Kernel launch that feeds an open timing window on s with the kernel's
// own start and end times (hipExtLaunchKernelGGL); a plain launch otherwise.
template <typename F, typename... Args>
inline void launch_k(F kernel, dim3 grid, dim3 block, uint32_t shm, hipStream_t s, Args... args) {
  hipEvent_t a, b;
  prof_kernel_events(s, &a, &b);
  hipExtLaunchKernelGGL(kernel, grid, block, shm, s, a, b, 0, args...);
}

// ---- router (router.hip)
int router_slices(int d);
bool router_split(int dtype, int N, int d, int E);
size_t router_ws_bytes(int dtype, int N, int d, int E);
hipError_t launch_router_logits(int dtype, const void* x, const void* w, int N, int d, int E,
                                bool split, float* out, hipStream_t s);
hipError_t launch_topk(const float* src, int n_partials, int N, int E, const float* bias,
                       int score, int k, int G, int TG, int norm, float scale,
                       float* logits_out, int32_t* ids, float* w, hipStream_t s);

// ---- dispatch (dispatch.hip)
size_t plan_ws_bytes(int N, int E);
// Fixed plan workspace of the allocation-free dispatch entry point: 4 MiB,
// enough for ceil(N / 64) * E <= 262144 (e.g. 32768 tokens over 512
// experts).  plan_scratch() gives its device address on the current device.
constexpr size_t kPlanScratchBytes = (size_t)4 << 20;
constexpr int kPlanScratchMaxDevices = 64;
hipError_t plan_scratch(void** out);
hipError_t launch_plan(const int32_t* ids, int N, int k, int E, int R, int32_t* counts,
                       int32_t* offsets, int32_t* rank_offsets, int32_t* slot_to_row,
                       int32_t* row_to_slot, void* ws, hipStream_t s);
hipError_t launch_pack(int dtype, const void* x, const int32_t* slot_to_row, int N, int k, int d,
                       void* send, hipStream_t s);
// FP8 rows: codes [N, d] bytes and one fp32 scale per row, to the send rows
// of slot_to_row (codes [rows, d], scales [rows]).
hipError_t launch_pack_fp8(const uint8_t* codes, const float* scales, const int32_t* slot_to_row,
                           int N, int k, int d, uint8_t* send_codes, float* send_scales,
                           hipStream_t s);
hipError_t launch_local_rows(const int32_t* offsets, const int32_t* rank_offsets,
                             const int32_t* row_to_slot, int N, int k, int E, int R, int r,
                             int32_t* local_tokens, int32_t* local_offsets, hipStream_t s);
hipError_t launch_receive_rows(const int32_t* src_counts, const int32_t* src_offsets, int R,
                               int E, int r, int64_t cap, int32_t* group_rows,
                               int32_t* group_offsets, hipStream_t s);

// ---- grouped SwiGLU FFN and dense linear (gemm.hip)
size_t ffn_ws_bytes(int dtype, int64_t max_rows, int ffn, int d);
// rows_in: gate/up reads input row rows_in[i] (NULL: row i); rows_out: down
// writes output row rows_out[i] (NULL: row i).
hipError_t launch_grouped_ffn(int dtype, int n_groups, int ffn, int d, const void* in,
                              const int32_t* rows_in, const int32_t* rows_out,
                              const int32_t* goff, int64_t max_rows,
                              const void* w_gate_up, const void* w_down, void* out, void* ws,
                              hipStream_t s, int prof_gate_up);  // profile id of gate/up, down = +1; -1: none
// FP8 (E4M3) experts: row quantisation, and the grouped SwiGLU FFN on
// quantised operands (x and the weights by row scales; H is quantised per
// row between the passes, inside the workspace).
// Row i of the output quantises source row gather[i] (or row i) for
// i < min(*row_count, rows) (or rows).
hipError_t launch_quantize_fp8(int dtype, const void* src, int64_t rows, int cols,
                               const int32_t* row_count, uint8_t* codes, float* scales,
                               hipStream_t s, const int32_t* gather = nullptr);
size_t ffn_fp8_ws_bytes(int64_t max_rows, int ffn, int d);
hipError_t launch_grouped_ffn_fp8(int n_groups, int ffn, int d, const uint8_t* x,
                                  const float* x_scale, const int32_t* rows_in,
                                  const int32_t* rows_out, const int32_t* goff, int64_t max_rows,
                                  const uint8_t* w_gate_up, const float* s_gate_up,
                                  const uint8_t* w_down, const float* s_down, void* out,
                                  void* ws, hipStream_t s, int prof_gate_up);
hipError_t launch_dense_linear(int dtype, int m, int n, int kdim, const void* a, const void* w,
                               void* out, hipStream_t s);
// Expert weights in MFMA fragment order: n_mats row-major [rows, cols] bf16
// matrices (rows % 32 == 0, cols % 16 == 0) to [rows/32][cols/16][64][8].
hipError_t launch_fragment_order(const void* src, int64_t n_mats, int rows, int cols, void* dst,
                                 hipStream_t s);
// FP8 fragment order of n_mats row-major [rows, cols] E4M3 code matrices
// (rows % 32 == 0, cols % 64 == 0).
hipError_t launch_fragment_order_fp8(const uint8_t* src, int64_t n_mats, int rows, int cols,
                                     uint8_t* dst, hipStream_t s);
// The FP8 grouped SwiGLU FFN on FP8-fragment-ordered weights (ffn % 128 == 0,
// d % 256 == 0); operands and workspace as launch_grouped_ffn_fp8.
hipError_t launch_grouped_ffn_fo_fp8(int G, int ffn, int d, const uint8_t* x, const float* x_scale,
                                     const int32_t* rows_in, const int32_t* rows_out,
                                     const int32_t* goff, int64_t max_rows,
                                     const uint8_t* w_gate_up_fo, const float* s_gate_up,
                                     const uint8_t* w_down_fo, const float* s_down, void* out,
                                     void* ws, hipStream_t s, int prof_gate_up);
// The grouped SwiGLU FFN on fragment-ordered weights (bf16; ffn % 128 == 0,
// d % 256 == 0); the workspace is that of launch_grouped_ffn.
hipError_t launch_grouped_ffn_fo(int G, int ffn, int d, const void* in, const int32_t* rows_in,
                                 const int32_t* rows_out, const int32_t* goff, int64_t max_rows,
                                 const void* w_gate_up_fo, const void* w_down_fo, void* out,
                                 void* ws, hipStream_t s, int prof_gate_up);

// ---- combine and residual (elementwise.hip)
// row_range (device, 2 ints) or NULL: only plan rows in [row_range[0],
// row_range[1]) contribute, read from y_ret at row - row_range[0].
hipError_t launch_combine(int dtype, const void* y_ret, const int32_t* slot_to_row,
                          const float* topk_w, const void* shared_out, void* routed_out,
                          void* residual, const int32_t* row_range, int N, int k, int d,
                          hipStream_t s);
hipError_t launch_residual(int dtype, void* out, const void* a, const void* b, const void* c,
                           int64_t n_elems, hipStream_t s);

// ---- stand-in collectives (standin.hip)
// Copy `bytes` from src to dst with `workgroups` workgroups, taking at least
// `seconds` (0: unpaced); see the kernel's comment for the schedule.
// Pointers and bytes must be multiples of 4 (else hipErrorInvalidValue).
hipError_t launch_paced_copy(void* dst, const void* src, size_t bytes, double seconds,
                             int workgroups, hipStream_t s);

}  // namespace fs
