// Link-paced stand-in copy: the one-GPU stand-in for a collective
// (the Dispatch and Combine all-to-alls of Section 2.1, the all-reduces of
// Section 4.2) that takes the time the collective would take on a node.
//
// On a node, the collective's kernels occupy a few CUs and move bytes no
// faster than the links allow; a device-to-device copy at HBM speed is
// neither.  This copy runs on a fixed number of workgroups and follows the
// byte schedule of a transfer at `rate`: byte b of the buffer is not read
// before t0 + b / rate, and a workgroup does not finish before its last
// chunk's due time, so the copy takes bytes / rate once it is resident (or
// longer, when the workgroups cannot keep up).  The bytes copied are the
// bytes of the buffer, bit for bit; only the timing is modelled.
//
// The wall clock (a constant-rate counter, queried on the host per device)
// paces each wave on its own: the wait is a sleep loop on a monotonic
// counter towards a finite due time, so every wave ends.

#include <mutex>

#include "common.hpp"
#include "internal.hpp"

namespace fs {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kCopyUnroll = 8;  // loads in flight per lane

__device__ __forceinline__ void wait_until(uint64_t due) {
  while (wall_clock64() < due) __builtin_amdgcn_s_sleep(2);
}

// T: the copy unit (16 or 4 bytes; both pointers aligned to it).  Chunk
// c covers units [c * CH, (c + 1) * CH), CH = 256 * kCopyUnroll; workgroup
// w takes chunks w, w + G, ...  Chunk c may start at t0 + c * ticks_chunk
// and is due at t0 + (c + 1) * ticks_chunk (the last one at the buffer's
// end); ticks_chunk = 0 copies unpaced.  The tail bytes past the last whole
// unit (4, 8 or 12 with 16-byte units) are copied bytewise by workgroup 0.
template <typename T>
__global__ __launch_bounds__(256) void paced_copy_kernel(const T* __restrict__ src,
                                                         T* __restrict__ dst, int64_t n_units,
                                                         const unsigned char* __restrict__ src_tail,
                                                         unsigned char* __restrict__ dst_tail,
                                                         int tail_bytes, double ticks_chunk,
                                                         double ticks_total) {
  constexpr int64_t CH = 256 * kCopyUnroll;
  const int64_t n_chunks = (n_units + CH - 1) / CH;
  const uint64_t t0 = wall_clock64();
  const int tid = threadIdx.x;
  for (int64_t c = blockIdx.x; c < n_chunks; c += gridDim.x) {
    if (ticks_chunk > 0.0) wait_until(t0 + (uint64_t)((double)c * ticks_chunk));
    const int64_t base = c * CH + tid;
    if ((c + 1) * CH <= n_units) {
      T v[kCopyUnroll];
#pragma unroll
      for (int u = 0; u < kCopyUnroll; ++u) v[u] = __builtin_nontemporal_load(src + base + u * 256);
#pragma unroll
      for (int u = 0; u < kCopyUnroll; ++u) __builtin_nontemporal_store(v[u], dst + base + u * 256);
    } else {
      for (int64_t i = base; i < n_units; i += 256) dst[i] = src[i];
    }
  }
  if (blockIdx.x == 0 && tid < tail_bytes) dst_tail[tid] = src_tail[tid];
  if (ticks_chunk > 0.0) {
    // this workgroup's last chunk is due at its end (the whole buffer's end
    // for the last chunk)
    const int64_t last = blockIdx.x + ((n_chunks - 1 - blockIdx.x) / gridDim.x) * gridDim.x;
    const double due = fmin((double)(last + 1) * ticks_chunk, ticks_total);
    if (last < n_chunks) wait_until(t0 + (uint64_t)due);
  }
}

std::mutex g_clock_mu;
int g_clock_khz[64] = {};

hipError_t wall_clock_khz(int* khz) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_clock_mu);
  if (g_clock_khz[dev] == 0) {
    e = hipDeviceGetAttribute(&g_clock_khz[dev], hipDeviceAttributeWallClockRate, dev);
    if (e != hipSuccess) return e;
    if (g_clock_khz[dev] <= 0) return hipErrorInvalidValue;
  }
  *khz = g_clock_khz[dev];
  return hipSuccess;
}

template <typename T>
void launch_typed(void* dst, const void* src, size_t bytes, int workgroups, double ticks_per_byte,
                  hipStream_t s) {
  const int64_t n_units = (int64_t)(bytes / sizeof(T));
  const int tail = (int)(bytes - (size_t)n_units * sizeof(T));
  const int64_t CH = 256 * kCopyUnroll;
  const int64_t n_chunks = (n_units + CH - 1) / CH;
  const int grid = (int)std::max<int64_t>(1, std::min<int64_t>(workgroups, n_chunks));
  const size_t head = (size_t)n_units * sizeof(T);
  launch_k(paced_copy_kernel<T>, dim3(grid), dim3(256), 0, s, static_cast<const T*>(src),
           static_cast<T*>(dst), n_units, static_cast<const unsigned char*>(src) + head,
           static_cast<unsigned char*>(dst) + head, tail,
           ticks_per_byte * (double)(CH * (int64_t)sizeof(T)), ticks_per_byte * (double)bytes);
}

}  // namespace

hipError_t launch_paced_copy(void* dst, const void* src, size_t bytes, double seconds,
                             int workgroups, hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  int khz = 0;
  hipError_t e = wall_clock_khz(&khz);
  if (e != hipSuccess) return e;
  const double ticks_per_byte = seconds > 0.0 ? seconds * (double)khz * 1e3 / (double)bytes : 0.0;
  const uintptr_t a = reinterpret_cast<uintptr_t>(dst) | reinterpret_cast<uintptr_t>(src);
  if (a % 4 != 0 || bytes % 4 != 0) return hipErrorInvalidValue;
  if (a % 16 == 0)
    launch_typed<u32x4>(dst, src, bytes, workgroups, ticks_per_byte, s);
  else
    launch_typed<unsigned int>(dst, src, bytes, workgroups, ticks_per_byte, s);
  return hipGetLastError();
}

}  // namespace fs
