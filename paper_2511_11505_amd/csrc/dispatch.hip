// Dispatch plan, pack and receive rows (Section 2.1, Dispatch).
//
// The plan is a stable counting sort of the N*k (token, expert) slots by
// expert, with no global atomics, so it is deterministic:
//   1. per 64-token tile, a bit mask per expert of the tile's tokens that
//      chose it (LDS OR, order-independent) and its population count;
//   2. one workgroup scans the per-tile counts into per-tile bases and the
//      expert offsets;
//   3. each slot's row = the expert's offset + its tile's base for the expert + the number of
//      earlier tokens of the tile with the same expert (popcount of the mask
//      below the token's lane).
// Up to a few thousand tokens, every tile's workgroup counts all slots
// itself and ranks its tile, in one launch; larger batches take the three
// kernels.
// Pack copies each token row once from HBM and writes it to its k rows with
// 16-byte vector accesses.
//
// With replicated activations (the inference variant) a rank keeps only the
// rows of its own experts: a contiguous block of the plan's rows, read back
// to token indices so the expert GEMM gathers them straight from x.

#include <mutex>

#include "common.hpp"
#include "internal.hpp"

// Plan workspace of the allocation-free dispatch entry point
// (fs_dispatch_pack_noalloc): a fixed device array that every device holding
// this library keeps until the process ends.  Host code never passes its
// name to a kernel (on the host the name is a stand-in, not a device
// address); it uses the per-device address plan_scratch() returns.
static __device__ __align__(256) unsigned char scratch[fs::kPlanScratchBytes];

namespace fs {
namespace {

constexpr int kTile = 64;  // tokens per plan tile (one wavefront)

__global__ __launch_bounds__(64) void plan_hist_kernel(const int32_t* __restrict__ ids, int N,
                                                       int k, int E, uint64_t* __restrict__ bits,
                                                       int32_t* __restrict__ hist) {
  extern __shared__ uint64_t sb[];
  const int tile = blockIdx.x, lane = threadIdx.x;
  for (int e = lane; e < E; e += 64) sb[e] = 0;
  __syncthreads();
  const int t = tile * kTile + lane;
  if (t < N) {
    for (int j = 0; j < k; ++j) {
      const int e = ids[(size_t)t * k + j];
      if ((unsigned)e < (unsigned)E) atomicOr((unsigned long long*)&sb[e], 1ull << lane);
    }
  }
  __syncthreads();
  for (int e = lane; e < E; e += 64) {
    const uint64_t b = sb[e];
    bits[(size_t)tile * E + e] = b;
    hist[(size_t)tile * E + e] = __popcll(b);
  }
}

// One workgroup of 512 threads (E <= 512).  Expert e gets P = 512 / EP
// threads (EP: E rounded up to a power of two), each summing one contiguous
// chunk of the tiles' counts, so a few experts still spread their tiles over
// the whole workgroup; the chunk sums are scanned per expert in LDS.
// Writes, per tile, the number of earlier tiles' slots on each expert
// (tile_base[tile][e]), the counts, the exclusive offsets and rank offsets.
// All sums are integer, so any grouping gives the same values.
__global__ __launch_bounds__(512) void plan_scan_kernel(const int32_t* __restrict__ hist,
                                                        int n_tiles, int E, int R,
                                                        int32_t* __restrict__ tile_base,
                                                        int32_t* __restrict__ counts,
                                                        int32_t* __restrict__ offsets,
                                                        int32_t* __restrict__ rank_offsets) {
  __shared__ int32_t part[512];
  __shared__ int32_t sc[512];
  const int tid = threadIdx.x;
  int EP = 1;
  while (EP < E) EP <<= 1;
  const int P = 512 / EP;
  const int e = tid % EP, c = tid / EP;
  const int tpc = (n_tiles + P - 1) / P;
  const int ta = min(n_tiles, c * tpc), tb = min(n_tiles, ta + tpc);
  // 1. this chunk's sum (loads sixteen at a time so they overlap)
  int sum = 0;
  if (e < E) {
    for (int t0 = ta; t0 < tb; t0 += 16) {
      int h[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) h[i] = (t0 + i < tb) ? hist[(size_t)(t0 + i) * E + e] : 0;
#pragma unroll
      for (int i = 0; i < 16; ++i) sum += h[i];
    }
  }
  part[tid] = sum;
  __syncthreads();
  // 2. inclusive scan of the chunk sums of each expert (stride EP in part)
  for (int o = 1; o < P; o <<= 1) {
    const int v = (c >= o) ? part[tid - o * EP] : 0;
    __syncthreads();
    part[tid] += v;
    __syncthreads();
  }
  // 3. the per-tile bases of this chunk (its counts again, now from L2)
  if (e < E) {
    int run = part[tid] - sum;
    for (int t0 = ta; t0 < tb; t0 += 16) {
      int h[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) h[i] = (t0 + i < tb) ? hist[(size_t)(t0 + i) * E + e] : 0;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        if (t0 + i < tb) tile_base[(size_t)(t0 + i) * E + e] = run;
        run += h[i];
      }
    }
  }
  // 4. expert totals (the last chunk's inclusive sums) and their scan
  const int run = (tid < E) ? part[(P - 1) * EP + tid] : 0;
  sc[tid] = run;
  __syncthreads();
  for (int o = 1; o < 512; o <<= 1) {
    const int v = (tid >= o) ? sc[tid - o] : 0;
    __syncthreads();
    sc[tid] += v;
    __syncthreads();
  }
  const int incl = sc[tid];
  if (tid < E) {
    counts[tid] = run;
    offsets[tid] = incl - run;
  }
  if (tid == E - 1) offsets[E] = incl;
  // rank_offsets[r] = offsets[r * E / R]
  if (tid <= R) {
    const int ge = tid * (E / R);
    rank_offsets[tid] = (ge == 0) ? 0 : sc[ge - 1];
  }
}

__global__ __launch_bounds__(64) void plan_rank_kernel(const int32_t* __restrict__ ids, int N,
                                                       int k, int E,
                                                       const uint64_t* __restrict__ bits,
                                                       const int32_t* __restrict__ tile_base,
                                                       const int32_t* __restrict__ offsets,
                                                       int32_t* __restrict__ slot_to_row,
                                                       int32_t* __restrict__ row_to_slot) {
  const int tile = blockIdx.x, lane = threadIdx.x;
  const int t = tile * kTile + lane;
  if (t >= N) return;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int j = 0; j < k; ++j) {
    const int slot = t * k + j;
    const int e = ids[slot];
    int row = -1;
    if ((unsigned)e < (unsigned)E) {
      const size_t te = (size_t)tile * E + e;
      row = offsets[e] + tile_base[te] + __popcll(bits[te] & below);
      row_to_slot[row] = slot;
    }
    slot_to_row[slot] = row;
  }
}

// The plan in one launch of one workgroup per 64-token tile, for batches
// whose slots every workgroup can afford to read (kPlanTileReads): each
// workgroup counts, over all N k slots, the slots on each expert before its
// tile and from its tile on (integer LDS adds, so their order does not
// matter).  Their sum is the expert's count, whose exclusive scan over the
// experts is its offset; the first part is the tile's base.  So no
// workgroup waits for another, and the rows are those of the kernels
// above.  Workgroup 0 writes the counts and offsets.  (Measured: DeepSeek-V3
// prefill, 4096 tokens top-8 of 256, 19.1 -> 10.0 us against the three
// kernels; a 64-token decode batch 6.3 -> 4.7 us against the same steps in
// one workgroup.)
constexpr int64_t kPlanTileReads = int64_t(1) << 23;   // tiles x slots (32 MB of ids)

__global__ __launch_bounds__(512) void plan_tile_kernel(const int32_t* __restrict__ ids, int N,
                                                        int k, int E, int R,
                                                        int32_t* __restrict__ counts,
                                                        int32_t* __restrict__ offsets,
                                                        int32_t* __restrict__ rank_offsets,
                                                        int32_t* __restrict__ slot_to_row,
                                                        int32_t* __restrict__ row_to_slot) {
  __shared__ int32_t pre[512], post[512], sc[512];
  __shared__ uint64_t sb[512];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int tile = blockIdx.x;
  pre[tid] = 0;
  post[tid] = 0;
  sb[tid] = 0;
  __syncthreads();
  // 1. per-expert slot counts before the tile and from it on; sixteen
  // coalesced loads per thread go out before their adds
  const int64_t nslots = (int64_t)N * k, lim = (int64_t)tile * kTile * k;
  for (int64_t q0 = 0; q0 < nslots; q0 += 16 * 512) {
    int e[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int64_t q = q0 + tid + 512 * i;
      e[i] = q < nslots ? ids[q] : -1;
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int64_t q = q0 + tid + 512 * i;
      if ((unsigned)e[i] < (unsigned)E) atomicAdd(q < lim ? &pre[e[i]] : &post[e[i]], 1);
    }
  }
  // the tile's masks: bit `lane` of sb[e] says token tile * 64 + lane chose e
  const int t = tile * kTile + lane;
  if (t < N)
    for (int j = wave; j < k; j += 8) {
      const int e = ids[(size_t)t * k + j];
      if ((unsigned)e < (unsigned)E) atomicOr((unsigned long long*)&sb[e], 1ull << lane);
    }
  __syncthreads();
  // 2. counts and their scan over the experts
  const int cnt = tid < E ? pre[tid] + post[tid] : 0;
  sc[tid] = cnt;
  __syncthreads();
  for (int o = 1; o < 512; o <<= 1) {
    const int v = (tid >= o) ? sc[tid - o] : 0;
    __syncthreads();
    sc[tid] += v;
    __syncthreads();
  }
  const int incl = sc[tid];
  // the first row of this tile's slots on expert tid
  if (tid < E) post[tid] = incl - cnt + pre[tid];
  if (blockIdx.x == 0) {
    if (tid < E) {
      counts[tid] = cnt;
      offsets[tid] = incl - cnt;
    }
    if (tid == E - 1) offsets[E] = incl;
    if (tid <= R) {
      const int ge = tid * (E / R);
      rank_offsets[tid] = (ge == 0) ? 0 : sc[ge - 1];
    }
  }
  __syncthreads();
  // 3. ranks: earlier tokens of the tile on the same expert
  if (t < N) {
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int j = wave; j < k; j += 8) {
      const int slot = t * k + j;
      const int e = ids[slot];
      int row = -1;
      if ((unsigned)e < (unsigned)E) {
        row = post[e] + __popcll(sb[e] & below);
        row_to_slot[row] = slot;
      }
      slot_to_row[slot] = row;
    }
  }
}

// Each lane moves one 16-byte chunk of one token row: it reads the chunk
// once and writes it to the token's k send rows.  Waves are laid out
// (token, 64-chunk block), so short batches still fill the machine.
// KC > 0 fixes k at compile time (all k row indices are read before the
// stores); KC = 0 loops over any k.  FP8 rows (T = uint8_t codes) also carry
// one fp32 scale per row: the lane of chunk 0 copies the token's scale to
// its k send rows.
template <typename T, int KC>
__global__ __launch_bounds__(256) void pack_kernel(const T* __restrict__ x,
                                                   const int32_t* __restrict__ slot_to_row, int N,
                                                   int k, int d, T* __restrict__ send,
                                                   const float* __restrict__ x_scale,
                                                   float* __restrict__ send_scale) {
  const int nch = d * (int)sizeof(T) / 16;
  const int nb = (nch + 63) / 64;
  const int64_t wave = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int t = (int)(wave / nb);
  const int c = (int)(wave % nb) * 64 + (threadIdx.x & 63);
  if (t >= N || c >= nch) return;
  if (x_scale && c == 0) {
    const float sc = x_scale[t];
    for (int j = 0; j < k; ++j) {
      const int row = slot_to_row[(size_t)t * k + j];
      if (row >= 0) send_scale[row] = sc;
    }
  }
  const uint4 v = reinterpret_cast<const uint4*>(x + (size_t)t * d)[c];
  if constexpr (KC > 0) {
    int rw[KC];
#pragma unroll
    for (int j = 0; j < KC; ++j) rw[j] = slot_to_row[(size_t)t * KC + j];
#pragma unroll
    for (int j = 0; j < KC; ++j)
      if (rw[j] >= 0) reinterpret_cast<uint4*>(send + (size_t)rw[j] * d)[c] = v;
    return;
  }
  for (int j = 0; j < k; ++j) {
    const int row = slot_to_row[(size_t)t * k + j];
    if (row >= 0) reinterpret_cast<uint4*>(send + (size_t)row * d)[c] = v;
  }
}

// One workgroup per local expert e.  Its rows start after all rows of the
// local experts before it; within e, source 0's rows come first.
__global__ __launch_bounds__(256) void receive_rows_kernel(const int32_t* __restrict__ counts,
                                                           const int32_t* __restrict__ offsets,
                                                           int R, int E, int r, int64_t cap,
                                                           int32_t* __restrict__ group_rows,
                                                           int32_t* __restrict__ goff) {
  __shared__ int red[256];
  const int E_loc = E / R;
  const int e = blockIdx.x;
  const int ge = r * E_loc + e;
  const int tid = threadIdx.x;
  int part = 0;
  for (int i = tid; i < e * R; i += 256) {
    const int ep = i / R, s = i % R;
    part += counts[(size_t)s * E + r * E_loc + ep];
  }
  red[tid] = part;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (tid < o) red[tid] += red[tid + o];
    __syncthreads();
  }
  int base = red[0];
  if (tid == 0) goff[e] = base;
  for (int s = 0; s < R; ++s) {
    const int c = counts[(size_t)s * E + ge];
    const int64_t start = (int64_t)s * cap + offsets[(size_t)s * (E + 1) + ge];
    for (int j = tid; j < c; j += 256) group_rows[base + j] = (int32_t)(start + j);
    base += c;
  }
  if (e == E_loc - 1 && tid == 0) goff[E_loc] = base;
}

// Rows [rank_offsets[r], rank_offsets[r+1]) of the plan belong to rank r's
// experts.  Thread i < that count writes the token of row lo + i; threads
// 0..E_loc write the local group offsets.
__global__ __launch_bounds__(256) void local_rows_kernel(const int32_t* __restrict__ offsets,
                                                         const int32_t* __restrict__ rank_offsets,
                                                         const int32_t* __restrict__ row_to_slot,
                                                         int k, int E_loc, int r,
                                                         int32_t* __restrict__ local_tokens,
                                                         int32_t* __restrict__ local_offsets) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int lo = rank_offsets[r], hi = rank_offsets[r + 1];
  if (i < hi - lo) local_tokens[i] = row_to_slot[lo + i] / k;
  if (i <= E_loc) local_offsets[i] = offsets[(size_t)r * E_loc + i] - lo;
}

}  // namespace

size_t plan_ws_bytes(int N, int E) {
  const size_t n_tiles = (size_t)(N + kTile - 1) / kTile;
  return n_tiles * E * (sizeof(uint64_t) + 2 * sizeof(int32_t));
}

// Device address of `scratch` on the current device, looked up once per
// device with that device current and kept.
hipError_t plan_scratch(void** out) {
  static std::mutex mu;
  static void* addr[kPlanScratchMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kPlanScratchMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *out = addr[dev];
  return hipSuccess;
}

hipError_t launch_plan(const int32_t* ids, int N, int k, int E, int R, int32_t* counts,
                       int32_t* offsets, int32_t* rank_offsets, int32_t* slot_to_row,
                       int32_t* row_to_slot, void* ws, hipStream_t s) {
  const int n_tiles = (N + kTile - 1) / kTile;
  uint64_t* bits = reinterpret_cast<uint64_t*>(ws);
  int32_t* hist = reinterpret_cast<int32_t*>(bits + (size_t)n_tiles * E);
  int32_t* tile_base = hist + (size_t)n_tiles * E;
  if ((int64_t)n_tiles * N * k <= kPlanTileReads) {
    launch_k(plan_tile_kernel, n_tiles, 512, 0, s, ids, N, k, E, R, counts, offsets, rank_offsets,
             slot_to_row, row_to_slot);
    return hipGetLastError();
  }
  launch_k(plan_hist_kernel, n_tiles, 64, E * sizeof(uint64_t), s, ids, N, k, E, bits, hist);
  launch_k(plan_scan_kernel, 1, 512, 0, s, hist, n_tiles, E, R, tile_base, counts, offsets,
                                     rank_offsets);
  launch_k(plan_rank_kernel, n_tiles, 64, 0, s, ids, N, k, E, bits, tile_base, offsets, slot_to_row,
                                          row_to_slot);
  return hipGetLastError();
}

hipError_t launch_pack(int dtype, const void* x, const int32_t* slot_to_row, int N, int k, int d,
                       void* send, hipStream_t s) {
  const int64_t nb = ((int64_t)d * (dtype == 0 ? 4 : 2) / 16 + 63) / 64;
  dim3 grid((unsigned)((N * nb + 3) / 4));
#define FS_PACK(T, KC)                                                                         \
  launch_k(pack_kernel<T, KC>, grid, 256, 0, s, (const T*)x, slot_to_row, N, k, d, (T*)send, \
           (const float*)nullptr, (float*)nullptr)
#define FS_PACK_T(T)                 \
  switch (k) {                       \
    case 1: FS_PACK(T, 1); break;    \
    case 2: FS_PACK(T, 2); break;    \
    case 4: FS_PACK(T, 4); break;    \
    case 6: FS_PACK(T, 6); break;    \
    case 8: FS_PACK(T, 8); break;    \
    default: FS_PACK(T, 0); break;   \
  }
  if (dtype == 0) {
    FS_PACK_T(float);
  } else {
    FS_PACK_T(bf16_t);
  }
#undef FS_PACK_T
#undef FS_PACK
  return hipGetLastError();
}

hipError_t launch_pack_fp8(const uint8_t* codes, const float* scales, const int32_t* slot_to_row,
                           int N, int k, int d, uint8_t* send_codes, float* send_scales,
                           hipStream_t s) {
  const int64_t nb = ((int64_t)d / 16 + 63) / 64;
  dim3 grid((unsigned)((N * nb + 3) / 4));
#define FS_PACK8(KC)                                                                        \
  launch_k(pack_kernel<uint8_t, KC>, grid, 256, 0, s, codes, slot_to_row, N, k, d, send_codes, \
           scales, send_scales)
  switch (k) {
    case 1: FS_PACK8(1); break;
    case 2: FS_PACK8(2); break;
    case 4: FS_PACK8(4); break;
    case 6: FS_PACK8(6); break;
    case 8: FS_PACK8(8); break;
    default: FS_PACK8(0); break;
  }
#undef FS_PACK8
  return hipGetLastError();
}

hipError_t launch_local_rows(const int32_t* offsets, const int32_t* rank_offsets,
                             const int32_t* row_to_slot, int N, int k, int E, int R, int r,
                             int32_t* local_tokens, int32_t* local_offsets, hipStream_t s) {
  const int E_loc = E / R;
  const int64_t rows = (int64_t)N * k, n = rows > E_loc + 1 ? rows : E_loc + 1;
  launch_k(local_rows_kernel, (unsigned)((n + 255) / 256), 256, 0, s,
      offsets, rank_offsets, row_to_slot, k, E_loc, r, local_tokens, local_offsets);
  return hipGetLastError();
}

hipError_t launch_receive_rows(const int32_t* src_counts, const int32_t* src_offsets, int R,
                               int E, int r, int64_t cap, int32_t* group_rows,
                               int32_t* group_offsets, hipStream_t s) {
  launch_k(receive_rows_kernel, E / R, 256, 0, s, src_counts, src_offsets, R, E, r, cap, group_rows,
                                            group_offsets);
  return hipGetLastError();
}

}  // namespace fs
