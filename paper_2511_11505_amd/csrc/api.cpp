// C ABI of libfarskip.so: argument checks, workspace layout, the two-phase
// FarSkip block driver and per-kernel timing.  Every check runs on the host
// before anything is enqueued.

#include <hip/hip_runtime.h>

#include <mutex>
#include <string>
#include <vector>

#include "../../include/farskip.h"
#include "internal.hpp"

namespace {

thread_local std::string g_msg;

fs_status fail(fs_status st, const std::string& m) {
  g_msg = m;
  return st;
}
fs_status hip_fail(hipError_t e, const char* where) {
  g_msg = std::string(where) + ": " + hipGetErrorString(e);
  return FS_ERR_HIP;
}
#define FS_HIP(expr, where)                     \
  do {                                          \
    hipError_t e_ = (expr);                     \
    if (e_ != hipSuccess) return hip_fail(e_, where); \
  } while (0)

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
bool aligned4(const void* p) { return ((uintptr_t)p & 3u) == 0; }

#define NEED(ptr, name)                                                                      \
  do {                                                                                       \
    if (!(ptr)) return fail(FS_ERR_INVALID, std::string(name) + " must not be NULL");        \
    if (!aligned16(ptr)) return fail(FS_ERR_INVALID, std::string(name) + " must be 16-byte aligned"); \
  } while (0)
// int32 index arrays and fp32 gate arrays are read element by element
#define NEED4(ptr, name)                                                                     \
  do {                                                                                       \
    if (!(ptr)) return fail(FS_ERR_INVALID, std::string(name) + " must not be NULL");        \
    if (!aligned4(ptr)) return fail(FS_ERR_INVALID, std::string(name) + " must be 4-byte aligned"); \
  } while (0)
#define OPT4(ptr, name)                                                                      \
  do {                                                                                       \
    if ((ptr) && !aligned4(ptr))                                                             \
      return fail(FS_ERR_INVALID, std::string(name) + " must be 4-byte aligned");            \
  } while (0)
#define OPT(ptr, name)                                                                       \
  do {                                                                                       \
    if ((ptr) && !aligned16(ptr))                                                            \
      return fail(FS_ERR_INVALID, std::string(name) + " must be 16-byte aligned");           \
  } while (0)

size_t elem(int dtype) { return dtype == FS_F32 ? 4 : 2; }
size_t align256(size_t b) { return (b + 255) / 256 * 256; }

fs_status check_desc(const fs_moe_desc* d) {
  if (!d) return fail(FS_ERR_INVALID, "desc must not be NULL");
  if (d->abi_version != FS_ABI_VERSION) return fail(FS_ERR_INVALID, "desc->abi_version mismatch");
  if (d->n_tokens < 0) return fail(FS_ERR_INVALID, "n_tokens must be >= 0");
  if (d->hidden <= 0) return fail(FS_ERR_INVALID, "hidden must be > 0");
  if (d->hidden % 128 != 0) return fail(FS_ERR_UNSUPPORTED, "hidden must be a multiple of 128");
  if (d->n_experts < 1) return fail(FS_ERR_INVALID, "n_experts must be >= 1");
  if (d->n_experts > 512) return fail(FS_ERR_UNSUPPORTED, "n_experts must be <= 512");
  if (d->top_k < 1 || d->top_k > d->n_experts)
    return fail(FS_ERR_INVALID, "top_k must be in [1, n_experts]");
  if (d->top_k > 32) return fail(FS_ERR_UNSUPPORTED, "top_k must be <= 32");
  if (d->n_groups < 1 || d->n_experts % d->n_groups != 0)
    return fail(FS_ERR_INVALID, "n_groups must divide n_experts");
  if (d->n_groups > 64) return fail(FS_ERR_UNSUPPORTED, "n_groups must be <= 64");
  if (d->n_groups > 1) {
    if (d->topk_groups < 1 || d->topk_groups > d->n_groups)
      return fail(FS_ERR_INVALID, "topk_groups must be in [1, n_groups]");
    if (d->top_k > d->topk_groups * (d->n_experts / d->n_groups))
      return fail(FS_ERR_INVALID, "top_k exceeds the experts of the kept groups");
  }
  if (d->score != FS_SOFTMAX && d->score != FS_SIGMOID)
    return fail(FS_ERR_INVALID, "score must be FS_SOFTMAX or FS_SIGMOID");
  if (d->norm_topk != 0 && d->norm_topk != 1) return fail(FS_ERR_INVALID, "norm_topk must be 0/1");
  if (!(d->routed_scale == d->routed_scale)) return fail(FS_ERR_INVALID, "routed_scale is NaN");
  if (d->ffn <= 0) return fail(FS_ERR_INVALID, "ffn must be > 0");
  if (d->ffn % 64 != 0) return fail(FS_ERR_UNSUPPORTED, "ffn must be a multiple of 64");
  if (d->n_shared < 0) return fail(FS_ERR_INVALID, "n_shared must be >= 0");
  if (d->n_shared > 0) {
    if (d->ffn_shared <= 0) return fail(FS_ERR_INVALID, "ffn_shared must be > 0");
    if ((int64_t)d->n_shared * d->ffn_shared % 64 != 0)
      return fail(FS_ERR_UNSUPPORTED, "n_shared * ffn_shared must be a multiple of 64");
  }
  if (d->ep_size < 1 || d->n_experts % d->ep_size != 0)
    return fail(FS_ERR_INVALID, "ep_size must divide n_experts");
  if (d->ep_rank < 0 || d->ep_rank >= d->ep_size) return fail(FS_ERR_INVALID, "ep_rank out of range");
  if (d->dtype != FS_F32 && d->dtype != FS_BF16) return fail(FS_ERR_INVALID, "dtype must be FS_F32 or FS_BF16");
  if ((int64_t)d->ep_size * d->n_tokens * d->top_k >= (int64_t)1 << 31)
    return fail(FS_ERR_UNSUPPORTED, "ep_size * n_tokens * top_k must be < 2^31");
  return FS_OK;
}

hipStream_t S(fs_stream s) { return reinterpret_cast<hipStream_t>(s); }

// ---------------------------------------------------------------- profiling
// A timing window per (kernel id, stream).  Kernels launched on the stream
// while its window is open (fs::launch_k) record the window's events from
// their dispatch packets: the first kernel's start and every kernel's end,
// so the window measures kernel time from the first start to the last end,
// without the launch latency before the first kernel.  A window with no
// kernel launch (a copy) falls back to events recorded on the stream.
struct ProfState {
  std::mutex mu;
  bool on = false;
  uint32_t mask = (1u << FS_K_COUNT) - 1;   // kernel ids that open windows
  struct Window {
    int kernel;
    hipStream_t s;
    hipEvent_t a, b, k0;  // stream-recorded start, end, first kernel start
    bool kern;
  };
  struct Rec {
    int kernel;
    hipEvent_t a, b, spare;
  };
  std::vector<Window> windows;   // open
  std::vector<Rec> open;         // closed, not yet read
  std::vector<hipEvent_t> pool;  // reusable events
  double total_ms[FS_K_COUNT] = {};
  int64_t count[FS_K_COUNT] = {};
};
ProfState& prof() {
  static ProfState p;
  return p;
}
hipEvent_t take_event(ProfState& p) {
  if (!p.pool.empty()) {
    hipEvent_t e = p.pool.back();
    p.pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// ---------------------------------------------------------------- workspace
struct Carve {
  char* base;
  size_t off = 0;
  void* take(size_t bytes) {
    void* p = base ? base + off : nullptr;
    off += align256(bytes);
    return p;
  }
};

size_t router_bytes(const fs_moe_desc* d) {
  return align256(fs::router_ws_bytes(d->dtype, d->n_tokens, d->hidden, d->n_experts));
}
size_t plan_bytes(const fs_moe_desc* d) { return align256(fs::plan_ws_bytes(d->n_tokens, d->n_experts)); }

// Workspace of one FFN inside the block: bf16, or FP8 (row codes and scales
// of the input, then the FP8 FFN's own workspace).
size_t block_ffn_bytes(const fs_moe_desc* d, int64_t rows, int ffn, bool fp8) {
  if (!fp8) return align256(fs::ffn_ws_bytes(d->dtype, rows, ffn, d->hidden));
  return align256((size_t)rows * d->hidden) + align256((size_t)rows * 4) +
         align256(fs::ffn_fp8_ws_bytes(rows, ffn, d->hidden));
}

// FP8 pack: the plan's workspace, then the N token rows' codes and scales.
size_t plan_fp8_bytes(const fs_moe_desc* d) {
  return plan_bytes(d) + align256((size_t)d->n_tokens * d->hidden) + align256((size_t)d->n_tokens * 4);
}

// Routed experts inside the block: bf16, or FP8 reading the received codes
// (the FFN's own workspace only).
size_t routed_ffn_bytes(const fs_moe_desc* d, int64_t max_rows, bool fp8) {
  if (!fp8) return block_ffn_bytes(d, max_rows, d->ffn, false);
  return align256(fs::ffn_fp8_ws_bytes(max_rows, d->ffn, d->hidden));
}

size_t block_bytes(const fs_moe_desc* d, int64_t max_rows, bool fp8_routed, bool fp8_shared) {
  size_t b = router_bytes(d) + (fp8_routed ? plan_fp8_bytes(d) : plan_bytes(d)) +
             routed_ffn_bytes(d, max_rows, fp8_routed);
  if (d->n_shared > 0) b += block_ffn_bytes(d, d->n_tokens, d->n_shared * d->ffn_shared, fp8_shared);
  return b;
}

// Link model of the stand-in collectives (fs_standin_link); links == 0:
// device-to-device copies at HBM speed.
struct LinkModel {
  int links = 0;
  double bytes_per_s = 0.0;
  int workgroups = 0;
};
std::mutex g_link_mu;
LinkModel g_link;

LinkModel link_model() {
  std::lock_guard<std::mutex> g(g_link_mu);
  return g_link;
}

// One stand-in copy of a collective moving `bytes` per GPU: `factor` 1 for
// an all-to-all (each of the links + 1 GPUs' shares crosses its own link,
// all links at once: bytes / ((links + 1) rate)), 2 for a ring all-reduce
// over every link (2 (n - 1) / n bytes out of each GPU over n - 1 links).
hipError_t standin_copy(void* dst, const void* src, size_t bytes, double factor, hipStream_t s) {
  const LinkModel m = link_model();
  if (m.links == 0) return hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, s);
  const double seconds = factor * (double)bytes / ((double)(m.links + 1) * m.bytes_per_s);
  return fs::launch_paced_copy(dst, src, bytes, seconds, m.workgroups, s);
}

}  // namespace

namespace fs {
void prof_begin(int kernel, hipStream_t s) {
  ProfState& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  if (!p.on || !((p.mask >> kernel) & 1u)) return;
  hipEvent_t a = take_event(p), b = take_event(p), k0 = take_event(p);
  if (!a || !b || !k0 || hipEventRecord(a, s) != hipSuccess) {
    for (hipEvent_t e : {a, b, k0})
      if (e) p.pool.push_back(e);
    return;
  }
  p.windows.push_back({kernel, s, a, b, k0, false});
}
void prof_kernel_events(hipStream_t s, hipEvent_t* start, hipEvent_t* stop) {
  *start = *stop = nullptr;
  ProfState& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  if (!p.on) return;
  for (auto it = p.windows.rbegin(); it != p.windows.rend(); ++it) {
    if (it->s != s) continue;
    *start = it->kern ? nullptr : it->k0;
    *stop = it->b;
    it->kern = true;
    return;
  }
}
void prof_end(int kernel, hipStream_t s) {
  ProfState& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  for (auto it = p.windows.begin(); it != p.windows.end(); ++it) {
    if (it->kernel != kernel || it->s != s) continue;
    const ProfState::Window w = *it;
    p.windows.erase(it);
    if (w.kern) {
      p.open.push_back({kernel, w.k0, w.b, w.a});
    } else if (hipEventRecord(w.b, s) == hipSuccess) {
      p.open.push_back({kernel, w.a, w.b, w.k0});
    } else {
      for (hipEvent_t e : {w.a, w.b, w.k0}) p.pool.push_back(e);
    }
    return;
  }
}
}  // namespace fs

extern "C" {

const char* fs_status_string(int32_t status) {
  switch (status) {
    case FS_OK: return "FS_OK";
    case FS_ERR_INVALID: return "FS_ERR_INVALID";
    case FS_ERR_UNSUPPORTED: return "FS_ERR_UNSUPPORTED";
    case FS_ERR_WORKSPACE: return "FS_ERR_WORKSPACE";
    case FS_ERR_HIP: return "FS_ERR_HIP";
    default: return "FS_ERR_UNKNOWN";
  }
}

const char* fs_last_error_message(void) { return g_msg.c_str(); }

int32_t fs_abi_version(void) { return FS_ABI_VERSION; }

fs_status fs_workspace_size(const fs_moe_desc* desc, int32_t op, int64_t max_rows, int32_t ffn,
                            size_t* bytes) {
  fs_status st = check_desc(desc);
  if (st != FS_OK) return st;
  if (!bytes) return fail(FS_ERR_INVALID, "bytes must not be NULL");
  if (max_rows < 0) return fail(FS_ERR_INVALID, "max_rows must be >= 0");
  switch (op) {
    case FS_OP_ROUTER_TOPK: *bytes = router_bytes(desc); return FS_OK;
    case FS_OP_DISPATCH_PACK: *bytes = plan_bytes(desc); return FS_OK;
    case FS_OP_GROUPED_FFN:
      if (ffn <= 0) return fail(FS_ERR_INVALID, "ffn must be > 0");
      *bytes = fs::ffn_ws_bytes(desc->dtype, max_rows, ffn, desc->hidden);
      return FS_OK;
    case FS_OP_GROUPED_FFN_FP8:
      if (ffn <= 0) return fail(FS_ERR_INVALID, "ffn must be > 0");
      *bytes = fs::ffn_fp8_ws_bytes(max_rows, ffn, desc->hidden);
      return FS_OK;
    case FS_OP_BLOCK: *bytes = block_bytes(desc, max_rows, false, false); return FS_OK;
    case FS_OP_DISPATCH_PACK_FP8: *bytes = plan_fp8_bytes(desc); return FS_OK;
    case FS_OP_BLOCK_FP8: {
      size_t a = block_bytes(desc, max_rows, true, true), b = block_bytes(desc, max_rows, true, false);
      size_t c = block_bytes(desc, max_rows, false, true);
      *bytes = a > b ? (a > c ? a : c) : (b > c ? b : c);
      return FS_OK;
    }
    default: return fail(FS_ERR_INVALID, "unknown op");
  }
}

// ---- router + top-k
static fs_status router_impl(const fs_moe_desc* d, const void* x, const void* w_router,
                             const float* sel_bias, const float* logits_in, float* logits_out,
                             int32_t* topk_ids, float* topk_w, void* ws, hipStream_t s) {
  const int N = d->n_tokens, D = d->hidden, E = d->n_experts;
  if (N == 0) return FS_OK;
  const float* src = logits_in;
  int n_partials = 0;
  float* lout = logits_out;
  if (!logits_in) {
    Carve c{reinterpret_cast<char*>(ws)};
    float* scratch_logits = reinterpret_cast<float*>(c.take((size_t)N * E * sizeof(float)));
    const bool split = fs::router_split(d->dtype, N, D, E);
    float* dst;
    if (split) {
      dst = reinterpret_cast<float*>(c.take((size_t)fs::router_slices(D) * N * E * sizeof(float)));
      n_partials = fs::router_slices(D);
    } else {
      dst = logits_out ? logits_out : scratch_logits;
      lout = nullptr;  // already written by the router kernel
    }
    fs::prof_begin(FS_K_ROUTER, s);
    FS_HIP(fs::launch_router_logits(d->dtype, x, w_router, N, D, E, split, dst, s), "router");
    fs::prof_end(FS_K_ROUTER, s);
    src = dst;
  } else {
    lout = (logits_out && logits_out != logits_in) ? logits_out : nullptr;
  }
  fs::prof_begin(FS_K_TOPK, s);
  FS_HIP(fs::launch_topk(src, n_partials, N, E, sel_bias, d->score, d->top_k, d->n_groups,
                         d->n_groups > 1 ? d->topk_groups : 1, d->norm_topk, d->routed_scale,
                         lout, topk_ids, topk_w, s),
         "topk");
  fs::prof_end(FS_K_TOPK, s);
  return FS_OK;
}

fs_status fs_router_topk(const fs_moe_desc* desc, const void* x, const void* w_router,
                         const float* sel_bias, const float* logits_in, float* logits_out,
                         int32_t* topk_ids, float* topk_w, void* ws, size_t ws_bytes,
                         fs_stream stream) {
  fs_status st = check_desc(desc);
  if (st != FS_OK) return st;
  if (desc->n_tokens == 0) return FS_OK;
  if (!logits_in) {
    NEED(x, "x");
    NEED(w_router, "w_router");
    if (ws_bytes < router_bytes(desc))
      return fail(FS_ERR_WORKSPACE, "workspace smaller than fs_workspace_size(FS_OP_ROUTER_TOPK)");
    NEED(ws, "ws");
  } else {
    OPT4(logits_in, "logits_in");
  }
  if (sel_bias && desc->score == FS_SOFTMAX)
    return fail(FS_ERR_UNSUPPORTED, "a selection bias is defined for sigmoid scoring only");
  OPT4(sel_bias, "sel_bias");
  OPT4(logits_out, "logits_out");
  NEED4(topk_ids, "topk_ids");
  NEED4(topk_w, "topk_w");
  return router_impl(desc, x, w_router, sel_bias, logits_in, logits_out, topk_ids, topk_w, ws,
                     S(stream));
}

// ---- dispatch plan + pack
static fs_status plan_pack_impl(const fs_moe_desc* d, const int32_t* ids, const void* x,
                                int32_t* counts, int32_t* offsets, int32_t* rank_offsets,
                                int32_t* s2r, int32_t* r2s, void* send, void* ws, hipStream_t s) {
  const int N = d->n_tokens;
  if (N == 0) return FS_OK;
  fs::prof_begin(FS_K_PLAN, s);
  FS_HIP(fs::launch_plan(ids, N, d->top_k, d->n_experts, d->ep_size, counts, offsets,
                         rank_offsets, s2r, r2s, ws, s),
         "plan");
  fs::prof_end(FS_K_PLAN, s);
  if (send) {
    fs::prof_begin(FS_K_PACK, s);
    FS_HIP(fs::launch_pack(d->dtype, x, s2r, N, d->top_k, d->hidden, send, s), "pack");
    fs::prof_end(FS_K_PACK, s);
  }
  return FS_OK;
}

// FP8 rows: quantise the N token rows once, plan, pack codes and scales.
static fs_status plan_pack_fp8_impl(const fs_moe_desc* d, const int32_t* ids, const void* x,
                                    int32_t* counts, int32_t* offsets, int32_t* rank_offsets,
                                    int32_t* s2r, int32_t* r2s, uint8_t* send_codes,
                                    float* send_scales, void* ws, hipStream_t s) {
  const int N = d->n_tokens, D = d->hidden;
  if (N == 0) return FS_OK;
  char* base = static_cast<char*>(ws) + plan_bytes(d);
  uint8_t* xq = reinterpret_cast<uint8_t*>(base);
  float* xs = reinterpret_cast<float*>(base + align256((size_t)N * D));
  fs::prof_begin(FS_K_QUANTIZE, s);
  FS_HIP(fs::launch_quantize_fp8(1, x, N, D, nullptr, xq, xs, s), "quantize_fp8");
  fs::prof_end(FS_K_QUANTIZE, s);
  fs_status st = plan_pack_impl(d, ids, nullptr, counts, offsets, rank_offsets, s2r, r2s, nullptr,
                                ws, s);
  if (st != FS_OK) return st;
  fs::prof_begin(FS_K_PACK, s);
  FS_HIP(fs::launch_pack_fp8(xq, xs, s2r, N, d->top_k, D, send_codes, send_scales, s), "pack_fp8");
  fs::prof_end(FS_K_PACK, s);
  return FS_OK;
}

fs_status fs_dispatch_pack_fp8(const fs_moe_desc* desc, const int32_t* topk_ids, const void* x,
                               int32_t* expert_counts, int32_t* expert_offsets,
                               int32_t* rank_offsets, int32_t* slot_to_row, int32_t* row_to_slot,
                               uint8_t* send_codes, float* send_scales, void* ws, size_t ws_bytes,
                               fs_stream stream) {
  fs_status st = check_desc(desc);
  if (st != FS_OK) return st;
  if (desc->dtype != FS_BF16) return fail(FS_ERR_UNSUPPORTED, "FP8 rows need a bf16 desc");
  if (desc->hidden % 16 != 0) return fail(FS_ERR_UNSUPPORTED, "FP8 rows need hidden % 16 == 0");
  if (desc->n_tokens == 0) return FS_OK;
  NEED4(topk_ids, "topk_ids");
  NEED4(expert_counts, "expert_counts");
  NEED4(expert_offsets, "expert_offsets");
  NEED4(rank_offsets, "rank_offsets");
  NEED4(slot_to_row, "slot_to_row");
  NEED4(row_to_slot, "row_to_slot");
  NEED(x, "x");
  NEED(send_codes, "send_codes");
  NEED4(send_scales, "send_scales");
  if (ws_bytes < plan_fp8_bytes(desc))
    return fail(FS_ERR_WORKSPACE, "workspace smaller than fs_workspace_size(FS_OP_DISPATCH_PACK_FP8)");
  NEED(ws, "ws");
  return plan_pack_fp8_impl(desc, topk_ids, x, expert_counts, expert_offsets, rank_offsets,
                            slot_to_row, row_to_slot, send_codes, send_scales, ws, S(stream));
}

fs_status fs_dispatch_pack(const fs_moe_desc* desc, const int32_t* topk_ids, const void* x,
                           int32_t* expert_counts, int32_t* expert_offsets,
                           int32_t* rank_offsets, int32_t* slot_to_row, int32_t* row_to_slot,
                           void* send, void* ws, size_t ws_bytes, fs_stream stream) {
  fs_status st = check_desc(desc);
  if (st != FS_OK) return st;
  if (desc->n_tokens == 0) return FS_OK;
  NEED4(topk_ids, "topk_ids");
  NEED4(expert_counts, "expert_counts");
  NEED4(expert_offsets, "expert_offsets");
  NEED4(rank_offsets, "rank_offsets");
  NEED4(slot_to_row, "slot_to_row");
  NEED4(row_to_slot, "row_to_slot");
  OPT(send, "send");
  if (send) NEED(x, "x");
  if (ws_bytes < plan_bytes(desc))
    return fail(FS_ERR_WORKSPACE, "workspace smaller than fs_workspace_size(FS_OP_DISPATCH_PACK)");
  NEED(ws, "ws");
  return plan_pack_impl(desc, topk_ids, x, expert_counts, expert_offsets, rank_offsets,
                        slot_to_row, row_to_slot, send, ws, S(stream));
}

fs_status fs_dispatch_pack_noalloc(const fs_moe_desc* desc, const int32_t* topk_ids,
                                   const void* x, int32_t* expert_counts,
                                   int32_t* expert_offsets, int32_t* rank_offsets,
                                   int32_t* slot_to_row, int32_t* row_to_slot, void* send,
                                   fs_stream stream) {
  fs_status st = check_desc(desc);
  if (st != FS_OK) return st;
  if (desc->n_tokens == 0) return FS_OK;
  NEED4(topk_ids, "topk_ids");
  NEED4(expert_counts, "expert_counts");
  NEED4(expert_offsets, "expert_offsets");
  NEED4(rank_offsets, "rank_offsets");
  NEED4(slot_to_row, "slot_to_row");
  NEED4(row_to_slot, "row_to_slot");
  OPT(send, "send");
  if (send) NEED(x, "x");
  const size_t need = fs::plan_ws_bytes(desc->n_tokens, desc->n_experts);
  if (need > fs::kPlanScratchBytes)
    return fail(FS_ERR_UNSUPPORTED,
                "fs_dispatch_pack_noalloc: the plan needs " + std::to_string(need) +
                    " bytes of scratch, more than its fixed " +
                    std::to_string(fs::kPlanScratchBytes) +
                    " (ceil(n_tokens / 64) * n_experts must be <= 262144); use fs_dispatch_pack");
  hipStream_t s = S(stream);
  if (s) {
    int cur = 0;
    hipDevice_t sdev = 0;
    FS_HIP(hipGetDevice(&cur), "hipGetDevice");
    FS_HIP(hipStreamGetDevice(s, &sdev), "hipStreamGetDevice");
    if ((int)sdev != cur)
      return fail(FS_ERR_INVALID, "fs_dispatch_pack_noalloc: the stream belongs to device " +
                                      std::to_string((int)sdev) + ", not the current device " +
                                      std::to_string(cur));
  }
  void* scratch = nullptr;
  FS_HIP(fs::plan_scratch(&scratch), "plan scratch address");
  // the plan kernels write every scratch word they later read, so the last
  // call's contents need no clearing; no timing windows are opened (they
  // may create events)
  FS_HIP(fs::launch_plan(topk_ids, desc->n_tokens, desc->top_k, desc->n_experts, desc->ep_size,
                         expert_counts, expert_offsets, rank_offsets, slot_to_row, row_to_slot,
                         scratch, s),
         "plan");
  if (send)
    FS_HIP(fs::launch_pack(desc->dtype, x, slot_to_row, desc->n_tokens, desc->top_k,
                           desc->hidden, send, s),
           "pack");
  return FS_OK;
}

fs_status fs_receive_rows(const fs_moe_desc* desc, const int32_t* src_counts,
                          const int32_t* src_offsets, int32_t* group_rows, int32_t* group_offsets,
                          fs_stream stream) {
  fs_status st = check_desc(desc);
  if (st != FS_OK) return st;
  NEED4(src_counts, "src_counts");
  NEED4(src_offsets, "src_offsets");
  NEED4(group_rows, "group_rows");
  NEED4(group_offsets, "group_offsets");
  FS_HIP(fs::launch_receive_rows(src_counts, src_offsets, desc->ep_size, desc->n_experts,
                                 desc->ep_rank, (int64_t)desc->n_tokens * desc->top_k,
                                 group_rows, group_offsets, S(stream)),
         "receive_rows");
  return FS_OK;
}

fs_status fs_local_rows(const fs_moe_desc* desc, const int32_t* expert_offsets,
                        const int32_t* rank_offsets, const int32_t* row_to_slot,
                        int32_t* local_tokens, int32_t* local_offsets, fs_stream stream) {
  fs_status st = check_desc(desc);
  if (st != FS_OK) return st;
  if (desc->n_tokens == 0) return FS_OK;
  NEED4(expert_offsets, "expert_offsets");
  NEED4(rank_offsets, "rank_offsets");
  NEED4(row_to_slot, "row_to_slot");
  NEED4(local_tokens, "local_tokens");
  NEED4(local_offsets, "local_offsets");
  FS_HIP(fs::launch_local_rows(expert_offsets, rank_offsets, row_to_slot, desc->n_tokens,
                               desc->top_k, desc->n_experts, desc->ep_size, desc->ep_rank,
                               local_tokens, local_offsets, S(stream)),
         "local_rows");
  return FS_OK;
}

// ---- grouped FFN
static fs_status ffn_checks(const fs_moe_desc* desc, int32_t n_groups, int32_t ffn,
                            const int32_t* group_offsets, int64_t max_rows) {
  fs_status st = check_desc(desc);
  if (st != FS_OK) return st;
  if (n_groups < 1) return fail(FS_ERR_INVALID, "n_groups must be >= 1");
  if (n_groups > 512) return fail(FS_ERR_UNSUPPORTED, "n_groups must be <= 512");
  if (ffn <= 0) return fail(FS_ERR_INVALID, "ffn must be > 0");
  if (ffn % 64 != 0) return fail(FS_ERR_UNSUPPORTED, "ffn must be a multiple of 64");
  if (max_rows < 0) return fail(FS_ERR_INVALID, "max_rows must be >= 0");
  if (max_rows >= ((int64_t)1 << 31)) return fail(FS_ERR_UNSUPPORTED, "max_rows must be < 2^31");
  if (!group_offsets && n_groups != 1)
    return fail(FS_ERR_INVALID, "group_offsets may be NULL only with n_groups == 1");
  return FS_OK;
}

fs_status fs_grouped_expert_ffn_gathered(const fs_moe_desc* desc, int32_t n_groups, int32_t ffn,
                                         const void* x, const int32_t* gather_rows,
                                         const int32_t* group_offsets, int64_t max_rows,
                                         const void* w_gate_up, const void* w_down, void* y,
                                         void* ws, size_t ws_bytes, fs_stream stream) {
  fs_status st = ffn_checks(desc, n_groups, ffn, group_offsets, max_rows);
  if (st != FS_OK) return st;
  if (max_rows == 0) return FS_OK;
  NEED(x, "x");
  NEED4(gather_rows, "gather_rows");
  OPT4(group_offsets, "group_offsets");
  NEED(w_gate_up, "w_gate_up");
  NEED(w_down, "w_down");
  NEED(y, "y");
  if (ws_bytes < fs::ffn_ws_bytes(desc->dtype, max_rows, ffn, desc->hidden))
    return fail(FS_ERR_WORKSPACE, "workspace smaller than fs_workspace_size(FS_OP_GROUPED_FFN)");
  NEED(ws, "ws");
  FS_HIP(fs::launch_grouped_ffn(desc->dtype, n_groups, ffn, desc->hidden, x, gather_rows,
                                nullptr, group_offsets, max_rows, w_gate_up, w_down, y, ws,
                                S(stream), FS_K_GATE_UP),
         "grouped_ffn_gathered");
  return FS_OK;
}

fs_status fs_quantize_fp8(int32_t dtype, int64_t rows, int32_t cols, const void* src,
                          uint8_t* codes, float* scales, fs_stream stream) {
  if (dtype != FS_F32 && dtype != FS_BF16) return fail(FS_ERR_INVALID, "dtype must be FS_F32 or FS_BF16");
  if (rows < 0 || cols <= 0) return fail(FS_ERR_INVALID, "rows >= 0 and cols > 0 required");
  if (cols % 16 != 0) return fail(FS_ERR_UNSUPPORTED, "cols must be a multiple of 16");
  if (rows == 0) return FS_OK;
  NEED(src, "src");
  NEED(codes, "codes");
  NEED4(scales, "scales");
  FS_HIP(fs::launch_quantize_fp8(dtype == FS_F32 ? 0 : 1, src, rows, cols, nullptr, codes, scales,
                                 S(stream)),
         "quantize_fp8");
  return FS_OK;
}

fs_status fs_grouped_expert_ffn_fp8(const fs_moe_desc* desc, int32_t n_groups, int32_t ffn,
                                    const uint8_t* x_codes, const float* x_scales,
                                    const int32_t* group_rows, const int32_t* group_offsets,
                                    int64_t max_rows, const uint8_t* w_gate_up,
                                    const float* s_gate_up, const uint8_t* w_down,
                                    const float* s_down, void* out_rows, void* ws, size_t ws_bytes,
                                    fs_stream stream) {
  fs_status st = ffn_checks(desc, n_groups, ffn, group_offsets, max_rows);
  if (st != FS_OK) return st;
  if (desc->dtype != FS_BF16) return fail(FS_ERR_UNSUPPORTED, "FP8 experts write bf16 rows (dtype FS_BF16)");
  if (ffn % 128 != 0 || desc->hidden % 256 != 0)
    return fail(FS_ERR_UNSUPPORTED, "FP8 experts need ffn % 128 == 0 and hidden % 256 == 0");
  if (max_rows == 0) return FS_OK;
  NEED(x_codes, "x_codes");
  NEED4(x_scales, "x_scales");
  OPT4(group_rows, "group_rows");
  OPT4(group_offsets, "group_offsets");
  NEED(w_gate_up, "w_gate_up");
  NEED4(s_gate_up, "s_gate_up");
  NEED(w_down, "w_down");
  NEED4(s_down, "s_down");
  NEED(out_rows, "out_rows");
  if (ws_bytes < fs::ffn_fp8_ws_bytes(max_rows, ffn, desc->hidden))
    return fail(FS_ERR_WORKSPACE, "workspace smaller than fs_workspace_size(FS_OP_GROUPED_FFN_FP8)");
  NEED(ws, "ws");
  FS_HIP(fs::launch_grouped_ffn_fp8(n_groups, ffn, desc->hidden, x_codes, x_scales, group_rows,
                                    group_rows, group_offsets, max_rows, w_gate_up, s_gate_up,
                                    w_down, s_down, out_rows, ws, S(stream),
                                    group_offsets ? FS_K_GATE_UP : FS_K_SHARED_GATE_UP),
         "grouped_ffn_fp8");
  return FS_OK;
}

fs_status fs_grouped_expert_ffn(const fs_moe_desc* desc, int32_t n_groups, int32_t ffn,
                                const void* in_rows, const int32_t* group_rows,
                                const int32_t* group_offsets, int64_t max_rows,
                                const void* w_gate_up, const void* w_down, void* out_rows,
                                void* ws, size_t ws_bytes, fs_stream stream) {
  fs_status st = ffn_checks(desc, n_groups, ffn, group_offsets, max_rows);
  if (st != FS_OK) return st;
  if (max_rows == 0) return FS_OK;
  NEED(in_rows, "in_rows");
  OPT4(group_rows, "group_rows");
  OPT4(group_offsets, "group_offsets");
  NEED(w_gate_up, "w_gate_up");
  NEED(w_down, "w_down");
  NEED(out_rows, "out_rows");
  if (ws_bytes < fs::ffn_ws_bytes(desc->dtype, max_rows, ffn, desc->hidden))
    return fail(FS_ERR_WORKSPACE, "workspace smaller than fs_workspace_size(FS_OP_GROUPED_FFN)");
  NEED(ws, "ws");
  // one group of max_rows rows (the shared-expert / dense form) is timed
  // apart from the grouped routed-expert form
  FS_HIP(fs::launch_grouped_ffn(desc->dtype, n_groups, ffn, desc->hidden, in_rows, group_rows,
                                group_rows, group_offsets, max_rows, w_gate_up, w_down, out_rows, ws,
                                S(stream), group_offsets ? FS_K_GATE_UP : FS_K_SHARED_GATE_UP),
         "grouped_ffn");
  return FS_OK;
}

fs_status fs_expert_weights_fragment_order(int32_t dtype, int64_t n_mats, int32_t rows,
                                           int32_t cols, const void* src, void* dst,
                                           fs_stream stream) {
  if (dtype != FS_BF16) return fail(FS_ERR_UNSUPPORTED, "fragment order is for bf16 weights");
  if (n_mats < 0 || rows <= 0 || cols <= 0) return fail(FS_ERR_INVALID, "bad matrix shape");
  if (rows % 32 != 0 || cols % 16 != 0)
    return fail(FS_ERR_UNSUPPORTED, "fragment order needs rows % 32 == 0 and cols % 16 == 0");
  if (n_mats == 0) return FS_OK;
  NEED(src, "src");
  NEED(dst, "dst");
  const size_t bytes = (size_t)n_mats * rows * cols * 2;
  const char *a = static_cast<const char*>(src), *b = static_cast<const char*>(dst);
  if (a < b + bytes && b < a + bytes) return fail(FS_ERR_INVALID, "src and dst overlap");
  FS_HIP(fs::launch_fragment_order(src, n_mats, rows, cols, dst, S(stream)), "fragment_order");
  return FS_OK;
}

static bool fo_shape_ok(const fs_moe_desc* d, int32_t ffn) {
  return d->dtype == FS_BF16 && ffn % 128 == 0 && d->hidden % 256 == 0;
}

fs_status fs_expert_weights_fragment_order_fp8(int64_t n_mats, int32_t rows, int32_t cols,
                                               const uint8_t* src, uint8_t* dst,
                                               fs_stream stream) {
  if (n_mats < 0 || rows <= 0 || cols <= 0) return fail(FS_ERR_INVALID, "bad matrix shape");
  if (rows % 32 != 0 || cols % 64 != 0)
    return fail(FS_ERR_UNSUPPORTED, "FP8 fragment order needs rows % 32 == 0 and cols % 64 == 0");
  if (n_mats == 0) return FS_OK;
  NEED(src, "src");
  NEED(dst, "dst");
  const size_t bytes = (size_t)n_mats * rows * cols;
  const char *a = reinterpret_cast<const char*>(src), *b = reinterpret_cast<const char*>(dst);
  if (a < b + bytes && b < a + bytes) return fail(FS_ERR_INVALID, "src and dst overlap");
  FS_HIP(fs::launch_fragment_order_fp8(src, n_mats, rows, cols, dst, S(stream)),
         "fragment_order_fp8");
  return FS_OK;
}

fs_status fs_grouped_expert_ffn_fp8_fo(const fs_moe_desc* desc, int32_t n_groups, int32_t ffn,
                                       const uint8_t* x_codes, const float* x_scales,
                                       const int32_t* group_rows, const int32_t* group_offsets,
                                       int64_t max_rows, const uint8_t* w_gate_up_fo,
                                       const float* s_gate_up, const uint8_t* w_down_fo,
                                       const float* s_down, void* out_rows, void* ws,
                                       size_t ws_bytes, fs_stream stream) {
  fs_status st = ffn_checks(desc, n_groups, ffn, group_offsets, max_rows);
  if (st != FS_OK) return st;
  if (!fo_shape_ok(desc, ffn))
    return fail(FS_ERR_UNSUPPORTED, "FP8 fragment-ordered experts write bf16 rows and need "
                                    "ffn % 128 == 0 and hidden % 256 == 0");
  if (max_rows == 0) return FS_OK;
  NEED(x_codes, "x_codes");
  NEED4(x_scales, "x_scales");
  OPT4(group_rows, "group_rows");
  OPT4(group_offsets, "group_offsets");
  NEED(w_gate_up_fo, "w_gate_up_fo");
  NEED4(s_gate_up, "s_gate_up");
  NEED(w_down_fo, "w_down_fo");
  NEED4(s_down, "s_down");
  NEED(out_rows, "out_rows");
  if (ws_bytes < fs::ffn_fp8_ws_bytes(max_rows, ffn, desc->hidden))
    return fail(FS_ERR_WORKSPACE, "workspace smaller than fs_workspace_size(FS_OP_GROUPED_FFN_FP8)");
  NEED(ws, "ws");
  FS_HIP(fs::launch_grouped_ffn_fo_fp8(n_groups, ffn, desc->hidden, x_codes, x_scales, group_rows,
                                       group_rows, group_offsets, max_rows, w_gate_up_fo,
                                       s_gate_up, w_down_fo, s_down, out_rows, ws, S(stream),
                                       group_offsets ? FS_K_GATE_UP : FS_K_SHARED_GATE_UP),
         "grouped_ffn_fp8_fo");
  return FS_OK;
}

fs_status fs_grouped_expert_ffn_fo(const fs_moe_desc* desc, int32_t n_groups, int32_t ffn,
                                   const void* in_rows, const int32_t* group_rows,
                                   const int32_t* group_offsets, int64_t max_rows,
                                   const void* w_gate_up_fo, const void* w_down_fo,
                                   void* out_rows, void* ws, size_t ws_bytes, fs_stream stream) {
  fs_status st = ffn_checks(desc, n_groups, ffn, group_offsets, max_rows);
  if (st != FS_OK) return st;
  if (!fo_shape_ok(desc, ffn))
    return fail(FS_ERR_UNSUPPORTED, "fragment-ordered experts need bf16, ffn % 128 == 0 and "
                                    "hidden % 256 == 0");
  if (max_rows == 0) return FS_OK;
  NEED(in_rows, "in_rows");
  OPT4(group_rows, "group_rows");
  OPT4(group_offsets, "group_offsets");
  NEED(w_gate_up_fo, "w_gate_up_fo");
  NEED(w_down_fo, "w_down_fo");
  NEED(out_rows, "out_rows");
  if (ws_bytes < fs::ffn_ws_bytes(desc->dtype, max_rows, ffn, desc->hidden))
    return fail(FS_ERR_WORKSPACE, "workspace smaller than fs_workspace_size(FS_OP_GROUPED_FFN)");
  NEED(ws, "ws");
  FS_HIP(fs::launch_grouped_ffn_fo(n_groups, ffn, desc->hidden, in_rows, group_rows, group_rows,
                                   group_offsets, max_rows, w_gate_up_fo, w_down_fo, out_rows, ws,
                                   S(stream), group_offsets ? FS_K_GATE_UP : FS_K_SHARED_GATE_UP),
         "grouped_ffn_fo");
  return FS_OK;
}

// ---- combine + residual
fs_status fs_combine_unpack(const fs_moe_desc* desc, const void* y_ret,
                            const int32_t* slot_to_row, const float* topk_w,
                            const void* shared_out, void* routed_out, void* residual,
                            fs_stream stream) {
  fs_status st = check_desc(desc);
  if (st != FS_OK) return st;
  if (desc->n_tokens == 0) return FS_OK;
  NEED(y_ret, "y_ret");
  NEED4(slot_to_row, "slot_to_row");
  NEED4(topk_w, "topk_w");
  OPT(shared_out, "shared_out");
  OPT(routed_out, "routed_out");
  OPT(residual, "residual");
  if (!routed_out && !residual) return fail(FS_ERR_INVALID, "routed_out and residual are both NULL");
  hipStream_t s = S(stream);
  fs::prof_begin(FS_K_COMBINE, s);
  FS_HIP(fs::launch_combine(desc->dtype, y_ret, slot_to_row, topk_w, shared_out, routed_out,
                            residual, nullptr, desc->n_tokens, desc->top_k, desc->hidden, s),
         "combine");
  fs::prof_end(FS_K_COMBINE, s);
  return FS_OK;
}

fs_status fs_combine_partial(const fs_moe_desc* desc, const void* y_local,
                             const int32_t* slot_to_row, const int32_t* rank_offsets,
                             const float* topk_w, void* partial_out, fs_stream stream) {
  fs_status st = check_desc(desc);
  if (st != FS_OK) return st;
  if (desc->n_tokens == 0) return FS_OK;
  NEED(y_local, "y_local");
  NEED4(slot_to_row, "slot_to_row");
  NEED4(rank_offsets, "rank_offsets");
  NEED4(topk_w, "topk_w");
  NEED(partial_out, "partial_out");
  hipStream_t s = S(stream);
  fs::prof_begin(FS_K_COMBINE, s);
  FS_HIP(fs::launch_combine(desc->dtype, y_local, slot_to_row, topk_w, nullptr, partial_out,
                            nullptr, rank_offsets + desc->ep_rank, desc->n_tokens, desc->top_k,
                            desc->hidden, s),
         "combine_partial");
  fs::prof_end(FS_K_COMBINE, s);
  return FS_OK;
}

fs_status fs_allreduce_standin(const fs_moe_desc* desc, void* out, const void* partial,
                               fs_stream stream) {
  fs_status st = check_desc(desc);
  if (st != FS_OK) return st;
  if (desc->n_tokens == 0) return FS_OK;
  NEED(out, "out");
  NEED(partial, "partial");
  const size_t bytes = (size_t)desc->n_tokens * desc->hidden * elem(desc->dtype);
  const char* o = static_cast<const char*>(out);
  const char* p = static_cast<const char*>(partial);
  if (o < p + bytes && p < o + bytes && o != p)
    return fail(FS_ERR_INVALID, "out and partial overlap");
  hipStream_t s = S(stream);
  if (o == p) return FS_OK;
  fs::prof_begin(FS_K_ALLREDUCE_COPY, s);
  FS_HIP(standin_copy(out, partial, bytes, 2.0, s), "allreduce stand-in copy");
  fs::prof_end(FS_K_ALLREDUCE_COPY, s);
  return FS_OK;
}

fs_status fs_standin_link(int32_t links, double link_bytes_per_s, int32_t workgroups) {
  if (links < 0 || links > 1023) return fail(FS_ERR_INVALID, "links must be in [0, 1023]");
  if (links > 0) {
    if (!(link_bytes_per_s >= 1e9 && link_bytes_per_s <= 1e15))
      return fail(FS_ERR_INVALID, "link_bytes_per_s must be in [1e9, 1e15]");
    if (workgroups < 1 || workgroups > 4096)
      return fail(FS_ERR_INVALID, "workgroups must be in [1, 4096]");
  }
  std::lock_guard<std::mutex> g(g_link_mu);
  g_link = links > 0 ? LinkModel{links, link_bytes_per_s, workgroups} : LinkModel{};
  return FS_OK;
}

fs_status fs_standin_link_get(int32_t* links, double* link_bytes_per_s, int32_t* workgroups) {
  if (!links || !link_bytes_per_s || !workgroups)
    return fail(FS_ERR_INVALID, "outputs must not be NULL");
  const LinkModel m = link_model();
  *links = m.links;
  *link_bytes_per_s = m.bytes_per_s;
  *workgroups = m.workgroups;
  return FS_OK;
}

fs_status fs_farskip_residual(const fs_moe_desc* desc, void* out, const void* residual,
                              const void* deferred, const void* extra, fs_stream stream) {
  fs_status st = check_desc(desc);
  if (st != FS_OK) return st;
  if (desc->n_tokens == 0) return FS_OK;
  NEED(out, "out");
  NEED(residual, "residual");
  NEED(deferred, "deferred");
  OPT(extra, "extra");
  FS_HIP(fs::launch_residual(desc->dtype, out, residual, deferred, extra,
                             (int64_t)desc->n_tokens * desc->hidden, S(stream)),
         "residual");
  return FS_OK;
}

// ---- dense linear
fs_status fs_dense_linear(int32_t dtype, int32_t m, int32_t n, int32_t kdim, const void* a,
                          const void* w, void* out, fs_stream stream) {
  if (dtype != FS_F32 && dtype != FS_BF16) return fail(FS_ERR_INVALID, "dtype must be FS_F32 or FS_BF16");
  if (m < 0 || n <= 0 || kdim <= 0) return fail(FS_ERR_INVALID, "m >= 0, n > 0, kdim > 0 required");
  if (kdim % 64 != 0) return fail(FS_ERR_UNSUPPORTED, "kdim must be a multiple of 64");
  if (n % (dtype == FS_BF16 ? 128 : 64) != 0)
    return fail(FS_ERR_UNSUPPORTED, "n must be a multiple of 128 (bf16) or 64 (fp32)");
  if (m == 0) return FS_OK;
  NEED(a, "a");
  NEED(w, "w");
  NEED(out, "out");
  fs::prof_begin(FS_K_DENSE, S(stream));
  FS_HIP(fs::launch_dense_linear(dtype, m, n, kdim, a, w, out, S(stream)), "dense_linear");
  fs::prof_end(FS_K_DENSE, S(stream));
  return FS_OK;
}

// ---- block sync
struct fs_block_sync {
  hipEvent_t packed = nullptr;      // send buffer ready (compute)
  hipEvent_t dispatched = nullptr;  // Dispatch copy done (comm)
  hipEvent_t computed = nullptr;    // expert outputs ready (compute)
  hipEvent_t returned = nullptr;    // Combine copy done (comm)
  bool have_dispatch = false;
  bool have_return = false;
};

fs_status fs_block_sync_create(fs_block_sync** out) {
  if (!out) return fail(FS_ERR_INVALID, "out must not be NULL");
  fs_block_sync* s = new (std::nothrow) fs_block_sync();
  if (!s) return fail(FS_ERR_INVALID, "out of host memory");
  hipError_t e = hipEventCreateWithFlags(&s->packed, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&s->dispatched, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&s->computed, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&s->returned, hipEventDisableTiming);
  if (e != hipSuccess) {
    (void)fs_block_sync_destroy(s);
    return hip_fail(e, "hipEventCreate");
  }
  *out = s;
  return FS_OK;
}

fs_status fs_block_sync_destroy(fs_block_sync* s) {
  if (!s) return FS_OK;
  if (s->packed) (void)hipEventDestroy(s->packed);
  if (s->dispatched) (void)hipEventDestroy(s->dispatched);
  if (s->computed) (void)hipEventDestroy(s->computed);
  if (s->returned) (void)hipEventDestroy(s->returned);
  delete s;
  return FS_OK;
}

// ---- the block
fs_status fs_moe_block_forward(const fs_moe_desc* desc, int32_t phase,
                               const fs_moe_weights* wt, const void* residual_in,
                               void* partial_out, void* residual_io, fs_block_buffers* b,
                               int64_t max_recv_rows, void* ws, size_t ws_bytes,
                               fs_block_sync* sync, fs_stream compute, fs_stream comm) {
  fs_status st = check_desc(desc);
  if (st != FS_OK) return st;
  if (phase < FS_PHASE_ALL || phase > FS_PHASE_COMBINE)
    return fail(FS_ERR_INVALID, "phase must be one of FS_PHASE_ALL .. FS_PHASE_COMBINE");
  if (!wt) return fail(FS_ERR_INVALID, "weights must not be NULL");
  if (!b) return fail(FS_ERR_INVALID, "buffers must not be NULL");
  if (comm && !sync) return fail(FS_ERR_INVALID, "a comm stream needs a sync object");
  const int N = desc->n_tokens, D = desc->hidden, K = desc->top_k, E = desc->n_experts;
  const int R = desc->ep_size, r = desc->ep_rank, E_loc = E / R;
  const int64_t cap = (int64_t)N * K;
  if (max_recv_rows < 0) return fail(FS_ERR_INVALID, "max_recv_rows must be >= 0");
  if (R == 1 && max_recv_rows < cap)
    return fail(FS_ERR_INVALID, "max_recv_rows must be >= n_tokens * top_k when ep_size == 1");
  if (max_recv_rows > (int64_t)R * cap)
    return fail(FS_ERR_INVALID, "max_recv_rows must be <= ep_size * n_tokens * top_k");
  const bool do_gate = phase == FS_PHASE_ALL || phase == FS_PHASE_BEGIN || phase == FS_PHASE_GATE;
  const bool do_shared = phase == FS_PHASE_ALL || phase == FS_PHASE_BEGIN || phase == FS_PHASE_SHARED;
  const bool do_experts = phase == FS_PHASE_ALL || phase == FS_PHASE_FINISH || phase == FS_PHASE_EXPERTS;
  const bool do_combine = phase == FS_PHASE_ALL || phase == FS_PHASE_FINISH || phase == FS_PHASE_COMBINE;
  const bool fp8_routed = wt->w_gate_up_fp8 != nullptr;
  const bool fp8_shared = desc->n_shared > 0 && wt->ws_gate_up_fp8 != nullptr;
  if (fp8_routed || fp8_shared) {
    if (desc->dtype != FS_BF16) return fail(FS_ERR_UNSUPPORTED, "FP8 experts need a bf16 block");
    if (D % 256 != 0) return fail(FS_ERR_UNSUPPORTED, "FP8 experts need hidden % 256 == 0");
    if (fp8_routed && desc->ffn % 128 != 0)
      return fail(FS_ERR_UNSUPPORTED, "FP8 routed experts need ffn % 128 == 0");
    if (fp8_shared && (desc->n_shared * desc->ffn_shared) % 128 != 0)
      return fail(FS_ERR_UNSUPPORTED, "FP8 shared experts need n_shared * ffn_shared % 128 == 0");
  }
  const size_t need = block_bytes(desc, max_recv_rows, fp8_routed, fp8_shared);
  if (ws_bytes < need)
    return fail(FS_ERR_WORKSPACE, fp8_routed || fp8_shared
                                      ? "workspace smaller than fs_workspace_size(FS_OP_BLOCK_FP8)"
                                      : "workspace smaller than fs_workspace_size(FS_OP_BLOCK)");
  if (N == 0) return FS_OK;
  NEED(ws, "ws");
  NEED(residual_in, "residual_in");
  if (do_gate) {
    NEED(wt->w_router, "weights->w_router");
    OPT4(wt->sel_bias, "weights->sel_bias");
    if (wt->sel_bias && desc->score == FS_SOFTMAX)
      return fail(FS_ERR_UNSUPPORTED, "a selection bias is defined for sigmoid scoring only");
    NEED(b->send, "buffers->send");
    NEED4(b->row_to_slot, "buffers->row_to_slot");
    OPT4(b->logits, "buffers->logits");
  }
  if (do_shared) {
    NEED(partial_out, "partial_out");
    if (desc->n_shared > 0) {
      if (fp8_shared) {
        NEED(wt->ws_gate_up_fp8, "weights->ws_gate_up_fp8");
        NEED4(wt->ss_gate_up, "weights->ss_gate_up");
        NEED(wt->ws_down_fp8, "weights->ws_down_fp8");
        NEED4(wt->ss_down, "weights->ss_down");
      } else {
        NEED(wt->ws_gate_up, "weights->ws_gate_up");
        NEED(wt->ws_down, "weights->ws_down");
      }
      NEED(b->shared_out, "buffers->shared_out");
    }
  }
  if (do_experts) {
    if (fp8_routed) {
      NEED(wt->w_gate_up_fp8, "weights->w_gate_up_fp8");
      NEED4(wt->s_gate_up, "weights->s_gate_up");
      NEED(wt->w_down_fp8, "weights->w_down_fp8");
      NEED4(wt->s_down, "weights->s_down");
      OPT(wt->w_gate_up_fp8_fo, "weights->w_gate_up_fp8_fo");
      OPT(wt->w_down_fp8_fo, "weights->w_down_fp8_fo");
    } else {
      NEED(wt->w_gate_up, "weights->w_gate_up");
      NEED(wt->w_down, "weights->w_down");
      OPT(wt->w_gate_up_fo, "weights->w_gate_up_fo");
      OPT(wt->w_down_fo, "weights->w_down_fo");
    }
    NEED(b->y, "buffers->y");
    if (R > 1) {
      NEED4(b->group_rows, "buffers->group_rows");
      NEED4(b->group_offsets, "buffers->group_offsets");
    }
    if (!b->recv) NEED(b->send, "buffers->send");
  }
  if (do_combine) {
    NEED(residual_io, "residual_io");
    if (!b->ret) NEED(b->y, "buffers->y");
  }
  OPT(b->ret, "buffers->ret");
  NEED4(b->topk_ids, "buffers->topk_ids");
  NEED4(b->topk_w, "buffers->topk_w");
  NEED4(b->src_counts, "buffers->src_counts");
  NEED4(b->src_offsets, "buffers->src_offsets");
  NEED4(b->rank_offsets, "buffers->rank_offsets");
  NEED4(b->slot_to_row, "buffers->slot_to_row");
  if (R > 1 || comm) NEED(b->recv, "buffers->recv");

  hipStream_t sc = S(compute), sm = S(comm);
  const size_t es = elem(desc->dtype);
  const size_t slot_bytes = (size_t)cap * D * es;
  Carve c{reinterpret_cast<char*>(ws)};
  void* ws_router = c.take(router_bytes(desc));
  void* ws_plan = c.take(fp8_routed ? plan_fp8_bytes(desc) : plan_bytes(desc));
  char* ws_ffn = static_cast<char*>(c.take(routed_ffn_bytes(desc, max_recv_rows, fp8_routed)));
  char* ws_shared =
      desc->n_shared > 0
          ? static_cast<char*>(c.take(block_ffn_bytes(desc, N, desc->n_shared * desc->ffn_shared, fp8_shared)))
          : nullptr;
  // FP8 parts of an FFN region: input codes, their scales, the FFN workspace
  auto fp8_parts = [&](char* base, int64_t rows, uint8_t** codes, float** scales, void** rest) {
    *codes = reinterpret_cast<uint8_t*>(base);
    *scales = reinterpret_cast<float*>(base + align256((size_t)rows * D));
    *rest = base + align256((size_t)rows * D) + align256((size_t)rows * 4);
  };
  int32_t* my_counts = b->src_counts + (size_t)r * E;
  int32_t* my_offsets = b->src_offsets + (size_t)r * (E + 1);
  char* recv_slot = b->recv ? reinterpret_cast<char*>(b->recv) + (size_t)r * slot_bytes : nullptr;
  // FP8 routed experts: send and recv are FP8 row buffers (codes, then
  // scales at a(rows * d)); slot s of recv is rows [s*cap, (s+1)*cap)
  uint8_t* send_codes = static_cast<uint8_t*>(b->send);
  float* send_scales =
      b->send ? reinterpret_cast<float*>(static_cast<char*>(b->send) + align256((size_t)cap * D))
              : nullptr;
  uint8_t* recv_codes = static_cast<uint8_t*>(b->recv);
  float* recv_scales =
      b->recv ? reinterpret_cast<float*>(static_cast<char*>(b->recv) + align256((size_t)R * cap * D))
              : nullptr;
  // the Dispatch stand-in: the whole send buffer into receive slot r
  auto dispatch_copy = [&](hipStream_t st) -> fs_status {
    fs::prof_begin(FS_K_DISPATCH_COPY, st);
    if (fp8_routed) {
      FS_HIP(standin_copy(recv_codes + (size_t)r * cap * D, send_codes, (size_t)cap * D, 1.0, st),
             "dispatch stand-in copy");
      FS_HIP(standin_copy(recv_scales + (size_t)r * cap, send_scales, (size_t)cap * 4, 1.0, st),
             "dispatch stand-in copy");
    } else {
      FS_HIP(standin_copy(recv_slot, b->send, slot_bytes, 1.0, st), "dispatch stand-in copy");
    }
    fs::prof_end(FS_K_DISPATCH_COPY, st);
    return FS_OK;
  };
  char* y_slot = b->y ? reinterpret_cast<char*>(b->y) + (size_t)r * slot_bytes : nullptr;

  if (do_gate) {
    // gate: router + top-k (not overlappable, Eq. 9), then plan + pack
    st = router_impl(desc, residual_in, wt->w_router, wt->sel_bias, nullptr, b->logits,
                     b->topk_ids, b->topk_w, ws_router, sc);
    if (st != FS_OK) return st;
    if (fp8_routed)
      st = plan_pack_fp8_impl(desc, b->topk_ids, residual_in, my_counts, my_offsets,
                              b->rank_offsets, b->slot_to_row, b->row_to_slot, send_codes,
                              send_scales, ws_plan, sc);
    else
      st = plan_pack_impl(desc, b->topk_ids, residual_in, my_counts, my_offsets, b->rank_offsets,
                          b->slot_to_row, b->row_to_slot, b->send, ws_plan, sc);
    if (st != FS_OK) return st;
    // Dispatch stand-in: the whole send buffer into receive slot r, on the
    // comm stream, else in order on compute
    if (sm) {
      FS_HIP(hipEventRecord(sync->packed, sc), "hipEventRecord");
      FS_HIP(hipStreamWaitEvent(sm, sync->packed, 0), "hipStreamWaitEvent");
      st = dispatch_copy(sm);
      if (st != FS_OK) return st;
      FS_HIP(hipEventRecord(sync->dispatched, sm), "hipEventRecord");
      sync->have_dispatch = true;
    } else if (recv_slot) {
      st = dispatch_copy(sc);
      if (st != FS_OK) return st;
    }
  }
  if (do_shared) {
    // shared experts on o_{k-1}, then the next layer's partial input
    if (fp8_shared) {
      uint8_t* xq;
      float* xs;
      void* rest;
      fp8_parts(ws_shared, N, &xq, &xs, &rest);
      fs::prof_begin(FS_K_QUANTIZE, sc);
      FS_HIP(fs::launch_quantize_fp8(1, residual_in, N, D, nullptr, xq, xs, sc), "quantize_fp8");
      fs::prof_end(FS_K_QUANTIZE, sc);
      FS_HIP(fs::launch_grouped_ffn_fp8(1, desc->n_shared * desc->ffn_shared, D, xq, xs, nullptr,
                                        nullptr, nullptr, N, wt->ws_gate_up_fp8, wt->ss_gate_up,
                                        wt->ws_down_fp8, wt->ss_down, b->shared_out, rest, sc,
                                        FS_K_SHARED_GATE_UP),
             "shared_ffn_fp8");
    } else if (desc->n_shared > 0) {
      FS_HIP(fs::launch_grouped_ffn(desc->dtype, 1, desc->n_shared * desc->ffn_shared, D,
                                    residual_in, nullptr, nullptr, nullptr, N, wt->ws_gate_up, wt->ws_down,
                                    b->shared_out, ws_shared, sc, FS_K_SHARED_GATE_UP),
             "shared_ffn");
    }
    FS_HIP(fs::launch_residual(desc->dtype, partial_out, residual_in,
                               desc->n_shared > 0 ? b->shared_out : nullptr, nullptr,
                               (int64_t)N * D, sc),
           "partial");
  }
  if (do_experts) {
    if (sm && sync->have_dispatch) {
      FS_HIP(hipStreamWaitEvent(sc, sync->dispatched, 0), "hipStreamWaitEvent");
      sync->have_dispatch = false;
    }
    const void* in_rows;
    const int32_t* rows;
    const int32_t* goff;
    if (R > 1) {
      FS_HIP(fs::launch_receive_rows(b->src_counts, b->src_offsets, R, E, r, cap, b->group_rows,
                                     b->group_offsets, sc),
             "receive_rows");
      in_rows = b->recv;
      rows = b->group_rows;
      goff = b->group_offsets;
    } else {
      in_rows = recv_slot ? recv_slot : b->send;
      rows = nullptr;
      goff = my_offsets;  // E + 1 entries = E_loc + 1 when R == 1
    }
    if (fp8_routed) {
      // the received codes and scales, gathered through the receive rows;
      // the outputs go back to their receive rows
      const uint8_t* xq = b->recv ? recv_codes : send_codes;
      const float* xs = b->recv ? recv_scales : send_scales;
      if (wt->w_gate_up_fp8_fo && wt->w_down_fp8_fo && fo_shape_ok(desc, desc->ffn) &&
          max_recv_rows <= (int64_t)64 * E_loc) {
        // groups of few rows (decode): stream the FP8-fragment-ordered codes
        FS_HIP(fs::launch_grouped_ffn_fo_fp8(E_loc, desc->ffn, D, xq, xs, rows, rows, goff,
                                             max_recv_rows, wt->w_gate_up_fp8_fo, wt->s_gate_up,
                                             wt->w_down_fp8_fo, wt->s_down, b->y, ws_ffn, sc,
                                             FS_K_GATE_UP),
               "grouped_ffn_fp8_fo");
      } else {
        FS_HIP(fs::launch_grouped_ffn_fp8(E_loc, desc->ffn, D, xq, xs, rows, rows, goff,
                                          max_recv_rows, wt->w_gate_up_fp8, wt->s_gate_up,
                                          wt->w_down_fp8, wt->s_down, b->y, ws_ffn, sc,
                                          FS_K_GATE_UP),
               "grouped_ffn_fp8");
      }
    } else if (wt->w_gate_up_fo && wt->w_down_fo && fo_shape_ok(desc, desc->ffn) &&
               max_recv_rows <= (int64_t)64 * E_loc) {
      // groups of few rows (decode): stream the fragment-ordered weights
      FS_HIP(fs::launch_grouped_ffn_fo(E_loc, desc->ffn, D, in_rows, rows, rows, goff,
                                       max_recv_rows, wt->w_gate_up_fo, wt->w_down_fo, b->y,
                                       ws_ffn, sc, FS_K_GATE_UP),
             "grouped_ffn_fo");
    } else {
      FS_HIP(fs::launch_grouped_ffn(desc->dtype, E_loc, desc->ffn, D, in_rows, rows, rows, goff,
                                    max_recv_rows, wt->w_gate_up, wt->w_down, b->y, ws_ffn, sc,
                                    FS_K_GATE_UP),
             "grouped_ffn");
    }
    // Combine stand-in: slot r of y (the rows this rank's tokens get back)
    // into ret, on the comm stream, else in order on compute
    if (b->ret) {
      if (sm) {
        FS_HIP(hipEventRecord(sync->computed, sc), "hipEventRecord");
        FS_HIP(hipStreamWaitEvent(sm, sync->computed, 0), "hipStreamWaitEvent");
        fs::prof_begin(FS_K_COMBINE_COPY, sm);
        FS_HIP(standin_copy(b->ret, y_slot, slot_bytes, 1.0, sm), "combine stand-in copy");
        fs::prof_end(FS_K_COMBINE_COPY, sm);
        FS_HIP(hipEventRecord(sync->returned, sm), "hipEventRecord");
        sync->have_return = true;
      } else {
        fs::prof_begin(FS_K_COMBINE_COPY, sc);
        FS_HIP(standin_copy(b->ret, y_slot, slot_bytes, 1.0, sc), "combine stand-in copy");
        fs::prof_end(FS_K_COMBINE_COPY, sc);
      }
    }
  }
  if (do_combine) {
    if (sm && sync->have_return) {
      FS_HIP(hipStreamWaitEvent(sc, sync->returned, 0), "hipStreamWaitEvent");
      sync->have_return = false;
    }
    const void* y_ret = b->ret ? b->ret : y_slot;
    fs::prof_begin(FS_K_COMBINE, sc);
    FS_HIP(fs::launch_combine(desc->dtype, y_ret, b->slot_to_row, b->topk_w, nullptr, nullptr,
                              residual_io, nullptr, N, K, D, sc),
           "combine");
    fs::prof_end(FS_K_COMBINE, sc);
  }
  return FS_OK;
}

// ---- profiling
fs_status fs_profile_enable(int32_t on) {
  ProfState& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  p.on = on != 0;
  return FS_OK;
}

fs_status fs_profile_select(uint32_t mask) {
  if (mask >> FS_K_COUNT) return fail(FS_ERR_INVALID, "mask has bits beyond FS_K_COUNT");
  ProfState& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  p.mask = mask;
  return FS_OK;
}

fs_status fs_profile_read(int32_t kernel, double* total_ms, int64_t* launches) {
  if (kernel < 0 || kernel >= FS_K_COUNT) return fail(FS_ERR_INVALID, "kernel id out of range");
  ProfState& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  for (auto& rec : p.open) {
    hipError_t e = hipEventSynchronize(rec.b);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, rec.a, rec.b);
    if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
    p.total_ms[rec.kernel] += ms;
    p.count[rec.kernel] += 1;
    p.pool.push_back(rec.a);
    p.pool.push_back(rec.b);
    p.pool.push_back(rec.spare);
  }
  p.open.clear();
  if (total_ms) *total_ms = p.total_ms[kernel];
  if (launches) *launches = p.count[kernel];
  return FS_OK;
}

fs_status fs_profile_reset(void) {
  ProfState& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  for (auto& rec : p.open) {
    (void)hipEventSynchronize(rec.b);
    p.pool.push_back(rec.a);
    p.pool.push_back(rec.b);
    p.pool.push_back(rec.spare);
  }
  p.open.clear();
  for (auto& w : p.windows) {
    (void)hipEventSynchronize(w.a);
    for (hipEvent_t e : {w.a, w.b, w.k0}) p.pool.push_back(e);
  }
  p.windows.clear();
  for (int k = 0; k < FS_K_COUNT; ++k) {
    p.total_ms[k] = 0;
    p.count[k] = 0;
  }
  return FS_OK;
}

}  // extern "C"
