/*
 * farskip.h -- C ABI of libfarskip.so: the forward pass of one FarSkip MoE
 * block on one expert-parallel (EP) rank's share, on an AMD Instinct MI355X
 * (gfx950).
 *
 * What is computed (arXiv 2511.11505):
 *   Section 2.1  MoE(A) = sum_j G(A)_j MLP^j(A), G(A) = s(A W_R^T); experts
 *                are split over EP ranks; Dispatch permutes A and sends each
 *                token row to the ranks of its experts; Combine returns the
 *                expert outputs and sums them with the gate weights; shared
 *                experts run on every token.  The expert MLP is read as
 *                SwiGLU: (SiLU(A Wg^T) * (A Wu^T)) Wd^T.
 *   Section 3    FarSkip residual (Eq. 7): the next layer reads an input
 *                that lacks this block's routed-expert output (the partial
 *                input of Eq. 8b: residual + shared-expert output); the MoE
 *                itself reads the outdated residual o_{k-1} (Eq. 8a); the
 *                routed output is added into the residual afterwards.
 *   Section 4.1  Dispatch overlaps the next computation; the gate and the
 *                routed experts are the parts that cannot overlap (Eq. 9).
 *   Section 4.2  The inference variant with replicated activations: every
 *                rank holds all N tokens and routes them, runs only its
 *                own experts (fs_local_rows, fs_grouped_expert_ffn_gathered,
 *                fs_combine_partial) and the per-rank partial sums are
 *                all-reduced; FarSkip defers the routed all-reduce to the
 *                next MoE and merges the attention and shared-expert
 *                partials into one all-reduce (Tab. 5).
 *
 * Conventions shared by every entry point
 *   Memory      Every array argument is DEVICE memory owned by the caller,
 *               row-major with the leading dimension stated.  The library
 *               never allocates or frees device memory; scratch space is a
 *               caller-provided workspace sized by fs_workspace_size().
 *   Alignment   Arrays of tokens, weights, expert outputs and residuals
 *               (accessed as 16-byte vectors) must be 16-byte aligned;
 *               int32 index arrays and fp32 logit / gate / bias arrays
 *               4-byte aligned.
 *   Element     FS_F32 or FS_BF16 selects the type of tokens, weights,
 *   types       expert outputs and residuals (desc->dtype); router logits,
 *               gate weights and the selection bias are always fp32;
 *               accumulation is always fp32; index arrays are int32.
 *   Streams     Calls enqueue work on the given HIP stream (a hipStream_t
 *               passed as void*, NULL = the null stream) and return without
 *               synchronising.
 *   Errors      Argument checks run on the host before anything is
 *               enqueued: FS_ERR_INVALID (bad value or pointer),
 *               FS_ERR_UNSUPPORTED (valid but outside what the kernels
 *               handle), FS_ERR_WORKSPACE (workspace too small).  A failing
 *               HIP call returns FS_ERR_HIP.  fs_last_error_message() gives
 *               the detail for the calling thread.  Device faults surface at
 *               the caller's next synchronisation.  The library never
 *               aborts and never prints.
 *   Shapes      hidden % 128 == 0, ffn % 64 == 0, 1 <= top_k <= min(E, 32),
 *               E <= 512, E % n_groups == 0, n_groups <= 64,
 *               top_k <= topk_groups * E / n_groups, E % ep_size == 0,
 *               ep_size * n_tokens * top_k < 2^31.  n_tokens == 0 is a
 *               valid no-op.
 */
#ifndef FARSKIP_H
#define FARSKIP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FS_ABI_VERSION 9

typedef enum {
  FS_OK = 0,
  FS_ERR_INVALID = 1,
  FS_ERR_UNSUPPORTED = 2,
  FS_ERR_WORKSPACE = 3,
  FS_ERR_HIP = 4
} fs_status;

typedef enum { FS_F32 = 0, FS_BF16 = 1 } fs_dtype;
typedef enum { FS_SOFTMAX = 0, FS_SIGMOID = 1 } fs_score;
typedef enum {
  FS_PHASE_ALL = 0,      /* GATE, SHARED, EXPERTS, COMBINE */
  FS_PHASE_BEGIN = 1,    /* GATE, SHARED */
  FS_PHASE_FINISH = 2,   /* EXPERTS, COMBINE */
  FS_PHASE_GATE = 3,     /* router + top-k, plan + pack, Dispatch started */
  FS_PHASE_SHARED = 4,   /* shared experts, partial_out */
  FS_PHASE_EXPERTS = 5,  /* Dispatch joined, routed experts, Combine started */
  FS_PHASE_COMBINE = 6   /* Combine joined, weighted sum + deferred add */
} fs_phase;
typedef enum {
  FS_OP_ROUTER_TOPK = 0,
  FS_OP_DISPATCH_PACK = 1,
  FS_OP_GROUPED_FFN = 2,
  FS_OP_BLOCK = 3,
  FS_OP_GROUPED_FFN_FP8 = 4,
  FS_OP_BLOCK_FP8 = 5,
  FS_OP_DISPATCH_PACK_FP8 = 6
} fs_op;

/* One MoE block on one EP rank (Section 2.1).  A plain host struct, read
 * only during the call. */
typedef struct {
  int32_t abi_version;   /* FS_ABI_VERSION */
  int32_t n_tokens;      /* N: tokens this rank routes (its own batch) */
  int32_t hidden;        /* d */
  int32_t n_experts;     /* E: routed experts over all ranks */
  int32_t top_k;         /* k */
  int32_t n_groups;      /* G: expert groups for group-limited routing; 1 = off */
  int32_t topk_groups;   /* groups kept per token when G > 1 */
  int32_t score;         /* fs_score */
  int32_t norm_topk;     /* 1: renormalise the k gate weights to sum to 1 */
  float routed_scale;    /* gate weights are multiplied by this last */
  int32_t ffn;           /* F: routed expert width */
  int32_t n_shared;      /* S: shared experts (0 = none) */
  int32_t ffn_shared;    /* width of each shared expert */
  int32_t ep_size;       /* R */
  int32_t ep_rank;       /* r: owns experts [r*E/R, (r+1)*E/R) */
  int32_t dtype;         /* fs_dtype */
} fs_moe_desc;

typedef void* fs_stream; /* a hipStream_t */

const char* fs_status_string(int32_t status);
const char* fs_last_error_message(void);
int32_t fs_abi_version(void);

/* Bytes of workspace an entry point needs.
 *   op = FS_OP_ROUTER_TOPK:   fs_router_topk (max_rows, ffn ignored)
 *   op = FS_OP_DISPATCH_PACK: fs_dispatch_pack (max_rows, ffn ignored)
 *   op = FS_OP_GROUPED_FFN:   fs_grouped_expert_ffn with up to max_rows rows
 *                             and width ffn
 *   op = FS_OP_BLOCK:         fs_moe_block_forward with up to max_rows rows
 *                             landing on local experts (ffn ignored)
 *   op = FS_OP_GROUPED_FFN_FP8: fs_grouped_expert_ffn_fp8 with up to
 *                             max_rows rows and width ffn
 *   op = FS_OP_BLOCK_FP8:     fs_moe_block_forward with FP8 routed and
 *                             shared experts (enough for either alone)
 *   op = FS_OP_DISPATCH_PACK_FP8: fs_dispatch_pack_fp8 (max_rows, ffn
 *                             ignored) */
fs_status fs_workspace_size(const fs_moe_desc* desc, int32_t op, int64_t max_rows,
                            int32_t ffn, size_t* bytes);

/* Router scoring and top-k (Section 2.1: G(A) = s(A W_R^T)).
 *   x          [N, d] dtype: the MoE input o_{k-1}
 *   w_router   [E, d] dtype
 *   sel_bias   [E] fp32 or NULL; sigmoid scoring only: the selection key is
 *              sigmoid(z) + bias, the gate weight the unbiased sigmoid(z)
 *   logits_in  [N, E] fp32 or NULL: when given, the logits are taken from
 *              here and x / w_router are not read
 *   logits_out [N, E] fp32 or NULL: receives the logits
 *   topk_ids   [N, k] int32 out: selected experts, descending key order,
 *              ties to the lower expert index
 *   topk_w     [N, k] fp32 out: gate weights (softmax over all E experts or
 *              sigmoid; renormalised over the k when norm_topk; * scale)
 * Logits are fp32 sums in a fixed order: the hidden dimension is cut into
 * slices of 256 consecutive elements, products are added one at a time in
 * ascending order within a slice, and slice sums are added in ascending
 * slice order; every operation rounds to fp32.  With G > 1 a group's score
 * is the sum of its two largest keys; the topk_groups best groups are kept
 * (ties to the lower group).  Inputs must be finite. */
fs_status fs_router_topk(const fs_moe_desc* desc, const void* x, const void* w_router,
                         const float* sel_bias, const float* logits_in, float* logits_out,
                         int32_t* topk_ids, float* topk_w, void* ws, size_t ws_bytes,
                         fs_stream stream);

/* Dispatch plan and pack (Section 2.1, Dispatch: the permutation of A that
 * precedes the all-to-all).  One send row per (token, selected expert);
 * rows are ordered by expert, then token, so the buffer is expert-contiguous
 * and, experts being rank-blocked, rank-contiguous.  Bit-exact and
 * deterministic (no global atomics).
 *   topk_ids       [N, k] int32 in: distinct ids in [0, E) per token
 *   x              [N, d] dtype
 *   expert_counts  [E] int32 out
 *   expert_offsets [E+1] int32 out: exclusive prefix sum of the counts
 *   rank_offsets   [R+1] int32 out: expert_offsets[r * E/R]
 *   slot_to_row    [N*k] int32 out: send row of slot t*k+j
 *   row_to_slot    [N*k] int32 out: its inverse
 *   send           [N*k, d] dtype out: send[slot_to_row[t*k+j]] = x[t];
 *                  NULL computes the plan only (x is then not read) */
fs_status fs_dispatch_pack(const fs_moe_desc* desc, const int32_t* topk_ids, const void* x,
                           int32_t* expert_counts, int32_t* expert_offsets,
                           int32_t* rank_offsets, int32_t* slot_to_row, int32_t* row_to_slot,
                           void* send, void* ws, size_t ws_bytes, fs_stream stream);

/* Dispatch plan and pack of FP8 rows, for FP8 routed experts (the FP8
 * experts of the paper's inference runs, Section 5.2).  Each token row of x
 * is quantised once, as fs_quantize_fp8, and its codes and scale go to the
 * token's k send rows: the send rows are what fs_quantize_fp8 gives for
 * the bf16 send rows of fs_dispatch_pack, in about half the bytes.
 *   x            [N, d] bf16 (desc->dtype FS_BF16, d % 16 == 0;
 *                FS_ERR_UNSUPPORTED otherwise)
 *   send_codes   [N*k, d] uint8 out, 16-byte aligned
 *   send_scales  [N*k] fp32 out
 * The plan outputs are those of fs_dispatch_pack.  Workspace:
 * FS_OP_DISPATCH_PACK_FP8 (the plan's, then the token codes and scales).
 * An FP8 row buffer of n rows (the block's send and recv with FP8 routed
 * experts) holds codes [n, d] at byte 0 and scales [n] at byte a(n*d),
 * where a(b) rounds b up to a multiple of 256; it fits in the bytes of a
 * bf16 [n, d] buffer. */
fs_status fs_dispatch_pack_fp8(const fs_moe_desc* desc, const int32_t* topk_ids, const void* x,
                               int32_t* expert_counts, int32_t* expert_offsets,
                               int32_t* rank_offsets, int32_t* slot_to_row,
                               int32_t* row_to_slot, uint8_t* send_codes, float* send_scales,
                               void* ws, size_t ws_bytes, fs_stream stream);

/* Dispatch plan and pack for callers that cannot allocate memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation.  Same arguments and results as fs_dispatch_pack without the
 * workspace: the plan's scratch is a fixed 4 MiB device array inside the
 * library, one per device, kept until the process ends; the call allocates
 * and frees nothing.  The plan kernels overwrite every scratch word they
 * read, so nothing carries over between calls.
 *   Limit     ceil(N / 64) * E <= 262144 (e.g. 32768 tokens over 512
 *             experts); larger shapes return FS_ERR_UNSUPPORTED before
 *             anything is enqueued.
 *   Device    The array of the current device is used; a non-NULL stream
 *             must belong to that device (FS_ERR_INVALID otherwise).
 *   Races     Every call on one device shares that device's array: calls
 *             whose work overlaps on one device (other streams, other
 *             threads) race and must be ordered by the caller.
 *   Timing    No fs_profile timing windows are opened. */
fs_status fs_dispatch_pack_noalloc(const fs_moe_desc* desc, const int32_t* topk_ids,
                                   const void* x, int32_t* expert_counts,
                                   int32_t* expert_offsets, int32_t* rank_offsets,
                                   int32_t* slot_to_row, int32_t* row_to_slot, void* send,
                                   fs_stream stream);

/* Rows landing on this rank's experts after Dispatch (Section 2.1).  The
 * receive buffer holds, for every source rank s, that rank's whole send
 * buffer at rows [s*N*k, (s+1)*N*k).
 *   src_counts    [R, E] int32 in: expert_counts of every source rank
 *   src_offsets   [R, E+1] int32 in: expert_offsets of every source rank
 *   group_rows    [R*N*k] int32 out: for each local expert e ascending, the
 *                 rows of source 0, 1, .. R-1 in that source's send order:
 *                 s*N*k + src_offsets[s][r*E/R + e] + j
 *   group_offsets [E/R + 1] int32 out: start of each local expert's rows */
fs_status fs_receive_rows(const fs_moe_desc* desc, const int32_t* src_counts,
                          const int32_t* src_offsets, int32_t* group_rows,
                          int32_t* group_offsets, fs_stream stream);

/* Rows of this rank's experts with replicated activations (Section 4.2:
 * every rank holds all N tokens; Section 2.1: rank r owns experts
 * [r*E/R, (r+1)*E/R)).  These are the plan rows [rank_offsets[r],
 * rank_offsets[r+1]) of fs_dispatch_pack (expert-major, tokens ascending),
 * read back to token indices so the expert GEMM gathers them from x.
 *   expert_offsets [E+1], rank_offsets [R+1], row_to_slot [N*k]: int32 in,
 *                  as written by fs_dispatch_pack for the same topk_ids
 *   local_tokens   [min(k, E/R) * N] int32 out: entry i < M_r is the token of
 *                  local row i, M_r = rank_offsets[r+1] - rank_offsets[r];
 *                  later entries are not written
 *   local_offsets  [E/R + 1] int32 out: expert_offsets[r*E/R + e] -
 *                  rank_offsets[r], the start of local expert e's rows
 * With N == 0 nothing is written (no rows). */
fs_status fs_local_rows(const fs_moe_desc* desc, const int32_t* expert_offsets,
                        const int32_t* rank_offsets, const int32_t* row_to_slot,
                        int32_t* local_tokens, int32_t* local_offsets, fs_stream stream);

/* Grouped SwiGLU expert FFN (Section 2.1, MLP^j read as SwiGLU): for each
 * group g and its rows X_g, Y_g = (SiLU(X_g Wg^T) * (X_g Wu^T)) Wd^T.
 * bf16 runs on MFMA with fp32 accumulation and the hidden activation
 * rounded to bf16; fp32 runs on the vector ALUs.
 *   n_groups      groups (local experts, or 1 for merged shared experts)
 *   ffn           F of every group
 *   in_rows       [*, d] dtype: row i of the grouped order is
 *                 in_rows[group_rows[i]] (or in_rows[i] when group_rows is
 *                 NULL)
 *   group_rows    [M] int32 or NULL
 *   group_offsets [n_groups+1] int32 device, non-decreasing, [0] = 0; NULL
 *                 only with n_groups == 1, meaning one group of max_rows rows
 *   max_rows      host-known bound on M = group_offsets[n_groups]; sizes the
 *                 launch and the workspace (any M <= max_rows is correct)
 *   w_gate_up     [n_groups, 2F, d] dtype: rows [0,F) gate, [F,2F) up
 *   w_down        [n_groups, d, F] dtype
 *   out_rows      [*, d] dtype out: output i goes to out_rows[group_rows[i]]
 *                 (or out_rows[i]) */
fs_status fs_grouped_expert_ffn(const fs_moe_desc* desc, int32_t n_groups, int32_t ffn,
                                const void* in_rows, const int32_t* group_rows,
                                const int32_t* group_offsets, int64_t max_rows,
                                const void* w_gate_up, const void* w_down, void* out_rows,
                                void* ws, size_t ws_bytes, fs_stream stream);

/* Expert weights in MFMA fragment order, a load-time layout transform for
 * weight streaming (decode: the MoE layer's experts, Section 2.1, whose
 * weights each routed pass reads once from HBM; the paper's decode is
 * memory-bound, Section 5.2).  n_mats row-major bf16 matrices [rows, cols]
 * (rows % 32 == 0, cols % 16 == 0) are rewritten as [rows/32][cols/16]
 * blocks of 1 KB: in block (g, c), the 16 bytes at lane l (0..63) are
 * row 32 g + l % 32, columns 16 c + 8 (l / 32) .. + 7, the B operand layout
 * of a 32 x 32 x 16 bf16 matrix instruction.  A block is one 1 KB load and
 * a 32-row group's whole column range is contiguous.
 *   src, dst   n_mats * rows * cols bf16 each, device, 16-byte aligned,
 *              not overlapping
 * FS_ERR_UNSUPPORTED for other dtypes or shapes. */
fs_status fs_expert_weights_fragment_order(int32_t dtype, int64_t n_mats, int32_t rows,
                                           int32_t cols, const void* src, void* dst,
                                           fs_stream stream);

/* fs_grouped_expert_ffn with fragment-ordered weights
 * (fs_expert_weights_fragment_order of w_gate_up as n_groups matrices
 * [2F, d] and of w_down as n_groups matrices [d, F]): the same rows,
 * groups, outputs and workspace (FS_OP_GROUPED_FFN), bf16 only, ffn % 128
 * == 0 and d % 256 == 0 (FS_ERR_UNSUPPORTED otherwise).  The weights
 * stream from memory straight into the matrix units' registers, 64 rows
 * per tile: meant for groups of few rows (decode), where the pass is
 * bound by reading every weight once; larger groups are correct but re-read
 * each weight panel once per 64 rows. */
fs_status fs_grouped_expert_ffn_fo(const fs_moe_desc* desc, int32_t n_groups, int32_t ffn,
                                   const void* in_rows, const int32_t* group_rows,
                                   const int32_t* group_offsets, int64_t max_rows,
                                   const void* w_gate_up_fo, const void* w_down_fo,
                                   void* out_rows, void* ws, size_t ws_bytes, fs_stream stream);

/* FP8 fragment order: n_mats row-major E4M3 code matrices [rows, cols]
 * (rows % 32 == 0, cols % 64 == 0; fs_quantize_fp8 codes) rewritten as
 * [rows/32][cols/64] fragments of 2 KB, each two 1 KB halves: in fragment
 * (g, c), half h, the 16 bytes at lane l (0..63) are row 32 g + l % 32,
 * columns 64 c + 32 (l / 32) + 16 h .. + 15 (lane l's 32 bytes are the B
 * operand of a 32 x 32 x 64 FP8 matrix instruction).  Same purpose as
 * fs_expert_weights_fragment_order: weight streaming in decode (Section
 * 5.2), here for the FP8 experts the paper's inference runs use.
 *   src, dst   n_mats * rows * cols bytes each, device, 16-byte aligned,
 *              not overlapping
 * FS_ERR_UNSUPPORTED for other shapes. */
fs_status fs_expert_weights_fragment_order_fp8(int64_t n_mats, int32_t rows, int32_t cols,
                                               const uint8_t* src, uint8_t* dst,
                                               fs_stream stream);

/* fs_grouped_expert_ffn_fp8 with FP8-fragment-ordered weight codes
 * (fs_expert_weights_fragment_order_fp8 of w_gate_up as n_groups matrices
 * [2F, d] and of w_down as n_groups matrices [d, F]; the row scales are
 * unchanged): the same operands, groups, outputs and workspace
 * (FS_OP_GROUPED_FFN_FP8), ffn % 128 == 0 and d % 256 == 0.  The MFMAs see
 * the operands of fs_grouped_expert_ffn_fp8's kernel, so a pass that kernel
 * runs without splitting K gives the same bits.  Meant for groups of few
 * rows (decode). */
fs_status fs_grouped_expert_ffn_fp8_fo(const fs_moe_desc* desc, int32_t n_groups, int32_t ffn,
                                       const uint8_t* x_codes, const float* x_scales,
                                       const int32_t* group_rows, const int32_t* group_offsets,
                                       int64_t max_rows, const uint8_t* w_gate_up_fo,
                                       const float* s_gate_up, const uint8_t* w_down_fo,
                                       const float* s_down, void* out_rows, void* ws,
                                       size_t ws_bytes, fs_stream stream);

/* The grouped SwiGLU FFN of fs_grouped_expert_ffn with the input gathered
 * and the output in grouped order: row i of the grouped order reads
 * x[gather_rows[i]] and writes y[i].  Used with replicated activations,
 * where the GEMM reads this rank's rows straight from the token matrix.
 *   x            [*, d] dtype
 *   gather_rows  [max_rows] int32: token of each row (local_tokens of
 *                fs_local_rows)
 *   y            [max_rows, d] dtype out
 * Other arguments, the workspace (FS_OP_GROUPED_FFN) and the arithmetic are
 * those of fs_grouped_expert_ffn. */
fs_status fs_grouped_expert_ffn_gathered(const fs_moe_desc* desc, int32_t n_groups, int32_t ffn,
                                         const void* x, const int32_t* gather_rows,
                                         const int32_t* group_offsets, int64_t max_rows,
                                         const void* w_gate_up, const void* w_down, void* y,
                                         void* ws, size_t ws_bytes, fs_stream stream);

/* FP8 experts (the paper's inference runs use FP8 experts, Section 5.2).
 * Row-wise OCP FP8 E4M3 quantisation of rows x [rows, cols] (activations:
 * one row per token or expert row; weights: one row per output channel):
 * amax = max |x_i|; scale = amax / 448 and inv = 448 / amax, each a
 * correctly rounded fp32 division; code_i = E4M3(clamp(x_i * inv, +-448))
 * rounded to nearest, ties to even (x_i * inv one fp32 rounding).  An
 * all-zero row gets scale 1 and zero codes.  The row stands for
 * dec(code_i) * scale.
 *   dtype   FS_F32 or FS_BF16: the type of src
 *   src     [rows, cols], cols % 16 == 0, 16-byte aligned
 *   codes   [rows, cols] uint8 out, 16-byte aligned
 *   scales  [rows] fp32 out */
fs_status fs_quantize_fp8(int32_t dtype, int64_t rows, int32_t cols, const void* src,
                          uint8_t* codes, float* scales, fs_stream stream);

/* Grouped SwiGLU expert FFN on FP8 operands: the data flow of
 * fs_grouped_expert_ffn with x and the weights as E4M3 codes and row
 * scales (fs_quantize_fp8).  gate and up are
 *   sum_k dec(x_mk) dec(w_nk) * x_scale[m] * s_gate_up[g][n]
 * (MFMA with fp32 accumulation); H = SiLU(gate) * up rounded to bf16; H is
 * quantised per row (as fs_quantize_fp8) inside the workspace; down is the
 * same scaled product of H and w_down; out rows are bf16.
 *   x_codes [*, d] uint8, x_scales [*] fp32: rows as in_rows of
 *           fs_grouped_expert_ffn (gathered through group_rows)
 *   w_gate_up [n_groups, 2F, d] uint8, s_gate_up [n_groups, 2F] fp32
 *   w_down [n_groups, d, F] uint8, s_down [n_groups, d] fp32
 *   out_rows [*, d] bf16 out (scattered through group_rows)
 * desc->dtype must be FS_BF16; F % 128 == 0 and d % 256 == 0
 * (FS_ERR_UNSUPPORTED otherwise).  Workspace: FS_OP_GROUPED_FFN_FP8; after
 * the call it holds, for the M = group_offsets[n_groups] rows in grouped
 * order, H as bf16 [max_rows, F] at byte 0, its codes [max_rows, F] at
 * byte a(2 max_rows F) and its scales [max_rows] fp32 at byte
 * a(2 max_rows F) + a(max_rows F), where a(n) rounds n up to a multiple
 * of 256. */
fs_status fs_grouped_expert_ffn_fp8(const fs_moe_desc* desc, int32_t n_groups, int32_t ffn,
                                    const uint8_t* x_codes, const float* x_scales,
                                    const int32_t* group_rows, const int32_t* group_offsets,
                                    int64_t max_rows, const uint8_t* w_gate_up,
                                    const float* s_gate_up, const uint8_t* w_down,
                                    const float* s_down, void* out_rows, void* ws, size_t ws_bytes,
                                    fs_stream stream);

/* Combine and unpack (Section 2.1, Combine: weighted sum of the returned
 * expert outputs), fused with the deferred residual add of Eq. 7.
 *   acc[t] = sum_{j<k} topk_w[t,j] * y_ret[slot_to_row[t*k+j]]  (fp32, j
 *            ascending) + shared_out[t] (when given)
 *   y_ret       [N*k, d] dtype: expert outputs in send order
 *   shared_out  [N, d] dtype or NULL
 *   routed_out  [N, d] dtype or NULL: receives acc
 *   residual    [N, d] dtype or NULL: residual[t] += acc[t], one rounding
 * At least one of routed_out / residual must be given. */
fs_status fs_combine_unpack(const fs_moe_desc* desc, const void* y_ret,
                            const int32_t* slot_to_row, const float* topk_w,
                            const void* shared_out, void* routed_out, void* residual,
                            fs_stream stream);

/* Partial Combine of rank r with replicated activations (Section 4.2):
 *   partial[t] = sum over j < k with lo <= slot_to_row[t*k+j] < hi of
 *                topk_w[t,j] * y_local[slot_to_row[t*k+j] - lo]
 * in fp32, j ascending, rounded once to dtype; lo = rank_offsets[r],
 * hi = rank_offsets[r+1] (device).  A token whose selections are all on
 * other ranks gets a zero row.  Summed over the R ranks (the all-reduce)
 * the partials are the routed MoE output.
 *   y_local      [M_r, d] dtype: fs_grouped_expert_ffn_gathered's y
 *   slot_to_row  [N*k], rank_offsets [R+1]: int32, from fs_dispatch_pack
 *   topk_w       [N, k] fp32
 *   partial_out  [N, d] dtype out */
fs_status fs_combine_partial(const fs_moe_desc* desc, const void* y_local,
                             const int32_t* slot_to_row, const int32_t* rank_offsets,
                             const float* topk_w, void* partial_out, fs_stream stream);

/* One-GPU stand-in for the all-reduce of an [N, d] dtype partial sum over
 * the R ranks (Section 4.2): with one participant the sum is the partial
 * itself, so out = partial as a stand-in copy on `stream` (the traffic and
 * the stream placement of the collective, and with fs_standin_link its
 * duration; on a node RCCL's all-reduce takes its place).  out == partial
 * is an in-place no-op; other overlaps are FS_ERR_INVALID. */
fs_status fs_allreduce_standin(const fs_moe_desc* desc, void* out, const void* partial,
                               fs_stream stream);

/* Link model of the one-GPU stand-in copies: the Dispatch and Combine
 * copies of fs_moe_block_forward (the all-to-alls of Section 2.1) and
 * fs_allreduce_standin (the all-reduces of Section 4.2).  Process-wide;
 * applies to copies enqueued after the call.
 *   links == 0 (the default): each stand-in copy is a device-to-device copy
 *     at HBM speed (the arguments after links are ignored).
 *   links > 0: each runs as a copy kernel on `workgroups` workgroups that
 *     takes the time the collective would take on a node of links + 1 GPUs,
 *     every pair joined by one link of link_bytes_per_s per direction:
 *     B / ((links + 1) * link_bytes_per_s) for an all-to-all of a B-byte
 *     send buffer (each peer's share on its own link, all links at once),
 *     twice that for a ring all-reduce of B bytes over every link.  Byte b
 *     of the buffer is read no earlier than b / rate after the kernel
 *     starts, so the copy takes HBM bandwidth and CUs as a transfer at that
 *     rate would; it takes longer when the workgroups cannot keep up.
 * The bytes copied are the same either way.  links in [0, 1023];
 * link_bytes_per_s in [1e9, 1e15] and workgroups in [1, 4096] when links > 0;
 * else FS_ERR_INVALID and the setting is unchanged.  No GPU work. */
fs_status fs_standin_link(int32_t links, double link_bytes_per_s, int32_t workgroups);
/* The current link model (links 0: HBM-speed copies). */
fs_status fs_standin_link_get(int32_t* links, double* link_bytes_per_s, int32_t* workgroups);

/* FarSkip residual add (Eq. 7): out = residual + deferred (+ extra), in
 * fp32 with one rounding.  out may equal residual (in place).  [N, d]
 * dtype each; extra may be NULL. */
fs_status fs_farskip_residual(const fs_moe_desc* desc, void* out, const void* residual,
                              const void* deferred, const void* extra, fs_stream stream);

/* Weights of one block.  Shared experts are passed merged into one SwiGLU
 * of width S*F_s: ws_gate_up [2*S*F_s, d] holds the gate rows of every
 * shared expert followed by their up rows; ws_down [d, S*F_s]. */
typedef struct {
  const void* w_router;   /* [E, d] */
  const float* sel_bias;  /* [E] or NULL */
  const void* w_gate_up;  /* [E/R, 2F, d]: this rank's experts */
  const void* w_down;     /* [E/R, d, F] */
  const void* ws_gate_up; /* NULL when S = 0 */
  const void* ws_down;
  /* FP8 experts (fs_quantize_fp8 codes and row scales; bf16 blocks only).
   * When w_gate_up_fp8 is given the routed experts run in FP8 and
   * w_gate_up / w_down are not read: the gate phase packs FP8 rows
   * (fs_dispatch_pack_fp8), so `send` and `recv` hold FP8 row buffers
   * (send: N*k rows; recv: R*N*k rows, slot s = rows [s*N*k, (s+1)*N*k)
   * of its codes and of its scales), Dispatch moves codes and scales, and
   * fs_grouped_expert_ffn_fp8 reads the received codes.  Likewise
   * ws_gate_up_fp8 for the shared experts, which quantise their N input
   * rows.  y and Combine stay bf16. */
  const uint8_t* w_gate_up_fp8;  /* [E/R, 2F, d] or NULL */
  const float* s_gate_up;        /* [E/R, 2F] */
  const uint8_t* w_down_fp8;     /* [E/R, d, F] */
  const float* s_down;           /* [E/R, d] */
  const uint8_t* ws_gate_up_fp8; /* [2 S F_s, d] or NULL */
  const float* ss_gate_up;       /* [2 S F_s] */
  const uint8_t* ws_down_fp8;    /* [d, S F_s] */
  const float* ss_down;          /* [d] */
  /* Fragment-ordered copies of w_gate_up and w_down
   * (fs_expert_weights_fragment_order), or NULL.  When given (bf16, ffn %
   * 128 == 0, d % 256 == 0), routed-expert passes whose groups average at
   * most 64 rows (decode) stream them with fs_grouped_expert_ffn_fo's
   * kernels; other passes read w_gate_up / w_down, which stay required. */
  const void* w_gate_up_fo;      /* [E/R, 2F, d] in fragment order */
  const void* w_down_fo;         /* [E/R, d, F] in fragment order */
  /* FP8-fragment-ordered copies of w_gate_up_fp8 and w_down_fp8
   * (fs_expert_weights_fragment_order_fp8), or NULL: with FP8 routed
   * experts, passes whose groups average at most 64 rows stream them with
   * fs_grouped_expert_ffn_fp8_fo's kernels; the FP8 fields above stay
   * required. */
  const uint8_t* w_gate_up_fp8_fo; /* [E/R, 2F, d] codes in FP8 fragment order */
  const uint8_t* w_down_fp8_fo;    /* [E/R, d, F] */
} fs_moe_weights;

/* Caller-owned buffers of one block (device memory). */
typedef struct {
  float* logits;          /* [N, E] or NULL */
  int32_t* topk_ids;      /* [N, k] */
  float* topk_w;          /* [N, k] */
  int32_t* src_counts;    /* [R, E]: row r written by BEGIN, other rows by the
                             caller before FINISH (the counts exchange) */
  int32_t* src_offsets;   /* [R, E+1]: likewise */
  int32_t* rank_offsets;  /* [R+1] */
  int32_t* slot_to_row;   /* [N*k] */
  int32_t* row_to_slot;   /* [N*k] */
  void* send;             /* [N*k, d] */
  void* recv;             /* [R*N*k, d]: slot s = source s's send buffer; the
                             caller fills slots s != r (R > 1); may be NULL
                             when R = 1 and no comm stream is given */
  int32_t* group_rows;    /* [R*N*k] (R > 1) */
  int32_t* group_offsets; /* [E/R+1] (R > 1) */
  void* y;                /* [R*N*k, d]: expert outputs at their receive row;
                             slot r is this rank's Combine return y_ret, whose
                             rows for other ranks' experts the caller fills */
  void* shared_out;       /* [N, d] (S > 0) */
  void* ret;              /* [N*k, d] or NULL: the Combine stand-in copies y's
                             slot r here and the weighted sum reads it; NULL:
                             no copy, the sum reads slot r of y */
} fs_block_buffers;

/* Events that order the two streams of one block. */
typedef struct fs_block_sync fs_block_sync;
fs_status fs_block_sync_create(fs_block_sync** out);
fs_status fs_block_sync_destroy(fs_block_sync* sync);

/* One FarSkip MoE block forward (Section 3 connectivity, Section 4.1
 * schedule), in phases that let the caller place other work between them.
 *   FS_PHASE_GATE on `compute`: router + top-k, plan + pack; then the
 *     Dispatch stand-in: on `comm` (after an event), a stand-in copy
 *     (fs_standin_link) of the whole send buffer into receive slot r.
 *   FS_PHASE_SHARED on `compute`: the shared experts on residual_in and
 *     partial_out = residual_in + shared_out (Eq. 8b: the next layer's input
 *     without the routed output).
 *   FS_PHASE_EXPERTS on `compute`: wait for the Dispatch copy, receive rows
 *     (R > 1), grouped SwiGLU experts; then, if buffers->ret is given, the
 *     Combine stand-in: on `comm` (after an event), a copy of y's slot r
 *     (the rows this rank's tokens get back) into ret.
 *   FS_PHASE_COMBINE on `compute`: wait for the Combine copy, then the
 *     weighted sum over each token's k rows and the deferred add
 *     residual_io += routed (Eq. 7).
 *   FS_PHASE_BEGIN = GATE + SHARED, FS_PHASE_FINISH = EXPERTS + COMBINE,
 *   FS_PHASE_ALL = all four.  Between BEGIN and FINISH the caller enqueues
 *   the far-skipped next computation on `compute`, reading partial_out; it
 *   overlaps the Dispatch copy.  In the two-window schedule of Section 4.1
 *   the phases of consecutive layers interleave: GATE_k, attention,
 *   EXPERTS_k, SHARED_k, the next layer's first attention part, COMBINE_k,
 *   GATE_{k+1}, ...; the Combine copy of layer k then overlaps SHARED_k and
 *   that attention part.
 * With comm == NULL each copy runs on `compute` in order (blocking, as in
 *   the regular schedule); the Dispatch copy is skipped when recv is NULL
 *   (R = 1: the experts read `send`), the Combine copy when ret is NULL.
 * residual_in [N, d] is o_{k-1}, the MoE input (Eq. 8a); partial_out [N, d];
 * residual_io [N, d] is updated in place (normally partial_out after the
 * caller added its next-layer output).  max_recv_rows bounds the rows
 * landing on local experts (N*k when R = 1).  sync may be NULL only with
 * comm == NULL.  Every phase of one block gets the same comm argument.  One
 * sync object serves one block at a time: the phases of one block are
 * enqueued in order (GATE before EXPERTS before COMBINE) before the next
 * GATE that uses the same object. */
fs_status fs_moe_block_forward(const fs_moe_desc* desc, int32_t phase,
                               const fs_moe_weights* weights, const void* residual_in,
                               void* partial_out, void* residual_io, fs_block_buffers* buffers,
                               int64_t max_recv_rows, void* ws, size_t ws_bytes,
                               fs_block_sync* sync, fs_stream compute, fs_stream comm);

/* Dense linear out[m, n] = a[m, :] . w[n, :] in dtype with fp32
 * accumulation; stands in for the next layer's computation.  a [m, kdim],
 * w [n, kdim], out [m, n]; kdim % 64 == 0; n % 128 == 0 for bf16, n % 64 == 0
 * for fp32 (else FS_ERR_UNSUPPORTED). */
fs_status fs_dense_linear(int32_t dtype, int32_t m, int32_t n, int32_t kdim, const void* a,
                          const void* w, void* out, fs_stream stream);

/* Per-kernel timing with HIP events recorded on the launch stream around
 * selected kernels.  fs_profile_read synchronises those events.
 * FS_K_GATE_UP / FS_K_DOWN time the routed experts' passes (and
 * fs_grouped_expert_ffn and fs_grouped_expert_ffn_fp8 with group_offsets,
 * and fs_grouped_expert_ffn_gathered; for FP8, FS_K_DOWN includes the
 * quantisation of H); FS_K_COMBINE fs_combine_unpack,
 * fs_combine_partial and the block's Combine; FS_K_SHARED_* the shared
 * experts' passes inside fs_moe_block_forward and fs_grouped_expert_ffn
 * without group_offsets (one group of max_rows rows);
 * FS_K_DISPATCH_COPY / FS_K_COMBINE_COPY the Dispatch and Combine stand-in
 * copies on the stream they run on; FS_K_DENSE fs_dense_linear;
 * FS_K_ALLREDUCE_COPY fs_allreduce_standin; FS_K_QUANTIZE the activation
 * quantisation of the block's FP8 experts. */
typedef enum {
  FS_K_ROUTER = 0,
  FS_K_TOPK = 1,
  FS_K_PLAN = 2,
  FS_K_PACK = 3,
  FS_K_GATE_UP = 4,
  FS_K_DOWN = 5,
  FS_K_COMBINE = 6,
  FS_K_SHARED_GATE_UP = 7,
  FS_K_SHARED_DOWN = 8,
  FS_K_DISPATCH_COPY = 9,
  FS_K_DENSE = 10,
  FS_K_COMBINE_COPY = 11,
  FS_K_ALLREDUCE_COPY = 12,
  FS_K_QUANTIZE = 13,
  FS_K_COUNT = 14
} fs_kernel_id;
fs_status fs_profile_enable(int32_t on);
/* Which kernels fs_profile_enable times: bit i of mask selects fs_kernel_id
 * i (all by default).  Every timed kernel adds a stream event, and on a
 * step of many short kernels those events slow the step itself, so a
 * caller that times the whole step can select only the kernels it needs.
 * Bits at or above FS_K_COUNT: FS_ERR_INVALID. */
fs_status fs_profile_select(uint32_t mask);
fs_status fs_profile_read(int32_t kernel, double* total_ms, int64_t* launches);
fs_status fs_profile_reset(void);

#ifdef __cplusplus
}
#endif

#endif /* FARSKIP_H */
