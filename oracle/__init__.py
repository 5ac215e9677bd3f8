"""CPU oracle for the FarSkip MoE block forward -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product path (the HIP library and its Python
binding) never imports, calls or links anything here, and this package
imports nothing from the product path.

What it computes is the plain definition of one FarSkip MoE block on one
expert-parallel rank's share (Section 2.1: the MoE layer, Dispatch and
Combine; Section 3: the FarSkip residual, Eq. 7 with the outdated input of
Eq. 8a for the MoE and the partial input of Eq. 8b for the next layer).
Floating point is fp64 on values decoded exactly from the fp32/bf16 inputs.
Routing decisions are taken from fp32 logits summed in the documented fixed
order (``logits_routing_f32``), because the kernel takes them in fp32.

Parity status per function (what pins it is in tests/test_oracle_pins.py):
  logits_f64, logits_routing_f32 ... pinned (exact integer cases, error bound)
  route ............................ pinned (brute force over subsets)
  dispatch_plan, pack .............. pinned (stable argsort, bijection)
  receive_rows ..................... pinned (per-source decomposition)
  swiglu ........................... pinned (closed forms)
  combine, moe_block ............... pinned (dense masked brute force)
  route_given ...................... pinned (route's own selection, slot order)
  moe_tokens_direct ................ pinned (dense gate-matrix mixture, the packed
                                     block with remote rows, a hand value)
  farskip_pair, regular_pair ....... pinned (zero-output equality, conservation)
  farskip_stack, regular_stack ..... pinned (zero-output equality, conservation,
                                     one layer = the block, the dropped dependency)

oracle.allreduce holds the replicated-activation inference variant (each
rank runs its own experts on every token; partial sums are all-reduced):
  local_rows ....................... pinned (the plan's rank blocks)
  routed_partial, combine_partial .. pinned (partials over R ranks sum to the
                                     all-to-all block; zero rows; two forms)
  shared_partial, attention_partial  pinned (partials sum to the full terms)
  farskip_ar_stack, regular_ar_stack pinned (R = 1 equals the all-to-all
                                     stacks; conservation; dropped dependency)
tests/test_oracle_allreduce.py holds those pins.

oracle.fp8 holds the FP8 (E4M3) experts: row quantisation, scaled GEMMs and
the FP8 SwiGLU expert:
  e4m3_decode / e4m3_encode ........ pinned (format constants, round trip,
                                     brute-force nearest with ties to even)
  quantize_rows, scaled_gemm ....... pinned (amax code, zero rows, error
                                     bound, hand value)
  swiglu_fp8 ....................... pinned (lossless quantisation reduces to
                                     the bf16-rounded SwiGLU)
tests/test_oracle_fp8.py holds those pins.
"""

from . import allreduce, fp8  # noqa: F401
from .moe import (  # noqa: F401
    ROUTER_SLICE,
    logits_f64,
    logits_routing_f32,
    route,
    route_given,
    dispatch_plan,
    pack,
    receive_rows,
    silu,
    swiglu,
    shared_ffn,
    combine,
    moe_block,
    moe_tokens_direct,
    farskip_pair,
    regular_pair,
    residual_add,
    dense_linear,
    attention_stand_in,
    farskip_stack,
    regular_stack,
)
