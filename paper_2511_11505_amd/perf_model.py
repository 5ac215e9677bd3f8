"""Analytic performance model of FarSkip prefill (App. B, Tab. 5, Fig. 9).

One MoE transformer layer of a DeepSeek-V3-like model serving a prefill
batch on an 8-accelerator node, attention and shared experts tensor-parallel
over the 8, routed experts expert-parallel over the 8 with perfect load
balance, activations replicated (the inference variant of Section 4.2):
after attention and after the MLP the activations are all-reduced.

Component runtimes are FLOPs / rate (GEMMs and attention at their own
rates) and message bytes / all-reduce bandwidth.  The exposed communication
of each all-reduce follows Tab. 5, with max(0, .) where the table prints
min(0, .) (an exposed time is never negative):
  regular:  attention all-reduce attn.comm, MLP all-reduce mlp.comm, both
            fully exposed;
  FarSkip:  attention + shared all-reduce (one message)
            max(0, as.comm - routed.runtime); routed all-reduce
            max(0, routed.comm - attn.runtime).
Sparsity s = routed experts / active routed experts; a model s/32 times
sparser than DeepSeek-V3 (s = 32) has s/32 times the experts, each
32/s times narrower, with the same 8 + 1 active experts: same parameters,
fewer routed FLOPs.

Pure arithmetic on the host; no GPU and no data.  ``measured_rates`` and
``calibrated_machine`` take the rates from a bench.py record of one MI355X
instead (``--bench FILE``).
"""

from dataclasses import dataclass, replace


@dataclass(frozen=True)
class Arch:
    """DeepSeek-V3 dimensions (the attention is multi-head latent)."""
    d: int = 7168
    heads: int = 128
    q_lora: int = 1536
    kv_lora: int = 512
    qk_nope: int = 128
    qk_rope: int = 64
    v_head: int = 128
    experts: int = 256
    active: int = 8
    ffn: int = 2048
    shared_ffn: int = 2048
    n_shared: int = 1

    def sparser(self, s):
        """The same parameter count at sparsity s (s = experts / active)."""
        ratio = s * self.active / self.experts
        return replace(self, experts=int(round(self.experts * ratio)),
                       ffn=int(round(self.ffn / ratio)))


@dataclass(frozen=True)
class Machine:
    """Sustained rates: FLOP/s for GEMMs and for attention, all-reduce bus
    bandwidth in bytes/s, node size.  The default is the hypothetical
    accelerator of App. B."""
    gemm_flops: float = 600e12
    attn_flops: float = 500e12
    allreduce_bw: float = 400e9
    gpus: int = 8
    gate_flops: float = 0.0     # the router's rate; 0: the GEMM rate

    def scaled(self, compute=1.0, attention=1.0, comm=1.0):
        return replace(self, gemm_flops=self.gemm_flops * compute,
                       attn_flops=self.attn_flops * compute * attention,
                       gate_flops=self.gate_flops * compute,
                       allreduce_bw=self.allreduce_bw * comm)


@dataclass(frozen=True)
class Batch:
    """Prefill batch: sequences x context, activations of `act_bytes`."""
    seqs: int = 32
    context: int = 2048
    act_bytes: int = 2

    @property
    def tokens(self):
        return self.seqs * self.context


def gemm_flops(m, k, n):
    return 2.0 * m * k * n


def attention_flops(a, b):
    """Whole-node FLOPs of one MLA attention layer on a causal prefill
    batch: the projections plus QK^T and PV over the lower triangle."""
    t = b.tokens
    proj = (gemm_flops(t, a.d, a.q_lora)
            + gemm_flops(t, a.q_lora, a.heads * (a.qk_nope + a.qk_rope))
            + gemm_flops(t, a.d, a.kv_lora + a.qk_rope)
            + gemm_flops(t, a.kv_lora, a.heads * (a.qk_nope + a.v_head))
            + gemm_flops(t, a.heads * a.v_head, a.d))
    pairs = b.seqs * b.context * (b.context + 1) / 2.0       # causal (query, key) pairs
    core = 2.0 * pairs * a.heads * (a.qk_nope + a.qk_rope) + 2.0 * pairs * a.heads * a.v_head
    return proj, core


def swiglu_flops(tokens, d, f):
    """Gate, up and down projections of one SwiGLU MLP."""
    return gemm_flops(tokens, d, 2 * f) + gemm_flops(tokens, f, d)


def allreduce_time(nbytes, m):
    """Ring all-reduce of nbytes over m.gpus at bus bandwidth m.allreduce_bw
    (bus bandwidth = algorithm bandwidth x 2 (n - 1) / n)."""
    n = m.gpus
    return nbytes * 2.0 * (n - 1) / n / m.allreduce_bw


def layer_times(a, m, b):
    """Per-accelerator runtimes of one layer's parts (seconds)."""
    t = b.tokens
    proj, core = attention_flops(a, b)
    attn = proj / m.gpus / m.gemm_flops + core / m.gpus / m.attn_flops
    shared = a.n_shared * swiglu_flops(t, a.d, a.shared_ffn) / m.gpus / m.gemm_flops
    routed = a.active * swiglu_flops(t, a.d, a.ffn) / m.gpus / m.gemm_flops
    gate = gemm_flops(t, a.d, a.experts) / m.gpus / (m.gate_flops or m.gemm_flops)
    msg = allreduce_time(t * a.d * b.act_bytes, m)            # one [tokens, d] all-reduce
    return dict(attn=attn, shared=shared, routed=routed, gate=gate, attn_comm=msg, mlp_comm=msg)


def exposed(comm, overlapped_compute):
    """Communication left exposed after overlapping it with a computation."""
    return max(0.0, comm - overlapped_compute)


def layer_runtime(parts, farskip):
    """Layer time (seconds): compute plus exposed communication (Tab. 5)."""
    compute = parts["attn"] + parts["shared"] + parts["routed"] + parts["gate"]
    if farskip:
        comm = (exposed(parts["attn_comm"], parts["routed"])     # attention + shared, one message
                + exposed(parts["mlp_comm"], parts["attn"]))     # routed experts
    else:
        comm = parts["attn_comm"] + parts["mlp_comm"]
    return compute + comm


def speedup(a, m, b):
    parts = layer_times(a, m, b)
    return layer_runtime(parts, False) / layer_runtime(parts, True)


SPARSITIES = (4, 8, 16, 32, 64, 128, 256, 512)

SCENARIOS = {
    "baseline": dict(),
    "2x compute": dict(compute=2.0),
    "2x attention": dict(attention=2.0),
    "2x communication": dict(comm=2.0),
    "2x compute + 2x communication": dict(compute=2.0, comm=2.0),
}


def sweep(machine=Machine(), batch=Batch(), arch=Arch(), sparsities=SPARSITIES):
    """{scenario: [(sparsity, speedup)]} (Fig. 9 and its scenarios)."""
    out = {}
    for name, kw in SCENARIOS.items():
        m = machine.scaled(**kw)
        out[name] = [(s, speedup(arch.sparser(s), m, batch)) for s in sparsities]
    return out


# ---------------------------------------------------------------- calibration
# Rates measured on one MI355X by bench.py replace the hypothetical
# accelerator's: the routed SwiGLU experts' sustained TFLOP/s for the
# model's GEMMs, the dense linear's (the attention stand-in's parts a and b)
# for attention, and the router's.  The all-reduce bandwidth of an
# 8 x MI355X node is not measurable on one GPU and stays a parameter.

@dataclass(frozen=True)
class Rates:
    """Sustained TFLOP/s of the kernels a bench.py record timed."""
    routed: float          # routed SwiGLU experts, gate/up + down
    shared: float          # shared experts, gate/up + down (0 without)
    dense: float           # dense d x d linear (attention stand-in)
    router: float          # router logits


def _record_shape(rec):
    c = rec["config"]
    N, d, E, k = c["tokens"], c["hidden"], c["experts"], c["top_k"]
    # rows on this rank's experts: recorded by block lines; a stacked-layer
    # line takes the balanced expectation N k (each of R ranks routes N
    # tokens to k experts, a 1/R share of which is local)
    rows = c.get("rows_local_experts", N * k)
    return N, d, E, k, c["ffn"], c.get("shared", 0), c.get("ffn_shared", 0), rows


def measured_rates(rec):
    """Rates of a bench.py JSON record (a block line, or a stacked-layer
    line of bench.py --layers), from its per-launch kernel times."""
    N, d, E, k, F, S, Fs, rows = _record_shape(rec)
    us = rec["kernels_us"]
    tflops = lambda flops, t_us: flops / (t_us * 1e-6) / 1e12
    routed = tflops(swiglu_flops(rows, d, F), us["gate_up"] + us["down"])
    shared = (tflops(S * swiglu_flops(N, d, Fs), us["shared_gate_up"] + us["shared_down"])
              if S and "shared_gate_up" in us else 0.0)
    dense = tflops(gemm_flops(N, d, d), us["next_layer"]) if "next_layer" in us else routed
    router = tflops(gemm_flops(N, d, E), us["router"])
    return Rates(routed, shared, dense, router)


STACK_KERNELS = ("router", "topk", "plan", "pack", "gate_up", "down", "combine",
                 "shared_gate_up", "shared_down")


def stack_layer_time(rec):
    """Modelled time (s) of one stacked layer of bench.py --layers: the
    attention stand-in's two dense linears and the block's kernels, in
    sequence, with the Dispatch and Combine stand-in copies hidden (the
    FarSkip schedule's windows, Eq. 9)."""
    us = rec["kernels_us"]
    t = sum(us.get(n, 0.0) for n in STACK_KERNELS) + 2 * us.get("next_layer", 0.0)
    return t * 1e-6


def calibrated_machine(rec, allreduce_bw, gpus=8):
    """The App. B node with one MI355X's measured rates: GEMMs at the
    routed experts' rate, attention at the dense linear's, the gate at the
    router's."""
    r = measured_rates(rec)
    return Machine(gemm_flops=r.routed * 1e12, attn_flops=r.dense * 1e12,
                   allreduce_bw=allreduce_bw, gpus=gpus, gate_flops=r.router * 1e12)


def main():
    import argparse
    import json
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gemm-tflops", type=float, default=600.0)
    ap.add_argument("--attn-tflops", type=float, default=500.0)
    ap.add_argument("--allreduce-gbs", type=float, default=400.0)
    ap.add_argument("--bench", default=None,
                    help="a bench.py JSON line (file): take the GEMM and attention rates from it")
    a = ap.parse_args()
    m = Machine(a.gemm_tflops * 1e12, a.attn_tflops * 1e12, a.allreduce_gbs * 1e9)
    if a.bench:
        rec = json.loads(open(a.bench).read().strip().splitlines()[-1])
        r = measured_rates(rec)
        m = calibrated_machine(rec, a.allreduce_gbs * 1e9)
        print(f"rates from {a.bench}: routed {r.routed:.1f}, shared {r.shared:.1f}, dense "
              f"{r.dense:.1f}, router {r.router:.1f} TFLOP/s; all-reduce {a.allreduce_gbs:.0f} GB/s")
        if "layers" in rec["config"]:
            per = rec["ms_per_step"] * 1e-3 / rec["config"]["layers"]
            print(f"stacked layer: modelled {stack_layer_time(rec) * 1e6:.1f} us, measured "
                  f"{per * 1e6:.1f} us")
    res = sweep(m)
    print("| scenario | " + " | ".join(f"{s}x" for s in SPARSITIES) + " |")
    print("|---|" + "---|" * len(SPARSITIES))
    for name, row in res.items():
        print(f"| {name} | " + " | ".join(f"{v:.3f}" for _, v in row) + " |")


if __name__ == "__main__":
    main()
