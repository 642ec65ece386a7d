"""Workload shapes and closed-form cost accounting.

The five workloads are synthetic single attention layers shaped like the
paper's models (Sec. 4: TinyLlama-1.1B, Llama-3.1-8B, a 12B-class GQA model)
and cache formats (Sec. 3.1: grouped affine, KIVI K2V2, Hadamard-rotated
K4V2 with symmetric codes).  There are no datasets or trained weights: every
tensor is drawn by :mod:`paper_2609_04263_amd.synth`.

Format dictionaries use the field names of ``kvq_format`` in ``include/kvq.h``.
"""
from __future__ import annotations

from dataclasses import dataclass, field

AFFINE, SYMMETRIC = 0, 1
PER_TOKEN, PER_CHANNEL = 0, 1


def make_format(k_bits=4, v_bits=4, k_mode=AFFINE, v_mode=AFFINE, k_axis=PER_TOKEN,
                v_axis=PER_TOKEN, k_group=64, v_group=64, residual=0, flush=0, rotate=0,
                meta_fp16=0, sink=0) -> dict:
    return dict(k_bits=k_bits, v_bits=v_bits, k_mode=k_mode, v_mode=v_mode, k_axis=k_axis,
                v_axis=v_axis, k_group=k_group, v_group=v_group, residual=residual,
                flush=flush, rotate=rotate, meta_fp16=meta_fp16, sink=sink)


@dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    B: int
    H_q: int
    H_kv: int
    D: int
    d_in: int
    rank: int
    alpha: float
    fmt: dict = field(hash=False)
    context: int           # tokens in the cache when decoding starts
    decode_steps: int
    chunk: int             # tokens per sequence per prefill projection call
    w_var: float           # variance of base weights
    outlier: tuple         # ("scale", count per kv head, factor) | ("student_t", nu)

    @property
    def G(self) -> int:
        return self.H_q // self.H_kv

    @property
    def d_q(self) -> int:
        return self.H_q * self.D

    @property
    def d_kv(self) -> int:
        return self.H_kv * self.D

    @property
    def d_qkv(self) -> int:
        return self.d_q + 2 * self.d_kv

    @property
    def lora_scale(self) -> float:
        return self.alpha / self.rank if self.rank else 0.0

    @property
    def T_max(self) -> int:
        return self.context + self.decode_steps


WORKLOADS = {
    # TinyLlama-shaped layer, batch 1: prefill 256 then 16 decode appends.
    "tiny_b1": Workload("tiny_b1", 1, 1, 32, 4, 64, 2048, 8, 16.0,
                        make_format(4, 4, k_group=32, v_group=32), 256, 16, 256,
                        1.0 / 2048, ("scale", 4, 20.0)),
    # TinyLlama-shaped layer, batch 16, context 4096, 128 decode steps.
    "tiny_b16": Workload("tiny_b16", 2, 16, 32, 4, 64, 2048, 16, 32.0,
                         make_format(4, 4, k_group=64, v_group=64), 4096, 128, 2048,
                         1.0 / 2048, ("scale", 4, 20.0)),
    # Llama-3.1-8B-shaped layer, batch 32, context 8192, KIVI K2V2.
    "llama8b_kivi": Workload("llama8b_kivi", 3, 32, 32, 8, 128, 4096, 16, 32.0,
                             make_format(2, 2, k_axis=PER_CHANNEL, k_group=32, v_group=32,
                                         residual=128, flush=32), 8192, 128, 2048,
                             1.0 / 4096, ("scale", 4, 20.0)),
    # 12B-class GQA layer, batch 8, context 8192, 2048-token prefill chunks.
    "gqa12b_b8": Workload("gqa12b_b8", 4, 8, 16, 8, 256, 3840, 32, 64.0,
                          make_format(4, 4, k_group=64, v_group=64), 8192, 256, 2048,
                          1.0 / 3840, ("scale", 8, 30.0)),
    # Llama-3.1-8B-shaped layer, batch 4, context 32768, Hadamard K4V2 symmetric.
    "llama8b_had": Workload("llama8b_had", 5, 4, 32, 8, 128, 4096, 64, 128.0,
                            make_format(4, 2, k_mode=SYMMETRIC, v_mode=SYMMETRIC, k_group=128,
                                        v_group=32, rotate=128), 32768, 64, 2048,
                            1.0 / 4096, ("student_t", 3.0)),
}

WORKLOAD_ORDER = ["tiny_b1", "tiny_b16", "llama8b_kivi", "gqa12b_b8", "llama8b_had"]


# --------------------------------------------------------------- accounting

def adapter_params(d_in: int, d_outs, rank: int) -> int:
    """Parameters of explicit rank-r adapters on projections with output
    widths ``d_outs``: r (d_in + d_out) each (Sec. 3.4).  The same number is
    the extra multiply-accumulates per processed token."""
    return sum(rank * (d_in + d) for d in d_outs)


def projection_flops(M: int, d_in: int, d_q: int, d_kv: int, rank: int) -> int:
    """Algorithmic flops of the adapted Q/K/V projection for M tokens:
    2 M [d_in (d_q + 2 d_kv) + sum_p r (d_in + d_out,p)]."""
    macs = d_in * (d_q + 2 * d_kv) + adapter_params(d_in, (d_q, d_kv, d_kv), rank)
    return 2 * M * macs


def projection_weight_bytes(d_in: int, d_q: int, d_kv: int, rank: int) -> int:
    """bf16 bytes of W_qkv, A and B (the decode projection streams them once)."""
    N = d_q + 2 * d_kv
    return 2 * (N * d_in + 3 * rank * d_in + N * rank)


def coded_bytes_per_token(D: int, bits: int, axis: int, group: int, affine: bool, meta_fp16: int = 0) -> float:
    """Cache bytes of one coded token of one KV head: packed codes plus
    metadata (scale, and offset when affine; fp32, or fp16 with meta_fp16).
    Per-channel groups share one scale/offset per channel across ``group``
    tokens."""
    meta = (8 if affine else 4) // (2 if meta_fp16 else 1)
    if axis == PER_TOKEN:
        return D * bits / 8 + (D // group) * meta
    return D * bits / 8 + D * meta / group


def num_coded(fmt: dict, n: int) -> int:
    """Tokens held as codes when n are cached (the rest sit in the fp16 sink
    or the fp16 window)."""
    n = max(0, n - fmt.get("sink", 0))
    if fmt["flush"] == 0:
        return n
    over = n - fmt["residual"]
    return 0 if over <= 0 else over // fmt["flush"] * fmt["flush"]


def attention_bytes(wl: Workload, n: int) -> int:
    """Algorithmic HBM bytes of one decode-attention step over n cached tokens:
    coded tokens (codes + metadata), fp16 sink and window tokens (K and V),
    the bf16 queries and the fp32 outputs.  Split-K partials are not
    counted."""
    f = wl.fmt
    nq = num_coded(f, n)
    m16 = f.get("meta_fp16", 0)
    bk = coded_bytes_per_token(wl.D, f["k_bits"], f["k_axis"], f["k_group"], f["k_mode"] == AFFINE, m16)
    bv = coded_bytes_per_token(wl.D, f["v_bits"], f["v_axis"], f["v_group"], f["v_mode"] == AFFINE, m16)
    per_head = nq * (bk + bv) + (n - nq) * 4 * wl.D
    return int(round(wl.B * wl.H_kv * per_head)) + 2 * wl.B * wl.H_q * wl.D + 4 * wl.B * wl.H_q * wl.D
