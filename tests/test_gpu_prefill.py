"""GPU chunked prefill attention vs the oracle on identical caches.

Each case appends a prefix and then the chunk on both sides from the same
bf16 K/V (the GPU image is first checked byte-equal to the oracle's), then
compares the GPU's fp32 output for the chunk's queries with the oracle's
fp64 causal attention over the reconstruction: |gpu - ref| <= 2e-3 +
1e-2 |ref| elementwise.  Cases cover every cache format of the decode tests
(fp16 windows, per-channel keys, rotation, head sizes 64/128/256), chunks of
one token, chunks not aligned to the 32-token blocks, chunks that are the
whole cache, grouped-query sizes that leave ragged query tiles, a
workload-shaped chunk, and workspaces that hold only some of the (sequence,
KV head) units (the call then runs the units in groups; outputs must not
change by a bit).  Workspaces start filled with 0xFF bytes (fp16 NaN), so an
image byte the reconstruction failed to write shows up in the output.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_04263_amd import configs, synth

from gpu_util import assert_close, dev_bf16, image
from test_gpu_append import CASES

pytestmark = pytest.mark.gpu

# Rotating formats at the shapes the shared cases leave out: head size 64
# (four-wave attention workgroups) and 32-channel key groups at 128.
EXTRA = {
    "had_d64_g32": (configs.make_format(4, 4, k_group=32, v_group=32, rotate=64), 64),
    "had_d128_g32": (configs.make_format(4, 2, k_mode=1, v_mode=1, k_group=32, v_group=32, rotate=128), 128),
}


def run(name, B, H, G, n, C, seed, sm=None, ws_units=None):
    from paper_2609_04263_amd import kvq
    fmt, D = CASES[name] if name in CASES else EXTRA[name]
    outlier = ("student_t", 3.0) if fmt["rotate"] else ("scale", 4, 20.0)
    K, V = synth.kv_tokens(seed, B, n, H, D, outlier=outlier)
    T = n + 8
    ref = oracle.Cache(fmt, B, H, D, T)
    gc = kvq.Cache(fmt, B, H, D, T)
    for lo, hi in ((0, n - C), (n - C, n)):
        if hi > lo:
            ref.append(K[:, lo:hi], V[:, lo:hi])
            gc.append(dev_bf16(K[:, lo:hi]), dev_bf16(V[:, lo:hi]))
    assert np.array_equal(image(gc), ref.image), "cache images differ"
    H_q = H * G
    Q = synth.normal_bf16(seed, ("chunk-q",), (B, C, H_q, D))
    sm = 1.0 / np.sqrt(D) if sm is None else sm
    O = torch.full((B, C, H_q, D), float("nan"), dtype=torch.float32, device="cuda")
    full = gc.prefill_workspace_bytes()
    assert full % (B * H) == 0
    nbytes = full if ws_units is None else ws_units * (full // (B * H))
    ws = torch.full((nbytes,), 0xFF, dtype=torch.uint8, device="cuda")
    gc.prefill_attn(dev_bf16(Q), C, H_q, sm, O, ws)
    torch.cuda.synchronize()
    ref_o = ref.prefill_attn(Q, sm)
    assert_close(O.cpu().numpy(), ref_o, what=f"{name} n={n} C={C} G={G} ws_units={ws_units}")
    return O.cpu().numpy()


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("n,C", [(33, 1), (150, 40), (300, 128), (64, 64)])
def test_prefill_matches_oracle(name, n, C):
    run(name, B=2, H=2, G=4, n=n, C=C, seed=90 + n + C)


@pytest.mark.parametrize("G", [1, 3, 8, 16])
def test_prefill_group_sizes(G):
    run("tiny_b16", B=1, H=2, G=G, n=200, C=37, seed=100 + G)
    run("kivi", B=1, H=2, G=G, n=230, C=70, seed=110 + G)


def test_prefill_peaked_and_flat_softmax():
    run("tiny_b16", B=1, H=2, G=4, n=260, C=50, seed=120, sm=4.0)
    run("hadamard", B=1, H=2, G=4, n=260, C=50, seed=121, sm=1e-4)


def test_prefill_workload_shape_chunk():
    # a 256-token chunk at the end of 1280 tokens, D = 256, G = 2 (the 12B layer's shape)
    run("gqa12b", B=1, H=2, G=2, n=1280, C=256, seed=130)


@pytest.mark.parametrize("name", list(EXTRA))
@pytest.mark.parametrize("n,C", [(33, 1), (150, 40), (300, 128)])
def test_prefill_rotated_other_shapes(name, n, C):
    run(name, B=2, H=2, G=3, n=n, C=C, seed=160 + n + C)


def test_prefill_rotated_outputs_near_zero():
    # rotated K4V2 with 128 sinks: outputs near zero missed the bar while
    # each value entered the products as a single fp16 rounding (the inverse
    # rotation sums the rounding errors of all D channels into every output)
    run("kvarn_sink", B=2, H=2, G=2, n=505, C=406, seed=346969)


@pytest.mark.parametrize("name", ["tiny_b16", "kivi", "kvarn_sink"])
def test_prefill_workspace_groups(name):
    # B H = 6 units: one pass, groups of 4 + 2, and one unit at a time
    outs = [run(name, B=3, H=2, G=2, n=170, C=60, seed=140, ws_units=u) for u in (None, 4, 1)]
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


def test_prefill_workspace_too_small():
    from paper_2609_04263_amd import kvq
    fmt, D = CASES["tiny_b16"]
    B, H, n = 2, 2, 64
    K, V = synth.kv_tokens(150, B, n, H, D)
    gc = kvq.Cache(fmt, B, H, D, n)
    gc.append(dev_bf16(K), dev_bf16(V))
    Q = dev_bf16(synth.normal_bf16(151, ("chunk-q",), (B, 8, 2 * H, D)))
    O = torch.empty((B, 8, 2 * H, D), dtype=torch.float32, device="cuda")
    share = gc.prefill_workspace_bytes() // (B * H)
    with pytest.raises(kvq.KvqError) as e:
        gc.prefill_attn(Q, 8, 2 * H, 0.125, O, torch.empty(share - 16, dtype=torch.uint8, device="cuda"))
    assert e.value.status == kvq.ERR_WORKSPACE
