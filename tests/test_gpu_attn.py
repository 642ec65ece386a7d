"""GPU decode attention vs the oracle on identical caches.

Each case builds the cache on both sides from the same bf16 K/V (the GPU
image is first checked byte-equal to the oracle's), then compares the GPU's
fp32 output with the oracle's fp64 attention over the reconstruction:
|gpu - ref| <= 2e-3 + 1e-2 |ref| elementwise.  Lengths cover one token,
ragged 32-token tails, several splits, KIVI caches that are all fp16 window
or mostly coded, and every grouped-query size up to 16.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_04263_amd import configs, synth

from gpu_util import assert_close, dev_bf16, image
from test_gpu_append import CASES

pytestmark = pytest.mark.gpu


def run(name, B, H, G, n, seed, sm=None, extra_appends=0):
    from paper_2609_04263_amd import kvq
    fmt, D = CASES[name]
    outlier = ("student_t", 3.0) if fmt["rotate"] else ("scale", 4, 20.0)
    K, V = synth.kv_tokens(seed, B, n, H, D, outlier=outlier)
    T = n + 8
    ref = oracle.Cache(fmt, B, H, D, T)
    ref.append(K, V)
    gc = kvq.Cache(fmt, B, H, D, T)
    gc.append(dev_bf16(K), dev_bf16(V))
    assert np.array_equal(image(gc), ref.image), "cache images differ"
    H_q = H * G
    Q = synth.queries(seed, B, H_q, D)
    sm = 1.0 / np.sqrt(D) if sm is None else sm
    O = torch.empty((B, H_q, D), dtype=torch.float32, device="cuda")
    ws = gc.decode_workspace(H_q)
    gc.decode_attn(dev_bf16(Q), H_q, sm, O, ws)
    torch.cuda.synchronize()
    ref_o = ref.decode_attn(Q, sm)
    return assert_close(O.cpu().numpy(), ref_o, what=f"{name} n={n} G={G}")


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("n", [1, 33, 257, 1500])
def test_attention_matches_oracle(name, n):
    run(name, B=2, H=2, G=4, n=n, seed=40 + n)


@pytest.mark.parametrize("G", [1, 2, 3, 8, 16])
def test_attention_group_sizes(G):
    run("tiny_b16", B=2, H=2, G=G, n=300, seed=50 + G)
    run("kivi", B=1, H=2, G=G, n=300, seed=60 + G)


@pytest.mark.parametrize("n", [100, 128, 159, 160, 161, 191, 192, 700])
def test_kivi_window_boundaries(n):
    run("kivi", B=2, H=2, G=4, n=n, seed=70 + n)


def test_split_boundaries_many_blocks():
    # enough tokens and few units so the planner uses many splits with a ragged last split
    run("tiny_b1", B=1, H=1, G=8, n=5000 + 17, seed=80)
    run("gqa12b", B=1, H=2, G=2, n=3001, seed=81)


def test_peaked_and_flat_softmax():
    run("tiny_b16", B=1, H=2, G=4, n=400, seed=82, sm=4.0)
    run("tiny_b16", B=1, H=2, G=4, n=400, seed=83, sm=1e-4)


def test_workspace_too_small_is_rejected():
    from paper_2609_04263_amd import kvq
    fmt, D = CASES["tiny_b1"]
    K, V = synth.kv_tokens(84, 1, 10, 1, D)
    gc = kvq.Cache(fmt, 1, 1, D, 10)
    gc.append(dev_bf16(K), dev_bf16(V))
    O = torch.empty((1, 8, D), dtype=torch.float32, device="cuda")
    ws = torch.empty(16, dtype=torch.uint8, device="cuda")
    Q = dev_bf16(synth.queries(84, 1, 8, D))
    with pytest.raises(kvq.KvqError) as e:
        gc.decode_attn(Q, 8, 0.125, O, ws)
    assert e.value.status == kvq.ERR_WORKSPACE
