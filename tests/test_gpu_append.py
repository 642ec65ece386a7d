"""GPU append vs the oracle: the storage image must match byte for byte.

Both sides code the same bf16 K/V.  The GPU appends in ragged chunks
(1 token, partial 32-token blocks, a bulk chunk) while the oracle appends
everything at once, so byte equality also checks chunking invariance of the
kernels.  Formats cover every workload plus 2-bit affine, symmetric codes
with an fp16 window, per-channel keys with a 64-token window,
head_dim-wide groups, fp16 metadata, 8-bit codes and fp16 sink tokens.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_04263_amd import configs, synth

from gpu_util import dev_bf16, image

pytestmark = pytest.mark.gpu

CASES = {
    "tiny_b1": (configs.WORKLOADS["tiny_b1"].fmt, 64),
    "tiny_b16": (configs.WORKLOADS["tiny_b16"].fmt, 64),
    "kivi": (configs.WORKLOADS["llama8b_kivi"].fmt, 128),
    "gqa12b": (configs.WORKLOADS["gqa12b_b8"].fmt, 256),
    "hadamard": (configs.WORKLOADS["llama8b_had"].fmt, 128),
    "affine2_g128": (configs.make_format(2, 2, k_group=128, v_group=64), 128),
    "sym4_window": (configs.make_format(4, 4, k_mode=1, v_mode=1, k_group=32, v_group=64,
                                        residual=32, flush=32), 64),
    "perch_k4v2_window64": (configs.make_format(4, 2, k_axis=1, k_group=32, v_group=32,
                                                residual=64, flush=64), 64),
    "had_affine_window": (configs.make_format(4, 4, k_group=64, v_group=64, residual=32, flush=32,
                                              rotate=256), 256),
    "g256": (configs.make_format(4, 4, k_group=256, v_group=256), 256),
    # fp16 scales and offsets, as the paper stores them
    "tiny_meta16": (dict(configs.WORKLOADS["tiny_b16"].fmt, meta_fp16=1), 64),
    "kivi_meta16": (dict(configs.WORKLOADS["llama8b_kivi"].fmt, meta_fp16=1), 128),
    "hadamard_meta16": (dict(configs.WORKLOADS["llama8b_had"].fmt, meta_fp16=1), 128),
    # 8-bit codes (the 8-bit ablation): the tiny model's format, symmetric
    # codes with a window at D = 256, per-channel keys with fp16 metadata
    "affine8": (configs.make_format(8, 8, k_group=64, v_group=64), 64),
    "sym8_window_d256": (configs.make_format(8, 8, k_mode=1, v_mode=1, k_group=64, v_group=128,
                                             residual=32, flush=32), 256),
    "perch8_meta16": (configs.make_format(8, 8, k_axis=1, k_group=32, v_group=32, residual=32,
                                          flush=32, meta_fp16=1), 128),
    # fp16 sink tokens: KVarN's K4V2 g128 with 128 sinks, a sink before a
    # KIVI window, a 64-token sink at D = 64
    "kvarn_sink": (configs.make_format(4, 2, k_group=128, v_group=128, rotate=128, sink=128), 128),
    "sink32_window": (configs.make_format(2, 2, k_axis=1, k_group=32, v_group=32, residual=64,
                                          flush=32, sink=32), 128),
    "sink64": (configs.make_format(4, 4, k_group=64, v_group=64, sink=64), 64),
}


def run_case(name, B, H, n, cuts, seed):
    fmt, D = CASES[name]
    from paper_2609_04263_amd import kvq
    outlier = ("student_t", 3.0) if fmt["rotate"] else ("scale", 4, 20.0)
    K, V = synth.kv_tokens(seed, B, n, H, D, outlier=outlier)
    T = n + 5
    ref = oracle.Cache(fmt, B, H, D, T)
    ref.append(K, V)
    gc = kvq.Cache(fmt, B, H, D, T)
    Kd, Vd = dev_bf16(K), dev_bf16(V)
    for a, b in zip(cuts[:-1], cuts[1:]):
        gc.append(Kd[:, a:b].contiguous(), Vd[:, a:b].contiguous())
    assert gc.length() == (n, ref.n_coded)
    img = image(gc)
    assert img.size == ref.image.size
    for i in range(10):
        o, ln = ref.offsets[i], ref.lengths[i]
        a, b = img[o:o + ln], ref.image[o:o + ln]
        if not np.array_equal(a, b):
            diff = np.nonzero(a != b)[0]
            raise AssertionError(f"{name}: section {i} differs at {diff.size} bytes, first at {diff[0]}")
    assert np.array_equal(img, ref.image)


@pytest.mark.parametrize("name", list(CASES))
def test_append_ragged_chunks_match_oracle(name):
    n = 233
    run_case(name, B=2, H=3, n=n, cuts=[0, 1, 2, 31, 64, 100, 131, 200, n], seed=31)


@pytest.mark.parametrize("name", ["tiny_b16", "kivi", "hadamard", "kvarn_sink", "sink32_window"])
def test_append_token_by_token(name):
    n = 170
    run_case(name, B=1, H=2, n=n, cuts=list(range(n + 1)), seed=32)


@pytest.mark.parametrize("name", ["tiny_b1", "kivi", "gqa12b"])
def test_append_bulk_multi_block(name):
    n = 1000
    run_case(name, B=2, H=2, n=n, cuts=[0, n], seed=33)


@pytest.mark.parametrize("name", ["tiny_b16", "affine2_g128", "sym4_window", "kivi", "affine8",
                                  "tiny_meta16", "kvarn_sink"])
def test_append_exact_rounding_ties(name):
    """Half-integer inputs whose groups hold 0 and 15 (keys) or -7 and 7
    (values): scales of 1 at 4 bits, so many quotients are exact ties (round
    half to even) or fall next to one."""
    from paper_2609_04263_amd import kvq
    fmt, D = CASES[name]
    B, H, n = 2, 2, 150
    b, t, h, d = np.meshgrid(np.arange(B), np.arange(n), np.arange(H), np.arange(D), indexing="ij")
    idx = 7 * d + 3 * t + 5 * h + 11 * b
    K = synth.to_bf16_bits(((idx % 31) / 2.0).astype(np.float32))
    V = synth.to_bf16_bits(((idx % 29 - 14) / 2.0).astype(np.float32))
    ref = oracle.Cache(fmt, B, H, D, n)
    ref.append(K, V)
    gc = kvq.Cache(fmt, B, H, D, n)
    for lo, hi in ((0, 1), (1, 70), (70, n)):
        gc.append(dev_bf16(K[:, lo:hi]), dev_bf16(V[:, lo:hi]))
    assert np.array_equal(image(gc), ref.image)


def test_append_after_reset_rewrites_live_region():
    from paper_2609_04263_amd import kvq
    fmt, D = CASES["tiny_b16"]
    B, H, n = 1, 2, 77
    K1, V1 = synth.kv_tokens(34, B, n, H, D)
    K2, V2 = synth.kv_tokens(35, B, 50, H, D)
    gc = kvq.Cache(fmt, B, H, D, n)
    gc.append(dev_bf16(K1), dev_bf16(V1))
    gc.reset()
    gc.append(dev_bf16(K2), dev_bf16(V2))
    ref = oracle.Cache(fmt, B, H, D, n)
    ref.append(K2, V2)
    kh_ref, vh_ref = ref.dequant()
    # decode the GPU image with the oracle's reconstruction over the 50 live tokens
    probe = oracle.Cache(fmt, B, H, D, n)
    probe.image[:] = image(gc)
    probe.n = 50
    kh, vh = probe.dequant()
    assert np.array_equal(kh, kh_ref) and np.array_equal(vh, vh_ref)


def test_append_capacity_error_changes_nothing():
    from paper_2609_04263_amd import kvq
    fmt, D = CASES["tiny_b1"]
    K, V = synth.kv_tokens(36, 1, 40, 1, D)
    gc = kvq.Cache(fmt, 1, 1, D, 40)
    gc.append(dev_bf16(K[:, :30]), dev_bf16(V[:, :30]))
    before = image(gc).copy()
    with pytest.raises(kvq.KvqError) as e:
        gc.append(dev_bf16(K[:, :11]), dev_bf16(V[:, :11]))
    assert e.value.status == kvq.ERR_CAPACITY
    assert gc.n == 30 and np.array_equal(image(gc), before)
