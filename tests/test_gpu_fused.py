"""GPU projection fused with the append (kvq_project_append) vs the oracle.

The fused call must leave the cache exactly as the oracle's append of the
projection's bf16 K and V leaves it: the unfused GPU projection supplies
those bf16 K and V (a code may flip on a one-ulp projection difference, so
codes are compared on identical inputs), the oracle appends them, and the
fused call's image must equal the oracle's byte for byte.  Its Q must equal
the unfused projection's Q bit for bit (the same tiled product).  Cases:
head sizes 64/128/256, 2/4/8-bit codes, symmetric codes, fp16 metadata, an
adapter and none, two calls in a row (the second starting at position 128).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_04263_amd import configs, synth

from gpu_util import dev_bf16, image

pytestmark = pytest.mark.gpu

CASES = {
    "d64_affine4": (configs.make_format(4, 4, k_group=64, v_group=32), 64, 16),
    "d128_affine2": (configs.make_format(2, 2, k_group=128, v_group=64), 128, 8),
    "d256_sym4_meta16": (configs.make_format(4, 4, k_mode=1, v_mode=1, k_group=64, v_group=256, meta_fp16=1),
                         256, 32),
    "d64_affine8_rank0": (configs.make_format(8, 8, k_group=32, v_group=64), 64, 0),
}


@pytest.mark.parametrize("name", list(CASES))
def test_fused_projection_append_matches_oracle(name):
    fmt, D, rank = CASES[name]
    check_fused(name, fmt, D, H=256 // D, rank=rank, B=2, n_new=128, calls=2, d_in=256, d_q=512,
                seed=140 + D + rank)


# Shapes with several K and V column tiles per projection (so the KV-head
# offset of a tile is not 0), row counts that are not a multiple of the
# 256-row tile (slices past M skipped, sequences crossing row tiles), and
# more than one row tile under the XCD-grouped tile order.
SHAPES = {
    "d128_h4_B3_n96": (configs.make_format(4, 4, k_group=64, v_group=64), 128, 4, 16, 3, 96, 512, 256),
    "d256_h4_B5_n160": (configs.make_format(2, 2, k_group=128, v_group=64), 256, 4, 8, 5, 160, 1024, 512),
    "d128_h8_B4_n224_sym": (configs.make_format(4, 2, k_mode=1, v_mode=1, k_group=128, v_group=32), 128, 8, 32,
                            4, 224, 1024, 384),
    "d64_h16_B6_n64_meta16": (configs.make_format(4, 4, k_group=32, v_group=64, meta_fp16=1), 64, 16, 0, 6, 64,
                              768, 128),
}


@pytest.mark.parametrize("name", list(SHAPES))
def test_fused_multi_tile_and_ragged_rows(name):
    fmt, D, H, rank, B, n_new, d_q, d_in = SHAPES[name]
    check_fused(name, fmt, D, H=H, rank=rank, B=B, n_new=n_new, calls=2, d_in=d_in, d_q=d_q, seed=170 + B)


def test_fused_benchmark_shape():
    """gqa12b_b8's prefill chunk as the benchmark runs it: M = 8 x 2048 rows,
    d_in 3840, d_q 4096, d_kv 2048 (eight KV heads of 256), rank 32."""
    wl = configs.WORKLOADS["gqa12b_b8"]
    check_fused("gqa12b_b8", wl.fmt, wl.D, H=wl.H_kv, rank=wl.rank, B=wl.B, n_new=wl.chunk, calls=1,
                d_in=wl.d_in, d_q=wl.d_q, seed=wl.seed, lora_scale=wl.lora_scale)


def check_fused(name, fmt, D, H, rank, B, n_new, calls, d_in, d_q, seed, lora_scale=2.0):
    from paper_2609_04263_amd import kvq
    d_kv = H * D
    N = d_q + 2 * d_kv
    W = dev_bf16(synth.normal_bf16(seed, "W", (N, d_in), std=1.0 / np.sqrt(d_in)))
    A = dev_bf16(synth.normal_bf16(seed, "A", (3 * max(rank, 1), d_in), std=1.0 / np.sqrt(d_in)))
    Bm = dev_bf16(synth.normal_bf16(seed, "B", (N, max(rank, 1)), std=0.14))
    scale = lora_scale
    T = n_new * calls
    ref = oracle.Cache(fmt, B, H, D, T)
    gc = kvq.Cache(fmt, B, H, D, T)
    M = B * n_new
    ws = torch.empty(max(16, kvq.project_workspace_bytes(M, rank)), dtype=torch.uint8, device="cuda")
    for call in range(calls):
        Hm = dev_bf16(synth.normal_bf16(seed, ("H", call), (M, d_in)))
        Qr = torch.empty((M, d_q), dtype=torch.bfloat16, device="cuda")
        Kr = torch.empty((M, d_kv), dtype=torch.bfloat16, device="cuda")
        Vr = torch.empty((M, d_kv), dtype=torch.bfloat16, device="cuda")
        kvq.project_qkv(Hm, W, A, Bm, rank, scale, d_q, d_kv, Qr, Kr, Vr, ws)
        Q = torch.full((M, d_q), float("nan"), dtype=torch.bfloat16, device="cuda")
        kvq.project_append(Hm, W, A, Bm, rank, scale, d_q, d_kv, Q, gc, n_new, ws)
        torch.cuda.synchronize()
        bits = lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)
        ref.append(bits(Kr).reshape(B, n_new, H, D), bits(Vr).reshape(B, n_new, H, D))
        assert np.array_equal(bits(Q), bits(Qr)), f"{name}: Q differs (call {call})"
        assert gc.length() == (ref.n, ref.n_coded)
        img = image(gc)
        for i in range(10):
            o, ln = ref.offsets[i], ref.lengths[i]
            a, b = img[o:o + ln], ref.image[o:o + ln]
            if not np.array_equal(a, b):
                diff = np.nonzero(a != b)[0]
                raise AssertionError(f"{name} call {call}: section {i} differs at {diff.size} bytes, "
                                     f"first at {diff[0]}")


# Decode steps of window formats (one new token per sequence, M = B <= 32):
# the projection writes K and V straight into the fp16 window and a due
# flush is coded from the window.  (format, D, H, rank, B, prefill tokens,
# decode steps): the steps cross at least two flushes.
WINDOW = {
    "kivi_d128_b4": (configs.make_format(2, 2, k_axis=configs.PER_CHANNEL, k_group=32, v_group=32,
                                         residual=32, flush=32), 128, 2, 16, 4, 40, 70),
    "kivi_d64_b32_r8": (configs.make_format(2, 2, k_axis=configs.PER_CHANNEL, k_group=32, v_group=32,
                                            residual=64, flush=32), 64, 4, 8, 32, 90, 70),
    "token_window_d256_b1_r32": (configs.make_format(4, 4, k_group=64, v_group=64, residual=32, flush=32), 256, 1,
                                 32, 1, 0, 100),
    "kivi_meta16_sym_d128_b3_rank0": (configs.make_format(4, 2, k_mode=1, v_mode=1, k_axis=configs.PER_CHANNEL,
                                                          k_group=32, v_group=32, residual=64, flush=32,
                                                          meta_fp16=1), 128, 2, 0, 3, 33, 100),
    "window8_d64_b5_r64": (configs.make_format(8, 8, k_group=32, v_group=64, residual=32, flush=32), 64, 2, 64,
                           5, 7, 95),
}


@pytest.mark.parametrize("name", list(WINDOW))
def test_fused_decode_window_steps(name):
    from paper_2609_04263_amd import kvq
    fmt, D, H, rank, B, n_pre, steps = WINDOW[name]
    seed = 300 + D + B
    d_in, d_q = 256, 256
    d_kv = H * D
    N = d_q + 2 * d_kv
    W = dev_bf16(synth.normal_bf16(seed, "W", (N, d_in), std=1.0 / np.sqrt(d_in)))
    A = dev_bf16(synth.normal_bf16(seed, "A", (3 * max(rank, 1), d_in), std=1.0 / np.sqrt(d_in)))
    Bm = dev_bf16(synth.normal_bf16(seed, "B", (N, max(rank, 1)), std=0.14))
    T = n_pre + steps
    ref = oracle.Cache(fmt, B, H, D, T)
    gc = kvq.Cache(fmt, B, H, D, T)
    bits = lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)
    if n_pre:
        M = B * n_pre
        ws = torch.empty(max(16, kvq.project_workspace_bytes(M, rank)), dtype=torch.uint8, device="cuda")
        Hm = dev_bf16(synth.normal_bf16(seed, "Hpre", (M, d_in)))
        Qp = torch.empty((M, d_q), dtype=torch.bfloat16, device="cuda")
        Kp = torch.empty((M, d_kv), dtype=torch.bfloat16, device="cuda")
        Vp = torch.empty((M, d_kv), dtype=torch.bfloat16, device="cuda")
        kvq.project_qkv(Hm, W, A, Bm, rank, 2.0, d_q, d_kv, Qp, Kp, Vp, ws)
        gc.append(Kp.view(B, n_pre, H, D), Vp.view(B, n_pre, H, D))
        torch.cuda.synchronize()
        ref.append(bits(Kp).reshape(B, n_pre, H, D), bits(Vp).reshape(B, n_pre, H, D))
    ws = torch.empty(max(16, kvq.project_workspace_bytes(B, rank)), dtype=torch.uint8, device="cuda")
    Hd = dev_bf16(synth.normal_bf16(seed, "Hdec", (steps, B, d_in)))
    flushes = 0
    for i in range(steps):
        Qr = torch.empty((B, d_q), dtype=torch.bfloat16, device="cuda")
        Kr = torch.empty((B, d_kv), dtype=torch.bfloat16, device="cuda")
        Vr = torch.empty((B, d_kv), dtype=torch.bfloat16, device="cuda")
        kvq.project_qkv(Hd[i], W, A, Bm, rank, 2.0, d_q, d_kv, Qr, Kr, Vr, ws)
        Q = torch.full((B, d_q), float("nan"), dtype=torch.bfloat16, device="cuda")
        coded_before = gc.length()[1]
        kvq.project_append(Hd[i], W, A, Bm, rank, 2.0, d_q, d_kv, Q, gc, 1, ws)
        torch.cuda.synchronize()
        ref.append(bits(Kr).reshape(B, 1, H, D), bits(Vr).reshape(B, 1, H, D))
        assert np.array_equal(bits(Q), bits(Qr)), f"{name}: Q differs at step {i}"
        assert gc.length() == (ref.n, ref.n_coded), f"{name}: lengths at step {i}"
        flushes += gc.length()[1] > coded_before
        if i % 7 == 6 or i == steps - 1 or gc.length()[1] > coded_before:
            img = image(gc)
            for s in range(10):
                o, ln = ref.offsets[s], ref.lengths[s]
                a, b = img[o:o + ln], ref.image[o:o + ln]
                if not np.array_equal(a, b):
                    diff = np.nonzero(a != b)[0]
                    raise AssertionError(f"{name} step {i}: section {s} differs at {diff.size} bytes, first at {diff[0]}")
    assert flushes >= 2, f"{name}: the steps crossed {flushes} flushes"


def test_fused_decode_window_unsupported_formats():
    from paper_2609_04263_amd import kvq
    B, H, D, rank, d_in, d_q = 2, 2, 64, 8, 256, 128
    d_kv = H * D
    N = d_q + 2 * d_kv
    W = torch.zeros((N, d_in), dtype=torch.bfloat16, device="cuda")
    A = torch.zeros((3 * rank, d_in), dtype=torch.bfloat16, device="cuda")
    Bm = torch.zeros((N, rank), dtype=torch.bfloat16, device="cuda")
    Hm = torch.zeros((B, d_in), dtype=torch.bfloat16, device="cuda")
    Q = torch.empty((B, d_q), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(kvq.project_workspace_bytes(B, rank), dtype=torch.uint8, device="cuda")
    for fmt in (configs.make_format(4, 4, k_mode=1, v_mode=1, k_group=64, v_group=64, residual=32, flush=32,
                                    rotate=64),
                configs.make_format(4, 4, k_group=64, v_group=64, residual=32, flush=32, sink=32)):
        gc = kvq.Cache(fmt, B, H, D, 64)
        with pytest.raises(kvq.KvqError) as e:
            kvq.project_append(Hm, W, A, Bm, rank, 2.0, d_q, d_kv, Q, gc, 1, ws)
        assert e.value.status == kvq.ERR_FORMAT
        assert gc.length() == (0, 0)
