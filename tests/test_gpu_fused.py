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
    from paper_2609_04263_amd import kvq
    fmt, D, rank = CASES[name]
    B, n_new, calls = 2, 128, 2
    d_in, d_kv = 256, 256
    H = d_kv // D
    d_q = 512
    N = d_q + 2 * d_kv
    seed = 140 + D + rank
    W = dev_bf16(synth.normal_bf16(seed, "W", (N, d_in), std=1.0 / 16))
    A = dev_bf16(synth.normal_bf16(seed, "A", (3 * max(rank, 1), d_in), std=1.0 / 16))
    Bm = dev_bf16(synth.normal_bf16(seed, "B", (N, max(rank, 1)), std=0.14))
    scale = 2.0
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
