"""GPU dense-merge deployment (W' = W + lora_scale * B_p A_p) vs the oracle.

The GPU accumulates the rank-r update in fp32 and rounds W' once to bf16;
the oracle does the same sum in fp64.  The bar: every element within half a
bf16 ulp of the fp64 value plus 2^-21 of |W| + |s| sum_k |B A| (the fp32
rounding of the update and of its sum with W, which cancellation can leave
large next to a small result), and at least 99.9% of the elements
bit-identical to the oracle's rounding (a difference is possible only next
to a rounding tie).  Shapes cover ragged
row and channel tiles (d_in not a multiple of the 128-channel tile, row
tiles straddling the Q/K/V boundaries), ranks that are and are not
multiples of 8 and of the 16-deep MFMA step, in-place merging, and two
workload shapes.  End to end, the rank-0 projection on the GPU's W' meets
the projection parity bar against the oracle's rank-0 projection on its
own merged bf16 weights, and differs from the explicit-adapter projection by
no more than the rounding of the merged weights to bf16 allows.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_04263_amd import configs, synth

from gpu_util import assert_close, dev_bf16, host_bits

pytestmark = pytest.mark.gpu


def f64(bits):
    return synth.bf16_bits_to_f32(bits).astype(np.float64)


def problem(seed, d_in, d_q, d_kv, r):
    g = np.random.default_rng(seed)
    N = d_q + 2 * d_kv
    W = synth.to_bf16_bits(g.standard_normal((N, d_in)) / np.sqrt(d_in))
    A = synth.to_bf16_bits(g.standard_normal((3 * r, d_in)) / np.sqrt(d_in))
    Bm = synth.to_bf16_bits(g.standard_normal((N, r)) * np.sqrt(0.02))
    return W, A, Bm


def gpu_merge(W, A, Bm, r, scale, d_q, d_kv, in_place=False):
    from paper_2609_04263_amd import kvq
    dW = dev_bf16(W)
    out = dW if in_place else torch.empty_like(dW)
    kvq.merge_adapter(dW, dev_bf16(A), dev_bf16(Bm), r, scale, d_q, d_kv, out)
    torch.cuda.synchronize()
    return host_bits(out)


def magnitude(W, A, Bm, r, scale, d_q, d_kv):
    """|W| + |scale| sum_k |B[n][k] A_p[k][i]|: the scale of the fp32 rounding error."""
    mag = np.abs(f64(W))
    Af, Bf = np.abs(f64(A)), np.abs(f64(Bm))
    rows = [(0, d_q), (d_q, d_q + d_kv), (d_q + d_kv, d_q + 2 * d_kv)]
    for p, (lo, hi) in enumerate(rows):
        mag[lo:hi] += abs(scale) * Bf[lo:hi] @ Af[p * r:(p + 1) * r]
    return mag


def check_merge(gpu_bits, Wd, Wb, mag, what):
    g = f64(gpu_bits)
    ulp_half = np.ldexp(1.0, np.frexp(np.abs(Wd))[1] - 9)  # half a bf16 ulp of |Wd|
    err = np.abs(g - Wd)
    # fp32 accumulation of the rank-r update and of the sum with W
    bound = ulp_half + mag * 2.0 ** -21 + 1e-30
    assert np.all(err <= bound), f"{what}: {int((err > bound).sum())} elements beyond half an ulp"
    same = np.mean(gpu_bits == Wb)
    assert same >= 0.999, f"{what}: only {same:.5f} bit-identical"


@pytest.mark.parametrize("r", [1, 8, 13, 16, 40, 64])
def test_merge_matches_oracle(r):
    d_in, d_q, d_kv = 320, 384, 96     # 2.5 channel tiles, 4.5 row tiles
    W, A, Bm = problem(r, d_in, d_q, d_kv, r)
    Wd, Wb = oracle.merge_adapter(W, A, Bm, r, 2.0, d_q, d_kv)
    mag = magnitude(W, A, Bm, r, 2.0, d_q, d_kv)
    check_merge(gpu_merge(W, A, Bm, r, 2.0, d_q, d_kv), Wd, Wb, mag, f"r={r}")


def test_merge_in_place_and_negative_scale():
    d_in, d_q, d_kv, r = 256, 128, 64, 16
    W, A, Bm = problem(7, d_in, d_q, d_kv, r)
    Wd, Wb = oracle.merge_adapter(W, A, Bm, r, -0.75, d_q, d_kv)
    got = gpu_merge(W, A, Bm, r, -0.75, d_q, d_kv, in_place=True)
    check_merge(got, Wd, Wb, magnitude(W, A, Bm, r, -0.75, d_q, d_kv), "in place")
    assert np.array_equal(got, gpu_merge(W, A, Bm, r, -0.75, d_q, d_kv))


def test_merged_projection_matches_explicit_adapter():
    from paper_2609_04263_amd import kvq
    d_in, d_q, d_kv, r, M = 256, 256, 64, 16, 24
    W, A, Bm = problem(3, d_in, d_q, d_kv, r)
    H = synth.to_bf16_bits(np.random.default_rng(4).standard_normal((M, d_in)))
    Wm = gpu_merge(W, A, Bm, r, 2.0, d_q, d_kv)
    Q = torch.empty((M, d_q), dtype=torch.bfloat16, device="cuda")
    K = torch.empty((M, d_kv), dtype=torch.bfloat16, device="cuda")
    V = torch.empty((M, d_kv), dtype=torch.bfloat16, device="cuda")
    kvq.project_qkv(dev_bf16(H), dev_bf16(Wm), None, None, 0, 0.0, d_q, d_kv, Q, K, V, None)
    torch.cuda.synchronize()
    y = synth.bf16_bits_to_f32(np.concatenate([host_bits(Q), host_bits(K), host_bits(V)], axis=1))
    # the same deployment on the oracle: its own bf16 merged weights, rank 0
    Wd, Wb = oracle.merge_adapter(W, A, Bm, r, 2.0, d_q, d_kv)
    ref, _ = oracle.project(H, Wb, None, None, 0, 0.0, d_q, d_kv)
    assert_close(y, ref, what="merged projection")
    # against the explicit adapter the difference is the rounding of the
    # merged weights to bf16: at most sum_i half an ulp of W'[n][i] times |h_i|
    exp, _ = oracle.project(H, W, A, Bm, r, 2.0, d_q, d_kv)
    half = np.ldexp(1.0, np.frexp(np.abs(Wd))[1] - 9)
    bound = np.abs(f64(H)) @ half.T
    yb_ulp = np.ldexp(1.0, np.frexp(np.abs(exp))[1] - 8)  # the bf16 output rounding (one ulp)
    assert np.all(np.abs(y - exp) <= bound + yb_ulp + 1e-6)


@pytest.mark.parametrize("name", ["tiny_b16", "llama8b_had"])
def test_merge_workload_shapes(name):
    wl = configs.WORKLOADS[name]
    W, A, Bm = problem(wl.seed, wl.d_in, wl.d_q, wl.d_kv, wl.rank)
    Wd, Wb = oracle.merge_adapter(W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv)
    mag = magnitude(W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv)
    check_merge(gpu_merge(W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv), Wd, Wb, mag, name)
