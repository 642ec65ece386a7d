"""GPU adapted Q/K/V projection vs the oracle (fp64, explicit adapter).

Covers the skinny decode kernel (M <= 32, including M = 1 and a ragged 17),
the tiled kernel (M > 32 with ragged row tiles), ranks 0..64, output widths
that are not multiples of the 128-column tile (so tiles straddle Q/K/V),
and the workload shapes on sampled rows.  Outputs are bf16; the bound is
|gpu - ref| <= 2e-3 + 1e-2 |ref| against the unrounded fp64 reference.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_04263_amd import configs, synth

from gpu_util import assert_close, dev_bf16, host_bits

pytestmark = pytest.mark.gpu


def problem(seed, M, d_in, d_q, d_kv, r, outlier=True):
    g = np.random.default_rng(seed)
    N = d_q + 2 * d_kv
    H = synth.to_bf16_bits(g.standard_normal((M, d_in)))
    Wf = g.standard_normal((N, d_in)) / np.sqrt(d_in)
    Bf = g.standard_normal((N, max(r, 1))) * np.sqrt(0.02)
    if outlier:   # a few key rows x20 as in the workloads
        rows = d_q + g.choice(d_kv, size=max(1, d_kv // 32), replace=False)
        Wf[rows] *= 20
        Bf[rows] *= 20
    W = synth.to_bf16_bits(Wf)
    A = synth.to_bf16_bits(g.standard_normal((3 * max(r, 1), d_in)) / np.sqrt(d_in))[:3 * r]
    Bm = synth.to_bf16_bits(Bf)[:, :r]
    return H, W, np.ascontiguousarray(A), np.ascontiguousarray(Bm)


def run_gpu(H, W, A, Bm, r, scale, d_q, d_kv):
    from paper_2609_04263_amd import kvq
    M = H.shape[0]
    Q = torch.empty((M, d_q), dtype=torch.bfloat16, device="cuda")
    K = torch.empty((M, d_kv), dtype=torch.bfloat16, device="cuda")
    V = torch.empty((M, d_kv), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(max(1, kvq.project_workspace_bytes(M, r)), dtype=torch.uint8, device="cuda")
    dA = dev_bf16(A) if r else None
    dB = dev_bf16(Bm) if r else None
    kvq.project_qkv(dev_bf16(H), dev_bf16(W), dA, dB, r, scale, d_q, d_kv, Q, K, V, ws)
    torch.cuda.synchronize()
    out = np.concatenate([host_bits(Q), host_bits(K), host_bits(V)], axis=1)
    return synth.bf16_bits_to_f32(out)


@pytest.mark.parametrize("M", [1, 5, 16, 17, 32, 33, 100, 300])
@pytest.mark.parametrize("r", [0, 8, 16, 64])
def test_projection_matches_oracle(M, r):
    d_in, d_q, d_kv = 256, 384, 80
    H, W, A, Bm = problem(M * 100 + r, M, d_in, d_q, d_kv, r)
    y = run_gpu(H, W, A, Bm, r, 2.0, d_q, d_kv)
    ref, _ = oracle.project(H, W, A if r else None, Bm if r else None, r, 2.0, d_q, d_kv)
    assert_close(y, ref, what=f"M={M} r={r}")


def test_projection_odd_scale_and_rank():
    d_in, d_q, d_kv, r = 128, 64, 16, 12
    for M in (3, 70):
        H, W, A, Bm = problem(7 + M, M, d_in, d_q, d_kv, r)
        y = run_gpu(H, W, A, Bm, r, 0.37, d_q, d_kv)
        ref, _ = oracle.project(H, W, A, Bm, r, 0.37, d_q, d_kv)
        assert_close(y, ref, what=f"M={M}")


@pytest.mark.parametrize("name", configs.WORKLOAD_ORDER)
@pytest.mark.parametrize("mode", ["decode", "prefill"])
def test_workload_shapes_sampled_rows(name, mode):
    wl = configs.WORKLOADS[name]
    W, A, Bm = synth.layer_weights(wl)
    M = wl.B if mode == "decode" else min(wl.B * wl.chunk, 4096)
    H = synth.hidden(wl, ("test", mode), M)
    y = run_gpu(H, W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv)
    rows = np.unique(np.random.default_rng(1).choice(M, size=min(M, 6), replace=False))
    rows = np.union1d(rows, [0, M - 1])
    ref, _ = oracle.project(H[rows], W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv)
    assert_close(y[rows], ref, what=f"{name} {mode}")
