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
def test_workload_shapes_decode_rows(name):
    wl = configs.WORKLOADS[name]
    W, A, Bm = synth.layer_weights(wl)
    H = synth.hidden(wl, ("test", "decode"), wl.B)
    y = run_gpu(H, W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv)
    ref, _ = oracle.project(H, W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv)
    assert_close(y, ref, what=f"{name} decode")


TILE_ROWS = 256  # row tile of the large-M kernel


@pytest.mark.parametrize("name", configs.WORKLOAD_ORDER)
def test_workload_prefill_chunk_every_tile(name):
    """The projection of one whole prefill chunk (M = B * chunk rows, the
    shape the benchmark runs), with the launch the benchmark uses.  One
    row at a random offset inside every 256-row tile is compared across all
    d_q + 2 d_kv columns, so every output tile of the XCD-ordered grid is
    checked (M = 16384 at gqa12b_b8: 64 row tiles x 32 column tiles)."""
    from paper_2609_04263_amd import kvq
    wl = configs.WORKLOADS[name]
    M = wl.B * min(wl.chunk, wl.context)
    W, A, Bm = synth.layer_weights(wl)
    Hd = synth.normal_bf16_device(wl.seed, ("test", "prefill-tiles"), (M, wl.d_in))
    Q = torch.empty((M, wl.d_q), dtype=torch.bfloat16, device="cuda")
    K = torch.empty((M, wl.d_kv), dtype=torch.bfloat16, device="cuda")
    V = torch.empty((M, wl.d_kv), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(max(1, kvq.project_workspace_bytes(M, wl.rank)), dtype=torch.uint8, device="cuda")
    kvq.project_qkv(Hd, dev_bf16(W), dev_bf16(A), dev_bf16(Bm), wl.rank, wl.lora_scale, wl.d_q, wl.d_kv,
                    Q, K, V, ws)
    torch.cuda.synchronize()
    g = np.random.default_rng(M)
    tiles = np.arange((M + TILE_ROWS - 1) // TILE_ROWS)
    rows = np.minimum(tiles * TILE_ROWS + g.integers(0, TILE_ROWS, size=tiles.size), M - 1)
    rows = np.union1d(rows, [0, M - 1])
    idx = torch.from_numpy(rows).to("cuda")
    H = host_bits(Hd[idx])
    y = synth.bf16_bits_to_f32(np.concatenate([host_bits(Q[idx]), host_bits(K[idx]), host_bits(V[idx])], axis=1))
    ref, _ = oracle.project(H, W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv)
    assert_close(y, ref, what=f"{name} prefill chunk M={M}, {rows.size} rows")
