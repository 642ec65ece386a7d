"""Pins of the oracle's dense-merge deployment (Sec. 3.4 "Deployment overhead":
the dense-base update folds into the weights, W <- W + (alpha/r) B A, leaving
the projection shapes unchanged).

* merge identity: projecting with the merged fp64 weights equals the oracle's
  explicit-adapter projection (itself pinned against numpy) to 1e-12;
* a closed form: with unit-vector rows of A, the update adds scale * B[n][k]
  to exactly one input column per adapter row;
* rank 0 returns W unchanged; the bf16 result is the fp64 one rounded once
  to nearest (ties to even).
"""
import numpy as np
import pytest

import oracle
from paper_2609_04263_amd import synth


def f64(bits):
    return synth.bf16_bits_to_f32(bits).astype(np.float64)


def problem(seed, d_in=128, d_q=256, d_kv=64, r=4, M=6):
    g = np.random.default_rng(seed)
    H = synth.to_bf16_bits(g.standard_normal((M, d_in)))
    W = synth.to_bf16_bits(g.standard_normal((d_q + 2 * d_kv, d_in)) / np.sqrt(d_in))
    A = synth.to_bf16_bits(g.standard_normal((3 * r, d_in)) / np.sqrt(d_in))
    Bm = synth.to_bf16_bits(g.standard_normal((d_q + 2 * d_kv, r)) * 0.14)
    return H, W, A, Bm


@pytest.mark.parametrize("r,scale", [(4, 2.0), (16, 0.37), (1, -1.5)])
def test_merged_weights_reproduce_the_explicit_branch(r, scale):
    d_q, d_kv = 256, 64
    H, W, A, Bm = problem(r, r=r)
    Wd, _ = oracle.merge_adapter(W, A, Bm, r, scale, d_q, d_kv)
    Y, _ = oracle.project(H, W, A, Bm, r, scale, d_q, d_kv)
    assert np.allclose(f64(H) @ Wd.T, Y, rtol=1e-12, atol=1e-12)


def test_unit_vector_adapter_rows_touch_one_column_each():
    d_in, d_q, d_kv, r, scale = 64, 32, 16, 3, 0.5
    _, W, _, Bm = problem(5, d_in=d_in, d_q=d_q, d_kv=d_kv, r=r)
    cols = [[3, 17, 40], [0, 63, 17], [5, 6, 7]]  # per projection, per adapter row
    A = np.zeros((3 * r, d_in), dtype=np.uint16)
    one = synth.to_bf16_bits(np.ones(1))[0]
    for p in range(3):
        for k in range(r):
            A[p * r + k, cols[p][k]] = one
    Wd, _ = oracle.merge_adapter(W, A, Bm, r, scale, d_q, d_kv)
    expect = f64(W)
    Bf = f64(Bm)
    rows = [(0, d_q), (d_q, d_q + d_kv), (d_q + d_kv, d_q + 2 * d_kv)]
    for p, (lo, hi) in enumerate(rows):
        for k in range(r):
            expect[lo:hi, cols[p][k]] += scale * Bf[lo:hi, k]
    assert np.array_equal(Wd, expect)


def test_rank_zero_and_rounding():
    d_q, d_kv = 256, 64
    _, W, A, Bm = problem(11)
    Wd0, Wb0 = oracle.merge_adapter(W, None, None, 0, 2.0, d_q, d_kv)
    assert np.array_equal(Wb0, W) and np.array_equal(Wd0, f64(W))
    Wd, Wb = oracle.merge_adapter(W, A, Bm, 4, 2.0, d_q, d_kv)
    # nearest bf16: neither neighbouring bit pattern is closer
    d0 = np.abs(f64(Wb) - Wd)
    for step in (1, -1):
        nb = (Wb.astype(np.int64) + step).astype(np.uint16)
        assert np.all(d0 <= np.abs(f64(nb) - Wd))
