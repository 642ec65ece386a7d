"""Pins of the oracle's decode attention over the reconstruction (Sec. 3.1-3.2).

* Agrees with torch's scaled_dot_product_attention (a library routine, fp64,
  grouped-query mode) run on the oracle's own reconstruction, for every
  format; for the rotated format, with the rotation applied by scipy's
  Hadamard matrix.
* Special cases: one token returns its value; identical keys or a zero query
  give the plain mean of the values; a huge softmax scale picks the value of
  the highest-scoring key.
* KIVI with at most 128 tokens is exact attention over fp16-rounded K/V.
"""
import numpy as np
import pytest
import scipy.linalg
import torch

import oracle
from paper_2609_04263_amd import configs, synth
from test_oracle_cache import FMTS


def f32(bits):
    return synth.bf16_bits_to_f32(bits)


def sdpa(q, k, v, sm):
    """q [B, Hq, D], k/v [B, H, n, D] fp64 -> [B, Hq, D] via torch (GQA mode)."""
    out = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[:, :, None, :], torch.from_numpy(k), torch.from_numpy(v),
        scale=sm, enable_gqa=True)
    return out[:, :, 0, :].numpy()


def build(name, B=2, H=2, G=4, n=150, seed=20):
    f = FMTS[name]
    D = 64 if f["k_axis"] == 0 else 128
    if f["rotate"]:
        D = f["rotate"]
    K, V = synth.kv_tokens(seed, B, n, H, D)
    c = oracle.Cache(f, B, H, D, n + 10)
    c.append(K, V)
    Q = synth.queries(seed, B, H * G, D)
    return c, K, V, Q, D


@pytest.mark.parametrize("name", list(FMTS))
def test_matches_library_attention_on_reconstruction(name):
    c, K, V, Q, D = build(name)
    sm = 1.0 / np.sqrt(D)
    O = c.decode_attn(Q, sm)
    kh, vh = c.dequant()
    q = f32(Q).astype(np.float64)
    if c.fmt["rotate"]:
        R = scipy.linalg.hadamard(D) / np.sqrt(D)
        ref = sdpa(q @ R.T, kh, vh, sm) @ R.T
    else:
        ref = sdpa(q, kh, vh, sm)
    assert np.allclose(O, ref, rtol=1e-10, atol=1e-12)


def test_single_token_returns_its_value():
    f = FMTS["affine4_g64"]
    K, V = synth.kv_tokens(21, 1, 1, 2, 64)
    c = oracle.Cache(f, 1, 2, 64, 4)
    c.append(K, V)
    _, vh = c.dequant()
    O = c.decode_attn(synth.queries(21, 1, 8, 64), 0.125)
    for hq in range(8):
        assert np.allclose(O[0, hq], vh[0, hq // 4, 0], rtol=0, atol=1e-15)


def test_equal_keys_and_zero_query_give_mean_value():
    f = FMTS["affine4_g32"]
    B, H, D, n = 1, 1, 64, 50
    K, V = synth.kv_tokens(22, B, n, H, D)
    K = np.repeat(K[:, :1], n, axis=1)          # every key identical
    c = oracle.Cache(f, B, H, D, n)
    c.append(K, V)
    _, vh = c.dequant()
    O = c.decode_attn(synth.queries(22, B, 4, D), 0.125)
    assert np.allclose(O[0], vh[0, 0].mean(0)[None], rtol=1e-12, atol=1e-12)
    c2 = oracle.Cache(f, B, H, D, n)
    K2, V2 = synth.kv_tokens(23, B, n, H, D)
    c2.append(K2, V2)
    _, vh2 = c2.dequant()
    Qz = np.zeros((B, 4, D), dtype=np.uint16)    # bf16 +0.0
    O2 = c2.decode_attn(Qz, 0.125)
    assert np.allclose(O2[0], vh2[0, 0].mean(0)[None], rtol=1e-12, atol=1e-12)


def test_huge_scale_selects_best_key():
    c, K, V, Q, D = build("affine4_g64", B=1, H=1, G=2, n=60, seed=24)
    kh, vh = c.dequant()
    O = c.decode_attn(Q, 1e6)
    for hq in range(2):
        scores = kh[0, 0] @ f32(Q[0, hq]).astype(np.float64)
        best = np.argmax(scores)
        assert np.allclose(O[0, hq], vh[0, 0, best], atol=1e-9)


def test_kivi_short_context_is_exact_fp16_attention():
    f = configs.WORKLOADS["llama8b_kivi"].fmt
    B, H, D, n, G = 1, 2, 128, 100, 4
    K, V = synth.kv_tokens(25, B, n, H, D)
    c = oracle.Cache(f, B, H, D, 200)
    c.append(K, V)
    Q = synth.queries(25, B, H * G, D)
    O = c.decode_attn(Q, 1 / np.sqrt(D))
    k16 = oracle.f16_to_f32(oracle.f32_to_f16(f32(K))).astype(np.float64).transpose(0, 2, 1, 3)
    v16 = oracle.f16_to_f32(oracle.f32_to_f16(f32(V))).astype(np.float64).transpose(0, 2, 1, 3)
    ref = sdpa(f32(Q).astype(np.float64), np.ascontiguousarray(k16), np.ascontiguousarray(v16),
               1 / np.sqrt(D))
    assert np.allclose(O, ref, rtol=1e-10, atol=1e-12)


def test_empty_cache_is_an_error():
    c = oracle.Cache(FMTS["affine4_g64"], 1, 1, 64, 8)
    with pytest.raises(oracle.OracleError):
        c.decode_attn(np.zeros((1, 1, 64), dtype=np.uint16), 0.125)
