"""Pins of the oracle's chunked prefill attention (Sec. 3.1: evaluation runs chunk
by chunk; the chunk's states are appended, then its queries attend over the
reconstruction, causally).

* Agrees with torch's scaled_dot_product_attention (fp64, grouped-query mode,
  an explicit causal mask offset by the tokens before the chunk) run on the
  oracle's own reconstruction, for every format; for the rotated format with
  scipy's Hadamard matrix applied to q and to the output.
* A chunk of one token is the decode attention of that token.
* Causality: without an fp16 window a token's codes depend only on its own
  values, so query i's row equals the decode attention of a cache that holds
  only the tokens up to it, and changing later tokens leaves it unchanged.
"""
import numpy as np
import pytest
import scipy.linalg
import torch

import oracle
from paper_2609_04263_amd import synth
from test_oracle_cache import FMTS


def f32(bits):
    return synth.bf16_bits_to_f32(bits)


def chunk_queries(seed, B, C, H_q, D):
    return synth.normal_bf16(seed, ("chunk-q",), (B, C, H_q, D))


def build(name, B=2, H=2, G=4, n=150, C=40, seed=30):
    f = FMTS[name]
    D = 64 if f["k_axis"] == 0 else 128
    if f["rotate"]:
        D = f["rotate"]
    K, V = synth.kv_tokens(seed, B, n, H, D)
    c = oracle.Cache(f, B, H, D, n + 10)
    c.append(K[:, :n - C], V[:, :n - C])
    c.append(K[:, n - C:], V[:, n - C:])   # the chunk
    Q = chunk_queries(seed, B, C, H * G, D)
    return c, K, V, Q, D


def sdpa_causal(q, k, v, sm, n):
    """q [B, C, Hq, D], k/v [B, H, n, D] fp64 -> [B, C, Hq, D]; query i sees keys <= n - C + i."""
    C = q.shape[1]
    mask = np.arange(n)[None, :] <= (n - C + np.arange(C))[:, None]
    out = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q).transpose(1, 2), torch.from_numpy(k), torch.from_numpy(v),
        attn_mask=torch.from_numpy(mask), scale=sm, enable_gqa=True)
    return out.transpose(1, 2).numpy()


@pytest.mark.parametrize("name", list(FMTS))
def test_matches_library_attention_on_reconstruction(name):
    c, K, V, Q, D = build(name)
    sm = 1.0 / np.sqrt(D)
    O = c.prefill_attn(Q, sm)
    kh, vh = c.dequant()
    q = f32(Q).astype(np.float64)
    if c.fmt["rotate"]:
        R = scipy.linalg.hadamard(D) / np.sqrt(D)
        ref = sdpa_causal(q @ R.T, kh, vh, sm, c.n) @ R.T
    else:
        ref = sdpa_causal(q, kh, vh, sm, c.n)
    assert np.allclose(O, ref, rtol=1e-10, atol=1e-12)


@pytest.mark.parametrize("name", ["affine4_g64", "kivi_k2v2", "had_k4v2"])
def test_single_token_chunk_is_decode_attention(name):
    c, K, V, Q, D = build(name, C=1)
    sm = 0.3
    assert np.array_equal(c.prefill_attn(Q, sm)[:, 0], c.decode_attn(Q[:, 0], sm))


@pytest.mark.parametrize("name", ["affine4_g32", "affine2_g64", "had_k4v2"])
def test_row_equals_decode_attention_of_the_prefix(name):
    B, H, G, n, C = 1, 2, 2, 70, 9
    c, K, V, Q, D = build(name, B=B, H=H, G=G, n=n, C=C)
    sm = 0.2
    O = c.prefill_attn(Q, sm)
    for i in (0, 4, C - 1):
        upto = n - C + i + 1
        p = oracle.Cache(FMTS[name], B, H, D, n + 10)
        p.append(K[:, :upto], V[:, :upto])
        assert np.array_equal(O[:, i], p.decode_attn(Q[:, i], sm)), i
    # later tokens do not reach earlier queries
    K2, V2 = K.copy(), V.copy()
    K2[:, n - 3:] ^= np.uint16(0x0040)
    V2[:, n - 3:] ^= np.uint16(0x0040)
    c2 = oracle.Cache(FMTS[name], B, H, D, n + 10)
    c2.append(K2, V2)
    O2 = c2.prefill_attn(Q, sm)
    assert np.array_equal(O2[:, :C - 3], O[:, :C - 3])
    assert not np.array_equal(O2[:, C - 1], O[:, C - 1])
