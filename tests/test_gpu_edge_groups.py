"""Eq. (3)'s edge cases on the GPU: groups the closed form treats specially.

Inputs are built so that every coding group (per-token groups along
head_dim and KIVI's per-channel groups of 32 tokens alike) is one of:
constant (any value, including large ones), all +0, a mix of -0 and +0,
a -0 minimum under positive values, a single one-ulp step, or a range (or
maximum magnitude, for symmetric codes) just below, at and just above the
point where the scale meets its floor (1e-8, and fp16's smallest subnormal
2^-24 when the metadata is fp16); ordinary normal groups are mixed in.  The
kind is fixed per (sequence, KV head, 32-token block), and the designated
extremes sit where (token + channel) % 32 is 0 or 1, so every per-token
group of 32 or more channels and every per-channel group of 32 tokens holds
both.  The GPU appends in ragged chunks; its storage image must equal the
oracle's byte for byte (codes, scales, offsets, the +0 canonical offset,
the fp16 window), then decode attention and chunked prefill attention over
that cache must match the oracle's fp64 attention at the float bar.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_04263_amd import configs, synth

from gpu_util import assert_close, dev_bf16, image

F32 = np.float32
FLOOR = F32(1e-8)
F16_TINY = F32(2.0 ** -24)


def bf16_near(x, span=12):
    """bf16-representable float32 values around x, ascending."""
    b = int(synth.to_bf16_bits(np.array([x], dtype=F32))[0])
    pats = np.arange(b - span, b + span + 1, dtype=np.int64)
    pats = pats[(pats >= 0) & (pats < 0x7F80)] if x >= 0 else pats
    vals = synth.bf16_bits_to_f32(pats.astype(np.uint16))
    return np.unique(vals[np.isfinite(vals)])


def threshold_pairs(mode, bits, thr):
    """(lo, hi) group extremes whose fp32 scale lands just below, at (when
    representable) and just above thr: affine groups [lo, hi] with
    s = (hi - lo) / (2^b - 1); symmetric groups with max |x| = hi, lo = -hi
    scaled by 1/3 so the sign of the extreme differs between rows."""
    out = []
    if mode == configs.AFFINE:
        qd = F32(2 ** bits - 1)
        lo = -synth.bf16_bits_to_f32(synth.to_bf16_bits(np.array([thr * qd / 2], dtype=F32)))[0]
        cands = bf16_near(thr * qd + lo)
        s = (cands - lo).astype(F32) / qd
        below, above = cands[s < thr], cands[s > thr]
        out += [(lo, below.max()), (lo, above.min())]
        at = cands[s == thr]
        if at.size:
            out.append((lo, at[0]))
    else:
        qm = F32(2 ** (bits - 1) - 1)
        cands = bf16_near(thr * qm)
        s = cands / qm
        below, above = cands[s < thr], cands[s > thr]
        out += [(-below.max() / 3, below.max()), (-above.min() / 3, above.min())]
        at = cands[s == thr]
        if at.size:
            out.append((-at[0] / 3, at[0]))
    return [(F32(a), F32(b)) for a, b in out]


def edge_tokens(seed, B, n, H, D, mode, bits, meta16, key):
    """K or V [B, n, H, D] as bf16 bits, one group kind per (b, h, block).
    The large constant is a large magnitude for values only: a constant key
    block of that size would dominate (or vanish from) every softmax.  It is
    -4352, so that the 128-point rotation of a constant row (a spike of
    sqrt(128) times the constant, 49233) stays inside binary16's range, which
    prefill attention's reconstructed operands require."""
    g = np.random.default_rng(seed)
    pairs = threshold_pairs(mode, bits, FLOOR)
    if meta16:
        pairs += threshold_pairs(mode, bits, F16_TINY)
    kinds = ["normal", "const", "zero", "signed_zero", "neg_zero_min", "one_ulp", "big_const"] + \
        [("pair", p) for p in pairs]
    X = np.zeros((B, n, H, D), dtype=F32)
    i_tok = np.arange(32)[:, None]
    d_ch = np.arange(D)[None, :]
    pos = (i_tok + d_ch) % 32
    k = 0
    for b in range(B):
        for h in range(H):
            for t0 in range(0, n, 32):
                m = min(32, n - t0)
                kind = kinds[k % len(kinds)]
                k += 1
                if kind == "normal":
                    tile = g.standard_normal((32, D)).astype(F32)
                elif kind == "const":
                    tile = np.full((32, D), F32(g.standard_normal() * 3), dtype=F32)
                elif kind == "big_const":
                    tile = np.full((32, D), F32(4.0 if key else -2.0 ** 12 - 2.0 ** 8), dtype=F32)
                elif kind == "zero":
                    tile = np.zeros((32, D), dtype=F32)
                elif kind == "signed_zero":
                    tile = np.where(g.random((32, D)) < 0.5, F32(-0.0), F32(0.0)).astype(F32)
                    tile[pos == 1] = F32(-0.0)
                elif kind == "neg_zero_min":
                    tile = g.random((32, D)).astype(F32) + F32(0.01)
                    tile[pos == 1] = F32(-0.0)
                elif kind == "one_ulp":
                    base = F32(0.75)
                    tile = np.full((32, D), base, dtype=F32)
                    tile[pos == 0] = F32(0.75 + 2.0 ** -8)  # bf16 ulp at 0.75
                else:
                    lo, hi = kind[1]
                    u = g.random((32, D)).astype(F32)
                    tile = lo + (hi - lo) * u
                    tile = synth.bf16_bits_to_f32(synth.to_bf16_bits(tile))
                    tile = np.clip(tile, lo, hi)
                    tile[pos == 0] = hi
                    tile[pos == 1] = lo
                X[b, t0:t0 + m, h, :] = tile[:m]
    return synth.to_bf16_bits(X)


FORMATS = {
    "affine4_g32": (configs.make_format(4, 4, k_group=32, v_group=32), 64),
    "affine2_g64_d128": (configs.make_format(2, 2, k_group=64, v_group=64), 128),
    "sym4_g64": (configs.make_format(4, 4, k_mode=1, v_mode=1, k_group=64, v_group=64), 64),
    "sym_k4v2_g128": (configs.make_format(4, 2, k_mode=1, v_mode=1, k_group=128, v_group=32), 128),
    "affine4_meta16": (configs.make_format(4, 4, k_group=64, v_group=64, meta_fp16=1), 64),
    "sym4_meta16_d256": (configs.make_format(4, 4, k_mode=1, v_mode=1, k_group=64, v_group=128, meta_fp16=1),
                         256),
    "kivi_k2v2": (configs.WORKLOADS["llama8b_kivi"].fmt, 128),
    "kivi_meta16": (dict(configs.WORKLOADS["llama8b_kivi"].fmt, meta_fp16=1), 128),
    "kivi_sym_k4v2": (configs.make_format(4, 2, k_mode=1, v_mode=1, k_axis=1, k_group=32, v_group=32,
                                          residual=64, flush=32), 64),
    "affine8": (configs.make_format(8, 8, k_group=64, v_group=64), 64),
    "sym8_meta16": (configs.make_format(8, 8, k_mode=1, v_mode=1, k_group=32, v_group=64, meta_fp16=1), 128),
    "hadamard_sym": (configs.WORKLOADS["llama8b_had"].fmt, 128),
}


def test_threshold_pairs_straddle_the_floor():
    # host-side check of the construction: fp32 scales below and above 1e-8
    for mode in (configs.AFFINE, configs.SYMMETRIC):
        for bits in (2, 4, 8):
            p = threshold_pairs(mode, bits, FLOOR)
            qd = F32(2 ** bits - 1) if mode == configs.AFFINE else F32(2 ** (bits - 1) - 1)
            s = [((hi - lo) if mode == configs.AFFINE else hi) / qd for lo, hi in p]
            assert s[0] < FLOOR < s[1], (mode, bits, s)


@pytest.mark.gpu
@pytest.mark.parametrize("name", list(FORMATS))
def test_edge_groups_append_decode_prefill(name):
    from paper_2609_04263_amd import kvq
    fmt, D = FORMATS[name]
    B, H, G, n = 2, 2, 4, 420
    K = edge_tokens(1000 + D, B, n, H, D, fmt["k_mode"], fmt["k_bits"], fmt["meta_fp16"], True)
    V = edge_tokens(2000 + D, B, n, H, D, fmt["v_mode"], fmt["v_bits"], fmt["meta_fp16"], False)
    assert (K == 0x8000).any() and (V == 0x8000).any(), "negative zeros must reach the coder"
    T = n + 12
    ref = oracle.Cache(fmt, B, H, D, T)
    ref.append(K, V)
    gc = kvq.Cache(fmt, B, H, D, T)
    Kd, Vd = dev_bf16(K), dev_bf16(V)
    for a, b in ((0, 1), (1, 33), (33, 200), (200, 201), (201, n)):
        gc.append(Kd[:, a:b].contiguous(), Vd[:, a:b].contiguous())
    img = image(gc)
    for i in range(10):
        o, ln = ref.offsets[i], ref.lengths[i]
        x, y = img[o:o + ln], ref.image[o:o + ln]
        if not np.array_equal(x, y):
            diff = np.nonzero(x != y)[0]
            raise AssertionError(f"{name}: section {i} differs at {diff.size} bytes, first at {diff[0]}")
    H_q = H * G
    sm = 1.0 / np.sqrt(D)
    Q = synth.queries(3000 + D, B, H_q, D)
    O = torch.empty((B, H_q, D), dtype=torch.float32, device="cuda")
    gc.decode_attn(dev_bf16(Q), H_q, sm, O, gc.decode_workspace(H_q))
    torch.cuda.synchronize()
    assert_close(O.cpu().numpy(), ref.decode_attn(Q, sm), what=f"{name} decode")
    C = 100
    Qc = synth.normal_bf16(3001 + D, "qc", (B, C, H_q, D))
    Oc = torch.empty((B, C, H_q, D), dtype=torch.float32, device="cuda")
    gc.prefill_attn(dev_bf16(Qc), C, H_q, sm, Oc, gc.prefill_workspace())
    torch.cuda.synchronize()
    assert_close(Oc.cpu().numpy(), ref.prefill_attn(Qc, sm), what=f"{name} prefill")
