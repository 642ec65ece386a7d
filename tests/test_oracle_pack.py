"""Pins of the oracle's bit packing and storage-image layout.

Sec. 3.1 stores "packed unsigned codes"; the bit order and section layout
are this implementation's (documented in the oracle's header and in
include/kvq.h).  Pinned by literal byte images, an exhaustive round trip,
and closed-form section sizes.
"""
import itertools

import numpy as np
import pytest

import oracle
from paper_2609_04263_amd import configs


def test_pack_byte_images():
    assert oracle.pack_word(np.arange(8), 4) == 0x76543210
    w = oracle.pack_word([1, 2, 3, 0] * 4, 2)
    assert w & 0xFF == 0x39
    assert w == 0x39393939
    assert oracle.pack_word([15] + [0] * 7, 4) == 0xF
    assert oracle.pack_word([0] * 7 + [15], 4) == 0xF0000000
    assert oracle.pack_word([0] * 15 + [3], 2) == 0xC0000000


@pytest.mark.parametrize("bits", [2, 4, 8])
def test_pack_round_trip_every_value_at_every_position(bits):
    n = 32 // bits
    for pos, val in itertools.product(range(n), range(2 ** bits)):
        codes = np.zeros(n, dtype=np.uint8)
        codes[pos] = val
        w = oracle.pack_word(codes, bits)
        assert w == val << (bits * pos)
        assert np.array_equal(oracle.unpack_word(w, bits), codes)
    rng = np.random.default_rng(bits)
    for _ in range(500):
        codes = rng.integers(0, 2 ** bits, n).astype(np.uint8)
        assert np.array_equal(oracle.unpack_word(oracle.pack_word(codes, bits), bits), codes)


@pytest.mark.parametrize("name", configs.WORKLOAD_ORDER)
def test_layout_sizes_closed_form(name):
    wl = configs.WORKLOADS[name]
    f = wl.fmt
    B, H, D, T = wl.B, wl.H_kv, wl.D, wl.T_max
    Ta = -(-T // 32) * 32
    off, ln, total = oracle.layout(f, B, H, D, T)
    assert all(o % 256 == 0 for o in off)
    assert ln[0] == B * H * Ta * D * f["k_bits"] // 8
    if f["k_axis"] == 0:
        assert ln[1] == B * H * Ta * (D // f["k_group"]) * 4
    else:
        assert ln[1] == B * H * (Ta // 32) * D * 4
    assert ln[2] == (ln[1] if f["k_mode"] == 0 else 0)
    assert ln[3] == B * H * Ta * D * f["v_bits"] // 8
    assert ln[4] == B * H * Ta * (D // f["v_group"]) * 4
    assert ln[5] == (ln[4] if f["v_mode"] == 0 else 0)
    ring = f["residual"] + f["flush"]
    assert ln[6] == ln[7] == B * H * ring * D * 2
    for i in range(7):
        assert off[i + 1] >= off[i] + ln[i]
    assert total >= off[7] + ln[7] and total % 256 == 0


def test_kivi_live_footprint_at_8192_tokens():
    # Sec. 3.1: footprint = packed codes + metadata + fp16 residual.  KIVI K2V2
    # on the Llama-shaped layer at n = 8192: 8064 coded tokens (64 + 64 bytes
    # per token per head) and 128 fp16 residual tokens (512 bytes).
    wl = configs.WORKLOADS["llama8b_kivi"]
    live = configs.attention_bytes(wl, 8192) - 6 * wl.B * wl.H_q * wl.D
    assert configs.num_coded(wl.fmt, 8192) == 8064
    assert live == 32 * 8 * (8064 * 128 + 128 * 512) == 281_018_368


@pytest.mark.parametrize("n,expect", [(0, 0), (100, 0), (128, 0), (159, 0), (160, 32), (191, 32),
                                      (192, 64), (8192, 8064), (8224, 8096)])
def test_kivi_coded_count(n, expect):
    f = configs.WORKLOADS["llama8b_kivi"].fmt
    assert oracle.num_coded(f, n) == expect == configs.num_coded(f, n)


def test_format_validation():
    good = configs.make_format()
    assert oracle.check_format(good, 64) == 0
    bad = [dict(good, k_bits=3), dict(good, v_mode=2), dict(good, v_axis=1),
           dict(good, k_group=48), dict(good, k_group=128), dict(good, rotate=32),
           dict(good, k_axis=1), dict(good, residual=128, flush=0), dict(good, flush=16)]
    for f in bad:
        assert oracle.check_format(f, 64) == 2, f
    assert oracle.check_format(good, 96) == 2
