"""The oracle's unit loops run on OpenMP threads; every result must be the
same for any thread count (each unit is computed by one thread in a fixed
order).  Checked bit for bit on append images, attention and projection."""
import numpy as np

import oracle
from paper_2609_04263_amd import configs, synth


def _run_all(threads):
    oracle.set_threads(threads)
    out = []
    for fmt, D in ((configs.WORKLOADS["llama8b_kivi"].fmt, 128), (configs.WORKLOADS["llama8b_had"].fmt, 128),
                   (configs.make_format(4, 4, k_group=64, v_group=64, sink=32), 64)):
        B, H, n = 3, 2, 300
        K, V = synth.kv_tokens(7, B, n, H, D)
        c = oracle.Cache(fmt, B, H, D, n)
        c.append(K[:, :131], V[:, :131])
        c.append(K[:, 131:], V[:, 131:])
        out.append(c.image.copy())
        Q = synth.queries(8, B, 4 * H, D)
        out.append(c.decode_attn(Q, 0.1))
        out.append(c.prefill_attn(synth.normal_bf16(9, "q", (B, 20, 4 * H, D)), 0.1))
        out += list(c.dequant())
    wl = configs.WORKLOADS["tiny_b1"]
    W, A, Bm = synth.layer_weights(wl)
    Hm = synth.hidden(wl, "threads", 37)
    out += list(oracle.project(Hm, W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv))
    out += list(oracle.merge_adapter(W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv))
    return out


def test_results_do_not_depend_on_thread_count():
    before = oracle.get_threads()
    try:
        one = _run_all(1)
        many = _run_all(max(4, before))
    finally:
        oracle.set_threads(before)
    assert len(one) == len(many)
    for a, b in zip(one, many):
        assert a.dtype == b.dtype and a.shape == b.shape
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8))
