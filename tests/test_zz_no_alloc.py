"""kvq_decode_attn_noalloc (split partials in the library's static scratch)
against kvq_decode_attn (partials in a caller workspace), through the C ABI.

Two calls in a row on one GPU, the second on a smaller cache, so the second
reuses scratch the first left dirty; with the uncapped plan both entry
points run the same kernels on the same plan and must agree bit for bit.
A cache whose partials would not fit is planned with fewer splits, down to
a single split that needs no partials (checked against the workspace entry
point at the float bar).
"""
import numpy as np
import pytest
import torch

from paper_2609_04263_amd import configs, synth

from gpu_util import assert_close, dev_bf16

pytestmark = pytest.mark.gpu


def filled_cache(fmt, B, H, D, n, seed):
    from paper_2609_04263_amd import kvq
    K, V = synth.kv_tokens(seed, B, n, H, D)
    gc = kvq.Cache(fmt, B, H, D, n)
    gc.append(dev_bf16(K), dev_bf16(V))
    return gc


def both(gc, H_q, seed):
    D = gc.D
    Q = dev_bf16(synth.queries(seed, gc.B, H_q, D))
    sm = 1.0 / np.sqrt(D)
    O_ws = torch.empty((gc.B, H_q, D), dtype=torch.float32, device="cuda")
    O_na = torch.full((gc.B, H_q, D), float("nan"), dtype=torch.float32, device="cuda")
    gc.decode_attn(Q, H_q, sm, O_ws, gc.decode_workspace(H_q))
    gc.decode_attn_noalloc(Q, H_q, sm, O_na)
    torch.cuda.synchronize()
    return O_na.cpu().numpy(), O_ws.cpu().numpy()


def test_noalloc_matches_workspace_entry_two_calls():
    kivi = configs.WORKLOADS["llama8b_kivi"].fmt
    tiny = configs.WORKLOADS["tiny_b16"].fmt
    # first call: KIVI window (an fp16 split), several splits per unit
    gc1 = filled_cache(kivi, B=4, H=8, D=128, n=3000, seed=500)
    na, ws = both(gc1, H_q=32, seed=501)
    assert_close(na, ws, what="noalloc vs workspace, KIVI B=4 n=3000")
    assert np.array_equal(na, ws), "same plan, same kernels: outputs must be identical"
    # second call, smaller: the scratch still holds the first call's partials
    gc2 = filled_cache(tiny, B=2, H=2, D=64, n=300, seed=502)
    na, ws = both(gc2, H_q=16, seed=503)
    assert_close(na, ws, what="noalloc vs workspace, tiny B=2 n=300")
    assert np.array_equal(na, ws)


def test_noalloc_caps_splits_to_the_scratch():
    tiny = configs.WORKLOADS["tiny_b16"].fmt
    # B * H_q = 512 rows of D = 128 (266 KB of partials per split): the
    # workspace entry point plans one split per resident workgroup slot
    # (16 per unit here), which would need more than the 4 MiB scratch, so
    # the no-alloc plan has fewer splits; the outputs agree at the float bar
    gc = filled_cache(tiny, B=4, H=8, D=128, n=2000, seed=504)
    na, ws = both(gc, H_q=128, seed=505)
    assert_close(na, ws, what="noalloc (capped splits) vs workspace")


def test_noalloc_single_split_when_two_do_not_fit():
    from paper_2609_04263_amd import kvq
    kivi = configs.WORKLOADS["llama8b_kivi"].fmt
    # 4096 rows of D = 128: two splits would need 4.26 MB of partials, more
    # than the 4 MiB scratch, so one split per unit writes the outputs
    B, H, H_q, D = 32, 8, 128, 128
    assert B * H_q * (D + 2) * 4 * 2 > kvq.SCRATCH_BYTES - 256
    gc = filled_cache(kivi, B=B, H=H, D=D, n=1200, seed=506)
    na, ws = both(gc, H_q=H_q, seed=507)
    assert_close(na, ws, what="noalloc (single split) vs workspace")
