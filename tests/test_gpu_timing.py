"""The measurement hook kvq_time_launches on the GPU (tests only): a decode
call timed by its kernels' own dispatch events gives a positive device time
no longer than the same call between two recorded marker events, leaves the
results unchanged, and stops timing once cleared."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2609_04263_amd import configs, kvq, synth

pytestmark = pytest.mark.gpu


class _Ev:
    _lib = None

    def __init__(self):
        if _Ev._lib is None:
            lib = ctypes.CDLL("libamdhip64.so")
            lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
            lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            lib.hipEventSynchronize.argtypes = [ctypes.c_void_p]
            lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
            lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
            _Ev._lib = lib
        self.ev = ctypes.c_void_p()
        assert _Ev._lib.hipEventCreate(ctypes.byref(self.ev)) == 0

    def record(self):
        assert _Ev._lib.hipEventRecord(self.ev, torch.cuda.current_stream().cuda_stream) == 0

    def ms_to(self, end) -> float:
        _Ev._lib.hipEventSynchronize(end.ev)
        ms = ctypes.c_float()
        assert _Ev._lib.hipEventElapsedTime(ctypes.byref(ms), self.ev, end.ev) == 0
        return ms.value

    def __del__(self):
        if self.ev:
            _Ev._lib.hipEventDestroy(self.ev)


def test_time_launches_decode_call():
    wl = configs.WORKLOADS["tiny_b16"]
    B, Hq, Hkv, D = wl.B, wl.H_q, wl.H_kv, wl.D
    cache = kvq.Cache(wl.fmt, B, Hkv, D, 2048)
    g = torch.Generator(device="cpu").manual_seed(5)
    K = torch.randn(B, 1500, Hkv, D, generator=g).to(torch.bfloat16).cuda()
    V = torch.randn(B, 1500, Hkv, D, generator=g).to(torch.bfloat16).cuda()
    cache.append(K, V)
    Q = torch.randn(B, Hq, D, generator=g).to(torch.bfloat16).cuda()
    ws = cache.decode_workspace(Hq)
    O_ref = torch.empty(B, Hq, D, dtype=torch.float32, device="cuda")
    O = torch.empty_like(O_ref)
    cache.decode_attn(Q, Hq, 1.0 / np.sqrt(D), O_ref, ws)
    m0, m1, d0, d1 = _Ev(), _Ev(), _Ev(), _Ev()
    torch.cuda.synchronize()
    m0.record()
    kvq.time_launches(d0.ev.value, d1.ev.value)
    cache.decode_attn(Q, Hq, 1.0 / np.sqrt(D), O, ws)
    kvq.time_launches(None, None)
    m1.record()
    torch.cuda.synchronize()
    dev_ms, mark_ms = d0.ms_to(d1), m0.ms_to(m1)
    assert 0.0 < dev_ms <= mark_ms, (dev_ms, mark_ms)
    assert torch.equal(O, O_ref)
    # cleared: a later call leaves the dispatch events where they were
    cache.decode_attn(Q, Hq, 1.0 / np.sqrt(D), O, ws)
    torch.cuda.synchronize()
    assert d0.ms_to(d1) == dev_ms

