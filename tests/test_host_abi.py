"""Host-side checks of the C ABI (no GPU needed).

* libkvq.so loads and exports every function include/kvq.h declares;
* the storage layout (total size and section offsets) matches the oracle's
  for every workload and a spread of formats;
* argument errors are reported before anything is enqueued and leave the
  cache handle unchanged (fake, never-dereferenced device addresses).
"""
import ctypes as C
import os
import re

import pytest

import oracle
from paper_2609_04263_amd import configs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 1 << 32          # 256-aligned address that host code never dereferences


@pytest.fixture(scope="module")
def kvq():
    from paper_2609_04263_amd import kvq as mod
    return mod


def declared_functions():
    text = open(os.path.join(ROOT, "include", "kvq.h")).read()
    return sorted(set(re.findall(r"^\s*(?:kvq_status|void|const char\*)\s+(kvq_\w+)\s*\(", text, re.M)))


def test_every_declared_symbol_is_exported(kvq):
    names = declared_functions()
    assert len(names) >= 13
    for name in names:
        assert hasattr(kvq.lib(), name), name
    assert set(names) == set(kvq.EXPORTED)


FORMATS = [wl.fmt for wl in configs.WORKLOADS.values()] + [
    configs.make_format(2, 4, k_mode=1, k_group=32, v_group=128),
    configs.make_format(4, 2, k_axis=1, k_group=32, v_group=64, residual=64, flush=64),
    configs.make_format(4, 4, k_group=256, v_group=256),
    configs.make_format(2, 4, k_axis=1, k_group=32, v_group=64, residual=128, flush=32, meta_fp16=1),
    configs.make_format(8, 8, k_group=64, v_group=128),
    configs.make_format(8, 8, k_mode=1, k_axis=1, k_group=32, v_group=32, residual=32, flush=32,
                        meta_fp16=1),
]


@pytest.mark.parametrize("kb,vb", [(8, 4), (4, 8), (8, 2), (3, 3), (16, 16)])
def test_code_widths_outside_the_kernels_are_rejected(kvq, kb, vb):
    # 8-bit codes are served only as K and V both 8-bit
    f = configs.make_format(kb, vb, k_group=64, v_group=64)
    with pytest.raises(kvq.KvqError) as e:
        kvq.cache_bytes(f, 1, 1, 64, 32)
    assert e.value.status == kvq.ERR_FORMAT


@pytest.mark.parametrize("fi", range(len(FORMATS)))
@pytest.mark.parametrize("dims", [(1, 1, 64, 1), (3, 2, 128, 77), (2, 5, 256, 300)])
def test_layout_matches_oracle(kvq, fi, dims):
    f = FORMATS[fi]
    B, H, D, T = dims
    if oracle.check_format(f, D) != 0:
        with pytest.raises(kvq.KvqError) as e:
            kvq.cache_bytes(f, B, H, D, T)
        assert e.value.status == kvq.ERR_FORMAT
        return
    off, ln, total = oracle.layout(f, B, H, D, T)
    assert kvq.cache_bytes(f, B, H, D, T) == total
    c = kvq.Cache(f, B, H, D, T, storage=FakeStorage(total))
    for i in range(10):
        assert c.section(i) == (off[i], ln[i])


class FakeStorage:
    """Stands in for a device tensor on hosts without a GPU."""

    def __init__(self, nbytes, addr=FAKE):
        self.nbytes, self.addr = nbytes, addr

    def data_ptr(self):
        return self.addr

    def numel(self):
        return self.nbytes

    def element_size(self):
        return 1


def test_errors_leave_cache_unchanged(kvq):
    f = configs.make_format(4, 4, k_group=64, v_group=64)
    B, H, D, T = 2, 2, 64, 40
    c = kvq.Cache(f, B, H, D, T, storage=FakeStorage(kvq.cache_bytes(f, B, H, D, T)))
    assert c.length() == (0, 0)
    fake_k = FakeStorage(0, FAKE + (1 << 30))
    # capacity
    with pytest.raises(kvq.KvqError) as e:
        c.append(fake_k, fake_k, n_new=41, stream=0)
    assert e.value.status == kvq.ERR_CAPACITY and c.length() == (0, 0)
    # format mismatch
    with pytest.raises(kvq.KvqError) as e:
        c.append(fake_k, fake_k, n_new=1, fmt=dict(f, k_bits=2), stream=0)
    assert e.value.status == kvq.ERR_FORMAT and c.length() == (0, 0)
    # misaligned input
    with pytest.raises(kvq.KvqError) as e:
        c.append(FakeStorage(0, FAKE + 8), fake_k, n_new=1, stream=0)
    assert e.value.status == kvq.ERR_ARG and c.length() == (0, 0)
    # empty append is a no-op
    c.append(fake_k, fake_k, n_new=0, stream=0)
    assert c.length() == (0, 0)
    # empty cache cannot be attended
    with pytest.raises(kvq.KvqError) as e:
        c.decode_attn(fake_k, 8, 0.125, fake_k, FakeStorage(1 << 20), stream=0)
    assert e.value.status == kvq.ERR_ARG
    # bad head grouping
    assert c.decode_workspace_bytes(8) > 0
    for bad in (3, 2 * 17 + 1, 2 * 17):
        with pytest.raises(kvq.KvqError):
            c.decode_workspace_bytes(bad)


def test_prefill_argument_checks(kvq):
    f = configs.make_format()
    c = kvq.Cache(f, 2, 2, 64, 64, storage=FakeStorage(kvq.cache_bytes(f, 2, 2, 64, 64)))
    q = FakeStorage(0, FAKE)
    ws = FakeStorage(1 << 20)
    # empty cache: no chunk can be attended
    with pytest.raises(kvq.KvqError) as e:
        c.prefill_attn(q, 1, 4, 0.125, q, ws, stream=0)
    assert e.value.status == kvq.ERR_ARG
    assert c.prefill_workspace_bytes() == 0
    c.restore(40)  # two 32-token blocks per (b, h) unit
    # workspace: one 192 D-byte image per visible block and unit
    full = c.prefill_workspace_bytes()
    assert full == 2 * 2 * 2 * 192 * 64
    # the same for a rotating format (its values are rotated back in the image)
    for D in (64, 256):
        fr = configs.make_format(rotate=D)
        cr = kvq.Cache(fr, 2, 2, D, 64, storage=FakeStorage(kvq.cache_bytes(fr, 2, 2, D, 64)))
        cr.restore(40)
        assert cr.prefill_workspace_bytes() == 2 * 2 * 2 * 192 * D
    # misaligned output, bad head grouping
    with pytest.raises(kvq.KvqError) as e:
        c.prefill_attn(q, 1, 4, 0.125, FakeStorage(0, FAKE + 4), ws, stream=0)
    assert e.value.status == kvq.ERR_ARG
    with pytest.raises(kvq.KvqError) as e:
        c.prefill_attn(q, 1, 3, 0.125, q, ws, stream=0)
    assert e.value.status == kvq.ERR_ARG
    # chunk longer than the cache
    with pytest.raises(kvq.KvqError) as e:
        c.prefill_attn(q, 41, 4, 0.125, q, ws, stream=0)
    assert e.value.status == kvq.ERR_ARG
    # workspace below one unit's share, misaligned or missing
    for bad in (FakeStorage(full // 4 - 16), FakeStorage(full, FAKE + 8), FakeStorage(full, 0)):
        with pytest.raises(kvq.KvqError) as e:
            c.prefill_attn(q, 1, 4, 0.125, q, bad, stream=0)
        assert e.value.status == kvq.ERR_WORKSPACE


def test_project_append_argument_checks(kvq):
    f = configs.make_format()
    B, H, D, T = 2, 4, 64, 512
    c = kvq.Cache(f, B, H, D, T, storage=FakeStorage(kvq.cache_bytes(f, B, H, D, T)))
    t = FakeStorage(0, FAKE)
    args = dict(d_in=256, d_q=512, d_kv=256, rank=0, n_new=128)

    def call(cache=c, M=None, **kw):
        a = dict(args, **kw)
        M = B * a["n_new"] if M is None else M
        return kvq.lib().kvq_project_append(FAKE, M, a["d_in"], FAKE, a["d_q"], a["d_kv"], FAKE, FAKE, a["rank"],
                                            2.0, FAKE, cache.handle, a["n_new"], FAKE, 1 << 20, None)
    assert call(n_new=100) == kvq.ERR_ARG              # tokens not a multiple of 32
    assert call(n_new=64) == kvq.ERR_ARG               # M = 128 < 256
    assert call(M=2 * 128 + 32) == kvq.ERR_ARG          # M != B n_new
    assert call(d_q=384) == kvq.ERR_ARG                 # d_q not a multiple of 256
    assert call(d_kv=512) == kvq.ERR_ARG                # d_kv != H D
    assert call(n_new=544) == kvq.ERR_CAPACITY          # 544 > T (checked after the shapes)
    for bad in (configs.WORKLOADS["llama8b_kivi"].fmt, configs.make_format(rotate=64), configs.make_format(sink=32)):
        cb = kvq.Cache(bad, B, H, D, T, storage=FakeStorage(kvq.cache_bytes(bad, B, H, D, T)))
        assert call(cache=cb) == kvq.ERR_FORMAT
    assert c.length() == (0, 0)


def test_rewind_only_without_window(kvq):
    f = configs.WORKLOADS["llama8b_kivi"].fmt
    c = kvq.Cache(f, 1, 1, 128, 64, storage=FakeStorage(kvq.cache_bytes(f, 1, 1, 128, 64)))
    with pytest.raises(kvq.KvqError) as e:
        c.rewind(0)
    assert e.value.status == kvq.ERR_FORMAT


def test_init_rejects_small_or_misaligned_storage(kvq):
    f = configs.make_format()
    n = kvq.cache_bytes(f, 1, 1, 64, 32)
    with pytest.raises(kvq.KvqError):
        kvq.Cache(f, 1, 1, 64, 32, storage=FakeStorage(n - 1))
    with pytest.raises(kvq.KvqError):
        kvq.Cache(f, 1, 1, 64, 32, storage=FakeStorage(n, FAKE + 128))


def test_projection_argument_checks(kvq):
    p = FakeStorage(0, FAKE)
    ws_small = FakeStorage(4, FAKE)
    # d_in must be a multiple of 64
    with pytest.raises(kvq.KvqError) as e:
        kvq.project_qkv(_Shape(4, 96), p, p, p, 8, 2.0, 64, 64, p, p, p, ws_small, stream=0)
    assert e.value.status == kvq.ERR_ARG
    # rank above 64
    with pytest.raises(kvq.KvqError) as e:
        kvq.project_qkv(_Shape(4, 128), p, p, p, 65, 2.0, 64, 64, p, p, p, ws_small, stream=0)
    assert e.value.status == kvq.ERR_ARG
    # workspace too small for M x 3r fp32
    with pytest.raises(kvq.KvqError) as e:
        kvq.project_qkv(_Shape(4, 128), p, p, p, 8, 2.0, 64, 64, p, p, p, ws_small, stream=0)
    assert e.value.status == kvq.ERR_WORKSPACE
    assert kvq.project_workspace_bytes(4, 8) == 16 * 4 * 24 * 4
    assert kvq.project_workspace_bytes(64, 8) == 64 * 24 * 4


def test_merge_argument_checks(kvq):
    p = FakeStorage(0, FAKE)
    mis = FakeStorage(0, FAKE + 8)
    cases = [
        (_Shape(96, 96), 8, 64, 64, p),    # d_in not a multiple of 64
        (_Shape(96, 128), 0, 64, 64, p),   # rank 0: nothing to merge
        (_Shape(96, 128), 65, 64, 64, p),  # rank above 64
        (_Shape(96, 128), 8, 48, 64, p),   # d_q not a multiple of 32
        (_Shape(96, 128), 8, 64, 16, p),   # d_kv below 32
        (_Shape(96, 128), 8, 64, 64, mis),  # misaligned output
    ]
    for W, rank, d_q, d_kv, out in cases:
        with pytest.raises(kvq.KvqError) as e:
            kvq.merge_adapter(W, p, p, rank, 2.0, d_q, d_kv, out, stream=0)
        assert e.value.status == kvq.ERR_ARG
    with pytest.raises(kvq.KvqError) as e:
        kvq.merge_adapter(_Shape(96, 128), p, p, 8, float("nan"), 64, 64, p, stream=0)
    assert e.value.status == kvq.ERR_ARG


class _Shape(FakeStorage):
    def __init__(self, M, d_in):
        super().__init__(0, FAKE)
        self.shape = (M, d_in)


def test_time_launches_argument_checks(kvq):
    """The measurement hook takes both events or neither; it launches nothing."""
    lib = kvq.lib()
    assert lib.kvq_time_launches(C.c_void_p(FAKE), None) == 1          # KVQ_ERR_ARG
    assert lib.kvq_time_launches(None, C.c_void_p(FAKE)) == 1
    assert lib.kvq_time_launches(None, None) == 0
