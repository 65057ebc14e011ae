"""C-ABI checks that need no GPU: the library loads, exports every entry point the
headers declare, and rejects bad arguments on the host before enqueueing anything."""

import ctypes
import glob
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    from paper_2608_27922_amd import api, build
    if not os.path.exists(api.LIB_PATH):
        build.build()
    return api.lib()


def declared_functions():
    names = []
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = open(h).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names += re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(densitykv_\w+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert len(names) >= 6
    from paper_2608_27922_amd import api
    assert set(names) == set(api.ENTRY_POINTS)
    for n in names:
        assert hasattr(L, n), n


def test_status_strings(L):
    for code in range(-7, 1):
        assert L.densitykv_status_string(code)
    assert L.densitykv_status_string(-99) == b"unknown status"


def _bank(api, **kw):
    f = dict(num_banks=12, group_size=12, head_dim=128, capacity=4680, dtype=0)
    f.update(kw)
    return api.DkvBank(f["num_banks"], f["group_size"], f["head_dim"], f["capacity"], f["dtype"],
                       *([1] * 8))  # non-null fake pointers: never dereferenced on error paths


def test_workspace_size_and_shape_checks(L):
    from paper_2608_27922_amd import api
    sz = ctypes.c_size_t()
    assert L.densitykv_workspace_size(ctypes.byref(_bank(api)), 4680, ctypes.byref(sz)) == 0
    small = sz.value
    assert L.densitykv_workspace_size(ctypes.byref(_bank(api, num_banks=360)), 4680, ctypes.byref(sz)) == 0
    assert sz.value > small
    assert L.densitykv_workspace_size(ctypes.byref(_bank(api, head_dim=96)), 10, ctypes.byref(sz)) == -3
    assert L.densitykv_workspace_size(ctypes.byref(_bank(api, group_size=5)), 10, ctypes.byref(sz)) == -2
    assert L.densitykv_workspace_size(ctypes.byref(_bank(api, capacity=40000)), 10, ctypes.byref(sz)) == -2
    # rows are 32-bit indices in the kernels: B * max(capacity, 8191) < 2^31
    assert L.densitykv_workspace_size(ctypes.byref(_bank(api, num_banks=65538, group_size=1, capacity=32767)), 10,
                                      ctypes.byref(sz)) == 0
    assert L.densitykv_workspace_size(ctypes.byref(_bank(api, num_banks=65539, group_size=1, capacity=32767)), 10,
                                      ctypes.byref(sz)) == -2
    assert L.densitykv_workspace_size(ctypes.byref(_bank(api, num_banks=262177, group_size=1, capacity=16)), 10,
                                      ctypes.byref(sz)) == -2
    assert L.densitykv_workspace_size(ctypes.byref(_bank(api, dtype=7)), 10, ctypes.byref(sz)) == -1
    assert L.densitykv_workspace_size(ctypes.byref(_bank(api)), 9000, ctypes.byref(sz)) == -2
    assert L.densitykv_workspace_size(None, 10, ctypes.byref(sz)) == -1


def test_update_rejects_bad_arguments_before_launch(L):
    from paper_2608_27922_amd import api
    b = _bank(api)
    seg = api.DkvSegment(100, 3, 1, 1)
    good = api.Params().c()
    ws = ctypes.c_void_p(1)
    upd = lambda bank, s, p, wsz: L.densitykv_update_bank(ctypes.byref(bank), ctypes.byref(s), ctypes.byref(p),
                                                          None, ws, wsz, None)
    assert upd(b, seg, api.Params(p=3).c(), 1 << 40) == -3
    assert upd(b, seg, api.Params(sigma2_log2=40).c(), 1 << 40) == -3
    assert upd(b, seg, api.Params(tau_num=1).c(), 1 << 40) == -5          # tau must exceed 1
    assert upd(b, seg, api.Params(tau_num=2, tau_log2_den=1).c(), 1 << 40) == -5
    assert upd(b, seg, api.Params(delta_q=0).c(), 1 << 40) == -5
    assert upd(b, seg, api.Params(flags=0x40).c(), 1 << 40) == -1          # unknown policy bits
    assert upd(b, seg, api.Params(flags=0x80000000).c(), 1 << 40) == -1
    both = api.POLICY_DENSEST_ONLY | api.POLICY_SOURCE_FILL
    assert upd(b, seg, api.Params(flags=both).c(), 1 << 40) == -1          # exclusive eviction policies
    kv = api.Params(flags=api.POLICY_KV_DESCRIPTOR).c()
    assert upd(_bank(api, dtype=1), seg, kv, 1 << 40) == -3                 # [K; V] geometry: bf16 banks only
    assert upd(b, api.DkvSegment(100, 3, 1, None), kv, 1 << 40) == -1       # ... and needs the values
    seq = api.POLICY_SEQUENTIAL
    for other in (api.POLICY_DENSEST_ONLY, api.POLICY_SOURCE_FILL, api.POLICY_KV_DESCRIPTOR):
        assert upd(b, seg, api.Params(flags=seq | other).c(), 1 << 40) == -1  # sequential combines with 0x1, 0x2 only
    assert upd(_bank(api, dtype=1), seg, api.Params(flags=seq).c(), 1 << 40) == -3   # bf16 banks only
    assert upd(_bank(api, num_banks=300, group_size=300), seg, api.Params(flags=seq).c(), 1 << 40) == -2
    sz, szs = ctypes.c_size_t(), ctypes.c_size_t()
    assert L.densitykv_workspace_size(ctypes.byref(b), 100, ctypes.byref(sz)) == 0
    assert L.densitykv_workspace_size_policy(ctypes.byref(b), 100, 0, ctypes.byref(szs)) == 0
    assert szs.value == sz.value
    assert L.densitykv_workspace_size_policy(ctypes.byref(b), 100, seq, ctypes.byref(szs)) == 0
    assert szs.value >= sz.value + 12 * (4680 + 100) ** 2 * 4               # the pairwise weights
    assert upd(b, seg, api.Params(flags=seq).c(), sz.value) == -4           # default-size workspace is too small
    assert upd(b, api.DkvSegment(9000, 3, 1, 1), good, 1 << 40) == -2
    assert upd(b, api.DkvSegment(100, -1, 1, 1), good, 1 << 40) == -5
    assert upd(b, api.DkvSegment(100, 3, None, 1), good, 1 << 40) == -1
    assert upd(b, seg, good, 16) == -4                                      # workspace too small
    nullk = api.DkvBank(12, 12, 128, 4680, 0, None, *([1] * 7))
    assert upd(nullk, seg, good, 1 << 40) == -1


def test_noalloc_update_rejects_before_launch(L):
    """The no-allocation update checks its arguments and the size of its static
    scratch on the host: bad arguments give the usual codes, a workspace need
    beyond the scratch gives DKV_ERR_SCRATCH, and nothing reaches the device."""
    from paper_2608_27922_amd import api
    seg = api.DkvSegment(4680, 3, 1, 1)
    upd = lambda bank, s, p: L.densitykv_update_bank_noalloc(ctypes.byref(bank), ctypes.byref(s), ctypes.byref(p),
                                                             None, None)
    assert upd(_bank(api), seg, api.Params(p=3).c()) == -3
    assert upd(_bank(api), api.DkvSegment(9000, 3, 1, 1), api.Params().c()) == -2
    big = _bank(api, num_banks=360)
    sz = ctypes.c_size_t()
    assert L.densitykv_workspace_size(ctypes.byref(big), 4680, ctypes.byref(sz)) == 0
    assert sz.value > api.NOALLOC_SCRATCH_BYTES
    assert upd(big, seg, api.Params().c()) == -7
    # the single-layer geometry (12 banks of 4,680 slots, 4,680 candidates) fits
    assert L.densitykv_workspace_size(ctypes.byref(_bank(api)), 4680, ctypes.byref(sz)) == 0
    assert sz.value <= api.NOALLOC_SCRATCH_BYTES
    # the sequential competition's pairwise weights do not fit at that size
    assert upd(_bank(api), seg, api.Params(flags=api.POLICY_SEQUENTIAL).c()) == -7


def test_attention_rejects_bad_arguments(L):
    from paper_2608_27922_amd import api
    b = _bank(api)
    att = lambda nq, nw, q, wk, scale: L.densitykv_bank_attention(ctypes.byref(b), q, nq, wk, wk, nw, q,
                                                                  ctypes.c_float(scale), None)
    assert att(-1, 0, 1, None, 0.1) == -2
    assert att(10, 5, 1, None, 0.1) == -1
    assert att(10, 0, None, None, 0.1) == -1
    assert att(10, 0, 1, None, 0.0) == -5
    assert att(10, 0, 1, None, float("nan")) == -5
    sink = lambda ns, sk: L.densitykv_bank_attention_sink(ctypes.byref(b), 1, 10, sk, sk, ns, None, None, 0, 1,
                                                          ctypes.c_float(0.1), None)
    assert sink(5, None) == -1                                               # sink missing
    assert sink(-1, None) == -2


def test_pair_weight_rejects_bad_arguments(L):
    from paper_2608_27922_amd import api
    p = api.Params().c()
    assert L.densitykv_pair_weight_q23(None, 5, ctypes.byref(p), None, None) == -1
    assert L.densitykv_pair_weight_q23(None, -1, ctypes.byref(p), None, None) == -2
    bad = api.Params(p=5).c()
    assert L.densitykv_pair_weight_q23(1, 5, ctypes.byref(bad), 1, None) == -3


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    from paper_2608_27922_amd import api
    monkeypatch.setattr(api, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(api, "_lib", None)
    with pytest.raises(RuntimeError):
        api.lib()
