"""The C-ABI library loads without a GPU, exports every entry point that
include/qmlp.h declares, and rejects invalid arguments before touching HIP
(every case below fails validation, so nothing is launched)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "qmlp.h")

OK, NULL, SHAPE, ALIGN, UNSUP, WS, HIP = range(7)


@pytest.fixture(scope="module")
def q():
    import paper_2606_04238_amd as qm
    return qm


@pytest.fixture(scope="module")
def lib(q):
    return q.library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(qmlp_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert "qmlp_forward" in names and "qmlp_pack_w2" in names
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings(lib):
    for s in range(7):
        assert lib.qmlp_status_string(s)
    assert lib.qmlp_status_string(99) == b"unknown status"


def test_size_queries(lib):
    assert lib.qmlp_codes_bytes(2, 9728, 2560) == 9728 * 2560 // 4
    assert lib.qmlp_codes_bytes(4, 2560, 9728) == 2560 * 9728 // 2
    assert lib.qmlp_codes_bytes(3, 16, 64) == 0
    assert lib.qmlp_codes_bytes(2, 16, 8) == 0          # k not a whole word
    assert lib.qmlp_meta_bytes(9728, 2560, 128) == 9728 * 20 * 4
    assert lib.qmlp_meta_bytes(16, 100, 64) == 0


FAKE = 0x100000          # 16-byte aligned, never dereferenced: validation fails first


def _qw(q, bits=2, n=512, k=256, g=64, codes=FAKE, meta=FAKE):
    return q.QWeightC(bits, n, k, g, codes, meta)


def _mlp(q, d=256, f=512, g=64, rank=8, **kw):
    A = kw.pop("A", FAKE)
    return q.MlpC(_qw(q, 2, f, d, g), _qw(q, 2, f, d, g), _qw(q, 4, d, f, g),
                  A, FAKE, FAKE, FAKE, rank, 1.0)


def _fwd(lib, m, M=1, dtype=0, x=FAKE, y=FAKE, ws=FAKE, wsb=1 << 30):
    return lib.qmlp_forward(ctypes.byref(m), ctypes.c_void_p(x), M, dtype, ctypes.c_void_p(y),
                            ctypes.c_void_p(ws), wsb, None)


def test_forward_validation(q, lib):
    assert lib.qmlp_forward(None, None, 1, 0, None, None, 0, None) == NULL
    m = _mlp(q)
    assert _fwd(lib, m, x=0) == NULL
    assert _fwd(lib, m, x=FAKE + 2) == ALIGN
    assert _fwd(lib, m, M=17) == UNSUP
    assert _fwd(lib, m, M=-1) == SHAPE
    assert _fwd(lib, m, dtype=1) == UNSUP
    assert _fwd(lib, m, ws=0) == WS
    assert _fwd(lib, m, wsb=16) == WS
    bad_rank = _mlp(q, rank=12)
    assert _fwd(lib, bad_rank) == UNSUP
    no_a = _mlp(q, A=0)
    assert _fwd(lib, no_a) == NULL
    m2 = _mlp(q)
    m2.down.bits = 2
    assert _fwd(lib, m2) == UNSUP
    m3 = _mlp(q)
    m3.up.n_out = 448
    assert _fwd(lib, m3) == SHAPE
    m4 = _mlp(q)
    m4.gate.codes = FAKE + 8
    assert _fwd(lib, m4) == ALIGN
    m5 = _mlp(q)
    m5.gate.group = 32
    assert _fwd(lib, m5) == UNSUP
    # M == 0 is a no-op that succeeds without touching the device
    assert _fwd(lib, m, M=0) == OK


def test_prefill_validation(q, lib):
    m = _mlp(q)                                     # d=256, f=512, g=64, r=8
    # bfloat16 runs the prefill-chunk path: M a multiple of 128, d of 128
    assert _fwd(lib, m, M=128, dtype=1, ws=0) == WS
    assert _fwd(lib, m, M=128, dtype=1, wsb=16) == WS
    assert _fwd(lib, m, M=100, dtype=1) == UNSUP
    assert _fwd(lib, m, M=128, dtype=0) == UNSUP    # binary16 decode stops at 16 tokens
    assert _fwd(lib, _mlp(q, d=320, f=448), M=128, dtype=1) == UNSUP
    assert _fwd(lib, m, M=0, dtype=1) == OK
    assert lib.qmlp_forward_launches(ctypes.byref(m), 256, 1) == 4
    assert lib.qmlp_forward_launches(ctypes.byref(_mlp(q, rank=0)), 256, 1) == 2
    assert lib.qmlp_forward_launches(ctypes.byref(m), 100, 1) == 0
    big = _mlp(q, d=6144, f=16384, g=128, rank=32)
    n = lib.qmlp_workspace_bytes(ctypes.byref(big), 512, 1)
    assert n >= 1024 + 512 * 16384 * 2 + 512 * 64 * 2 + 512 * 64 * 4
    w = _qw(q, bits=4, n=256, k=512)
    assert lib.qmlp_down_w4(ctypes.byref(w), ctypes.c_void_p(FAKE), 100, 1,
                            ctypes.c_void_p(FAKE), None) == UNSUP
    assert lib.qmlp_down_w4(ctypes.byref(w), None, 128, 1, ctypes.c_void_p(FAKE), None) == NULL


def test_workspace_bytes(q, lib):
    m = _mlp(q, d=2560, f=9728, g=128, rank=16)
    n = lib.qmlp_workspace_bytes(ctypes.byref(m), 1, 0)
    assert n >= 9728 * 2 + 2 * 16 * 4
    assert lib.qmlp_workspace_bytes(ctypes.byref(m), 17, 0) == 0
    assert lib.qmlp_workspace_bytes(None, 1, 0) == 0


def test_pack_validation(q, lib):
    out = _qw(q)
    assert lib.qmlp_pack_w2(None, 16, 256, 64, ctypes.byref(out), None, None) == NULL
    assert lib.qmlp_pack_w2(ctypes.c_void_p(FAKE), 16, 256, 96, ctypes.byref(out), None, None) == UNSUP
    assert lib.qmlp_pack_w2(ctypes.c_void_p(FAKE), 16, 200, 64, ctypes.byref(out), None, None) == SHAPE
    assert lib.qmlp_pack_w4(ctypes.c_void_p(FAKE + 4), 16, 256, 64, ctypes.byref(out), None, None) == ALIGN
    assert lib.qmlp_pack_w4(ctypes.c_void_p(FAKE), 0, 256, 64, ctypes.byref(out), None, None) == SHAPE
    assert lib.qmlp_pack_w4(ctypes.c_void_p(FAKE), 16, 256, 64, ctypes.byref(out),
                            ctypes.c_void_p(FAKE + 2), None) == ALIGN


def test_down_and_inspect_validation(q, lib):
    w = _qw(q, bits=4, n=256, k=512)
    assert lib.qmlp_down_w4(ctypes.byref(w), None, 1, 0, ctypes.c_void_p(FAKE), None) == NULL
    w2 = _qw(q, bits=2, n=256, k=512)
    assert lib.qmlp_down_w4(ctypes.byref(w2), ctypes.c_void_p(FAKE), 1, 0, ctypes.c_void_p(FAKE), None) == UNSUP
    assert lib.qmlp_unpack(ctypes.byref(w), None, None, None, None) == NULL
    w3 = _qw(q, bits=3)
    assert lib.qmlp_dequant(ctypes.byref(w3), ctypes.c_void_p(FAKE), None) == UNSUP
    assert lib.qmlp_dequant(ctypes.byref(w), ctypes.c_void_p(FAKE + 1), None) == ALIGN


def test_binding_fails_loudly_without_library(q, monkeypatch, tmp_path):
    monkeypatch.setattr(q, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(q, "_LIB", None)
    with pytest.raises(ImportError):
        q.library()


def _stack_arr(q, *mlps):
    return (q.MlpC * len(mlps))(*mlps)


def test_stack_validation(q, lib):
    m = _mlp(q)
    arr = _stack_arr(q, m, _mlp(q))
    P = ctypes.c_void_p

    def fs(a, L, M=1, x=FAKE, y=FAKE, ws=FAKE, wsb=1 << 30):
        return lib.qmlp_forward_stack(a, L, P(x), M, 0, P(y), None, P(ws), wsb, None)

    assert lib.qmlp_forward_stack(None, 2, None, 1, 0, None, None, None, 0, None) == NULL
    assert fs(arr, 0) == SHAPE
    assert fs(arr, 2, x=0) == NULL
    assert fs(arr, 2, y=FAKE + 8) == ALIGN
    assert fs(arr, 2, M=17) == UNSUP
    assert fs(arr, 2, ws=0) == WS
    assert fs(arr, 2, wsb=16) == WS
    # layers of different shapes are rejected
    odd = _stack_arr(q, m, _mlp(q, d=320, f=448))
    assert fs(odd, 2) == SHAPE
    assert lib.qmlp_stack_workspace_bytes(odd, 2, 1, 0) == 0
    assert lib.qmlp_stack_launches(odd, 2, 1, 0) == 0
    # an invalid block anywhere in the stack is reported
    bad = _stack_arr(q, m, _mlp(q, rank=7))
    assert fs(bad, 2) == UNSUP
    # the stack workspace covers at least the per-block workspace
    assert lib.qmlp_stack_workspace_bytes(arr, 2, 1, 0) >= lib.qmlp_workspace_bytes(ctypes.byref(m), 1, 0)


def test_layers_validation(q, lib):
    """qmlp_forward_layers: the same host-side checks as the stack, bfloat16
    accepted (it runs per block), and the persistent workspace starts with
    the control block."""
    m = _mlp(q)
    arr = _stack_arr(q, m, _mlp(q))
    P = ctypes.c_void_p

    def fl(a, L, M=1, x=FAKE, y=FAKE, ws=FAKE, wsb=1 << 30, dt=0):
        return lib.qmlp_forward_layers(a, L, P(x), M, dt, P(y), P(ws), wsb, None)

    assert lib.qmlp_forward_layers(None, 2, None, 1, 0, None, None, 0, None) == NULL
    assert fl(arr, 0) == SHAPE
    assert fl(arr, 2, x=0) == NULL
    assert fl(arr, 2, y=FAKE + 8) == ALIGN
    assert fl(arr, 2, ws=FAKE + 8) == ALIGN
    assert fl(arr, 2, M=17) == UNSUP
    assert fl(arr, 2, ws=0) == WS
    assert fl(arr, 2, wsb=16) == WS
    assert fl(arr, 2, M=0) == 0                     # nothing to do
    odd = _stack_arr(q, m, _mlp(q, d=320, f=448))
    assert fl(odd, 2) == SHAPE
    assert lib.qmlp_layers_workspace_bytes(odd, 2, 1, 0) == 0
    assert lib.qmlp_layers_launches(odd, 2, 1, 0) == 0
    bad = _stack_arr(q, m, _mlp(q, rank=7))
    assert fl(bad, 2) == UNSUP
    # without a GPU no shape runs persistently: one forward per block, and
    # the workspace is the per-block one
    assert lib.qmlp_layers_launches(arr, 2, 1, 0) == 2 * lib.qmlp_forward_launches(ctypes.byref(m), 1, 0)
    assert lib.qmlp_layers_workspace_bytes(arr, 2, 1, 0) == lib.qmlp_workspace_bytes(ctypes.byref(m), 1, 0)
    assert lib.qmlp_layers_workspace_bytes(arr, 2, 1, 1) == lib.qmlp_workspace_bytes(ctypes.byref(m), 1, 1)
