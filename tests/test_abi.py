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
    assert lib.qmlp_codes_bytes(5, 16, 64) == 0
    assert lib.qmlp_codes_bytes(3, 16, 128) == 16 * 128 * 3 // 8        # the two-plane 3-bit rows
    assert lib.qmlp_codes_bytes(3, 16, 64) == 0                         # rows not 16-byte aligned
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
    m2.down.bits = 3
    assert _fwd(lib, m2) == UNSUP
    m2.down.bits, m2.down.group = 2, 32             # 2-bit down needs whole 64-code units per group
    assert _fwd(lib, m2) == UNSUP
    m3 = _mlp(q)
    m3.up.n_out = 448
    assert _fwd(lib, m3) == SHAPE
    m4 = _mlp(q)
    m4.gate.codes = FAKE + 8
    assert _fwd(lib, m4) == ALIGN
    m5 = _mlp(q)
    m5.gate.group = 32                              # gate and up must share the group
    assert _fwd(lib, m5) == SHAPE
    m5.gate.group = m5.up.group = 96
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
    # LoRA-A, its reduction, gate/up, down over slices of f, the slices' sum
    assert lib.qmlp_forward_launches(ctypes.byref(m), 256, 1) == 5
    assert lib.qmlp_forward_launches(ctypes.byref(_mlp(q, rank=0)), 256, 1) == 3
    # f = 448 is not a multiple of 128: down runs unsplit
    assert lib.qmlp_forward_launches(ctypes.byref(_mlp(q, d=256, f=448)), 256, 1) == 4
    assert lib.qmlp_forward_launches(ctypes.byref(m), 100, 1) == 0
    big = _mlp(q, d=6144, f=16384, g=128, rank=32)
    n = lib.qmlp_workspace_bytes(ctypes.byref(big), 512, 1)
    # h, T, t and the down slices' fp32 partial sums (4 slices of 512 x 6144)
    assert n >= 1024 + 512 * 16384 * 2 + 512 * 64 * 2 + 512 * 64 * 4 + 4 * 512 * 6144 * 4
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
    w3 = _qw(q, bits=5)
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
    assert lib.qmlp_stack_error_offset(odd, 2, 1, 0) == 0
    # without a GPU the blocks never run persistently: no error word; with
    # one, the word lies inside the workspace past the per-layer part
    off = lib.qmlp_stack_error_offset(arr, 2, 1, 0)
    assert off == 0 or (lib.qmlp_workspace_bytes(ctypes.byref(m), 1, 0) < off
                        <= lib.qmlp_stack_workspace_bytes(arr, 2, 1, 0) - 4)
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
    # without a GPU no shape runs persistently: binary16 blocks run as one
    # batch on the stand-alone kernels (LoRA-A, gate/up, down of every block),
    # the workspace holding the control block, t and h of every block
    assert lib.qmlp_layers_launches(arr, 2, 1, 0) == 3
    r256 = lambda v: (v + 255) // 256 * 256
    assert lib.qmlp_layers_workspace_bytes(arr, 2, 3, 0) == 1024 + r256(2 * 3 * 16 * 4) + r256(2 * 3 * 512 * 2)
    big = _stack_arr(q, *[_mlp(q) for _ in range(41)])
    assert lib.qmlp_layers_launches(big, 41, 1, 0) == 6        # batches of at most 40 blocks
    assert lib.qmlp_layers_workspace_bytes(big, 41, 1, 0) == 1024 + r256(40 * 16 * 4) + r256(40 * 512 * 2)
    # bfloat16 runs qmlp_forward per block
    assert lib.qmlp_layers_workspace_bytes(arr, 2, 128, 1) == lib.qmlp_workspace_bytes(ctypes.byref(m), 128, 1)
    assert lib.qmlp_layers_launches(arr, 2, 128, 1) == 2 * lib.qmlp_forward_launches(ctypes.byref(m), 128, 1)


def _variant(q, bg=2, gg=64, bd=4, gd=64, d=256, f=512, rank=8):
    m = _mlp(q, d=d, f=f, rank=rank)
    m.gate.bits = m.up.bits = bg
    m.gate.group = m.up.group = gg
    m.down.bits, m.down.group = bd, gd
    return m


def test_precision_variants_validation(q, lib):
    """Uniform W4, uniform W2 and 2-bit group 32 (Sec. 5.2, Sec. 3.3) are
    accepted on the binary16 decode path and run on the stand-alone kernels
    (never the one-kernel layer); they are rejected on the prefill path, by
    qmlp_gateup_w2_lora at 4 bits, and in a stack mixing widths."""
    P = ctypes.c_void_p
    for kw in (dict(bg=4, gg=128, bd=4, gd=128), dict(bg=2, bd=2), dict(bg=2, gg=32),
               dict(bg=4, gg=32, bd=4, gd=32)):
        m = _variant(q, **kw)
        assert lib.qmlp_workspace_bytes(ctypes.byref(m), 1, 0) > 0, kw
        assert lib.qmlp_forward_launches(ctypes.byref(m), 1, 0) == 3, kw    # LoRA-A, gate/up, down
        m.rank = 0
        assert lib.qmlp_forward_launches(ctypes.byref(m), 4, 0) == 2, kw
        assert lib.qmlp_workspace_bytes(ctypes.byref(m), 256, 1) == 0, kw   # no prefill form
        assert _fwd(lib, m, M=256, dtype=1) == UNSUP, kw
        assert _fwd(lib, m, M=0) == OK
    w4 = _variant(q, bg=4)
    assert lib.qmlp_gateup_w2_lora(ctypes.byref(w4), P(FAKE), 1, 0, P(FAKE), P(FAKE), 1 << 30,
                                   None) == UNSUP
    g32 = _variant(q, gg=32)
    assert lib.qmlp_gateup_w2_lora(ctypes.byref(g32), P(FAKE), 1, 0, P(FAKE), P(0), 1 << 30,
                                   None) == WS
    assert _fwd(lib, _variant(q, bg=4, gg=128, d=320), M=1) == SHAPE   # d not a multiple of g
    # the 4-bit down entry takes group 32 on the decode path, not on the prefill path
    w = _qw(q, bits=4, n=256, k=512, g=32)
    assert lib.qmlp_down_w4(ctypes.byref(w), None, 1, 0, P(FAKE), None) == NULL
    assert lib.qmlp_down_w4(ctypes.byref(w), P(FAKE), 128, 1, P(FAKE), None) == UNSUP
    # pack at group 32
    out = _qw(q)
    assert lib.qmlp_pack_w2(P(FAKE), 16, 200, 32, ctypes.byref(out), None, None) == SHAPE
    # every block of a stack / layer list has the same widths
    mixed = _stack_arr(q, _mlp(q), _variant(q, bg=4))
    assert lib.qmlp_forward_layers(mixed, 2, P(FAKE), 1, 0, P(FAKE), P(FAKE), 1 << 30, None) == SHAPE
    same = _stack_arr(q, _variant(q, bg=4, rank=0), _variant(q, bg=4, rank=0))
    assert lib.qmlp_layers_launches(same, 2, 1, 0) == 2               # one batch, no LoRA-A


def test_batch_validation(q, lib):
    """qmlp_forward_batch: binary16 only; workspace = control block + t + h of
    at most 40 blocks."""
    P = ctypes.c_void_p
    arr = _stack_arr(q, _mlp(q), _mlp(q), _mlp(q))

    def fb(a, L, M=1, dt=0, x=FAKE, y=FAKE, ws=FAKE, wsb=1 << 30):
        return lib.qmlp_forward_batch(a, L, P(x), M, dt, P(y), P(ws), wsb, None)

    assert lib.qmlp_forward_batch(None, 3, None, 1, 0, None, None, 0, None) == NULL
    assert fb(arr, 0) == SHAPE
    assert fb(arr, 3, dt=1, M=128) == UNSUP
    assert fb(arr, 3, x=0) == NULL
    assert fb(arr, 3, y=FAKE + 4) == ALIGN
    assert fb(arr, 3, M=0) == OK
    need = lib.qmlp_batch_workspace_bytes(arr, 3, 2, 0)
    assert need == 1024 + 512 + 3 * 2 * 512 * 2            # t: 3 x 2 x 16 fp32 in 256-B units
    assert fb(arr, 3, M=2, wsb=need - 1) == WS
    assert fb(arr, 3, M=2, ws=FAKE + 16 * 3 + 8) == ALIGN
    assert lib.qmlp_batch_workspace_bytes(arr, 3, 128, 1) == 0
    mixed = _stack_arr(q, _mlp(q), _variant(q, bd=2))
    assert fb(mixed, 2) == SHAPE


def test_three_bit_validation(q, lib):
    """3-bit codes (Appendix B): two-plane rows of a multiple of 128 codes, for
    gate/up only, on the binary16 decode path; not through the 2-bit entry."""
    P = ctypes.c_void_p
    assert lib.qmlp_codes_bytes(3, 9728, 2560) == 9728 * 2560 * 3 // 8
    assert lib.qmlp_codes_bytes(3, 16, 96) == 0                   # not whole 128-code runs
    out = _qw(q)
    assert lib.qmlp_pack_w3(P(FAKE), 16, 96, 32, ctypes.byref(out), None, None) == SHAPE
    assert lib.qmlp_pack_w3(P(FAKE), 16, 256, 48, ctypes.byref(out), None, None) == UNSUP
    w3 = _variant(q, bg=3, gg=32)
    assert lib.qmlp_workspace_bytes(ctypes.byref(w3), 1, 0) > 0
    assert lib.qmlp_forward_launches(ctypes.byref(w3), 1, 0) == 3
    assert _fwd(lib, w3, M=256, dtype=1) == UNSUP
    assert lib.qmlp_gateup_w2_lora(ctypes.byref(w3), P(FAKE), 1, 0, P(FAKE), P(FAKE), 1 << 30,
                                   None) == UNSUP
    d3 = _variant(q, bd=3)
    assert _fwd(lib, d3) == UNSUP
    odd = _variant(q, bg=3, gg=32, d=320)                        # 320 codes: not whole 128-code runs
    assert _fwd(lib, odd) == SHAPE


def test_linear_batch_validation(q, lib):
    """qmlp_linear_batch: 1..40 linears of one shape and width (4, or 2 at
    group 64/128), binary16 decode, n and k multiples of 64."""
    P = ctypes.c_void_p

    def arr(*ws):
        return (q.QWeightC * len(ws))(*ws)

    w = _qw(q, bits=4, n=512, k=256)
    assert lib.qmlp_linear_batch(None, 1, P(FAKE), 1, 0, P(FAKE), None) == NULL
    assert lib.qmlp_linear_batch(arr(w), 0, P(FAKE), 1, 0, P(FAKE), None) == SHAPE
    assert lib.qmlp_linear_batch(arr(*[w] * 41), 41, P(FAKE), 1, 0, P(FAKE), None) == SHAPE
    assert lib.qmlp_linear_batch(arr(w, _qw(q, bits=4, n=448, k=256)), 2, P(FAKE), 1, 0, P(FAKE),
                                 None) == SHAPE
    assert lib.qmlp_linear_batch(arr(w), 1, P(FAKE), 17, 0, P(FAKE), None) == UNSUP
    assert lib.qmlp_linear_batch(arr(w), 1, P(FAKE), 1, 1, P(FAKE), None) == UNSUP
    assert lib.qmlp_linear_batch(arr(_qw(q, bits=3, n=512, k=256)), 1, P(FAKE), 1, 0, P(FAKE),
                                 None) == UNSUP
    assert lib.qmlp_linear_batch(arr(_qw(q, bits=2, n=512, k=256, g=32)), 1, P(FAKE), 1, 0,
                                 P(FAKE), None) == UNSUP
    assert lib.qmlp_linear_batch(arr(w), 1, None, 1, 0, P(FAKE), None) == NULL
    assert lib.qmlp_linear_batch(arr(w), 1, P(FAKE + 8), 1, 0, P(FAKE), None) == ALIGN
    assert lib.qmlp_linear_batch(arr(w), 1, P(FAKE), 0, 0, P(FAKE), None) == OK


def test_moe_validation(q, lib):
    """qmlp_forward_moe: 1..40 experts of one shape, 1 <= k <= E, M*k <= 40,
    binary16; routing arrays are device pointers checked for NULL and
    alignment only."""
    P = ctypes.c_void_p
    E = 8
    arr = _stack_arr(q, *[_mlp(q) for _ in range(E)])

    def fm(a, n, M=1, k=2, x=FAKE, idx=FAKE, w=FAKE, y=FAKE, ws=FAKE, wsb=1 << 30, dt=0):
        return lib.qmlp_forward_moe(a, n, P(x), M, dt, P(idx), P(w), k, P(y), P(ws), wsb, None)

    assert fm(arr, E, k=0) == SHAPE
    assert fm(arr, E, k=9) == SHAPE
    assert fm(arr, E, M=-1) == SHAPE
    assert fm(arr, E, M=17) == UNSUP
    assert fm(arr, E, M=11, k=4) == UNSUP                    # 44 instances
    assert fm(arr, E, dt=1) == UNSUP
    assert fm(arr, E, M=0) == OK
    assert fm(arr, E, idx=0) == NULL
    assert fm(arr, E, w=FAKE + 2) == ALIGN
    need = lib.qmlp_moe_workspace_bytes(arr, E, 3, 2, 0)
    r256 = lambda v: (v + 255) // 256 * 256
    # control block, t as tagged 64-bit words, h, the instances' outputs
    assert need == 1024 + r256(6 * 16 * 8) + r256(6 * 512 * 2) + r256(6 * 256 * 2)
    assert fm(arr, E, M=3, wsb=need - 1) == WS
    big = _stack_arr(q, *[_mlp(q) for _ in range(41)])
    assert fm(big, 41) == SHAPE
    odd = _stack_arr(q, _mlp(q), _mlp(q, d=320, f=448))
    assert fm(odd, 2, k=1) == SHAPE


def test_stream_probe_validation(lib):
    P = ctypes.c_void_p
    f = lib.qmlp_probe_stream_read
    assert f(None, 1 << 20, P(FAKE), 256, 1, None) == NULL
    assert f(P(FAKE), 1 << 20, None, 256, 1, None) == NULL
    assert f(P(FAKE), 0, P(FAKE), 256, 1, None) == SHAPE
    assert f(P(FAKE), (1 << 20) + 8, P(FAKE), 256, 1, None) == SHAPE      # not whole 16-byte units
    assert f(P(FAKE), 1 << 20, P(FAKE), 0, 1, None) == SHAPE
    assert f(P(FAKE), 1 << 20, P(FAKE), 65537, 0, None) == SHAPE
    assert f(P(FAKE + 8), 1 << 20, P(FAKE), 256, 1, None) == ALIGN
    assert f(P(FAKE), 1 << 20, P(FAKE + 2), 256, 1, None) == ALIGN


def test_noalloc_validation(q, lib):
    """The no-allocation entry checks as qmlp_forward does, then rejects
    blocks whose workspace exceeds its array, before any HIP call."""
    assert lib.qmlp_noalloc_scratch_bytes() == 1 << 20
    m = _mlp(q)
    P = ctypes.c_void_p
    f = lib.qmlp_forward_noalloc
    assert f(None, P(FAKE), 1, 0, P(FAKE), None) == NULL
    assert f(ctypes.byref(m), None, 1, 0, P(FAKE), None) == NULL
    assert f(ctypes.byref(m), P(FAKE + 4), 1, 0, P(FAKE), None) == ALIGN
    assert f(ctypes.byref(m), P(FAKE), 0, 0, P(FAKE), None) == OK           # M = 0: nothing to do
    assert f(ctypes.byref(m), P(FAKE), 17, 0, P(FAKE), None) != OK
    big = q.MlpC(_qw(q, 2, 32768, 8192, 128), _qw(q, 2, 32768, 8192, 128), _qw(q, 4, 8192, 32768, 128),
                 FAKE, FAKE, FAKE, FAKE, 32, 1.0)
    assert lib.qmlp_workspace_bytes(ctypes.byref(big), 7, 0) <= 1 << 20
    assert lib.qmlp_workspace_bytes(ctypes.byref(big), 8, 0) > 1 << 20
    assert f(ctypes.byref(big), P(FAKE), 8, 0, P(FAKE), None) == WS
    assert f(ctypes.byref(big), P(FAKE), 8, 1, P(FAKE), None) == UNSUP     # bfloat16


@pytest.mark.parametrize("d,f,gu_bits,dn_bits,M,k,cus,want", [
    # GPT-OSS-20B-class experts, top-4, one token, 256 compute units:
    # W4/W2-GateUp gate/up 8 -> 16 lanes; down forms the routing sum at the
    # fewest lanes with at most three units each (W4: 90 units -> 32 lanes)
    (2880, 2880, 2, 4, 1, 4, 256, (16, 32, "sum")),
    (2880, 2880, 2, 2, 1, 4, 256, (16, 16, "sum")),    # uniform W2 down: 45 units -> 16
    (2880, 2880, 4, 4, 1, 4, 256, (16, 32, "sum")),    # uniform W4 gate/up keeps 16
    (1024, 768, 2, 4, 1, 1, 256, (16, 8, "sum")),
    (1024, 768, 2, 4, 1, 2, 256, (16, 8, "sum")),
    (2048, 768, 2, 4, 1, 2, 256, (32, 8, "sum")),      # gate/up: one 16-byte unit per lane
    # the gate/up rule counts the device's compute units, not a fixed 256
    (2880, 2880, 2, 4, 1, 4, 80, (8, 32, "sum")),
    # enough instances to fill the chip: no doubling
    (2880, 2880, 2, 4, 10, 4, 256, (8, 32, "sum")),
    # past four slots: the pipelined down kernel (its lanes double while the
    # grid has fewer than two workgroups per CU) and a combine launch
    (2880, 2880, 2, 4, 1, 5, 256, (16, 64, "pipe")),
    (2880, 2880, 2, 4, 8, 5, 256, (8, 16, "pipe")),
    # f past the folded kernel's staging at k = 4 (U = 128 units of 4 bits);
    # 4096 gate/up rows at 8 lanes are already 512 workgroups: no doubling
    (2880, 4096, 2, 4, 1, 4, 256, (8, 64, "pipe")),
])
def test_moe_lane_choice(q, d, f, gu_bits, dn_bits, M, k, cus, want):
    """The lanes per row of qmlp_forward_moe's launches (host-only query)."""
    assert q.moe_lanes(d, f, gu_bits, dn_bits, M, k, cus) == want


def test_moe_lane_choice_rejects(q, lib):
    g, dn = ctypes.c_int(0), ctypes.c_int(0)
    for args in [(2880, 2880, 3, 4, 1, 4, 256), (2880, 2880, 2, 4, 0, 4, 256), (2880, 2880, 2, 4, 1, 0, 256),
                 (2880, 2880, 2, 4, 9, 5, 256), (2880, 2880, 2, 4, 1, 4, 0), (2890, 2880, 2, 4, 1, 4, 256)]:
        assert lib.qmlp_moe_lanes(*args, ctypes.byref(g), ctypes.byref(dn)) == -1
    assert lib.qmlp_moe_lanes(2880, 2880, 2, 4, 1, 4, 256, None, ctypes.byref(dn)) == -1
