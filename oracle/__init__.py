"""fp64 CPU oracle for the W4/W2-GateUp decode MLP -- TEST INFRASTRUCTURE ONLY.

Only the test-suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never touches it and shares no code with it.

The arithmetic lives in ``qmlp_oracle.c`` (plain C, fp64, no FMA contraction);
this module only marshals numpy arrays through ctypes.  Every function cites
the passage of the paper it follows in the C source:

* quantizer (Sec. 3.3, Sec. 4.1: INT2 gate/up, INT4 down, group-wise along the
  input dimension; round-to-nearest min-max with an integer zero point and
  fp16 scale/zero is this library's reading);
* dequantization (Sec. 6.3, quantize-dequantize semantics);
* LoRA-augmented linear (Sec. 3.1, Eq. (1)), adapters kept unmerged (Sec. 4.2);
* fused gate-activation-down with an fp64, unrounded intermediate (Sec. 5);
* the decoder context of a stack of blocks: unit-gain RMSNorm of the
  residual stream before each block and the residual add after it.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libqmlp_oracle.so")
SRC_PATH = os.path.join(_HERE, "qmlp_oracle.c")

_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    # QMLP_ORACLE_LIB points the pins at a deliberately broken copy of the
    # oracle (the mutation test); normally unset.
    path = os.environ.get("QMLP_ORACLE_LIB", LIB_PATH)
    if path == LIB_PATH and (not os.path.exists(LIB_PATH)
                             or os.path.getmtime(LIB_PATH) < os.path.getmtime(SRC_PATH)):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    L = ctypes.c_long
    I = ctypes.c_int
    D = ctypes.c_double
    lib.orc_f16_to_f64.restype = D
    lib.orc_f16_to_f64.argtypes = [ctypes.c_uint16]
    lib.orc_bf16_to_f64.restype = D
    lib.orc_bf16_to_f64.argtypes = [ctypes.c_uint16]
    lib.orc_f64_to_f16.restype = ctypes.c_uint16
    lib.orc_f64_to_f16.argtypes = [D]
    lib.orc_quantize.restype = L
    lib.orc_quantize.argtypes = [P, L, L, L, I, P, P, P]
    lib.orc_pack.restype = None
    lib.orc_pack.argtypes = [P, L, L, I, P]
    lib.orc_unpack.restype = None
    lib.orc_unpack.argtypes = [P, L, L, I, P]
    lib.orc_meta_interleave.restype = None
    lib.orc_meta_interleave.argtypes = [P, P, L, P]
    lib.orc_dequant.restype = None
    lib.orc_dequant.argtypes = [P, P, P, L, L, L, P]
    lib.orc_dequant_f16.restype = None
    lib.orc_dequant_f16.argtypes = [P, P, P, L, L, L, P]
    lib.orc_lora_a.restype = None
    lib.orc_lora_a.argtypes = [P, P, L, L, L, I, P]
    lib.orc_gateup.restype = I
    lib.orc_gateup.argtypes = [L, L, L, L] + [P] * 6 + [P] * 4 + [L, D, I, P, P, P, P]
    lib.orc_down.restype = I
    lib.orc_down.argtypes = [L, L, L, L, P, P, P, P, P]
    lib.orc_down_act.restype = I
    lib.orc_down_act.argtypes = [L, L, L, L, P, P, P, P, I, P]
    lib.orc_forward.restype = I
    lib.orc_forward.argtypes = [L, L, L, L, L] + [P] * 9 + [P] * 4 + [L, D, I, P, P, P]
    lib.orc_rmsnorm_f16.restype = None
    lib.orc_rmsnorm_f16.argtypes = [P, L, L, D, P]
    lib.orc_residual_f16.restype = None
    lib.orc_residual_f16.argtypes = [P, P, L, P]
    _lib = lib
    return lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


# ---------------------------------------------------------------- conversions
def f16_to_f64(bits) -> float:
    return _load().orc_f16_to_f64(int(bits))


def bf16_to_f64(bits) -> float:
    return _load().orc_bf16_to_f64(int(bits))


def f64_to_f16(v) -> int:
    return int(_load().orc_f64_to_f16(float(v)))


_TABLES = {}


def act_to_f64(bits: np.ndarray, bf16: bool) -> np.ndarray:
    """Activation bits (uint16) -> exact float64 values (table built from the C routine)."""
    if bf16 not in _TABLES:
        lib = _load()
        conv = lib.orc_bf16_to_f64 if bf16 else lib.orc_f16_to_f64
        _TABLES[bf16] = np.array([conv(i) for i in range(65536)], dtype=np.float64)
    flat = np.asarray(bits, dtype=np.uint16).ravel()
    return _TABLES[bf16][flat].reshape(np.shape(bits))


# ---------------------------------------------------------------- quantizer
class QTensor:
    """Oracle-side quantized matrix: canonical codes + separate scale/zero."""

    def __init__(self, codes, scale, zero, bits, group, bad):
        self.codes = codes      # uint8 [n][k]
        self.scale = scale      # uint16 (binary16 bits) [n][k/g]
        self.zero = zero        # uint16 (binary16 bits) [n][k/g]
        self.bits = bits
        self.group = group
        self.bad = bad          # number of invalid groups

    @property
    def shape(self):
        return self.codes.shape

    def packed(self) -> np.ndarray:
        return pack(self.codes, self.bits)

    def meta(self) -> np.ndarray:
        return meta_interleave(self.scale, self.zero)

    def dequant(self) -> np.ndarray:
        return dequant(self)

    def dequant_f16(self) -> np.ndarray:
        return dequant_f16(self)


def quantize(W: np.ndarray, bits: int, group: int) -> QTensor:
    """Group-wise RTN min-max quantization of fp32 W [n][k] (see qmlp_oracle.c)."""
    W = _c(W, np.float32)
    n, k = W.shape
    if k % group:
        raise ValueError("k must be a multiple of the group size")
    codes = np.empty((n, k), np.uint8)
    scale = np.empty((n, k // group), np.uint16)
    zero = np.empty((n, k // group), np.uint16)
    bad = _load().orc_quantize(_p(W), n, k, group, bits, _p(codes), _p(scale), _p(zero))
    return QTensor(codes, scale, zero, bits, group, int(bad))


def pack(codes: np.ndarray, bits: int) -> np.ndarray:
    """Codes [n][k] -> the packed words of the storage format (see qmlp_oracle.c;
    at 3 bits the two-plane layout, k a multiple of 64)."""
    codes = _c(codes, np.uint8)
    n, k = codes.shape
    if bits == 3 and k % 64:
        raise ValueError("3-bit rows hold a multiple of 64 codes")
    words = np.empty((n, k * bits // 32), np.uint32)
    _load().orc_pack(_p(codes), n, k, bits, _p(words))
    return words


def unpack(words: np.ndarray, k: int, bits: int) -> np.ndarray:
    words = _c(words, np.uint32)
    n = words.shape[0]
    codes = np.empty((n, k), np.uint8)
    _load().orc_unpack(_p(words), n, k, bits, _p(codes))
    return codes


def meta_interleave(scale: np.ndarray, zero: np.ndarray) -> np.ndarray:
    scale = _c(scale, np.uint16)
    zero = _c(zero, np.uint16)
    meta = np.empty(scale.shape + (2,), np.uint16)
    _load().orc_meta_interleave(_p(scale), _p(zero), scale.size, _p(meta))
    return meta


def dequant(q: QTensor) -> np.ndarray:
    n, k = q.codes.shape
    w = np.empty((n, k), np.float64)
    _load().orc_dequant(_p(q.codes), _p(q.scale), _p(q.zero), n, k, q.group, _p(w))
    return w


def dequant_f16(q: QTensor) -> np.ndarray:
    n, k = q.codes.shape
    w = np.empty((n, k), np.uint16)
    _load().orc_dequant_f16(_p(q.codes), _p(q.scale), _p(q.zero), n, k, q.group, _p(w))
    return w


# ---------------------------------------------------------------- forward
def lora_a(A: np.ndarray, x: np.ndarray, bf16: bool = False) -> np.ndarray:
    A = _c(A, np.uint16)
    x = _c(x, np.uint16)
    r, d = A.shape
    M = x.shape[0]
    t = np.empty((M, r), np.float64)
    _load().orc_lora_a(_p(A), _p(x), M, d, r, int(bf16), _p(t))
    return t


def gateup(qg: QTensor, qu: QTensor, Ag, Bg, Au, Bu, x, lora_scale=1.0, bf16=False,
           return_gu=False):
    """h = SiLU(W2g x + s B_g A_g x) * (W2u x + s B_u A_u x), fp64 [M][f]."""
    f, d = qg.shape
    x = _c(x, np.uint16)
    M = x.shape[0]
    rank = 0 if Ag is None else Ag.shape[0]
    Ag = _c(Ag, np.uint16) if rank else None
    Bg = _c(Bg, np.uint16) if rank else None
    Au = _c(Au, np.uint16) if rank else None
    Bu = _c(Bu, np.uint16) if rank else None
    h = np.empty((M, f), np.float64)
    G = np.empty((M, f), np.float64)
    U = np.empty((M, f), np.float64)
    rc = _load().orc_gateup(M, d, f, qg.group, _p(qg.codes), _p(qg.scale), _p(qg.zero),
                            _p(qu.codes), _p(qu.scale), _p(qu.zero),
                            _p(Ag), _p(Bg), _p(Au), _p(Bu), rank, float(lora_scale), int(bf16),
                            _p(x), _p(h), _p(G), _p(U))
    if rc:
        raise MemoryError("oracle gateup failed")
    return (h, G, U) if return_gu else h


def down(qd: QTensor, h: np.ndarray) -> np.ndarray:
    """y = W4down h on an fp64 intermediate h [M][f]."""
    d, f = qd.shape
    h = _c(h, np.float64)
    M = h.shape[0]
    y = np.empty((M, d), np.float64)
    rc = _load().orc_down(M, d, f, qd.group, _p(qd.codes), _p(qd.scale), _p(qd.zero), _p(h), _p(y))
    if rc:
        raise MemoryError("oracle down failed")
    return y


def down_act(qd: QTensor, h_bits: np.ndarray, bf16: bool = False) -> np.ndarray:
    """y = W4down h with h given as activation bits [M][f]."""
    d, f = qd.shape
    h_bits = _c(h_bits, np.uint16)
    M = h_bits.shape[0]
    y = np.empty((M, d), np.float64)
    rc = _load().orc_down_act(M, d, f, qd.group, _p(qd.codes), _p(qd.scale), _p(qd.zero),
                              _p(h_bits), int(bf16), _p(y))
    if rc:
        raise MemoryError("oracle down failed")
    return y


def forward(qg: QTensor, qu: QTensor, qd: QTensor, Ag, Bg, Au, Bu, x, lora_scale=1.0,
            bf16=False, return_h=False):
    """y = W4down(SiLU(G) * U) in fp64 [M][d]; optionally the fp64 intermediate."""
    f, d = qg.shape
    x = _c(x, np.uint16)
    M = x.shape[0]
    rank = 0 if Ag is None else Ag.shape[0]
    Ag = _c(Ag, np.uint16) if rank else None
    Bg = _c(Bg, np.uint16) if rank else None
    Au = _c(Au, np.uint16) if rank else None
    Bu = _c(Bu, np.uint16) if rank else None
    y = np.empty((M, d), np.float64)
    h = np.empty((M, f), np.float64) if return_h else None
    rc = _load().orc_forward(M, d, f, qg.group, qd.group,
                             _p(qg.codes), _p(qg.scale), _p(qg.zero),
                             _p(qu.codes), _p(qu.scale), _p(qu.zero),
                             _p(qd.codes), _p(qd.scale), _p(qd.zero),
                             _p(Ag), _p(Bg), _p(Au), _p(Bu), rank, float(lora_scale), int(bf16),
                             _p(x), _p(y), _p(h))
    if rc:
        raise MemoryError("oracle forward failed")
    return (y, h) if return_h else y


def moe_forward(experts, topk_idx, topk_w, x, lora_scale=1.0):
    """The routed-expert MLP (Sec. 5, the MoE decoder): token m's output is
    sum_j topk_w[m][j] * forward(expert topk_idx[m][j], x[m]) in fp64.
    experts: list of (qg, qu, qd, Ag, Bg, Au, Bu); x [M][d] binary16 bits."""
    x = _c(x, np.uint16)
    M = x.shape[0]
    y = None
    for m in range(M):
        ym = 0.0
        for e, w in zip(np.asarray(topk_idx)[m], np.asarray(topk_w, np.float64)[m]):
            qg, qu, qd, Ag, Bg, Au, Bu = experts[int(e)]
            ym = ym + w * forward(qg, qu, qd, Ag, Bg, Au, Bu, x[m:m + 1], lora_scale=lora_scale)[0]
        y = np.empty((M, ym.shape[0]), np.float64) if y is None else y
        y[m] = ym
    return y


def max_rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    """max |got - ref| / max |ref| over all elements, in fp64."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.max(np.abs(ref))
    return float(np.max(np.abs(got - ref)) / den) if den > 0 else float(np.max(np.abs(got)))


# ---------------------------------------------------------------- stack context
RMS_EPS = 1e-6


def rmsnorm_f16(x: np.ndarray, eps: float = RMS_EPS) -> np.ndarray:
    """u = x / sqrt(mean(x^2) + eps) per row, binary16 bits in and out."""
    x = _c(x, np.uint16)
    M, d = x.reshape(-1, x.shape[-1]).shape
    u = np.empty_like(x)
    _load().orc_rmsnorm_f16(_p(x), M, d, float(eps), _p(u))
    return u


def residual_f16(x: np.ndarray, y: np.ndarray) -> np.ndarray:
    """x + y of binary16 bits, rounded once."""
    x = _c(x, np.uint16)
    y = _c(y, np.uint16)
    out = np.empty_like(x)
    _load().orc_residual_f16(_p(x), _p(y), x.size, _p(out))
    return out
