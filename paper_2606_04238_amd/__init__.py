"""Python binding of libqmlp, the MI355X (gfx950) W4/W2-GateUp decode-MLP library.

Argument marshalling only: every step of the hot path runs in the HIP
kernels behind ``include/qmlp.h``.  PyTorch provides device memory and the
current stream.  The module fails loudly if the built library is missing;
there is no CPU fallback.

Functions keep the names of the C entry points:

* ``pack_w2`` / ``pack_w4``       -- quantize fp32 weights to packed 2/4-bit (Sec. 4.1, Sec. 7)
* ``gateup_w2_lora``              -- h = SiLU(W2g x + s B_g A_g x) * (W2u x + s B_u A_u x)
* ``down_w4``                     -- y = W4down h
* ``forward``                     -- the whole block x -> y
* ``forward_layers``              -- L independent blocks, y_l = block_l(x_l)
* ``forward_stack``               -- L blocks on a residual stream, x_{l+1} = x_l + block_l(RMSNorm(x_l))
* ``unpack`` / ``dequant``        -- inspection of a packed matrix (not timed)
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# QMLP_LIB_PATH: another build of the same sources (the host-sanitized one
# of build.py --host-sanitize); by default the library next to this file
LIB_PATH = os.environ.get("QMLP_LIB_PATH") or os.path.join(_HERE, "libqmlp.so")

F16, BF16 = 0, 1
_STATUS = {0: "QMLP_OK", 1: "QMLP_ERR_NULL", 2: "QMLP_ERR_SHAPE", 3: "QMLP_ERR_ALIGN",
           4: "QMLP_ERR_UNSUPPORTED", 5: "QMLP_ERR_WORKSPACE", 6: "QMLP_ERR_HIP"}


class QmlpError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s: %s (%s)" % (where, _STATUS.get(status, status),
                                          _lib().qmlp_status_string(status).decode()))


class QWeightC(ctypes.Structure):
    _fields_ = [("bits", ctypes.c_int32), ("n_out", ctypes.c_int32), ("k_in", ctypes.c_int32),
                ("group", ctypes.c_int32), ("codes", ctypes.c_void_p), ("meta", ctypes.c_void_p)]


class MlpC(ctypes.Structure):
    _fields_ = [("gate", QWeightC), ("up", QWeightC), ("down", QWeightC),
                ("A_gate", ctypes.c_void_p), ("B_gate", ctypes.c_void_p),
                ("A_up", ctypes.c_void_p), ("B_up", ctypes.c_void_p),
                ("rank", ctypes.c_int32), ("lora_scale", ctypes.c_float)]


_LIB = None


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libqmlp.so is not built (run __graft_entry__.build()); "
                              "there is no fallback path: %s" % LIB_PATH)
        lib = ctypes.CDLL(LIB_PATH)
        P, I, Z = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
        pq = ctypes.POINTER(QWeightC)
        pm = ctypes.POINTER(MlpC)
        sig = {
            "qmlp_codes_bytes": (Z, [I, I, I]),
            "qmlp_meta_bytes": (Z, [I, I, I]),
            "qmlp_workspace_bytes": (Z, [pm, I, I]),
            "qmlp_pack_w2": (I, [P, I, I, I, pq, P, P]),
            "qmlp_pack_w3": (I, [P, I, I, I, pq, P, P]),
            "qmlp_pack_w4": (I, [P, I, I, I, pq, P, P]),
            "qmlp_gateup_w2_lora": (I, [pm, P, I, I, P, P, Z, P]),
            "qmlp_down_w4": (I, [pq, P, I, I, P, P]),
            "qmlp_forward": (I, [pm, P, I, I, P, P, Z, P]),
            "qmlp_unpack": (I, [pq, P, P, P, P]),
            "qmlp_dequant": (I, [pq, P, P]),
            "qmlp_forward_launches": (I, [pm, I, I]),
            "qmlp_stack_workspace_bytes": (Z, [pm, I, I, I]),
            "qmlp_forward_stack": (I, [pm, I, P, I, I, P, P, P, Z, P]),
            "qmlp_stack_launches": (I, [pm, I, I, I]),
            "qmlp_stack_error_offset": (Z, [pm, I, I, I]),
            "qmlp_moe_lanes": (I, [I, I, I, I, I, I, I, ctypes.POINTER(I), ctypes.POINTER(I)]),
            "qmlp_layers_workspace_bytes": (Z, [pm, I, I, I]),
            "qmlp_forward_layers": (I, [pm, I, P, I, I, P, P, Z, P]),
            "qmlp_layers_launches": (I, [pm, I, I, I]),
            "qmlp_batch_workspace_bytes": (Z, [pm, I, I, I]),
            "qmlp_linear_batch": (I, [ctypes.POINTER(QWeightC), I, P, I, I, P, P]),
            "qmlp_moe_workspace_bytes": (Z, [pm, I, I, I, I]),
            "qmlp_forward_moe": (I, [pm, I, P, I, I, P, P, I, P, P, Z, P]),
            "qmlp_forward_batch": (I, [pm, I, P, I, I, P, P, Z, P]),
            "qmlp_status_string": (ctypes.c_char_p, [I]),
            "qmlp_probe_stream_read": (I, [P, Z, P, I, I, P]),
            "qmlp_forward_noalloc": (I, [pm, P, I, I, P, P]),
            "qmlp_layers_path": (I, [pm, I, I, I]),
            "qmlp_noalloc_scratch_bytes": (Z, []),
        }
        for name, (res, args) in sig.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = lib
    return _LIB


def library():
    """The loaded ctypes library (raises if it is not built)."""
    return _lib()


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _check(status: int, where: str):
    if status != 0:
        raise QmlpError(status, where)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float16:
        return F16
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError("activations must be float16 or bfloat16, got %s" % t.dtype)


def codes_bytes(bits: int, n_out: int, k_in: int) -> int:
    return int(_lib().qmlp_codes_bytes(bits, n_out, k_in))


def meta_bytes(n_out: int, k_in: int, group: int) -> int:
    return int(_lib().qmlp_meta_bytes(n_out, k_in, group))


class QWeight:
    """A packed quantized matrix: device tensors ``codes`` and ``meta`` plus its C view."""

    def __init__(self, bits, n_out, k_in, group, codes, meta, status=None):
        self.bits, self.n_out, self.k_in, self.group = bits, n_out, k_in, group
        self.codes = codes          # uint8 device tensor, codes_bytes() long
        self.meta = meta            # uint8 device tensor, meta_bytes() long
        self.status = status        # int32 device tensor set by the packer (bit 0: invalid group)

    def c(self) -> QWeightC:
        return QWeightC(self.bits, self.n_out, self.k_in, self.group,
                        self.codes.data_ptr(), self.meta.data_ptr())

    def invalid_groups(self) -> bool:
        """True if the packer flagged a non-finite weight or an overflowing scale (syncs)."""
        return bool(self.status is not None and int(self.status.item()) & 1)

    @property
    def nbytes(self) -> int:
        return self.codes.numel() + self.meta.numel()


def _pack(bits: int, W: torch.Tensor, group: int) -> QWeight:
    if W.dtype != torch.float32 or not W.is_cuda or W.dim() != 2:
        raise TypeError("W must be a 2-D float32 CUDA tensor")
    W = W.contiguous()
    n, k = W.shape
    cb, mb = codes_bytes(bits, n, k), meta_bytes(n, k, group)
    if cb == 0 or mb == 0:
        raise QmlpError(2, "pack_w%d" % bits)
    codes = torch.empty(cb, dtype=torch.uint8, device=W.device)
    meta = torch.empty(mb, dtype=torch.uint8, device=W.device)
    status = torch.zeros(1, dtype=torch.int32, device=W.device)
    qw = QWeightC(0, 0, 0, 0, codes.data_ptr(), meta.data_ptr())
    fn = {2: _lib().qmlp_pack_w2, 3: _lib().qmlp_pack_w3, 4: _lib().qmlp_pack_w4}[bits]
    _check(fn(_ptr(W), n, k, group, ctypes.byref(qw), _ptr(status), _stream()), "pack_w%d" % bits)
    return QWeight(qw.bits, qw.n_out, qw.k_in, qw.group, codes, meta, status)


def pack_w2(W: torch.Tensor, group: int) -> QWeight:
    """Quantize fp32 W [n][k] (device) to 2-bit codes + fp16 scale/zero per group."""
    return _pack(2, W, group)


def pack_w3(W: torch.Tensor, group: int) -> QWeight:
    """Quantize fp32 W [n][k] (device) to 3-bit codes (two-plane layout) + fp16 scale/zero."""
    return _pack(3, W, group)


def pack_w4(W: torch.Tensor, group: int) -> QWeight:
    """Quantize fp32 W [n][k] (device) to 4-bit codes + fp16 scale/zero per group."""
    return _pack(4, W, group)


class MLP:
    """One W4/W2-GateUp block with Recover-LoRA adapters (device tensors); the
    decode path also takes the uniform-W4 / uniform-W2 comparison widths and
    group 32 (see qmlp_mlp in include/qmlp.h)."""

    def __init__(self, gate: QWeight, up: QWeight, down: QWeight, A_gate=None, B_gate=None,
                 A_up=None, B_up=None, lora_scale: float = 1.0):
        self.gate, self.up, self.down = gate, up, down
        self.A_gate, self.B_gate, self.A_up, self.B_up = A_gate, B_gate, A_up, B_up
        self.rank = 0 if A_gate is None else int(A_gate.shape[0])
        self.lora_scale = float(lora_scale)
        self._c = MlpC(gate.c(), up.c(), down.c(), _ptr(A_gate), _ptr(B_gate), _ptr(A_up),
                       _ptr(B_up), self.rank, self.lora_scale)

    @property
    def d(self):
        return self.gate.k_in

    @property
    def f(self):
        return self.gate.n_out

    def c(self) -> MlpC:
        return self._c

    def with_lora_scale(self, lora_scale: float) -> "MLP":
        return MLP(self.gate, self.up, self.down, self.A_gate, self.B_gate, self.A_up, self.B_up,
                   lora_scale)


def workspace_bytes(mlp: MLP, M: int, dtype=torch.float16) -> int:
    code = F16 if dtype == torch.float16 else BF16
    return int(_lib().qmlp_workspace_bytes(ctypes.byref(mlp.c()), M, code))


def forward_launches(mlp: MLP, M: int, dtype=torch.float16) -> int:
    """Kernels qmlp_forward launches for this block at M tokens (1 = fused layer kernel)."""
    code = F16 if dtype == torch.float16 else BF16
    return int(_lib().qmlp_forward_launches(ctypes.byref(mlp.c()), M, code))


def workspace(mlp: MLP, M: int, dtype=torch.float16, device="cuda") -> torch.Tensor:
    """A zeroed workspace (it must start at zero; zero it again before it
    serves a block of another shape or after an error bit)."""
    n = workspace_bytes(mlp, M, dtype)
    return torch.zeros(max(n, 1024), dtype=torch.uint8, device=device)


def workspace_errors(ws: torch.Tensor) -> int:
    """Sticky error bits of a workspace's control block (syncs)."""
    return int(ws[640:644].view(torch.int32).item())


def gateup_w2_lora(mlp: MLP, x: torch.Tensor, h: torch.Tensor | None = None,
                   ws: torch.Tensor | None = None) -> torch.Tensor:
    M = x.shape[0]
    if h is None:
        h = torch.empty((M, mlp.f), dtype=x.dtype, device=x.device)
    if ws is None:
        ws = workspace(mlp, M, x.dtype, x.device)
    _check(_lib().qmlp_gateup_w2_lora(ctypes.byref(mlp.c()), _ptr(x), M, _dtype_code(x), _ptr(h),
                                      _ptr(ws), ws.numel(), _stream()), "gateup_w2_lora")
    return h


def down_w4(down: QWeight, h: torch.Tensor, y: torch.Tensor | None = None) -> torch.Tensor:
    M = h.shape[0]
    if y is None:
        y = torch.empty((M, down.n_out), dtype=h.dtype, device=h.device)
    qc = down.c()
    _check(_lib().qmlp_down_w4(ctypes.byref(qc), _ptr(h), M, _dtype_code(h), _ptr(y), _stream()),
           "down_w4")
    return y


def forward(mlp: MLP, x: torch.Tensor, y: torch.Tensor | None = None,
            ws: torch.Tensor | None = None) -> torch.Tensor:
    M = x.shape[0]
    if y is None:
        y = torch.empty((M, mlp.d), dtype=x.dtype, device=x.device)
    if ws is None:
        ws = workspace(mlp, M, x.dtype, x.device)
    _check(_lib().qmlp_forward(ctypes.byref(mlp.c()), _ptr(x), M, _dtype_code(x), _ptr(y),
                               _ptr(ws), ws.numel(), _stream()), "forward")
    return y


def forward_noalloc(mlp: MLP, x: torch.Tensor, y: torch.Tensor | None = None) -> torch.Tensor:
    """The whole block x -> y with the library's own per-GPU scratch array as
    workspace (qmlp_forward_noalloc): nothing is allocated by the call."""
    M = x.shape[0]
    if y is None:
        y = torch.empty((M, mlp.d), dtype=x.dtype, device=x.device)
    c = mlp.c()
    _check(_lib().qmlp_forward_noalloc(ctypes.byref(c), _ptr(x), M, _dtype_code(x), _ptr(y), _stream()),
           "qmlp_forward_noalloc")
    return y


def noalloc_scratch_bytes() -> int:
    return int(_lib().qmlp_noalloc_scratch_bytes())


def unpack(w: QWeight):
    """(codes uint8 [n][k], scale bits int16 [n][k/g], zero bits int16 [n][k/g]) on the device."""
    dev = w.codes.device
    codes = torch.empty((w.n_out, w.k_in), dtype=torch.uint8, device=dev)
    scales = torch.empty((w.n_out, w.k_in // w.group), dtype=torch.int16, device=dev)
    zeros = torch.empty_like(scales)
    qc = w.c()
    _check(_lib().qmlp_unpack(ctypes.byref(qc), _ptr(codes), _ptr(scales), _ptr(zeros), _stream()),
           "unpack")
    return codes, scales, zeros


def dequant(w: QWeight) -> torch.Tensor:
    """The dequantized weight as float16 [n][k] (one RNE rounding of scale*(q-zero))."""
    out = torch.empty((w.n_out, w.k_in), dtype=torch.float16, device=w.codes.device)
    qc = w.c()
    _check(_lib().qmlp_dequant(ctypes.byref(qc), _ptr(out), _stream()), "dequant")
    return out


class Layers:
    """L blocks of one shape; holds the C descriptor array that the
    multi-block entry points take."""

    def __init__(self, mlps):
        self.mlps = list(mlps)
        self._arr = (MlpC * len(self.mlps))(*[m.c() for m in self.mlps])

    def __len__(self):
        return len(self.mlps)

    def c(self):
        return self._arr


class Stack(Layers):
    """L blocks of one shape on a residual stream (x_{l+1} = x_l + y_l,
    y_l = block_l(RMSNorm(x_l)))."""


def layers_workspace_bytes(layers: Layers, M: int, dtype=torch.float16) -> int:
    code = F16 if dtype == torch.float16 else BF16
    return int(_lib().qmlp_layers_workspace_bytes(layers.c(), len(layers), M, code))


LAYERS_PATHS = {0: "rejected", 1: "streamed", 2: "batched", 3: "per-block", 4: "mfma"}


def layers_path(layers: Layers, M: int, dtype=torch.float16) -> str:
    """The path qmlp_forward_layers takes (qmlp_layers_path)."""
    code = F16 if dtype == torch.float16 else BF16
    return LAYERS_PATHS[int(_lib().qmlp_layers_path(layers.c(), len(layers), M, code))]


def layers_launches(layers: Layers, M: int, dtype=torch.float16) -> int:
    """Launches forward_layers makes (three per batch of up to 40 blocks on
    the streamed and batched paths, or those of one forward per block)."""
    code = F16 if dtype == torch.float16 else BF16
    return int(_lib().qmlp_layers_launches(layers.c(), len(layers), M, code))


def layers_workspace(layers: Layers, M: int, dtype=torch.float16, device="cuda") -> torch.Tensor:
    """A zeroed workspace for forward_layers."""
    n = layers_workspace_bytes(layers, M, dtype)
    return torch.zeros(max(n, 1024), dtype=torch.uint8, device=device)


def forward_layers(layers: Layers, x: torch.Tensor, y: torch.Tensor | None = None,
                   ws: torch.Tensor | None = None) -> torch.Tensor:
    """y [L][M][d]: y_l = block_l(x_l) for x [L][M][d], every block on its own input."""
    L, M, d = x.shape
    if L != len(layers) or d != layers.mlps[0].d:
        raise ValueError("x must be [L][M][d] for the L blocks")
    if y is None:
        y = torch.empty_like(x)
    if ws is None:
        ws = layers_workspace(layers, M, x.dtype, x.device)
    _check(_lib().qmlp_forward_layers(layers.c(), L, _ptr(x), M, _dtype_code(x), _ptr(y), _ptr(ws),
                                      ws.numel(), _stream()), "forward_layers")
    return y


def batch_workspace_bytes(layers: Layers, M: int, dtype=torch.float16) -> int:
    code = F16 if dtype == torch.float16 else BF16
    return int(_lib().qmlp_batch_workspace_bytes(layers.c(), len(layers), M, code))


def batch_workspace(layers: Layers, M: int, dtype=torch.float16, device="cuda") -> torch.Tensor:
    """A zeroed workspace for forward_batch."""
    n = batch_workspace_bytes(layers, M, dtype)
    return torch.zeros(max(n, 1024), dtype=torch.uint8, device=device)


def forward_batch(layers: Layers, x: torch.Tensor, y: torch.Tensor | None = None,
                  ws: torch.Tensor | None = None) -> torch.Tensor:
    """forward_layers on the stand-alone kernels whatever the shape: LoRA-A,
    gate/up and down of every block of a batch of up to 40, three launches."""
    L, M, d = x.shape
    if L != len(layers) or d != layers.mlps[0].d:
        raise ValueError("x must be [L][M][d] for the L blocks")
    if y is None:
        y = torch.empty_like(x)
    if ws is None:
        ws = batch_workspace(layers, M, x.dtype, x.device)
    _check(_lib().qmlp_forward_batch(layers.c(), L, _ptr(x), M, _dtype_code(x), _ptr(y), _ptr(ws),
                                     ws.numel(), _stream()), "forward_batch")
    return y


def linear_batch(ws, x: torch.Tensor, y: torch.Tensor | None = None) -> torch.Tensor:
    """y [L][M][n] = W_l x_l for L quantized linears of one shape (QWeight list)
    and x [L][M][k] binary16: one launch."""
    L, M, k = x.shape
    if L != len(ws) or k != ws[0].k_in:
        raise ValueError("x must be [L][M][k] for the L linears")
    if y is None:
        y = torch.empty((L, M, ws[0].n_out), dtype=x.dtype, device=x.device)
    arr = (QWeightC * L)(*[w.c() for w in ws])
    _check(_lib().qmlp_linear_batch(arr, L, _ptr(x), M, _dtype_code(x), _ptr(y), _stream()),
           "linear_batch")
    return y


def moe_workspace_bytes(experts: Layers, M: int, k: int, dtype=torch.float16) -> int:
    code = F16 if dtype == torch.float16 else BF16
    return int(_lib().qmlp_moe_workspace_bytes(experts.c(), len(experts), M, k, code))


def moe_lanes(d: int, f: int, gu_bits: int, dn_bits: int, M: int, k: int, cus: int):
    """(gate/up lanes per row, down lanes per row, down form) of
    qmlp_forward_moe's launches for M tokens with k experts each on `cus`
    compute units (qmlp_moe_lanes; host-only).  Down form: "sum" (the down
    launch forms the routing sum), "pipe" or "plain" (a combine follows)."""
    g, dn = ctypes.c_int(0), ctypes.c_int(0)
    r = int(_lib().qmlp_moe_lanes(d, f, gu_bits, dn_bits, M, k, cus, ctypes.byref(g), ctypes.byref(dn)))
    if r < 0:
        raise ValueError("qmlp_moe_lanes rejected its arguments")
    return g.value, dn.value, ("plain", "pipe", "sum")[r]


def forward_moe(experts: Layers, x: torch.Tensor, topk_idx: torch.Tensor, topk_w: torch.Tensor,
                y: torch.Tensor | None = None, ws: torch.Tensor | None = None) -> torch.Tensor:
    """y [M][d] = sum_j topk_w[m][j] * expert_{topk_idx[m][j]}(x[m]); topk_idx int32
    and topk_w float32 [M][k] on the device."""
    M, d = x.shape
    k = topk_idx.shape[1]
    if topk_idx.dtype != torch.int32 or topk_w.dtype != torch.float32 or topk_w.shape != topk_idx.shape:
        raise ValueError("topk_idx int32 and topk_w float32, both [M][k]")
    if y is None:
        y = torch.empty_like(x)
    if ws is None:
        ws = torch.zeros(max(moe_workspace_bytes(experts, M, k, x.dtype), 1024), dtype=torch.uint8,
                         device=x.device)
    _check(_lib().qmlp_forward_moe(experts.c(), len(experts), _ptr(x), M, _dtype_code(x),
                                   _ptr(topk_idx), _ptr(topk_w), k, _ptr(y), _ptr(ws), ws.numel(),
                                   _stream()), "forward_moe")
    return y


def stack_workspace_bytes(stack: Stack, M: int, dtype=torch.float16) -> int:
    code = F16 if dtype == torch.float16 else BF16
    return int(_lib().qmlp_stack_workspace_bytes(stack.c(), len(stack), M, code))


def stack_launches(stack: Stack, M: int, dtype=torch.float16) -> int:
    """Launches forward_stack makes (persistent launches, or the per-layer kernels)."""
    code = F16 if dtype == torch.float16 else BF16
    return int(_lib().qmlp_stack_launches(stack.c(), len(stack), M, code))


def stack_workspace(stack: Stack, M: int, dtype=torch.float16, device="cuda") -> torch.Tensor:
    """A zeroed workspace for forward_stack."""
    n = stack_workspace_bytes(stack, M, dtype)
    return torch.zeros(max(n, 1024), dtype=torch.uint8, device=device)


def stack_errors(stack: Stack, ws: torch.Tensor, M: int = 1, dtype=torch.float16) -> int:
    """Sticky error bits of the persistent stack launch (syncs): 1/2/4 = a wait for
    the activation / h / the cross-XCD partials gave up, 8 = a workgroup had no place."""
    code = F16 if dtype == torch.float16 else BF16
    off = int(_lib().qmlp_stack_error_offset(stack.c(), len(stack), M, code))
    if off == 0:
        return 0
    return int(ws[off: off + 4].view(torch.int32).item())


def forward_stack(stack: Stack, x: torch.Tensor, y: torch.Tensor | None = None,
                  ws: torch.Tensor | None = None, x_out: torch.Tensor | None = None) -> torch.Tensor:
    """y [L][M][d]: every block's output y_l = block_l(RMSNorm(x_l)) on the
    residual stream x_{l+1} = x_l + y_l (x_out, if given, receives x_L)."""
    M = x.shape[0]
    d = stack.mlps[0].d
    if y is None:
        y = torch.empty((len(stack), M, d), dtype=x.dtype, device=x.device)
    if ws is None:
        ws = stack_workspace(stack, M, x.dtype, x.device)
    _check(_lib().qmlp_forward_stack(stack.c(), len(stack), _ptr(x), M, _dtype_code(x), _ptr(y),
                                     _ptr(x_out), _ptr(ws), ws.numel(), _stream()), "forward_stack")
    return y


def probe_stream_read(buf: torch.Tensor, blocks: int, nontemporal: bool = True,
                      out: torch.Tensor | None = None) -> torch.Tensor:
    """Read all of `buf` once with 128-bit loads (measurement hook; see
    qmlp_probe_stream_read).  Returns the per-wave XOR words."""
    if out is None:
        out = torch.empty(4 * blocks, dtype=torch.int32, device=buf.device)
    _check(_lib().qmlp_probe_stream_read(_ptr(buf), buf.numel() * buf.element_size(), _ptr(out),
                                         blocks, int(bool(nontemporal)), _stream()),
           "qmlp_probe_stream_read")
    return out
