"""GPU parity of the precision variants against the fp64 oracle: the uniform
W4 and uniform W2 blocks that bracket W4/W2-GateUp in the throughput
comparison (Sec. 5.2: Gain and Capture are measured between them), the
paper's own INT2 grouping, 2-bit gate/up at group 32 (Sec. 3.3, Sec. 4.1),
and the 3-bit gate/up of Appendix B (W3, group 32; two-plane code layout).

They run on the stand-alone decode kernels (LoRA-A, gate/up, down).  The
oracle is bit-width agnostic (it dequantizes s * (q - z) from unpacked
codes), so each case quantizes the same fp32 weights at the variant's widths
on both sides: packing is compared bit for bit, outputs at the output bar
max|y - y_ref| / max|y_ref| <= 1e-2.  Each case prints its name before it
touches the GPU.
"""
import numpy as np
import pytest
import torch

import oracle as orc
import workloads as wl
from qmlp_testutil import act_tensor, bits_of, values_of

pytestmark = pytest.mark.gpu

Y_TOL = 1e-2

# (gate/up bits, gate/up group, down bits, down group); None = the workload's group
VARIANTS = {
    "w4_uniform": (4, None, 4, None),
    "w2_uniform": (2, None, 2, None),
    "w2g32_lora": (2, 32, 4, None),
    "w4g32_uniform": (4, 32, 4, 32),
    "w3g32_lora": (3, 32, 4, None),
    "w3_lora": (3, None, 4, None),
}


@pytest.fixture(scope="module")
def q():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_04238_amd as qm
    qm.library()
    return qm


def _announce(*what):
    print("\n[case]", *what, flush=True)


def _widths(cfg, variant):
    bg, gg, bd, gd = VARIANTS[variant]
    return bg, gg or cfg.g, bd, gd or cfg.g


def _pack(q, W, bits, group):
    t = torch.from_numpy(W).cuda()
    return {2: q.pack_w2, 3: q.pack_w3, 4: q.pack_w4}[bits](t, group)


def _block(q, lay, variant, rank=True):
    cfg = lay.cfg
    bg, gg, bd, gd = _widths(cfg, variant)
    g, u, d = (_pack(q, lay.W_gate, bg, gg), _pack(q, lay.W_up, bg, gg),
               _pack(q, lay.W_down, bd, gd))
    if not rank:
        return q.MLP(g, u, d, lora_scale=cfg.lora_scale)
    return q.MLP(g, u, d, act_tensor(lay.A_gate), act_tensor(lay.B_gate), act_tensor(lay.A_up),
                 act_tensor(lay.B_up), lora_scale=cfg.lora_scale)


def _oracle(lay, variant, rank=True, x=None):
    cfg = lay.cfg
    bg, gg, bd, gd = _widths(cfg, variant)
    qg, qu, qd = (orc.quantize(lay.W_gate, bg, gg), orc.quantize(lay.W_up, bg, gg),
                  orc.quantize(lay.W_down, bd, gd))
    lo = (lay.A_gate, lay.B_gate, lay.A_up, lay.B_up) if rank else (None,) * 4
    return orc.forward(qg, qu, qd, *lo, lay.x if x is None else x, lora_scale=cfg.lora_scale,
                       return_h=True), (qg, qu, qd)


def _check_packed(w, qt):
    assert np.array_equal(w.codes.cpu().numpy().view(np.uint32).reshape(w.n_out, -1), qt.packed())
    assert np.array_equal(w.meta.cpu().numpy().view(np.uint16).reshape(qt.scale.shape + (2,)),
                          qt.meta())


@pytest.mark.parametrize("variant", list(VARIANTS))
@pytest.mark.parametrize("M", [1, 3, 16])
def test_variant_tiny_matches_oracle(q, variant, M):
    cfg = wl.Config("tiny_var", M=M, d=512, f=1536, g=64, r=8, L=1)
    _announce("variant", variant, cfg.name, "M", M)
    lay = wl.layer(cfg, 0)
    rank = variant.endswith("_lora") or M == 3          # adapters also on the uniform blocks
    mlp = _block(q, lay, variant, rank=rank)
    assert q.forward_launches(mlp, M) == (3 if rank else 2)
    (y_ref, h_ref), (qg, qu, qd) = _oracle(lay, variant, rank=rank)
    _check_packed(mlp.gate, qg)
    _check_packed(mlp.down, qd)
    y = q.forward(mlp, act_tensor(lay.x))
    torch.cuda.synchronize()
    err = orc.max_rel_err(values_of(y), y_ref)
    print("max-rel error %.2e" % err)
    assert err <= Y_TOL


@pytest.mark.parametrize("variant", list(VARIANTS))
def test_variant_ragged_units(q, variant):
    """d = 704 (640 at 3 bits, whose rows take multiples of 128 codes) and
    f = 1600: 11 or 10 (2/3-bit) / 22 (4-bit) units per gate/up row and 25 / 50
    per down row, so the lanes of a row hold different unit counts."""
    g = 32 if variant == "w4g32_uniform" else 64
    d = 640 if variant.startswith("w3") else 704
    cfg = wl.Config("ragged_var", M=5, d=d, f=1600, g=g, r=16, L=1)
    _announce("variant", variant, cfg.name)
    lay = wl.layer(cfg, 2)
    mlp = _block(q, lay, variant)
    (y_ref, _), _ = _oracle(lay, variant)
    y = q.forward(mlp, act_tensor(lay.x))
    torch.cuda.synchronize()
    assert orc.max_rel_err(values_of(y), y_ref) <= Y_TOL


@pytest.mark.parametrize("variant", ["w4_uniform", "w2_uniform", "w2g32_lora", "w3g32_lora"])
@pytest.mark.parametrize("M", [1, 4])
def test_variant_qwen3_4b_matches_oracle(q, variant, M):
    """The Qwen3-4B block shape (d 2560, f 9728, group 128) at each width."""
    base = wl.CONFIGS["qwen3_4b"]
    cfg = wl.Config("qwen3_4b_var", M=M, d=base.d, f=base.f, g=base.g, r=base.r, L=1)
    _announce("variant", variant, cfg.name, "M", M)
    lay = wl.layer(cfg, 1)
    rank = variant.endswith("_lora")
    mlp = _block(q, lay, variant, rank=rank)
    (y_ref, h_ref), (qg, qu, qd) = _oracle(lay, variant, rank=rank)
    _check_packed(mlp.gate, qg)
    _check_packed(mlp.up, qu)
    _check_packed(mlp.down, qd)
    y = q.forward(mlp, act_tensor(lay.x))
    torch.cuda.synchronize()
    err = orc.max_rel_err(values_of(y), y_ref)
    print("max-rel error %.2e" % err)
    assert err <= Y_TOL


def test_w2g32_gateup_entry_and_unpack(q):
    """qmlp_gateup_w2_lora at group 32 gives h within the bar; unpack returns
    the oracle's codes, scales and zeros exactly."""
    cfg = wl.Config("g32", M=2, d=512, f=1536, g=64, r=8, L=1)
    _announce("w2 g32 gate/up entry", cfg.name)
    lay = wl.layer(cfg, 4)
    mlp = _block(q, lay, "w2g32_lora")
    (_, h_ref), (qg, _, _) = _oracle(lay, "w2g32_lora")
    h = q.gateup_w2_lora(mlp, act_tensor(lay.x))
    torch.cuda.synchronize()
    assert orc.max_rel_err(values_of(h), h_ref) <= Y_TOL
    codes, scales, zeros = q.unpack(mlp.gate)
    assert np.array_equal(codes.cpu().numpy(), qg.codes)
    assert np.array_equal(scales.cpu().numpy().view(np.uint16), qg.scale)
    assert np.array_equal(zeros.cpu().numpy().view(np.uint16), qg.zero)


def test_variant_layers_run_batched(q):
    """forward_layers over uniform-W4 blocks runs them as one batch on the
    stand-alone kernels (gate/up of every block, then down of every block)."""
    cfg = wl.Config("layers_w4", M=1, d=512, f=1536, g=64, r=8, L=3)
    _announce("variant layers", cfg.name)
    lays = [wl.layer(cfg, i) for i in range(3)]
    mlps = [_block(q, lay, "w4_uniform", rank=False) for lay in lays]
    layers = q.Layers(mlps)
    assert q.layers_launches(layers, 1) == 2
    x = torch.stack([act_tensor(lay.x) for lay in lays])
    y = q.forward_layers(layers, x)
    torch.cuda.synchronize()
    for i, lay in enumerate(lays):
        (y_ref, _), _ = _oracle(lay, "w4_uniform", rank=False)
        assert orc.max_rel_err(orc.act_to_f64(bits_of(y[i]), False), y_ref) <= Y_TOL


@pytest.mark.parametrize("group", [32, 128])
def test_w3_pack_unpack_dequant_match_oracle(q, group):
    """pack_w3 writes the oracle's two-plane words and metadata bit for bit;
    unpack returns its codes, scales and zeros, dequant its binary16 image."""
    cfg = wl.Config("w3pack", M=1, d=640, f=384, g=64, r=8, L=1)
    _announce("w3 pack", "group", group)
    W = wl.weight(cfg, 0, 0)                                     # [f][d]
    w = q.pack_w3(torch.from_numpy(W).cuda(), group)
    qt = orc.quantize(W, 3, group)
    torch.cuda.synchronize()
    assert not w.invalid_groups()
    _check_packed(w, qt)
    codes, scales, zeros = q.unpack(w)
    assert np.array_equal(codes.cpu().numpy(), qt.codes)
    assert np.array_equal(scales.cpu().numpy().view(np.uint16), qt.scale)
    assert np.array_equal(zeros.cpu().numpy().view(np.uint16), qt.zero)
    deq = q.dequant(w)
    assert np.array_equal(deq.cpu().numpy().view(np.uint16), qt.dequant_f16())
