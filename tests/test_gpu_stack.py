"""GPU parity of the layer stack (qmlp_forward_stack) against the fp64 oracle.

The stack runs L blocks on a residual stream: x_0 = x, u_l = RMSNorm(x_l),
y_l = block_l(u_l), x_{l+1} = x_l + y_l (binary16; the sum of two binary16
values computed in fp32 and rounded once equals the exactly rounded sum, so
the stream is recomputed here bit for bit from the GPU's y_l).  Each block's
output is compared with the oracle's forward of that block's quantized
weights on the oracle's RMSNorm of the same stream state, at the output bar
max|y - y_ref| / max|y_ref| <= 1e-2.  The oracle quantizes the fp32 weights
itself, normalizes in fp64 and keeps h in fp64.  Each case
prints its name and shape before touching the GPU.
"""
import numpy as np
import pytest
import torch

import oracle as orc
import workloads as wl
from qmlp_testutil import act_tensor, bits_of, gpu_mlp, oracle_q, values_of

pytestmark = pytest.mark.gpu

Y_TOL = 1e-2


@pytest.fixture(scope="module")
def q():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_04238_amd as qm
    qm.library()
    return qm


def _announce(*what):
    print("\n[case]", *what, flush=True)


def _stack(q, cfg, L, seed=0, lora_scale=None, rank=True, first=0):
    layers = [wl.layer(cfg, first + i, seed) for i in range(L)]
    mlps = [gpu_mlp(lay, lora_scale=lora_scale, rank=rank) for lay in layers]
    return layers, mlps, q.Stack(mlps)


def _residual(x_bits, y_bits):
    """x + y of two binary16 arrays, rounded once (the oracle's residual add)."""
    return orc.residual_f16(x_bits, y_bits)


def _check_chain(layers, y, x_bits, lora_scale=None, rank=True, tol=Y_TOL, x_out=None):
    """Per-block parity: block l against the oracle on RMSNorm(x_l)
    (x_0 = x, x_{l+1} = x_l + y_l from the GPU's y_l)."""
    cfg = layers[0].cfg
    ys = bits_of(y).reshape(len(layers), cfg.M, cfg.d)
    errs = []
    prev = np.ascontiguousarray(x_bits).reshape(cfg.M, cfg.d)
    for lay, yb in zip(layers, ys):
        qg, qu, qd = oracle_q(lay)
        ls = cfg.lora_scale if lora_scale is None else lora_scale
        lo = (lay.A_gate, lay.B_gate, lay.A_up, lay.B_up) if rank else (None,) * 4
        ref = orc.forward(qg, qu, qd, *lo, orc.rmsnorm_f16(prev), lora_scale=ls, bf16=False)
        err = orc.max_rel_err(orc.act_to_f64(yb, False), ref)
        errs.append(err)
        assert err <= tol, (len(errs) - 1, err)
        prev = _residual(prev, yb)
    if x_out is not None:
        assert np.array_equal(bits_of(x_out).reshape(prev.shape), prev)
    return errs


@pytest.mark.parametrize("L", [1, 4])
def test_stack_tiny_matches_chained_oracle(q, L):
    cfg = wl.CONFIGS["tiny"]
    _announce("stack", cfg.name, "L", L)
    layers, mlps, st = _stack(q, cfg, L)
    assert q.stack_launches(st, 1) == 1          # the persistent launch serves this shape
    x = act_tensor(layers[0].x)
    ws = q.stack_workspace(st, 1)
    xo = torch.empty_like(x)
    y = q.forward_stack(st, x, ws=ws, x_out=xo)
    torch.cuda.synchronize()
    assert q.stack_errors(st, ws) == 0
    errs = _check_chain(layers, y, layers[0].x, x_out=xo)
    print("max-rel errors per block:", ["%.2e" % e for e in errs])


def test_stack_qwen3_4b_matches_chained_oracle(q):
    cfg = wl.CONFIGS["qwen3_4b"]
    _announce("stack", cfg.name, "L", 3)
    layers, mlps, st = _stack(q, cfg, 3)
    assert q.stack_launches(st, 1) == 1
    x = act_tensor(layers[0].x)
    ws = q.stack_workspace(st, 1)
    y = q.forward_stack(st, x, ws=ws)
    torch.cuda.synchronize()
    assert q.stack_errors(st, ws) == 0
    errs = _check_chain(layers, y, layers[0].x)
    print("max-rel errors per block:", ["%.2e" % e for e in errs])


def test_stack_deterministic_across_calls_and_matches_per_layer_path(q):
    """Repeated calls on one workspace (the hand-off tags advance) give the
    same bits; the per-layer qmlp_forward chain agrees within the bar."""
    cfg = wl.CONFIGS["qwen3_4b"]
    _announce("stack determinism", cfg.name, "L", 4)
    layers, mlps, st = _stack(q, cfg, 4, first=10)
    x = act_tensor(layers[0].x)
    ws = q.stack_workspace(st, 1)
    outs = []
    for _ in range(3):
        outs.append(q.forward_stack(st, x, ws=ws).clone())
    torch.cuda.synchronize()
    assert q.stack_errors(st, ws) == 0
    for o in outs[1:]:
        assert torch.equal(o.view(torch.int16), outs[0].view(torch.int16))
    # per-layer forward on the stack's own inputs
    wsl = q.workspace(mlps[0], 1)
    prev = bits_of(x)
    for i, m in enumerate(mlps):
        yl = q.forward(m, act_tensor(orc.rmsnorm_f16(prev)), ws=wsl)
        ref = values_of(outs[0][i])
        assert orc.max_rel_err(values_of(yl), ref) <= Y_TOL
        prev = _residual(prev, bits_of(outs[0][i]))


def test_stack_more_layers_than_one_launch(q):
    """44 blocks: two persistent launches, the second reading the stream the first left."""
    cfg = wl.CONFIGS["tiny"]
    _announce("stack", cfg.name, "L", 44)
    layers, mlps, st = _stack(q, cfg, 44)
    assert q.stack_launches(st, 1) == 2
    x = act_tensor(layers[0].x)
    ws = q.stack_workspace(st, 1)
    xo = torch.empty_like(x)
    y = q.forward_stack(st, x, ws=ws, x_out=xo)
    torch.cuda.synchronize()
    assert q.stack_errors(st, ws) == 0
    _check_chain(layers, y, layers[0].x, x_out=xo)


def test_stack_without_adapter_and_zero_B(q):
    """Rank 0 matches the oracle without LoRA; B = 0 gives the same bits as
    lora_scale = 0 (the LoRA term is exactly +-0)."""
    cfg = wl.CONFIGS["tiny"]
    _announce("stack rank 0 / B = 0", cfg.name)
    layers, mlps, st = _stack(q, cfg, 3, rank=False)
    x = act_tensor(layers[0].x)
    y = q.forward_stack(st, x)
    torch.cuda.synchronize()
    _check_chain(layers, y, layers[0].x, rank=False)
    # zero B vs zero scale on the same weights
    base = [gpu_mlp(lay) for lay in layers]
    zb = [q.MLP(m.gate, m.up, m.down, m.A_gate, torch.zeros_like(m.B_gate), m.A_up,
                torch.zeros_like(m.B_up)) for m in base]
    zs = [m.with_lora_scale(0.0) for m in base]
    y_zb = q.forward_stack(q.Stack(zb), x)
    y_zs = q.forward_stack(q.Stack(zs), x)
    torch.cuda.synchronize()
    assert torch.equal(y_zb.view(torch.int16), y_zs.view(torch.int16))


def test_stack_graph_replays_match_eager(q):
    """The stack captured in a HIP graph and replayed several times, with
    eager work in between, reproduces the eager outputs bit for bit."""
    cfg = wl.CONFIGS["qwen3_4b"]
    _announce("stack graph replay", cfg.name, "L", 3)
    layers, mlps, st = _stack(q, cfg, 3, first=20)
    x = act_tensor(layers[0].x)
    ws = q.stack_workspace(st, 1)
    y = torch.empty((3, 1, cfg.d), dtype=torch.float16, device="cuda")
    q.forward_stack(st, x, y=y, ws=ws)
    torch.cuda.synchronize()
    eager = y.clone()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            q.forward_stack(st, x, y=y, ws=ws)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for rep in range(4):
        y.fill_(0)
        junk = torch.randn(1 << 20, device="cuda").sum()
        g.replay()
        torch.cuda.synchronize()
        assert float(junk) == float(junk)
        assert torch.equal(y.view(torch.int16), eager.view(torch.int16)), rep
    assert q.stack_errors(st, ws) == 0


def test_stack_qwen3_8b_matches_chained_oracle(q):
    cfg = wl.CONFIGS["qwen3_8b_m1"]
    _announce("stack", cfg.name, "L", 2)
    layers, mlps, st = _stack(q, cfg, 2)
    x = act_tensor(layers[0].x)
    ws = q.stack_workspace(st, 1)
    y = q.forward_stack(st, x, ws=ws)
    torch.cuda.synchronize()
    if q.stack_launches(st, 1) == 1:
        assert q.stack_errors(st, ws) == 0
    _check_chain(layers, y, layers[0].x)


def test_stack_fallback_shapes_chain_per_layer(q):
    """Shapes outside the persistent kernel (M > 1) run per layer, chained."""
    cfg = wl.CONFIGS["qwen3_8b_m4"]
    small = wl.Config("stack_m4", M=4, d=512, f=1536, g=64, r=8, L=3)
    _announce("stack fallback", small.name)
    layers, mlps, st = _stack(q, small, 3)
    assert q.stack_launches(st, 4) == 3 * (q.forward_launches(mlps[0], 4) + 2) - 1
    x = act_tensor(layers[0].x)
    xo = torch.empty_like(x)
    y = q.forward_stack(st, x, x_out=xo)
    torch.cuda.synchronize()
    _check_chain(layers, y, layers[0].x, x_out=xo)
    assert cfg.M == 4


def test_stack_qwen3_4b_full_depth_sampled(q):
    """The benchmark's 36-layer Qwen3-4B stack in its launch configuration
    (one persistent launch); layers 0, 17 and 35 against the oracle on the
    norm of their stream state, and the final stream x_36 recomputed bit for
    bit from the GPU outputs."""
    cfg = wl.CONFIGS["qwen3_4b"]
    _announce("stack full depth", cfg.name, "L", cfg.L)
    layers = [wl.layer(cfg, i, 0) for i in range(cfg.L)]
    mlps = [gpu_mlp(lay) for lay in layers]
    st = q.Stack(mlps)
    assert q.stack_launches(st, 1) == 1
    x = act_tensor(layers[0].x)
    ws = q.stack_workspace(st, 1)
    xo = torch.empty_like(x)
    y = q.forward_stack(st, x, ws=ws, x_out=xo)
    torch.cuda.synchronize()
    assert q.stack_errors(st, ws) == 0
    ys = bits_of(y).reshape(cfg.L, 1, cfg.d)
    prev = np.ascontiguousarray(layers[0].x).reshape(1, cfg.d)
    for i in range(cfg.L):
        if i in (0, 17, 35):
            qg, qu, qd = oracle_q(layers[i])
            lay = layers[i]
            ref = orc.forward(qg, qu, qd, lay.A_gate, lay.B_gate, lay.A_up, lay.B_up,
                              orc.rmsnorm_f16(prev), lora_scale=cfg.lora_scale, bf16=False)
            err = orc.max_rel_err(orc.act_to_f64(ys[i], False), ref)
            print("layer", i, "max-rel err %.2e" % err)
            assert err <= Y_TOL
        prev = _residual(prev, ys[i])
    assert np.array_equal(bits_of(xo).reshape(prev.shape), prev)
