"""qmlp_forward_noalloc (the block with the library's own per-GPU scratch
array as workspace) against qmlp_forward on a caller workspace, through the
C ABI: two calls in a row, the second with a smaller input, each bit-equal
to qmlp_forward on the same block and within the output bar of the oracle."""
import numpy as np
import pytest
import torch

import oracle as orc
import workloads as wl

pytestmark = pytest.mark.gpu


def _act(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.float16).to(dev)


def _block(q, cfg, index, dev):
    lay = wl.layer(cfg, index)
    mlp = q.MLP(q.pack_w2(torch.from_numpy(lay.W_gate).to(dev), cfg.g),
                q.pack_w2(torch.from_numpy(lay.W_up).to(dev), cfg.g),
                q.pack_w4(torch.from_numpy(lay.W_down).to(dev), cfg.g),
                _act(lay.A_gate, dev), _act(lay.B_gate, dev), _act(lay.A_up, dev), _act(lay.B_up, dev))
    return lay, mlp


def _oracle(cfg, lay, x_bits):
    qg, qu, qd = (orc.quantize(lay.W_gate, 2, cfg.g), orc.quantize(lay.W_up, 2, cfg.g),
                  orc.quantize(lay.W_down, 4, cfg.g))
    return orc.forward(qg, qu, qd, lay.A_gate, lay.B_gate, lay.A_up, lay.B_up, x_bits)


def _bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def test_noalloc_matches_forward_two_calls_second_smaller():
    import paper_2606_04238_amd as q
    dev = torch.device("cuda:0")
    print("noalloc: qwen3_4b-shaped block at M=4, then the tiny block at M=1", flush=True)
    big = wl.Config("nb", M=4, d=2560, f=9728, g=128, r=16, L=1)
    small = wl.Config("ns", M=1, d=512, f=1536, g=64, r=8, L=1)
    for cfg, seed_layer in ((big, 3), (small, 0)):
        lay, mlp = _block(q, cfg, seed_layer, dev)
        x = _act(wl.activations(cfg, seed_layer, M=cfg.M), dev)
        y_ws = q.forward(mlp, x)
        y_na = q.forward_noalloc(mlp, x)
        torch.cuda.synchronize()
        assert torch.equal(y_na.view(torch.int16), y_ws.view(torch.int16)), cfg.name
        ref = _oracle(cfg, lay, _bits(x))
        err = orc.max_rel_err(orc.act_to_f64(_bits(y_na), False), ref)
        print("%s M=%d max-rel err %.3e" % (cfg.name, cfg.M, err), flush=True)
        assert err <= 1e-2


def test_noalloc_repeated_calls_and_m1_headline_shape():
    """The one-kernel layer path (M = 1 at the headline shape) runs on the
    array several times in a row and after a call of another shape."""
    import paper_2606_04238_amd as q
    dev = torch.device("cuda:0")
    cfg = wl.Config("nh", M=1, d=2560, f=9728, g=128, r=16, L=1)
    lay, mlp = _block(q, cfg, 5, dev)
    x = _act(wl.activations(cfg, 5, M=1), dev)
    y_ws = q.forward(mlp, x)
    outs = [q.forward_noalloc(mlp, x) for _ in range(3)]
    torch.cuda.synchronize()
    for y in outs:
        assert torch.equal(y.view(torch.int16), y_ws.view(torch.int16))
    ref = _oracle(cfg, lay, _bits(x))
    assert orc.max_rel_err(orc.act_to_f64(_bits(outs[-1]), False), ref) <= 1e-2
