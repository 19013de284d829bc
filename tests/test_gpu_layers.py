"""GPU parity of L independent blocks (qmlp_forward_layers) against the fp64
oracle.

Every block has its own seeded weights and its own seeded input x_l, and
y_l = block_l(x_l) is compared with the oracle's forward of that block's
quantized weights on x_l at the output bar max|y - y_ref| / max|y_ref| <=
1e-2 (the oracle quantizes the fp32 weights itself and keeps h in fp64).
At one token the blocks stream: every workgroup of the gate/up launch and
of the down launch owns a contiguous range of the batch's rows flattened
over blocks, so ranges straddle block boundaries; a mix-up of blocks, of the
staged activations of a range or of the row walk would pair an output with
the wrong block's oracle and fail.  Each case prints its name and shape
before touching the GPU.
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


def _blocks(q, cfg, L, seed=0, lora_scale=None, rank=True, first=0):
    layers = [wl.layer(cfg, first + i, seed) for i in range(L)]
    mlps = [gpu_mlp(lay, lora_scale=lora_scale, rank=rank) for lay in layers]
    x = torch.stack([act_tensor(lay.x) for lay in layers])          # [L][M][d]
    return layers, mlps, q.Layers(mlps), x


def _check(layers, y, which=None, lora_scale=None, rank=True, tol=Y_TOL):
    """Block l's output against the oracle on block l's own input."""
    cfg = layers[0].cfg
    ys = bits_of(y).reshape(len(layers), cfg.M, cfg.d)
    errs = {}
    for i in (range(len(layers)) if which is None else which):
        lay = layers[i]
        qg, qu, qd = oracle_q(lay)
        ls = cfg.lora_scale if lora_scale is None else lora_scale
        lo = (lay.A_gate, lay.B_gate, lay.A_up, lay.B_up) if rank else (None,) * 4
        ref = orc.forward(qg, qu, qd, *lo, lay.x, lora_scale=ls, bf16=False)
        errs[i] = orc.max_rel_err(orc.act_to_f64(ys[i], False), ref)
        assert errs[i] <= tol, (i, errs[i])
    return errs


@pytest.mark.parametrize("L", [1, 2, 3, 4, 7])
def test_layers_tiny_match_oracle(q, L):
    """Batches from one block (fewer rows than compute units) up to seven."""
    cfg = wl.CONFIGS["tiny"]
    _announce("layers", cfg.name, "L", L)
    layers, mlps, ls, x = _blocks(q, cfg, L)
    assert q.layers_path(ls, 1) == "streamed" and q.layers_launches(ls, 1) == 2
    ws = q.layers_workspace(ls, 1)
    y = q.forward_layers(ls, x, ws=ws)
    torch.cuda.synchronize()
    errs = _check(layers, y)
    print("max-rel errors per block:", ["%.2e" % e for e in errs.values()])


def test_layers_qwen3_4b_match_oracle(q):
    cfg = wl.CONFIGS["qwen3_4b"]
    _announce("layers", cfg.name, "L", 5)
    layers, mlps, ls, x = _blocks(q, cfg, 5)
    assert q.layers_path(ls, 1) == "streamed" and q.layers_launches(ls, 1) == 2
    ws = q.layers_workspace(ls, 1)
    y = q.forward_layers(ls, x, ws=ws)
    torch.cuda.synchronize()
    errs = _check(layers, y)
    print("max-rel errors per block:", ["%.2e" % e for e in errs.values()])


def test_layers_deterministic_and_match_per_block_forward(q):
    """Repeated calls on one workspace give the same bits; qmlp_forward of
    each block on its input agrees within the bar."""
    cfg = wl.CONFIGS["qwen3_4b"]
    _announce("layers determinism", cfg.name, "L", 4)
    layers, mlps, ls, x = _blocks(q, cfg, 4, first=10)
    ws = q.layers_workspace(ls, 1)
    outs = [q.forward_layers(ls, x, ws=ws).clone() for _ in range(3)]
    torch.cuda.synchronize()
    for o in outs[1:]:
        assert torch.equal(o.view(torch.int16), outs[0].view(torch.int16))
    # the streamed gate/up launch's waits for t all ended with this call's
    # tag, and the down launch advanced the call counter once per call
    assert q.workspace_errors(ws) == 0
    assert int(ws[0:4].view(torch.int32).item()) == 3
    wsl = q.workspace(mlps[0], 1)
    for i, m in enumerate(mlps):
        yl = q.forward(m, x[i], ws=wsl)
        assert orc.max_rel_err(values_of(yl), values_of(outs[0][i])) <= Y_TOL


def test_layers_calls_of_different_lengths_share_a_workspace(q):
    """Calls with 5, 1, 2 and 5 blocks in a row on one workspace: every call
    reads only what its own launches wrote (t and h of the batch)."""
    cfg = wl.CONFIGS["tiny"]
    _announce("layers varying L", cfg.name)
    layers, mlps, ls, x = _blocks(q, cfg, 5, first=3)
    ws = q.layers_workspace(ls, 1)
    for L in (5, 1, 2, 5):
        sub = q.Layers(mlps[:L])
        y = q.forward_layers(sub, x[:L].contiguous(), ws=ws)
        torch.cuda.synchronize()
        _check(layers[:L], y)


def test_layers_more_than_one_launch(q):
    """44 blocks: two batches of 40 and 4 blocks (two streamed launches
    each, LoRA-A inside the gate/up one) that reuse t and h."""
    cfg = wl.CONFIGS["tiny"]
    _announce("layers", cfg.name, "L", 44)
    layers, mlps, ls, x = _blocks(q, cfg, 44)
    assert q.layers_launches(ls, 1) == 4
    ws = q.layers_workspace(ls, 1)
    y = q.forward_layers(ls, x, ws=ws)
    torch.cuda.synchronize()
    _check(layers, y)


def test_layers_without_adapter_and_zero_B(q):
    """Rank 0 matches the oracle without LoRA; B = 0 gives the same bits as
    lora_scale = 0."""
    cfg = wl.CONFIGS["tiny"]
    _announce("layers rank 0 / B = 0", cfg.name)
    layers, mlps, ls, x = _blocks(q, cfg, 3, rank=False)
    y = q.forward_layers(ls, x)
    torch.cuda.synchronize()
    _check(layers, y, rank=False)
    base = [gpu_mlp(lay) for lay in layers]
    zb = [q.MLP(m.gate, m.up, m.down, m.A_gate, torch.zeros_like(m.B_gate), m.A_up,
                torch.zeros_like(m.B_up)) for m in base]
    zs = [m.with_lora_scale(0.0) for m in base]
    y_zb = q.forward_layers(q.Layers(zb), x)
    y_zs = q.forward_layers(q.Layers(zs), x)
    torch.cuda.synchronize()
    assert torch.equal(y_zb.view(torch.int16), y_zs.view(torch.int16))


def test_layers_graph_replays_match_eager(q):
    """Captured in a HIP graph and replayed several times, with eager work in
    between: every replay reproduces the eager outputs bit for bit."""
    cfg = wl.CONFIGS["qwen3_4b"]
    _announce("layers graph replay", cfg.name, "L", 4)
    layers, mlps, ls, x = _blocks(q, cfg, 4, first=20)
    ws = q.layers_workspace(ls, 1)
    y = torch.empty_like(x)
    q.forward_layers(ls, x, y=y, ws=ws)
    torch.cuda.synchronize()
    eager = y.clone()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            q.forward_layers(ls, x, y=y, ws=ws)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for rep in range(4):
        y.fill_(0)
        junk = torch.randn(1 << 20, device="cuda").sum()
        g.replay()
        torch.cuda.synchronize()
        assert float(junk) == float(junk)
        assert torch.equal(y.view(torch.int16), eager.view(torch.int16)), rep


def test_layers_qwen3_8b_match_oracle(q):
    cfg = wl.CONFIGS["qwen3_8b_m1"]
    _announce("layers", cfg.name, "L", 3)
    layers, mlps, ls, x = _blocks(q, cfg, 3)
    ws = q.layers_workspace(ls, 1)
    assert q.layers_path(ls, 1) == "streamed"
    y = q.forward_layers(ls, x, ws=ws)
    torch.cuda.synchronize()
    _check(layers, y)


@pytest.mark.parametrize("M,L,d", [(2, 3, 512), (2, 41, 512), (4, 3, 640), (13, 5, 640)])
def test_layers_batched_shapes_match_oracle(q, M, L, d):
    """Shapes outside the streamed and matrix-core paths (M = 2, or d not a
    multiple of four groups) run in batches of up to 40 blocks on the
    stand-alone kernels (LoRA-A, gate/up and down of every block of a
    batch); 41 blocks take two batches that reuse t and h."""
    small = wl.Config("layers_m%d" % M, M=M, d=d, f=1536, g=64, r=8, L=L)
    _announce("layers batched", small.name, "d", d, "L", L)
    layers, mlps, ls, x = _blocks(q, small, L)
    assert q.layers_path(ls, M) == "batched"
    assert q.layers_launches(ls, M) == 3 * ((L + 39) // 40)
    y = q.forward_layers(ls, x)
    torch.cuda.synchronize()
    _check(layers, y, which=None if L <= 5 else (0, 1, 39, 40))
    wsl = q.workspace(mlps[0], M)
    for i in ((0, L - 1) if L > 5 else range(L)):
        yl = q.forward(mlps[i], x[i], ws=wsl)
        assert orc.max_rel_err(values_of(y[i]), values_of(yl)) <= Y_TOL


def test_layers_qwen3_4b_full_depth_sampled(q):
    """The benchmark's 36 Qwen3-4B blocks in its launch configuration (the
    streamed launches); blocks 0, 1, 17, 34 and 35 against the oracle, and
    every block against qmlp_forward on its input."""
    cfg = wl.CONFIGS["qwen3_4b"]
    _announce("layers full depth", cfg.name, "L", cfg.L)
    layers, mlps, ls, x = _blocks(q, cfg, cfg.L)
    assert q.layers_path(ls, 1) == "streamed" and q.layers_launches(ls, 1) == 2
    ws = q.layers_workspace(ls, 1)
    y = q.forward_layers(ls, x, ws=ws)
    torch.cuda.synchronize()
    errs = _check(layers, y, which=(0, 1, 17, 34, 35))
    print("max-rel errors:", {k: "%.2e" % v for k, v in errs.items()})
    wsl = q.workspace(mlps[0], 1)
    worst = 0.0
    for i, m in enumerate(mlps):
        yl = q.forward(m, x[i], ws=wsl)
        worst = max(worst, orc.max_rel_err(values_of(y[i]), values_of(yl)))
    print("max-rel vs per-block forward: %.2e" % worst)
    assert worst <= Y_TOL
    assert np.isfinite(values_of(y)).all()


def test_forward_batch_forces_standalone_kernels(q):
    """forward_batch runs the 4B blocks (a streamed shape for forward_layers)
    as one batch on the stand-alone kernels; both match the oracle and each
    other within the bar; a second call on the same workspace repeats the
    bits."""
    cfg = wl.CONFIGS["qwen3_4b"]
    _announce("forward_batch", cfg.name, "L", 5)
    layers, mlps, ls, x = _blocks(q, cfg, 5, first=7)
    ws = q.batch_workspace(ls, 1)
    y1 = q.forward_batch(ls, x, ws=ws).clone()
    y2 = q.forward_batch(ls, x, ws=ws)
    yl = q.forward_layers(ls, x)
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))
    _check(layers, y1)
    assert orc.max_rel_err(values_of(y1), values_of(yl)) <= Y_TOL


@pytest.mark.parametrize("d,f,g,r,L", [
    (512, 1536, 64, 0, 9),          # no adapter, group 64
    (512, 1536, 128, 32, 40),       # a full batch: ranges of 30 items straddle blocks
    (1024, 2048, 64, 8, 3),         # JC = 2
    (1536, 1280, 128, 16, 17),      # JC = 3, f not a multiple of 256
    (2048, 3072, 64, 32, 6),        # JC = 4
    (3072, 1024, 128, 8, 2),        # two steps per row (JC = 3), few rows
    (4096, 1536, 64, 16, 5),        # two steps per row (JC = 4)
    (3072, 1024, 128, 32, 36),      # 2304 LoRA-A rows over 256 workgroups of 8 waves: 9 per workgroup
])
def test_layers_streamed_shapes_match_oracle(q, d, f, g, r, L):
    """The streamed launches over widths of one and two steps per row, ranks
    0 to 32, groups 64 and 128, and batches from a few rows to a full batch
    whose workgroup ranges span two or three blocks."""
    cfg = wl.Config("stream_%d_%d" % (d, f), M=1, d=d, f=f, g=g, r=r, L=L)
    _announce("layers streamed", cfg.name, "g", g, "r", r, "L", L)
    layers, mlps, ls, x = _blocks(q, cfg, L, rank=r > 0)
    assert q.layers_path(ls, 1) == "streamed" and q.layers_launches(ls, 1) == 2 * ((L + 39) // 40)
    y = q.forward_layers(ls, x)
    torch.cuda.synchronize()
    _check(layers, y, rank=r > 0, which=None if L <= 9 else (0, 1, L // 2, L - 2, L - 1))


@pytest.mark.parametrize("M,d,f,g,r,L", [
    (3, 512, 1536, 64, 8, 1),       # the fewest tokens, one block: fewer items than compute units
    (4, 512, 6400, 128, 16, 3),     # MT = 4: f over two h' chunks of 6144 codes, the second short
    (5, 1536, 2560, 64, 0, 9),      # MT = 8, no adapter: h' chunks of 1536 codes, the last short
    (8, 1024, 2048, 128, 32, 40),   # a full batch: ranges straddle blocks
    (9, 512, 1536, 64, 16, 41),     # MT = 16, two batches
    (16, 2048, 3072, 64, 8, 6),     # all sixteen token rows
])
def test_layers_mfma_shapes_match_oracle(q, M, d, f, g, r, L):
    """3 <= M <= 16 runs on the matrix cores (LoRA-A, then one gate/up and
    one down launch per batch): token counts on both sides of each padded
    tile height (4, 8, 16), groups 64 and 128, ranks 0 to 32, batches from
    one block to two batches; d from 512 to 2048 gives each LoRA-A wave 1 to
    4 steps of 32 (a partial group of four at 1536).  Every block against the oracle (sampled for
    long batches) and against the stand-alone kernels on the same input."""
    cfg = wl.Config("mfma_m%d_%d_%d" % (M, d, f), M=M, d=d, f=f, g=g, r=r, L=L)
    _announce("layers mfma", cfg.name, "g", g, "r", r, "L", L)
    layers, mlps, ls, x = _blocks(q, cfg, L, rank=r > 0)
    assert q.layers_path(ls, M) == "mfma"
    assert q.layers_launches(ls, M) == (3 if r > 0 else 2) * ((L + 39) // 40)
    # control block, four slices of LoRA-A partial sums t, then h of a batch
    nb, r256 = min(L, 40), (lambda v: (v + 255) // 256 * 256)
    assert q.layers_workspace_bytes(ls, M) == 1024 + r256(4 * nb * M * 2 * r * 4) + r256(nb * M * f * 2)
    ws = q.layers_workspace(ls, M)
    y = q.forward_layers(ls, x, ws=ws)
    yb = q.forward_batch(ls, x)
    torch.cuda.synchronize()
    errs = _check(layers, y, rank=r > 0, which=None if L <= 9 else (0, 1, L // 2, L - 2, L - 1))
    print("max-rel errors:", {k: "%.2e" % v for k, v in errs.items()})
    assert orc.max_rel_err(values_of(y), values_of(yb)) <= Y_TOL
    assert np.isfinite(values_of(y)).all()
    # a second call on the same workspace repeats the bits
    y2 = q.forward_layers(ls, x, ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16), y2.view(torch.int16))


@pytest.mark.parametrize("name", ["qwen3_8b_m4", "qwen3_8b_m16", "dense14b_m8"])
def test_layers_mfma_full_depth_sampled(q, name):
    """The benchmark's several-token workloads in its launch configuration:
    every block of the model (36 or 40, each with its own weights and input)
    in one qmlp_forward_layers call on the matrix cores; the first, middle
    and last blocks against the oracle, every block against the stand-alone
    kernels on its input."""
    import concurrent.futures
    cfg = wl.CONFIGS[name]
    _announce("layers mfma full depth", cfg.name, "M", cfg.M, "L", cfg.L)
    with concurrent.futures.ThreadPoolExecutor(max_workers=8) as ex:
        layers = list(ex.map(lambda i: wl.layer(cfg, i, 0), range(cfg.L)))
    mlps = [gpu_mlp(lay) for lay in layers]
    x = torch.stack([act_tensor(lay.x) for lay in layers])
    ls = q.Layers(mlps)
    assert q.layers_path(ls, cfg.M) == "mfma" and q.layers_launches(ls, cfg.M) == 3
    ws = q.layers_workspace(ls, cfg.M)
    y = q.forward_layers(ls, x, ws=ws)
    yb = q.forward_batch(ls, x)
    torch.cuda.synchronize()
    errs = _check(layers, y, which=(0, cfg.L // 2, cfg.L - 1))
    print("max-rel errors:", {k: "%.2e" % v for k, v in errs.items()})
    worst = max(orc.max_rel_err(values_of(y[i]), values_of(yb[i])) for i in range(cfg.L))
    print("max-rel vs stand-alone kernels: %.2e" % worst)
    assert worst <= Y_TOL


def test_layers_streamed_graph_replays_match_eager(q):
    """The streamed launches captured in a HIP graph and replayed several
    times, with eager work in between: the call counter that tags t advances
    on the device, so every replay reads its own t and gives the eager
    bits; the error bits stay clear and the counter counts every call."""
    cfg = wl.CONFIGS["qwen3_4b"]
    _announce("layers streamed graph replay", cfg.name, "L", 4)
    layers, mlps, ls, x = _blocks(q, cfg, 4, first=20)
    assert q.layers_path(ls, 1) == "streamed"
    ws = q.layers_workspace(ls, 1)
    y = torch.empty_like(x)
    q.forward_layers(ls, x, y=y, ws=ws)
    torch.cuda.synchronize()
    ey = y.clone()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            q.forward_layers(ls, x, y=y, ws=ws)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for rep in range(4):
        y.fill_(0)
        junk = torch.randn(1 << 20, device="cuda").sum()
        g.replay()
        torch.cuda.synchronize()
        assert float(junk) == float(junk)
        assert torch.equal(y.view(torch.int16), ey.view(torch.int16)), rep
    assert q.workspace_errors(ws) == 0
    # the eager call, the captured one (capture runs nothing) and four replays
    assert int(ws[0:4].view(torch.int32).item()) == 5
