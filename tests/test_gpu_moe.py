"""GPU parity of qmlp_forward_moe (the routed-expert MLP of the MoE decoder,
Sec. 5) against the oracle's routing-weighted sum of expert blocks, at the
output bar max|y - y_ref| / max|y_ref| <= 1e-2.  Routing (expert ids and
weights) is synthetic and lives on the device."""
import numpy as np
import pytest
import torch

import oracle as orc
import workloads as wl
from qmlp_testutil import act_tensor, gpu_mlp, oracle_q, values_of

pytestmark = pytest.mark.gpu

Y_TOL = 1e-2


@pytest.fixture(scope="module")
def q():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_04238_amd as qm
    qm.library()
    return qm


def _run(q, cfg, E, k, M, layer=0, idx=None, w=None):
    lays = [wl.layer(cfg, e) for e in range(E)]
    experts = q.Layers([gpu_mlp(lay) for lay in lays])
    x = wl.activations(cfg, 100 + layer, 0, M=M)
    if idx is None:
        idx, w = wl.routing(M, E, k, layer)
    y = q.forward_moe(experts, act_tensor(x), torch.from_numpy(idx).cuda(),
                      torch.from_numpy(w).cuda())
    torch.cuda.synchronize()
    oq = [oracle_q(lay) + (lay.A_gate, lay.B_gate, lay.A_up, lay.B_up) for lay in lays]
    ref = orc.moe_forward(oq, idx, w, x, lora_scale=cfg.lora_scale)
    return orc.max_rel_err(values_of(y), ref)


@pytest.mark.parametrize("E,k,M", [(8, 2, 1), (8, 4, 3), (5, 1, 16), (32, 4, 10)])
def test_moe_tiny_matches_oracle(q, E, k, M):
    cfg = wl.Config("moe_tiny", M=1, d=512, f=768, g=64, r=8, L=1)
    print("\n[case] moe tiny E %d k %d M %d" % (E, k, M), flush=True)
    err = _run(q, cfg, E, k, M)
    print("max-rel %.2e" % err)
    assert err <= Y_TOL


def test_moe_gptoss20b_shape_matches_oracle(q):
    """32 GPT-OSS-20B-class experts (d = f = 2880, group 64, rank 16), top-4,
    one decode token."""
    mc = wl.MOE["gptoss20b_moe"]
    print("\n[case] moe", mc.name, flush=True)
    err = _run(q, mc.block, mc.experts, mc.topk, 1, layer=3)
    print("max-rel %.2e" % err)
    assert err <= Y_TOL


@pytest.mark.parametrize("d", [1024, 2048])
def test_moe_few_instances_take_more_lanes_per_row(q, d):
    """One token routed to one or two experts fills fewer than two workgroups
    per CU, so the gate/up launch doubles its lanes per row (16, then 32 at
    d = 2048, one 16-byte unit per lane); down forms the routing sum at 8
    lanes over f = 768 (k = 1: one wave per row group, four row groups;
    k = 2: two).  The picks are pinned on the CPU
    (test_abi.test_moe_lane_choice); here the results match the oracle."""
    cfg = wl.Config("moe_wide_tiny", M=1, d=d, f=768, g=64, r=8, L=1)
    for k in (1, 2):
        print("\n[case] moe d %d E 4 k %d M 1" % (d, k), flush=True)
        err = _run(q, cfg, 4, k, 1, layer=k)
        print("max-rel %.2e" % err)
        assert err <= Y_TOL


def test_moe_repeated_expert_and_single_slot(q):
    """Two tokens routed to the same expert with weight 1 each (k = 1) give
    that expert's qmlp_forward outputs."""
    cfg = wl.Config("moe_rep", M=1, d=512, f=768, g=64, r=8, L=1)
    print("\n[case] moe repeated expert", flush=True)
    E = 3
    lays = [wl.layer(cfg, e) for e in range(E)]
    mlps = [gpu_mlp(lay) for lay in lays]
    x = act_tensor(wl.activations(cfg, 7, 0, M=2))
    idx = torch.tensor([[1], [1]], dtype=torch.int32, device="cuda")
    w = torch.ones((2, 1), dtype=torch.float32, device="cuda")
    y = q.forward_moe(q.Layers(mlps), x, idx, w)
    yr = q.forward(mlps[1], x)
    torch.cuda.synchronize()
    assert orc.max_rel_err(values_of(y), values_of(yr)) <= 1e-3


def test_moe_and_batch_graph_replays_match_eager(q):
    """qmlp_forward_moe and qmlp_forward_batch captured in a HIP graph and
    replayed several times, with eager work in between: every replay gives
    the eager bits."""
    cfg = wl.Config("moe_graph", M=1, d=512, f=768, g=64, r=8, L=1)
    print("\n[case] moe / batch graph replay", flush=True)
    E, k, M = 6, 2, 3
    lays = [wl.layer(cfg, e) for e in range(E)]
    experts = q.Layers([gpu_mlp(lay) for lay in lays])
    x = act_tensor(wl.activations(cfg, 11, 0, M=M))
    idx, w = wl.routing(M, E, k, 4)
    idx, w = torch.from_numpy(idx).cuda(), torch.from_numpy(w).cuda()
    ws = torch.zeros(q.moe_workspace_bytes(experts, M, k), dtype=torch.uint8, device="cuda")
    y = torch.empty_like(x)
    xb = torch.stack([act_tensor(lay.x) for lay in lays])
    wsb = q.batch_workspace(experts, 1)
    yb = torch.empty_like(xb)

    def run():
        q.forward_moe(experts, x, idx, w, y=y, ws=ws)
        q.forward_batch(experts, xb, y=yb, ws=wsb)
    run()
    torch.cuda.synchronize()
    ey, eb = y.clone(), yb.clone()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            run()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for rep in range(4):
        y.fill_(0)
        yb.fill_(0)
        junk = torch.randn(1 << 20, device="cuda").sum()
        g.replay()
        torch.cuda.synchronize()
        assert float(junk) == float(junk)
        assert torch.equal(y.view(torch.int16), ey.view(torch.int16)), rep
        assert torch.equal(yb.view(torch.int16), eb.view(torch.int16)), rep


def test_moe_route_ids_outside_the_table_are_clamped(q):
    """Expert ids beyond the table read the last expert, negative ids the
    first (the kernels clamp; nothing is read outside the table)."""
    cfg = wl.Config("moe_clamp", M=1, d=512, f=768, g=64, r=8, L=1)
    print("\n[case] moe clamped ids", flush=True)
    E = 3
    lays = [wl.layer(cfg, e) for e in range(E)]
    experts = q.Layers([gpu_mlp(lay) for lay in lays])
    x = act_tensor(wl.activations(cfg, 12, 0, M=2))
    w = torch.ones((2, 1), dtype=torch.float32, device="cuda")
    bad = q.forward_moe(experts, x, torch.tensor([[7], [-5]], dtype=torch.int32, device="cuda"), w)
    good = q.forward_moe(experts, x, torch.tensor([[2], [0]], dtype=torch.int32, device="cuda"), w)
    torch.cuda.synchronize()
    assert torch.equal(bad.view(torch.int16), good.view(torch.int16))



@pytest.mark.parametrize("k", [3, 6])
def test_moe_repeated_calls_on_one_workspace(q, k):
    """Up to four slots per token the down launch also adds the slots (each
    workgroup runs all k instances of its rows; at k = 3 one wave of four
    only stages); past four a combine launch adds them.  Both forms, over
    three calls with other inputs and routing on one workspace (LoRA-A runs
    in the gate/up launch: each call's t words carry a new tag)."""
    cfg = wl.Config("moe_reuse", M=1, d=1024, f=768, g=64, r=8, L=1)
    E, M = 8, 4
    lays = [wl.layer(cfg, e) for e in range(E)]
    experts = q.Layers([gpu_mlp(lay) for lay in lays])
    oq = [oracle_q(lay) + (lay.A_gate, lay.B_gate, lay.A_up, lay.B_up) for lay in lays]
    ws = torch.zeros(q.moe_workspace_bytes(experts, M, k), dtype=torch.uint8, device="cuda")
    for call in range(3):
        print("\n[case] moe k %d call %d" % (k, call), flush=True)
        x = wl.activations(cfg, 40 + call, 0, M=M)
        idx, w = wl.routing(M, E, k, call)
        y = q.forward_moe(experts, act_tensor(x), torch.from_numpy(idx).cuda(),
                          torch.from_numpy(w).cuda(), ws=ws)
        torch.cuda.synchronize()
        err = orc.max_rel_err(values_of(y), orc.moe_forward(oq, idx, w, x, lora_scale=cfg.lora_scale))
        print("max-rel %.2e" % err)
        assert err <= Y_TOL
    # the gate/up launch's waits for the LoRA-A words all ended with this
    # call's tag, and the call counter advanced once per call
    assert q.workspace_errors(ws) == 0
    assert int(ws[0:4].view(torch.int32).item()) == 3


def test_moe_wide_activation_takes_the_chunked_staging(q):
    """Routed gate/up loads the activation ahead of the weights when one
    staging pass of at most two words per thread holds it (d <= 8192 at
    2 bits); a wider activation takes the chunk loop.  d = 8704 here."""
    cfg = wl.Config("moe_wide_x", M=1, d=8704, f=256, g=64, r=8, L=1)
    print("\n[case] moe d 8704 E 3 k 2 M 2", flush=True)
    err = _run(q, cfg, 3, 2, 2, layer=5)
    print("max-rel %.2e" % err)
    assert err <= Y_TOL


@pytest.mark.parametrize("r,k,M", [(32, 4, 2), (16, 2, 5), (0, 4, 1)])
def test_moe_ranks_and_slots(q, r, k, M):
    """Rank 32 (sixteen LoRA-A columns per instance, t read by 64 threads),
    rank 16 at two slots and five tokens (two row groups per down
    workgroup), and rank 0 (no LoRA-A columns, no t) against the oracle,
    with the control block's error bits clear afterwards."""
    cfg = wl.Config("moe_r%d" % r, M=1, d=1024, f=1536, g=64, r=r or 8, L=1)
    print("\n[case] moe r %d k %d M %d" % (r, k, M), flush=True)
    E = 6
    lays = [wl.layer(cfg, e) for e in range(E)]
    experts = q.Layers([gpu_mlp(lay, rank=r > 0) for lay in lays])
    ws = torch.zeros(q.moe_workspace_bytes(experts, M, k), dtype=torch.uint8, device="cuda")
    x = wl.activations(cfg, 60 + r, 0, M=M)
    idx, w = wl.routing(M, E, k, r)
    y = q.forward_moe(experts, act_tensor(x), torch.from_numpy(idx).cuda(), torch.from_numpy(w).cuda(), ws=ws)
    torch.cuda.synchronize()
    oq = [oracle_q(lay) + ((lay.A_gate, lay.B_gate, lay.A_up, lay.B_up) if r > 0 else (None,) * 4)
          for lay in lays]
    err = orc.max_rel_err(values_of(y), orc.moe_forward(oq, idx, w, x, lora_scale=cfg.lora_scale))
    print("max-rel %.2e" % err)
    assert err <= Y_TOL
    assert q.workspace_errors(ws) == 0
