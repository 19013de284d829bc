"""GPU parity of the HIP path against the fp64 oracle, through the C ABI.

Bar (the tolerances are derived next to their constants below):
  * packing, unpacking, scales, zeros and dequantized binary16 weights: bit-exact;
  * intermediate h of the gate/up kernel: max|h - h_ref| / max|h_ref| <= 2e-3;
  * block output y: max|y - y_ref| / max|y_ref| <= 1e-2 (fp16 outputs, fp32 accumulation).
The oracle quantizes the same fp32 weights independently; its forward keeps
h in fp64.  Each case prints its name, seed and shape before touching the GPU.
"""
import numpy as np
import pytest
import torch

import oracle as orc
import workloads as wl
from qmlp_testutil import act_tensor, bits_of, gpu_mlp, oracle_forward, oracle_q, values_of

pytestmark = pytest.mark.gpu

# h is stored in binary16: one rounding is at most 2^-11 ~ 4.9e-4 of the
# element; the fp32 accumulation over d terms, with the 1024 offset of the
# dequantization removed per group, adds about 2^-24 * 64 * sqrt(d) ~ 2e-5 of
# max|G|.  2e-3 leaves a 4x margin over the binary16 floor, while dropping the
# LoRA term (about 1e-2 of h on these inputs) fails it.
H_TOL = 2e-3
# the output bar for binary16 outputs with fp32 accumulation
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


DECODE_CASES = {
    "tiny": wl.CONFIGS["tiny"],
    "qwen3_4b": wl.CONFIGS["qwen3_4b"],
    "qwen3_8b_m1": wl.CONFIGS["qwen3_8b_m1"],
    "qwen3_8b_m4": wl.CONFIGS["qwen3_8b_m4"],
    "qwen3_8b_m16": wl.CONFIGS["qwen3_8b_m16"],
    "dense14b_m8": wl.CONFIGS["dense14b_m8"],
    # ragged shapes: units per row not a multiple of the lanes per row (idle
    # lanes, lanes with one unit more than others), odd M padded to the next
    # token tile
    "ragged_g64_m3": wl.Config("ragged_g64_m3", M=3, d=320, f=448, g=64, r=8, L=1),
    "ragged_g128_m5": wl.Config("ragged_g128_m5", M=5, d=640, f=1152, g=128, r=16, L=1),
    "ragged_r32_m13": wl.Config("ragged_r32_m13", M=13, d=1152, f=960, g=64, r=32, L=1),
}


# ------------------------------------------------------------- packing
def _check_pack(q, W, bits, group, ref=None):
    qw = (q.pack_w2 if bits == 2 else q.pack_w4)(torch.from_numpy(W).cuda(), group)
    ref = ref if ref is not None else orc.quantize(W, bits, group)
    codes = qw.codes.cpu().numpy()
    meta = qw.meta.cpu().numpy()
    assert np.array_equal(codes.view(np.uint32).reshape(ref.codes.shape[0], -1), ref.packed())
    assert np.array_equal(meta.view(np.uint16).reshape(ref.scale.shape + (2,)), ref.meta())
    c, s, z = q.unpack(qw)
    assert np.array_equal(c.cpu().numpy(), ref.codes)
    assert np.array_equal(s.cpu().numpy().view(np.uint16), ref.scale)
    assert np.array_equal(z.cpu().numpy().view(np.uint16), ref.zero)
    assert np.array_equal(bits_of(q.dequant(qw)), ref.dequant_f16())
    assert qw.invalid_groups() == (ref.bad > 0)
    return qw


@pytest.mark.parametrize("name", ["tiny", "qwen3_4b", "dense14b_m8", "prefill20b"])
def test_pack_bit_exact(q, name):
    cfg = wl.CONFIGS[name]
    for which, bits in ((0, 2), (2, 4)):
        _announce("pack", name, "matrix", which, "bits", bits, "seed 0 layer 0")
        W = wl.weight(cfg, 0, which)
        _check_pack(q, W, bits, cfg.g)


@pytest.mark.parametrize("bits", [2, 4])
@pytest.mark.parametrize("group", [64, 128])
def test_pack_edge_groups_bit_exact(q, bits, group):
    """All-zero groups, single-sign groups, subnormal scales, ties, the
    largest finite scale and overflowing / non-finite groups."""
    _announce("pack edge", bits, group)
    rng = np.random.default_rng(11)
    n, k = 40, 4 * group
    W = (0.02 * rng.standard_normal((n, k))).astype(np.float32)
    W[0, :group] = 0.0                                     # all-zero group
    W[1, :group] = np.abs(W[1, :group])                    # single-sign (positive)
    W[2, group:2 * group] = -np.abs(W[2, group:2 * group])  # single-sign (negative)
    W[3, :group] = 0.0
    W[3, 5] = 3e-7                                         # subnormal scale
    W[4, :group] = rng.integers(-2, 3, size=group) * 0.5   # exact halves: ties
    W[4, 0], W[4, 1] = -1.0, 2.0 if bits == 2 else 14.0   # scale 1.0, so +-0.5 are ties
    W[5, :group] = 0.0
    W[5, 1] = 196559.0 if bits == 2 else 982799.0          # largest finite scale
    W[6, :group] = rng.standard_normal(group).astype(np.float32) * 1e6   # overflow -> invalid
    W[7, 2 * group + 3] = np.nan                           # non-finite -> invalid
    W[8, 3 * group + 1] = np.inf
    W[9, :] = 1e-30                                        # range underflows: scale 1.0
    ref = orc.quantize(W, bits, group)
    assert ref.bad >= 3
    _check_pack(q, W, bits, group, ref)


def test_pack_status_clear_for_finite_weights(q):
    _announce("pack status")
    W = wl.weight(wl.CONFIGS["tiny"], 0, 0)
    qw = q.pack_w2(torch.from_numpy(W).cuda(), 64)
    assert not qw.invalid_groups()


# ------------------------------------------------------------- gate/up + down
@pytest.mark.parametrize("name", sorted(DECODE_CASES))
def test_gateup_matches_oracle(q, name):
    cfg = DECODE_CASES[name]
    _announce("gateup", name, "M", cfg.M, "d", cfg.d, "f", cfg.f, "g", cfg.g, "r", cfg.r)
    L = wl.layer(cfg, 0)
    mlp = gpu_mlp(L)
    x = act_tensor(L.x)
    h = q.gateup_w2_lora(mlp, x)
    torch.cuda.synchronize()
    h_ref = orc.gateup(*oracle_q(L)[:2], L.A_gate, L.B_gate, L.A_up, L.B_up, L.x,
                       lora_scale=cfg.lora_scale)
    err = orc.max_rel_err(values_of(h), h_ref)
    print("h max-rel err %.3e" % err)
    assert err <= H_TOL


@pytest.mark.parametrize("name", sorted(DECODE_CASES))
def test_forward_matches_oracle(q, name):
    cfg = DECODE_CASES[name]
    _announce("forward", name, "M", cfg.M, "d", cfg.d, "f", cfg.f, "g", cfg.g, "r", cfg.r)
    L = wl.layer(cfg, 0)
    mlp = gpu_mlp(L)
    x = act_tensor(L.x)
    y = q.forward(mlp, x)
    torch.cuda.synchronize()
    y_ref, _ = oracle_forward(L)
    err = orc.max_rel_err(values_of(y), y_ref)
    print("y max-rel err %.3e" % err)
    assert err <= Y_TOL


@pytest.mark.parametrize("name", ["tiny", "qwen3_4b", "ragged_g128_m5"])
def test_down_alone_matches_oracle_on_same_h(q, name):
    """qmlp_down_w4 on a given binary16 h against the oracle's down on exactly
    that h: isolates the 4-bit kernel from the gate/up error."""
    cfg = DECODE_CASES[name]
    _announce("down", name)
    L = wl.layer(cfg, 0)
    mlp = gpu_mlp(L)
    rng = np.random.default_rng(5)
    h_bits = wl.f32_to_f16_bits(rng.standard_normal((cfg.M, cfg.f)).astype(np.float32))
    y = q.down_w4(mlp.down, act_tensor(h_bits))
    torch.cuda.synchronize()
    y_ref = orc.down_act(oracle_q(L)[2], h_bits)
    err = orc.max_rel_err(values_of(y), y_ref)
    print("y max-rel err %.3e" % err)
    assert err <= 2e-3


# ------------------------------------------------------------- LoRA isolation
def test_zero_B_equals_zero_scale_bitwise_and_rank0_within_tol(q):
    """B = 0 makes the LoRA term exactly 0, so y(B=0) is bit-equal to
    y(lora_scale=0) from the same kernels, and within tolerance of the
    rank-0 path.  Also catches reads of an uninitialised t."""
    cfg = wl.CONFIGS["qwen3_4b"]
    _announce("lora B=0", cfg.name)
    L = wl.layer(cfg, 1)
    L0 = wl.Layer(cfg, 1, L.W_gate, L.W_up, L.W_down, L.A_gate, np.zeros_like(L.B_gate),
                  L.A_up, np.zeros_like(L.B_up), L.x)
    x = act_tensor(L.x)
    m_zero_b = gpu_mlp(L0)
    m_zero_scale = gpu_mlp(L, lora_scale=0.0)
    m_rank0 = gpu_mlp(L, rank=False)
    ws = q.workspace(m_zero_b, cfg.M)
    # garbage after the control block: its tags (0x7F7F) never match the
    # first call's tag (1), so nothing stale can be taken for t or h
    ws[1024:].fill_(0x7F)
    y0 = q.forward(m_zero_b, x, ws=ws)
    y1 = q.forward(m_zero_scale, x)
    y2 = q.forward(m_rank0, x)
    torch.cuda.synchronize()
    assert torch.equal(y0.view(torch.int16), y1.view(torch.int16))
    assert q.workspace_errors(ws) == 0
    y_ref, _ = oracle_forward(L, rank=False)
    assert orc.max_rel_err(values_of(y2), y_ref) <= Y_TOL
    assert orc.max_rel_err(values_of(y0), y_ref) <= Y_TOL


@pytest.mark.parametrize("amplify", [1.0, 25.0])
def test_lora_only_path(q, amplify):
    """W_gate = W_up = 0 pack to scale 1, zero 0, codes 0, so h is the pure
    low-rank term; with B amplified x25 the adapter dominates y."""
    cfg = wl.scaled(wl.CONFIGS["qwen3_4b"], M=2)
    _announce("lora only", amplify)
    L = wl.layer(cfg, 2)
    zero = np.zeros_like(L.W_gate)
    Bg = wl.f32_to_f16_bits(orc.act_to_f64(L.B_gate, False).astype(np.float32) * amplify)
    Bu = wl.f32_to_f16_bits(orc.act_to_f64(L.B_up, False).astype(np.float32) * amplify)
    L2 = wl.Layer(cfg, 2, zero, zero, L.W_down, L.A_gate, Bg, L.A_up, Bu, L.x)
    mlp = gpu_mlp(L2, lora_scale=2.0)
    x = act_tensor(L.x)
    h = q.gateup_w2_lora(mlp, x)
    y = q.forward(mlp, x)
    torch.cuda.synchronize()
    y_ref, h_ref = oracle_forward(L2, lora_scale=2.0)
    assert np.abs(h_ref).max() > 0
    assert orc.max_rel_err(values_of(h), h_ref) <= H_TOL
    assert orc.max_rel_err(values_of(y), y_ref) <= Y_TOL


def test_lora_term_matters_at_h(q):
    """Dropping the adapter moves h by more than the stage tolerance, so the
    h comparisons above do test the LoRA path."""
    cfg = wl.CONFIGS["qwen3_4b"]
    L = wl.layer(cfg, 3)
    _, h_ref = oracle_forward(L)
    _, h_nolora = oracle_forward(L, rank=False)
    assert orc.max_rel_err(h_nolora, h_ref) > 2 * H_TOL


# ------------------------------------------------------------- invariants
def test_rows_independent_and_deterministic(q):
    cfg = wl.CONFIGS["qwen3_8b_m16"]
    _announce("row independence", cfg.name)
    L = wl.layer(cfg, 0, M=8)
    mlp = gpu_mlp(L)
    x = act_tensor(L.x)
    y8 = q.forward(mlp, x)
    y8b = q.forward(mlp, x)
    rows = [q.forward(mlp, x[m:m + 1].contiguous()) for m in range(8)]
    torch.cuda.synchronize()
    assert torch.equal(y8.view(torch.int16), y8b.view(torch.int16))
    y_ref, _ = oracle_forward(L)
    for m in range(8):
        assert orc.max_rel_err(values_of(rows[m]), y_ref[m:m + 1]) <= Y_TOL
        assert orc.max_rel_err(values_of(rows[m]), values_of(y8[m:m + 1])) <= 2 * Y_TOL


def test_outputs_leave_guard_bands_untouched(q):
    cfg = DECODE_CASES["ragged_g128_m5"]
    _announce("guard bands", cfg.name)
    L = wl.layer(cfg, 0)
    mlp = gpu_mlp(L)
    x = act_tensor(L.x)
    pad = 4096
    ybuf = torch.full((cfg.M * cfg.d + 2 * pad,), 12345, dtype=torch.int16, device="cuda")
    hbuf = torch.full((cfg.M * cfg.f + 2 * pad,), 12345, dtype=torch.int16, device="cuda")
    y = ybuf[pad:pad + cfg.M * cfg.d].view(torch.float16).view(cfg.M, cfg.d)
    h = hbuf[pad:pad + cfg.M * cfg.f].view(torch.float16).view(cfg.M, cfg.f)
    q.forward(mlp, x, y=y)
    q.gateup_w2_lora(mlp, x, h=h)
    torch.cuda.synchronize()
    for buf in (ybuf, hbuf):
        assert bool((buf[:pad] == 12345).all()) and bool((buf[-pad:] == 12345).all())
    y_ref, h_ref = oracle_forward(L)
    assert orc.max_rel_err(values_of(y), y_ref) <= Y_TOL
    assert orc.max_rel_err(values_of(h), h_ref) <= H_TOL


def test_empty_batch_is_a_noop(q):
    cfg = wl.CONFIGS["tiny"]
    L = wl.layer(cfg, 0)
    mlp = gpu_mlp(L)
    x = torch.empty((0, cfg.d), dtype=torch.float16, device="cuda")
    y = q.forward(mlp, x, ws=torch.zeros(1024, dtype=torch.uint8, device="cuda"))
    assert y.shape == (0, cfg.d)


def test_full_stack_sampled_layers(q):
    """The 36 Qwen3-4B-shaped blocks exactly as the benchmark times them (one
    qmlp_forward_layers call over every block's own input, the bench's
    workspace and stream); blocks 0, 17 and 35 checked in full against the
    oracle."""
    cfg = wl.CONFIGS["qwen3_4b"]
    _announce("full stack", cfg.name, "L", cfg.L)
    import bench
    stack = bench.build_stack(cfg, seed=0)
    ys = bench.run_blocks_once(stack)
    torch.cuda.synchronize()
    assert q.layers_path(stack.lay, 1) == "streamed"
    for i in (0, 17, cfg.L - 1):
        L = wl.layer(cfg, i)
        y_ref, _ = oracle_forward(L)
        err = orc.max_rel_err(values_of(ys[i]), y_ref)
        print("layer %d y max-rel err %.3e" % (i, err))
        assert err <= Y_TOL


# ------------------------------------------------------------- fused layer kernel
@pytest.mark.parametrize("name", ["tiny", "qwen3_4b", "qwen3_8b_m4"])
def test_fused_forward_control_block(q, name):
    """The one-kernel-per-layer forward hands t and h between compute units
    as words tagged with the call counter (control word 0); after n calls the
    counter reads n, the finish count (word 32) is back to zero, no error bit
    is set, the rest of the control block is untouched, and repeated calls
    give bit-identical y."""
    cfg = DECODE_CASES[name]
    _announce("fused control block", name)
    L = wl.layer(cfg, 0)
    mlp = gpu_mlp(L)
    assert q.forward_launches(mlp, cfg.M) == 1
    x = act_tensor(L.x)
    ws = q.workspace(mlp, cfg.M)
    ys = [q.forward(mlp, x, ws=ws) for _ in range(5)]
    torch.cuda.synchronize()
    ctl = ws[:1024].view(torch.int32).cpu().numpy()
    assert ctl[0] == 5 and ctl[32] == 0 and q.workspace_errors(ws) == 0
    assert np.count_nonzero(ctl) == 1
    for y in ys[1:]:
        assert torch.equal(y.view(torch.int16), ys[0].view(torch.int16))
    y_ref, _ = oracle_forward(L)
    assert orc.max_rel_err(values_of(ys[0]), y_ref) <= Y_TOL


def test_fused_tags_across_token_counts_and_counter_wrap(q):
    """Stale hand-off words never pass for current ones: one workspace serves
    calls at 4, 1, 2 and 4 tokens (rows left over from an earlier call carry
    an older tag), and the call counter wraps its 16-bit tag (65534, 65535,
    65536 -> tags 65535, 1, 2)."""
    cfg = wl.CONFIGS["qwen3_8b_m4"]
    _announce("fused tags", cfg.name)
    L = wl.layer(cfg, 2)
    mlp = gpu_mlp(L)
    ws = q.workspace(mlp, 4)
    y_ref, _ = oracle_forward(L)
    for start in (0, 65534):
        ws[:4] = torch.tensor([start], dtype=torch.int32).view(torch.uint8).cuda()
        for M in (4, 1, 2, 4):
            assert q.forward_launches(mlp, M) == 1
            y = q.forward(mlp, act_tensor(L.x[:M]), ws=ws)
            torch.cuda.synchronize()
            assert q.workspace_errors(ws) == 0
            assert orc.max_rel_err(values_of(y), y_ref[:M]) <= Y_TOL
        assert int(ws[:4].view(torch.int32).item()) == start + 4


def test_graph_replays_match_eager(q):
    """A HIP graph of three layers' forwards, replayed several times with
    eager work and synchronizations in between, reproduces the eager outputs
    bit for bit on every replay."""
    cfg = wl.CONFIGS["qwen3_4b"]
    _announce("graph replay", cfg.name)
    layers = [wl.layer(cfg, i) for i in range(3)]
    mlps = [gpu_mlp(L) for L in layers]
    xs = [act_tensor(L.x) for L in layers]
    ws = q.workspace(mlps[0], cfg.M)
    ys = [torch.empty((cfg.M, cfg.d), dtype=torch.float16, device="cuda") for _ in layers]
    for m, x, y in zip(mlps, xs, ys):
        q.forward(m, x, y=y, ws=ws)
    torch.cuda.synchronize()
    eager = [y.clone() for y in ys]
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            for m, x, y in zip(mlps, xs, ys):
                q.forward(m, x, y=y, ws=ws)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for rep in range(4):
        for y in ys:
            y.fill_(0)
        junk = torch.randn(1 << 20, device="cuda").sum()      # eager work between replays
        g.replay()
        torch.cuda.synchronize()
        assert float(junk) == float(junk)
        for y, e in zip(ys, eager):
            assert torch.equal(y.view(torch.int16), e.view(torch.int16)), rep
    assert q.workspace_errors(ws) == 0
