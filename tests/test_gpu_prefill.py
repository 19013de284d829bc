"""GPU parity of the prefill-chunk path (M a multiple of 128, bfloat16
activations, MFMA) against the fp64 oracle, through the C ABI.

Bar:
  * h: max|h - h_ref| / max|h_ref| <= 8e-3.  h is stored in bfloat16
    (relative step 2^-8, so up to 2^-9 ~ 1.95e-3 of an element per rounding);
    the dequantized weights enter the matrix cores as bfloat16 (one rounding
    of scale * (q - zero) each, random errors of relative size <= 2^-9 that
    add up to ~2^-9 / sqrt(3) of a dot product) and t enters the LoRA product
    as bfloat16 of lora_scale * t.  2 x 2^-9 + 2^-9 / sqrt(3) + 2^-9 ~ 7e-3
    bounds what is expected; 8e-3 is the bar.
  * y: max|y - y_ref| / max|y_ref| <= 1e-2, the block's output bar.
The oracle keeps everything in fp64 and does not round h.
"""
import numpy as np
import pytest
import torch

import oracle as orc
import workloads as wl
from qmlp_testutil import act_tensor, bits_of, gpu_mlp, oracle_forward, oracle_q, values_of

pytestmark = pytest.mark.gpu

H_TOL = 8e-3
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


def _down_slices(M, d, f):
    """Slices of f the chunk's down projection takes (the library's rule:
    double while under 512 token x row tiles and f stays whole 128-wide
    steps per slice, at most 8)."""
    S = 1
    while S < 8 and (M // 128) * (d // 128) * S < 512 and f % (2 * S * 64) == 0:
        S *= 2
    return S


PREFILL_CASES = {
    # several 128-token tiles, several 64-column tiles of h and 128-row tiles
    # of y, groups of 64 and 128, ranks 8 / 16 / 32 (8 and 16 exercise the
    # zero-padded LoRA step), more than one split of the LoRA-A reduction
    "pf_m128_r8_g64": wl.Config("pf_m128_r8_g64", M=128, d=256, f=512, g=64, r=8, L=1, act="bf16"),
    "pf_m256_r16_g64": wl.Config("pf_m256_r16_g64", M=256, d=384, f=320, g=64, r=16, L=1,
                                 act="bf16"),
    "pf_m128_r32_g128": wl.Config("pf_m128_r32_g128", M=128, d=512, f=640, g=128, r=32, L=1,
                                  act="bf16"),
    "pf_m384_r32_g128_out": wl.Config("pf_m384_r32_g128_out", M=384, d=768, f=1024, g=128, r=32,
                                      L=1, act="bf16", outliers=True),
    # 256-token tiles with 128 columns of h per block (f % 128 == 0), two
    # token tiles, down over slices of f
    "pf_m512_r16_g128_wide": wl.Config("pf_m512_r16_g128_wide", M=512, d=512, f=768, g=128, r=16,
                                       L=1, act="bf16"),
}


@pytest.mark.parametrize("name", sorted(PREFILL_CASES))
def test_prefill_gateup_matches_oracle(q, name):
    cfg = PREFILL_CASES[name]
    _announce("prefill gateup", name, "M", cfg.M, "d", cfg.d, "f", cfg.f, "g", cfg.g, "r", cfg.r)
    L = wl.layer(cfg, 0)
    mlp = gpu_mlp(L)
    x = act_tensor(L.x, "bf16")
    h = q.gateup_w2_lora(mlp, x)
    torch.cuda.synchronize()
    h_ref = orc.gateup(*oracle_q(L)[:2], L.A_gate, L.B_gate, L.A_up, L.B_up, L.x,
                       lora_scale=cfg.lora_scale, bf16=True)
    err = orc.max_rel_err(values_of(h, "bf16"), h_ref)
    print("h max-rel err %.3e" % err)
    assert err <= H_TOL


@pytest.mark.parametrize("name", sorted(PREFILL_CASES))
def test_prefill_forward_matches_oracle(q, name):
    cfg = PREFILL_CASES[name]
    _announce("prefill forward", name, "M", cfg.M, "d", cfg.d, "f", cfg.f, "g", cfg.g, "r", cfg.r)
    L = wl.layer(cfg, 0)
    mlp = gpu_mlp(L)
    S = _down_slices(cfg.M, cfg.d, cfg.f)
    assert q.forward_launches(mlp, cfg.M, torch.bfloat16) == 4 + (S > 1)
    print("down slices", S)
    y = q.forward(mlp, act_tensor(L.x, "bf16"))
    torch.cuda.synchronize()
    y_ref, _ = oracle_forward(L)
    err = orc.max_rel_err(values_of(y, "bf16"), y_ref)
    print("y max-rel err %.3e" % err)
    assert err <= Y_TOL


def test_prefill_down_alone_matches_oracle_on_same_h(q):
    cfg = PREFILL_CASES["pf_m256_r16_g64"]
    _announce("prefill down alone", cfg.name)
    L = wl.layer(cfg, 0)
    mlp = gpu_mlp(L)
    h = q.gateup_w2_lora(mlp, act_tensor(L.x, "bf16"))
    y = q.down_w4(mlp.down, h)
    torch.cuda.synchronize()
    y_ref = orc.down_act(oracle_q(L)[2], bits_of(h), bf16=True)
    err = orc.max_rel_err(values_of(y, "bf16"), y_ref)
    print("y max-rel err %.3e" % err)
    assert err <= Y_TOL


def test_prefill_without_adapter(q):
    cfg = PREFILL_CASES["pf_m128_r8_g64"]
    _announce("prefill rank 0", cfg.name)
    L = wl.layer(cfg, 0)
    mlp = gpu_mlp(L, rank=False)
    assert q.forward_launches(mlp, cfg.M, torch.bfloat16) == 2 + (_down_slices(cfg.M, cfg.d, cfg.f) > 1)
    y = q.forward(mlp, act_tensor(L.x, "bf16"))
    torch.cuda.synchronize()
    y_ref, _ = oracle_forward(L, rank=False)
    err = orc.max_rel_err(values_of(y, "bf16"), y_ref)
    print("y max-rel err %.3e" % err)
    assert err <= Y_TOL


def test_prefill_zero_B_equals_zero_scale_bitwise(q):
    cfg = PREFILL_CASES["pf_m128_r32_g128"]
    _announce("prefill B=0 vs lora_scale=0", cfg.name)
    L = wl.layer(cfg, 0)
    mlp = gpu_mlp(L)
    x = act_tensor(L.x, "bf16")
    zB = q.MLP(mlp.gate, mlp.up, mlp.down, mlp.A_gate, torch.zeros_like(mlp.B_gate), mlp.A_up,
               torch.zeros_like(mlp.B_up), lora_scale=1.0)
    y1 = q.forward(zB, x)
    y2 = q.forward(mlp.with_lora_scale(0.0), x)
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))


def test_prefill_deterministic_and_tiles_independent(q):
    cfg = PREFILL_CASES["pf_m256_r16_g64"]
    _announce("prefill determinism", cfg.name)
    L = wl.layer(cfg, 0)
    mlp = gpu_mlp(L)
    x = act_tensor(L.x, "bf16")
    y1 = q.forward(mlp, x)
    y2 = q.forward(mlp, x)
    # the second 128-token tile alone gives the same rows
    y3 = q.forward(mlp, x[128:].contiguous())
    torch.cuda.synchronize()
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))
    assert torch.equal(y1[128:].view(torch.int16), y3.view(torch.int16))


def test_prefill_full_size_sampled_tokens(q):
    """The 20B-width prefill chunk (M=512, d=6144, f=16384, g128, r32) in the
    launch configuration the benchmark times (down over four slices of f);
    the oracle computes one sampled token of every 128-token tile (rows are
    independent)."""
    cfg = wl.CONFIGS["prefill20b"]
    _announce("prefill full size", cfg.name, "M", cfg.M, "d", cfg.d, "f", cfg.f)
    L = wl.layer(cfg, 0)
    mlp = gpu_mlp(L)
    y = q.forward(mlp, act_tensor(L.x, "bf16"))
    torch.cuda.synchronize()
    assert _down_slices(cfg.M, cfg.d, cfg.f) == 4
    rows = [0, 211, 300, 511]
    yv = values_of(y, "bf16")[rows]
    y_ref, _ = oracle_forward(L, x=np.ascontiguousarray(L.x[rows]))
    err = orc.max_rel_err(yv, y_ref)
    print("sampled y max-rel err %.3e" % err)
    assert err <= Y_TOL
    assert np.isfinite(values_of(y, "bf16")).all()
