#!/usr/bin/env python3
"""Benchmark of the W4/W2-GateUp decode MLP on one MI355X.

A step is one pass over the 36 independently seeded MLP blocks of the
Qwen3-4B-shaped workload (d=2560, f=9728, 2-bit gate/up and 4-bit down at
group 128, LoRA rank 16, M=1 token, every block with its own weights and
its own input x ~ N(0,1) in binary16), run back to back through
qmlp_forward_layers (three streamed launches at this shape).  Inputs are
packed and resident in HBM before the timed region.  Prints one JSON line:

  value    = achieved HBM GB/s = L * B(M) / t_step, where B(M) are the
             algorithmic bytes of one MLP step (packed codes + fp16
             scale/zero + LoRA factors + x in + y out; the intermediate h
             excluded, as the fused gate-activation-down keeps it on-chip);
  roofline = the step's algorithmic bytes over its duration (HIP events
             on the launch stream around the K back-to-back steps; a step is
             one qmlp_forward_layers call: the LoRA-A launch, then the
             gate/up and down launches over every block); traffic = HBM bytes
             of those launches from the rocprofv3 byte counters summarized
             under profiles/, reported only while the HIP sources match the
             ones profiled;
  cpu_baseline = the fp64 oracle timed on a bounded sample of the same
             blocks on this host (reported baseline only).

For context the same blocks are also timed as a decoder stack on a
residual stream (x_{l+1} = x_l + block_l(RMSNorm(x_l)), each block's input
depending on the previous block's output, qmlp_forward_stack) and one
qmlp_forward launch per block.

precision_comparison: the MLP-level analogue of the paper's Gain and
Capture (Sec. 5.2) on this GPU.  The same fp32 weights are packed as uniform
W4 (gate/up and down at 4 bits), uniform W2, W4/W2-GateUp with its LoRA
adapters, W4/W2-GateUp with the paper's INT2 group of 32, and the 3-bit
gate/up of Appendix B at group 32; all five run on the same stand-alone
decode kernels (qmlp_forward_batch: LoRA-A, gate/up and down of every block
in one launch each; one pass over the 36 blocks captured in a HIP graph), so
the comparison isolates the bit widths:  Gain = TPS_mix / TPS_W4 - 1,
Capture = (TPS_mix - TPS_W4) / (TPS_W2 - TPS_W4), TPS = 1 / (us per MLP step).

decoder_model: the same comparison for a whole Qwen3-4B-shaped decoder token
(attention projections, MLPs, LM head, and a KV-cache read standing in for
attention; Sec. 5.2's method with measured times).
"""
from __future__ import annotations

import argparse
import concurrent.futures
import dataclasses
import json
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workloads as wl  # noqa: E402
from paper_2606_04238_amd.profiling import read_traffic  # noqa: E402

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, 8 TB/s
# the kernels of one step of qmlp_forward_layers on each path, as named in
# the kernel trace (profile summaries); the streamed gate/up launch also
# computes LoRA-A
STEP_KERNELS = {"streamed": "gu_stream_kernel|dn_stream_kernel",
                "mfma": "mf_lora_kernel|mf_gu_kernel|mf_dn_kernel"}
METRIC = BASE_METRIC = ("achieved HBM GB/s (% of MI355X peak) and µs per W4/W2-GateUp MLP "
                        "decode step")


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


# --------------------------------------------------------------------- stack
class Stack:
    def __init__(self, cfg, mlps, xs, ys, ws, variants=None):
        self.cfg, self.mlps, self.xs, self.ys, self.ws = cfg, mlps, xs, ys, ws
        self.variants = variants or {}                 # name -> [MLP] at other widths
        import torch
        import paper_2606_04238_amd as q
        self.st = q.Stack(mlps)
        self.Y = torch.empty((len(mlps), cfg.M, cfg.d), dtype=ys[0].dtype, device="cuda")
        self.sws = q.stack_workspace(self.st, cfg.M, ys[0].dtype) if cfg.M > 0 and not cfg.bf16 else None
        self.lay = q.Layers(mlps)
        self.X = torch.stack(xs)                       # [L][M][d]: every block's own input
        self.YL = torch.empty_like(self.X)
        self.lws = q.layers_workspace(self.lay, cfg.M, ys[0].dtype)


def _gen_layer(cfg, i, seed):
    return wl.layer(cfg, i, seed)


# The precision comparison (Sec. 5.2): (gate/up bits, gate/up group, down
# bits, down group, adapters); group None = the workload's group.
VARIANTS = {
    "w4_uniform": (4, None, 4, None, False),
    "w2_uniform": (2, None, 2, None, False),
    "w4w2_gateup_lora": (2, None, 4, None, True),
    "w4w2_gateup_g32_lora": (2, 32, 4, None, True),
    "w4w3_gateup_g32_lora": (3, 32, 4, None, True),        # the W3 variant of Appendix B
}


def variant_widths(cfg: wl.Config, name: str):
    bg, gg, bd, gd, lora = VARIANTS[name]
    return bg, gg or cfg.g, bd, gd or cfg.g, lora


def variant_bytes(cfg: wl.Config, name: str) -> int:
    """Algorithmic bytes of one MLP step at a variant's widths: codes
    (2 f d bg/8 + d f bd/8), fp16 scale+zero (8 f d/gg + 4 d f/gd), the
    LoRA factors when the variant carries adapters, x in and y out."""
    bg, gg, bd, gd, lora = variant_widths(cfg, name)
    f, d, M, r = cfg.f, cfg.d, cfg.M, cfg.r
    n = 2 * f * d * bg // 8 + d * f * bd // 8 + 8 * f * d // gg + 4 * d * f // gd + 4 * M * d
    return n + (4 * r * (d + f) if lora else 0)


def build_stack(cfg: wl.Config, seed: int = 0, layers: int | None = None, threads: int = 16,
                variants: bool = False) -> Stack:
    """Generate the seeded layers on the host (parallel), pack them on the GPU
    (with `variants`, also at the other widths of the precision comparison)."""
    import torch
    import paper_2606_04238_amd as q
    L = cfg.L if layers is None else layers
    mlps, xs, ys = [], [], []
    var = {k: [] for k in VARIANTS} if variants else {}
    t0 = time.time()
    with concurrent.futures.ThreadPoolExecutor(max_workers=threads) as ex:
        futs = [ex.submit(_gen_layer, cfg, i, seed) for i in range(L)]
        for fut in futs:
            lay = fut.result()
            dt = torch.bfloat16 if cfg.bf16 else torch.float16

            def act(a):
                return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(dt).cuda()
            Wg, Wu, Wd = (torch.from_numpy(w).cuda() for w in (lay.W_gate, lay.W_up, lay.W_down))
            g = q.pack_w2(Wg, cfg.g)
            u = q.pack_w2(Wu, cfg.g)
            d = q.pack_w4(Wd, cfg.g)
            lo = (act(lay.A_gate), act(lay.B_gate), act(lay.A_up), act(lay.B_up))
            mlps.append(q.MLP(g, u, d, *lo, lora_scale=cfg.lora_scale))
            for name in var:
                bg, gg, bd, gd, lora = variant_widths(cfg, name)
                pk = {2: q.pack_w2, 3: q.pack_w3, 4: q.pack_w4}
                vg, vu, vd = pk[bg](Wg, gg), pk[bg](Wu, gg), pk[bd](Wd, gd)
                var[name].append(q.MLP(vg, vu, vd, *(lo if lora else ()),
                                       lora_scale=cfg.lora_scale))
            del Wg, Wu, Wd
            xs.append(act(lay.x))
            ys.append(torch.empty((cfg.M, cfg.d), dtype=dt, device="cuda"))
            fut._result = None          # drop the fp32 host copies
    torch.cuda.synchronize()
    for m in mlps + [v for vs in var.values() for v in vs]:
        for w in (m.gate, m.up, m.down):
            if w.invalid_groups():
                raise RuntimeError("packer flagged invalid groups")
    ws = q.workspace(mlps[0], cfg.M, ys[0].dtype)
    log("built %d layers%s in %.1f s" % (L, " (+%d width variants)" % len(var) if var else "",
                                         time.time() - t0))
    return Stack(cfg, mlps, xs, ys, ws, var)


def run_blocks_once(stack: Stack):
    """One step: every block on its own input, back to back (qmlp_forward_layers)."""
    import paper_2606_04238_amd as q
    q.forward_layers(stack.lay, stack.X, y=stack.YL, ws=stack.lws)
    return stack.YL


def run_stack_once(stack: Stack):
    """The blocks as a decoder stack on the residual stream from layer 0's x."""
    import paper_2606_04238_amd as q
    q.forward_stack(stack.st, stack.xs[0], y=stack.Y, ws=stack.sws)
    return stack.Y


def run_layers_once(stack: Stack):
    """The per-layer path for comparison: one qmlp_forward per layer, each on
    its own seeded input."""
    import paper_2606_04238_amd as q
    for m, x, y in zip(stack.mlps, stack.xs, stack.ys):
        q.forward(m, x, y=y, ws=stack.ws)
    return stack.ys


def run_variant_once(stack: Stack, name: str):
    """One pass of a width variant over every block: qmlp_forward_batch, the
    stand-alone decode kernels in batches of up to 40 blocks (LoRA-A,
    gate/up and down of every block of a batch)."""
    import paper_2606_04238_amd as q
    lay, ws = stack.variant_layers[name]
    return q.forward_batch(lay, stack.X, y=stack.YB, ws=ws)


def precision_comparison(stack: Stack, seed: int, steps: int, min_warm_s: float, mix_us: float):
    """us per MLP step of each width variant (graph replay of one pass over
    the blocks), its achieved GB/s, the oracle parity of block 0 and block
    L-1, and the MLP-level Gain / Capture of the two W4/W2-GateUp variants;
    beside them the Gain of the streamed W4/W2-GateUp path (mix_us, the
    headline) over uniform W4 on the batched kernels."""
    import torch
    import oracle as orc
    import paper_2606_04238_amd as q
    cfg = stack.cfg
    L = len(stack.mlps)
    stack.YB = torch.empty_like(stack.X)
    stack.variant_layers = {}
    samples = {i: wl.layer(cfg, i, seed) for i in (0, L - 1)}
    res = {}
    for name in VARIANTS:
        lay = q.Layers(stack.variants[name])
        stack.variant_layers[name] = (lay, q.batch_workspace(lay, cfg.M))
        g = capture(lambda: run_variant_once(stack, name))
        ms, _ = time_passes(g.replay, steps, 2, min_warm_s)
        us = sum(ms) / len(ms) * 1e3 / L
        run_variant_once(stack, name)
        torch.cuda.synchronize()
        Y = stack.YB.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
        bg, gg, bd, gd, lora = variant_widths(cfg, name)
        errs = []
        for i, ly in samples.items():
            qg, qu, qd = (orc.quantize(ly.W_gate, bg, gg), orc.quantize(ly.W_up, bg, gg),
                          orc.quantize(ly.W_down, bd, gd))
            lo = (ly.A_gate, ly.B_gate, ly.A_up, ly.B_up) if lora else (None,) * 4
            y_ref = orc.forward(qg, qu, qd, *lo, ly.x, lora_scale=cfg.lora_scale)
            errs.append(orc.max_rel_err(orc.act_to_f64(Y[i], False), y_ref))
        b = variant_bytes(cfg, name)
        res[name] = {"us_per_mlp_step": round(us, 3), "alg_bytes_per_mlp_step": b,
                     "gbs": round(b / (us * 1e-6) / 1e9, 1),
                     "frac_of_hbm_peak": round(b / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                     "launches_per_step": (L + 39) // 40 * (3 if lora else 2),
                     "parity_max_rel_err_blocks_0_last": float("%.3e" % max(errs))}
    t4, t2 = res["w4_uniform"]["us_per_mlp_step"], res["w2_uniform"]["us_per_mlp_step"]
    b4, b2 = variant_bytes(cfg, "w4_uniform"), variant_bytes(cfg, "w2_uniform")
    out = {"mlp_us": {k: v["us_per_mlp_step"] for k, v in res.items()},
           "kernels": "qmlp_forward_batch: stand-alone decode kernels, one launch each for "
                      "LoRA-A, gate/up and down of up to 40 blocks; HIP graph over %d blocks" % L,
           "variants": res}
    for name in ("w4w2_gateup_lora", "w4w2_gateup_g32_lora", "w4w3_gateup_g32_lora"):
        tm, bm = res[name]["us_per_mlp_step"], variant_bytes(cfg, name)
        out[name] = {
            "gain_pct": round((t4 / tm - 1) * 100, 1),
            "capture_pct": round((1 / tm - 1 / t4) / (1 / t2 - 1 / t4) * 100, 1),
            # the same two figures if every variant moved its bytes at one bandwidth
            "bytes_model_gain_pct": round((b4 / bm - 1) * 100, 1),
            "bytes_model_capture_pct": round((1 / bm - 1 / b4) / (1 / b2 - 1 / b4) * 100, 1)}
    out["streamed_w4w2_gateup_lora"] = {
        "us_per_mlp_step": round(mix_us, 3),
        "gain_pct_over_batched_w4": round((t4 / mix_us - 1) * 100, 1),
        "capture_pct_batched_w2_w4": round((1 / mix_us - 1 / t4) / (1 / t2 - 1 / t4) * 100, 1)}
    return out


def decoder_model(stack: Stack, seed: int, steps: int, min_warm_s: float, mlp_us: dict,
                  threads: int = 16):
    """Whole-model decode throughput of W4, W2 and W4/W2-GateUp on this GPU,
    the method of Sec. 5.2 (per-token time summed over the operators, TPS =
    1 / time) with measured times: per layer the q/k/v projection
    (one [q + 2 kv][d] matrix) and the o projection (qmlp_linear_batch over
    the layers; 4-bit, or 2-bit for W2), the MLP (mlp_us: the precision
    comparison's pass), and the read of a BF16 KV cache of ctx positions (a
    read-only pass of this library's streaming kernel over that many bytes
    stands in for attention, which is not built); per token the LM head at
    the linears' width.  The weight part of
    a token is timed as one graph per width; the per-operator times are
    reported beside it."""
    import torch
    import oracle as orc
    import paper_2606_04238_amd as q
    cfg = stack.cfg
    dims = wl.DECODERS[cfg.name]
    L, d, g = len(stack.mlps), cfg.d, cfg.g
    shapes = {"qkv": (dims.qkv_rows(), d, wl.TID_QKV), "o": (d, dims.o_cols(), wl.TID_O)}
    packs = {b: {k: [] for k in shapes} for b in (4, 2)}
    t0 = time.time()
    with concurrent.futures.ThreadPoolExecutor(max_workers=threads) as ex:
        for name, (n, k, tid) in shapes.items():
            futs = [ex.submit(wl.linear_weight, n, k, i, tid, seed) for i in range(L)]
            for fut in futs:
                W = torch.from_numpy(fut.result()).cuda()
                packs[4][name].append(q.pack_w4(W, g))
                packs[2][name].append(q.pack_w2(W, g))
                del W
                fut._result = None
    W = torch.from_numpy(wl.linear_weight(dims.vocab, d, 0, wl.TID_LM_HEAD, seed)).cuda()
    lm = {4: q.pack_w4(W, g), 2: q.pack_w2(W, g)}
    del W
    torch.cuda.synchronize()
    log("packed the attention projections and the LM head in %.1f s" % (time.time() - t0))
    xs = {name: torch.stack([torch.from_numpy(wl.linear_input(1, k, i, tid, seed).view(np.int16))
                             .view(torch.float16) for i in range(L)]).cuda()
          for name, (n, k, tid) in shapes.items()}
    xl = torch.from_numpy(wl.linear_input(1, d, 0, wl.TID_LM_HEAD, seed).view(np.int16)).view(
        torch.float16).cuda().reshape(1, 1, d)
    us = {}
    for b in (4, 2):
        for name in shapes:
            ys = torch.empty((L, 1, shapes[name][0]), dtype=torch.float16, device="cuda")
            gr = capture(lambda: q.linear_batch(packs[b][name], xs[name], y=ys))
            ms, _ = time_passes(gr.replay, steps, 2, min_warm_s)
            us[(b, name)] = sum(ms) / len(ms) * 1e3
            if b == 4 or name == "o":           # parity of layer 0 against the oracle
                n, k, tid = shapes[name]
                qt = orc.quantize(wl.linear_weight(n, k, 0, tid, seed), b, g)
                ref = orc.down_act(qt, wl.linear_input(1, k, 0, tid, seed))
                got = ys[0].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
                err = orc.max_rel_err(orc.act_to_f64(got, False), ref)
                if not err <= 1e-2:
                    raise RuntimeError("linear %s at %d bits: max-rel %.3e" % (name, b, err))
        yl = torch.empty((1, 1, dims.vocab), dtype=torch.float16, device="cuda")
        gr = capture(lambda: q.linear_batch([lm[b]], xl, y=yl))
        ms, _ = time_passes(gr.replay, steps, 2, min_warm_s)
        us[(b, "lm_head")] = sum(ms) / len(ms) * 1e3
    # the KV stand-in: one read-only pass over the BF16 bytes (pairs of 1.0)
    # with the streaming probe's 128-bit non-temporal loads, timed eagerly;
    # every wave reads an even number of equal words, so their XORs are zero
    kv = torch.full((L * dims.kv_bytes_per_layer() // 4,), 0x3F803F80, dtype=torch.int32, device="cuda")
    kvo = torch.empty(4 * 256, dtype=torch.int32, device="cuda")
    ms, _ = time_passes(lambda: q.probe_stream_read(kv, 256, True, kvo), steps, 2, min_warm_s)
    kv_us = sum(ms) / len(ms) * 1e3
    torch.cuda.synchronize()
    if torch.any(kvo != 0):
        raise RuntimeError("KV read stand-in read unexpected data")
    del kv, kvo
    widths = {"w4_uniform": 4, "w2_uniform": 2, "w4w2_gateup_lora": 4}
    out = {"dims": dataclasses.asdict(dims),
           "ops_us_per_token": {"qkv_4bit": round(us[(4, "qkv")], 2), "o_4bit": round(us[(4, "o")], 2),
                                "qkv_2bit": round(us[(2, "qkv")], 2), "o_2bit": round(us[(2, "o")], 2),
                                "lm_head_4bit": round(us[(4, "lm_head")], 2),
                                "lm_head_2bit": round(us[(2, "lm_head")], 2),
                                "kv_read_bf16": round(kv_us, 2)}}
    # the token step as one graph per width (the linears and the MLP of every
    # layer, the LM head): a long replay, steadier than the short per-operator
    # launches above, whose times vary with the clocks between repeats
    ys = {name: torch.empty((L, 1, shapes[name][0]), dtype=torch.float16, device="cuda")
          for name in shapes}
    yl = torch.empty((1, 1, dims.vocab), dtype=torch.float16, device="cuda")
    tps = {}
    for name, b in widths.items():
        lay, ws = stack.variant_layers[name]

        def token():
            q.linear_batch(packs[b]["qkv"], xs["qkv"], y=ys["qkv"])
            q.linear_batch(packs[b]["o"], xs["o"], y=ys["o"])
            q.forward_batch(lay, stack.X, y=stack.YB, ws=ws)
            q.linear_batch([lm[b]], xl, y=yl)
        gr = capture(token)
        ms, _ = time_passes(gr.replay, steps, 2, min_warm_s)
        t_w = sum(ms) / len(ms) * 1e3
        t = t_w + kv_us
        tps[name] = 1e6 / t
        out[name] = {"us_per_token": round(t, 1), "weights_graph_us": round(t_w, 1),
                     "sum_of_operator_us": round(mlp_us[name] * L + us[(b, "qkv")] + us[(b, "o")]
                                                 + us[(b, "lm_head")] + kv_us, 1),
                     "tokens_per_s": round(tps[name], 1)}
    t4, t2, tm = tps["w4_uniform"], tps["w2_uniform"], tps["w4w2_gateup_lora"]
    out["gain_pct"] = round((tm - t4) / t4 * 100, 1)
    out["capture_pct"] = round((tm - t4) / (t2 - t4) * 100, 1)
    return out


def capture(fn):
    """fn captured once in a HIP graph on a side stream."""
    import torch
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=s):
            fn()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    return g


# --------------------------------------------------------------------- timing
def time_passes(fn, steps: int, warmup: int, min_warm_s: float = 0.25):
    """Per-pass durations (ms) with HIP events on the current stream.  The
    untimed warmup runs at least `warmup` passes and at least `min_warm_s`
    seconds of passes, so that the GPU has left its idle clocks before the
    timed region (tens of milliseconds of one step are not enough)."""
    import torch
    t_end = time.perf_counter() + min_warm_s
    done = 0
    while done < warmup or time.perf_counter() < t_end:
        fn()
        done += 1
        if done % 8 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    st = torch.cuda.current_stream()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    t0 = time.perf_counter()
    evs[0].record(st)
    for i in range(steps):
        fn()
        evs[i + 1].record(st)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return [evs[i].elapsed_time(evs[i + 1]) for i in range(steps)], wall


def time_block(fn, steps: int, warmup: int, min_warm_s: float = 0.25):
    """Milliseconds per pass over `steps` passes launched back to back, with
    one event before the first and one after the last (after the same warmup
    as time_passes): nothing else is enqueued between the passes, so the
    figure holds only the GPU's own gaps between them."""
    import torch
    t_end = time.perf_counter() + min_warm_s
    done = 0
    while done < warmup or time.perf_counter() < t_end:
        fn()
        done += 1
        if done % 8 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    st = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(st)
    for _ in range(steps):
        fn()
    e1.record(st)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


# --------------------------------------------------------------------- cpu baseline
def cpu_baseline(cfg: wl.Config, seed: int, budget_s: float = 12.0, max_layers: int | None = None):
    """The fp64 oracle forward (single thread) over the first layers of the
    same stack until ~budget_s of CPU time; quantization is untimed."""
    import oracle as orc
    L = cfg.L if max_layers is None else max_layers
    total_t, n = 0.0, 0
    for i in range(L):
        lay = wl.layer(cfg, i, seed)
        qg, qu, qd = (orc.quantize(lay.W_gate, 2, cfg.g), orc.quantize(lay.W_up, 2, cfg.g),
                      orc.quantize(lay.W_down, 4, cfg.g))
        t0 = time.perf_counter()
        orc.forward(qg, qu, qd, lay.A_gate, lay.B_gate, lay.A_up, lay.B_up, lay.x,
                    lora_scale=cfg.lora_scale, bf16=cfg.bf16)
        total_t += time.perf_counter() - t0
        n += 1
        if total_t >= budget_s:
            break
    gbs = n * cfg.alg_bytes() / total_t / 1e9
    return {"value": round(gbs, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": "oracle forward (fp64, one thread) over layers 0..%d of the %d-layer stack, "
                      "%.2f s; quantization untimed; us per MLP step %.0f" % (n - 1, cfg.L, total_t,
                                                                            total_t / n * 1e6)}


def parity_blocks(stack: Stack, seed: int, sample=(0,)):
    """Max-rel error of the sampled blocks' outputs of the last timed step
    against the oracle on each block's own input."""
    import torch
    import oracle as orc
    cfg = stack.cfg
    Y = stack.YL.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    out = {}
    for i in sample:
        lay = wl.layer(cfg, i, seed)
        qg, qu, qd = (orc.quantize(lay.W_gate, 2, cfg.g), orc.quantize(lay.W_up, 2, cfg.g),
                      orc.quantize(lay.W_down, 4, cfg.g))
        y_ref = orc.forward(qg, qu, qd, lay.A_gate, lay.B_gate, lay.A_up, lay.B_up, lay.x,
                            lora_scale=cfg.lora_scale, bf16=cfg.bf16)
        out[i] = orc.max_rel_err(orc.act_to_f64(Y[i], cfg.bf16), y_ref)
    return out


def parity_sampled(stack: Stack, seed: int, sample=(0,)):
    """Max-rel error of the sampled layers' outputs of the last timed step
    against the oracle on the norm of each layer's stream state (recomputed
    from x_0 and the GPU outputs: x_{l+1} = x_l + y_l, binary16)."""
    import torch
    import oracle as orc
    cfg = stack.cfg
    Y = stack.Y.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    x = stack.xs[0].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    out = {}
    for i in range(max(sample) + 1):
        if i in sample:
            lay = wl.layer(cfg, i, seed)
            qg, qu, qd = (orc.quantize(lay.W_gate, 2, cfg.g), orc.quantize(lay.W_up, 2, cfg.g),
                          orc.quantize(lay.W_down, 4, cfg.g))
            y_ref = orc.forward(qg, qu, qd, lay.A_gate, lay.B_gate, lay.A_up, lay.B_up,
                                orc.rmsnorm_f16(x), lora_scale=cfg.lora_scale, bf16=cfg.bf16)
            out[i] = orc.max_rel_err(orc.act_to_f64(Y[i], cfg.bf16), y_ref)
        x = orc.residual_f16(x, Y[i])
    return out


# --------------------------------------------------------------------- prefill
MFMA_BF16_PEAK_TFLOPS = 2500.0     # MI355X dense bf16 matrix peak


def prefill_flops(cfg: wl.Config):
    """Algorithmic FLOPs of one prefill chunk: gate/up (4 M f d), down
    (2 M f d), LoRA A and B for gate and up (4 M r (d + f))."""
    M, d, f, r = cfg.M, cfg.d, cfg.f, cfg.r
    gateup = 4 * M * f * d + 4 * M * r * (d + f)
    down = 2 * M * f * d
    return gateup, down


def moe_main(mc: wl.MoeConfig, args):
    """The routed-expert MLP of an MoE decoder (GPT-OSS-20B-class: 24 layers of
    32 experts, top-4, one decode token): one step is qmlp_forward_moe over
    every layer, each layer on its own input and synthetic routing, at three
    widths (uniform W4, uniform W2, W4/W2-GateUp with adapters) for the MoE
    Gain / Capture.  Routing is fixed per layer, so only the 4 routed experts
    of a layer are ever read: those carry their own seeded weights, the other
    28 descriptors of the layer share one packed expert (never read)."""
    import torch
    import oracle as orc
    import paper_2606_04238_amd as q
    cfg = mc.block
    L, E, k, M = cfg.L, mc.experts, mc.topk, cfg.M
    routes = [wl.routing(M, E, k, l, args.seed) for l in range(L)]
    widths = {"w4_uniform": (4, 4, False), "w2_uniform": (2, 2, False),
              "w4w2_gateup_lora": (2, 4, True)}
    pk = {2: q.pack_w2, 4: q.pack_w4}

    def act(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.float16).cuda()

    t0 = time.time()
    filler = wl.layer(cfg, 10_000, args.seed)
    expert_lays = {}
    mlps = {v: [] for v in widths}
    with concurrent.futures.ThreadPoolExecutor(max_workers=16) as ex:
        need = sorted({(l, int(e)) for l in range(L) for e in routes[l][0].reshape(-1)})
        futs = {key: ex.submit(wl.layer, cfg, 1000 * key[0] + key[1], args.seed) for key in need}
        for key, fut in futs.items():
            expert_lays[key] = fut.result()
    dev = {}
    for key, lay in list(expert_lays.items()) + [(None, filler)]:
        Wg, Wu, Wd = (torch.from_numpy(w).cuda() for w in (lay.W_gate, lay.W_up, lay.W_down))
        lo = tuple(act(a) for a in (lay.A_gate, lay.B_gate, lay.A_up, lay.B_up))
        for v, (bg, bd, lora) in widths.items():
            dev[(key, v)] = q.MLP(pk[bg](Wg, cfg.g), pk[bg](Wu, cfg.g), pk[bd](Wd, cfg.g),
                                  *(lo if lora else ()), lora_scale=cfg.lora_scale)
        del Wg, Wu, Wd
    layers = {v: [q.Layers([dev[((l, e), v)] if (l, e) in expert_lays else dev[(None, v)]
                            for e in range(E)]) for l in range(L)] for v in widths}
    torch.cuda.synchronize()
    log("built %d routed experts (+1 shared filler) at 3 widths in %.1f s"
        % (len(expert_lays), time.time() - t0))
    xs = [act(wl.activations(cfg, 5000 + l, args.seed, M=M)) for l in range(L)]
    idx = [torch.from_numpy(r[0]).cuda() for r in routes]
    wts = [torch.from_numpy(r[1]).cuda() for r in routes]
    ys = [torch.empty_like(x) for x in xs]
    res = {}
    for v, (bg, bd, lora) in widths.items():
        wss = [torch.zeros(q.moe_workspace_bytes(layers[v][l], M, k), dtype=torch.uint8, device="cuda")
               for l in range(L)]

        def step():
            for l in range(L):
                q.forward_moe(layers[v][l], xs[l], idx[l], wts[l], y=ys[l], ws=wss[l])
        g = capture(step)
        ms, _ = time_passes(g.replay, args.steps, args.warmup, args.min_warm_s)
        us = sum(ms) / len(ms) * 1e3 / L
        step()
        torch.cuda.synchronize()
        errs = []
        for l in (0, L - 1):
            oq = []
            for e in range(E):
                lay = expert_lays.get((l, e), filler)
                oq.append((orc.quantize(lay.W_gate, bg, cfg.g), orc.quantize(lay.W_up, bg, cfg.g),
                           orc.quantize(lay.W_down, bd, cfg.g))
                          + ((lay.A_gate, lay.B_gate, lay.A_up, lay.B_up) if lora else (None,) * 4)
                          if (l, e) in expert_lays else None)
            ref = orc.moe_forward(oq, routes[l][0], routes[l][1],
                                  wl.activations(cfg, 5000 + l, args.seed, M=M),
                                  lora_scale=cfg.lora_scale)
            got = ys[l].contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
            errs.append(orc.max_rel_err(orc.act_to_f64(got, False), ref))
        f, d = cfg.f, cfg.d
        b_exp = 2 * f * d * bg // 8 + d * f * bd // 8 + 12 * f * d // cfg.g + \
            (4 * cfg.r * (d + f) if lora else 0)
        b = k * M * b_exp + 4 * M * d
        res[v] = {"us_per_moe_layer": round(us, 3), "alg_bytes_per_moe_layer": b,
                  "gbs": round(b / (us * 1e-6) / 1e9, 1),
                  "frac_of_hbm_peak": round(b / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                  "parity_max_rel_err_layers_0_last": float("%.3e" % max(errs))}
        if not max(errs) <= 1e-2:
            raise RuntimeError("moe parity %s: %.3e" % (v, max(errs)))
    t4, t2, tm = (res[v]["us_per_moe_layer"] for v in ("w4_uniform", "w2_uniform", "w4w2_gateup_lora"))
    mix = res["w4w2_gateup_lora"]
    out = {
        "metric": METRIC, "value": mix["gbs"], "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(tm * L / 1e3, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f16", "data": "synthetic",
        "config": {"workload": "%s: %d MoE layers of %d experts (d=%d, f=%d, group %d, LoRA rank %d), "
                               "top-%d routing, M=%d, every layer on its own input and routing"
                               % (mc.name, L, E, cfg.d, cfg.f, cfg.g, cfg.r, k, M),
                   "path": "qmlp_forward_moe (two launches over the routed instances: gate/up with LoRA-A, down with the routing-weighted sum)",
                   "widths": res,
                   "gain_pct": round((t4 / tm - 1) * 100, 1),
                   "capture_pct": round((1 / tm - 1 / t4) / (1 / t2 - 1 / t4) * 100, 1)},
        "roofline": {"bound": "hbm", "kernel": "MoE layer step (gate/up with LoRA-A, down with the routing-weighted sum)",
                     "achieved": mix["gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": mix["frac_of_hbm_peak"], "traffic": None},
    }
    calibrations(args)
    print(json.dumps(out), flush=True)
    return 0


def prefill_main(cfg: wl.Config, args):
    """One prefill chunk per step: qmlp_forward at M tokens (bf16, MFMA)."""
    import torch
    import paper_2606_04238_amd as q
    stack = build_stack(cfg, args.seed, layers=1)
    m, x, y, ws = stack.mlps[0], stack.xs[0], stack.ys[0], stack.ws
    st = torch.cuda.current_stream()
    ms, _ = time_passes(lambda: q.forward(m, x, y=y, ws=ws), args.steps, args.warmup)
    t_step = sum(ms) / len(ms)
    # per-half durations: events around the gate/up half (qmlp_gateup_w2_lora:
    # LoRA-A, its reduction, gate/up) and around the whole chunk; the down
    # half (down over slices of f and the slices' sum, which only the
    # chunk's workspace holds) is their difference
    h = torch.empty((cfg.M, cfg.f), dtype=x.dtype, device="cuda")
    a_us, c_us = [], []
    for _ in range(max(3, args.steps // 4)):
        e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        e0.record(st)
        q.gateup_w2_lora(m, x, h=h, ws=ws)
        e1.record(st)
        q.forward(m, x, y=y, ws=ws)
        e2.record(st)
        torch.cuda.synchronize()
        a_us.append(e0.elapsed_time(e1) * 1e3)
        c_us.append(e1.elapsed_time(e2) * 1e3)
    fg, fd = prefill_flops(cfg)
    tflops = (fg + fd) / (t_step * 1e-3) / 1e12
    gu_us = statistics.mean(a_us)
    dn_us = statistics.mean(c_us) - gu_us
    dom_us, dom_f, dom_name = (gu_us, fg, "prefill gate/up half (LoRA-A + MFMA gate/up)") \
        if gu_us >= dn_us else (dn_us, fd, "prefill down half (pf_down_kernel over slices of f + their sum)")
    achieved = dom_f / (dom_us * 1e-6) / 1e12
    out = {
        "metric": "achieved TFLOP/s (% of MI355X dense bf16 MFMA peak) of the W4/W2-GateUp MLP "
                  "prefill chunk",
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(t_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "%s prefill chunk: M=%d, d=%d, f=%d, group %d, LoRA rank %d"
                        % (cfg.name, cfg.M, cfg.d, cfg.f, cfg.g, cfg.r),
            "flops_per_step": fg + fd,
            "kernel_us": {"gateup_half": round(gu_us, 3), "down_half": round(dn_us, 3)},
            "launches": q.forward_launches(m, cfg.M, x.dtype),
            "frac_of_mfma_peak": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4),
        },
        "roofline": {
            "bound": "mfma",
            "kernel": dom_name,
            "achieved": round(achieved, 2),
            "peak": MFMA_BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4),
            "traffic": None,
        },
    }
    calibrations(args)
    print(json.dumps(out), flush=True)
    return 0


# --------------------------------------------------------------------- main
# --------------------------------------------------------------------- HBM read rate
PROBE_BLOCKS = (256, 512, 1024, 2048, 4096, 8192)


def stream_probe_main(args):
    """The read rate this GPU sustains: one read-only pass over a buffer far
    larger than the 256 MB Infinity Cache, 128-bit loads, no arithmetic.
    Context for the decode roofline, not its denominator (that stays the
    8 TB/s peak)."""
    import torch
    import paper_2606_04238_amd as q
    n = args.stream_probe_mib << 20
    buf = torch.empty(n // 4, dtype=torch.int32, device="cuda").fill_(0x01020304)
    torch.cuda.synchronize()
    res = {}
    for nt in (True, False):
        for blocks in PROBE_BLOCKS:
            out = torch.empty(4 * blocks, dtype=torch.int32, device="cuda")
            ms, _ = time_passes(lambda: q.probe_stream_read(buf, blocks, nt, out),
                                max(5, args.steps // 4), 3, 0.25)
            med = statistics.median(ms)
            res["%s_%d" % ("nt" if nt else "plain", blocks)] = round(n / (med * 1e-3) / 1e9, 1)
            if torch.any(out != 0):         # every word XORs an even number of equal words
                raise RuntimeError("stream probe read unexpected data")
    best = max(res, key=res.get)
    line = {"stream_probe": {"mib": args.stream_probe_mib, "gbs": res, "best": best,
                             "best_gbs": res[best], "frac_of_hbm_peak": round(res[best] / HBM_PEAK_GBS, 4),
                             "threads_per_block": 256, "loads_in_flight_per_thread": 8}}
    print(json.dumps(line), flush=True)
    return 0


def stream_calibration(mib: int):
    """One non-temporal and one plain pass of the streaming probe over `mib`
    MiB (reference dispatches of known read size for the byte counters)."""
    import torch
    import paper_2606_04238_amd as q
    n = mib << 20
    buf = torch.empty(n // 4, dtype=torch.int32, device="cuda").fill_(7)
    torch.cuda.synchronize()
    for nt in (True, False):
        q.probe_stream_read(buf, 1024, nt)
        torch.cuda.synchronize()
    log("stream calibration: %d bytes read with non-temporal loads, then %d with plain loads" % (n, n))
    del buf


def calibrations(args):
    """The reference dispatches of known size that the byte counters are
    scaled by (after the timing, so they never enter it)."""
    import torch
    if args.calibrate_stream_mib > 0:
        stream_calibration(args.calibrate_stream_mib)
    if args.calibrate_copy_mib > 0:
        n = args.calibrate_copy_mib << 20
        src = torch.ones(n // 2, dtype=torch.float16, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        log("copy calibration: %d bytes read, %d bytes written" % (n, n))
        del src, dst


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="qwen3_4b", choices=sorted(wl.CONFIGS) + sorted(wl.MOE))
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--mode", default="eager", choices=["graph", "eager"],
                    help="how the timed steps are launched: back-to-back launches on the stream (eager) or replays of a captured HIP graph")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--min-warm-s", type=float, default=0.25,
                    help="untimed warmup lasts at least this long (and at least --warmup steps)")
    ap.add_argument("--no-precision-comparison", action="store_true",
                    help="skip the uniform-W4 / uniform-W2 / W4/W2-GateUp comparison (Sec. 5.2)")
    ap.add_argument("--stream-probe", action="store_true",
                    help="only measure the HBM read rate this GPU sustains: the read-only "
                         "streaming probe over --stream-probe-mib MiB at several grid sizes, with "
                         "non-temporal and plain 128-bit loads; prints one JSON line")
    ap.add_argument("--stream-probe-mib", type=int, default=4096)
    ap.add_argument("--calibrate-stream-mib", type=int, default=0,
                    help="after timing, run the read-only streaming probe once over this many MiB "
                         "with non-temporal loads and once with plain loads, as reference "
                         "dispatches for HBM byte counters")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="after timing, run one copy-like elementwise kernel over this many MiB "
                         "(read N, write N) as the reference dispatch for HBM byte counters")
    args = ap.parse_args(argv)

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this library's decode MLP runs on a single "
              "MI355X (data-parallel scale-out needs no communication); run with --gpus 1.",
              file=sys.stderr)
        return 2

    import torch
    import paper_2606_04238_amd as q
    q.library()
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        return 2
    if args.stream_probe:
        return stream_probe_main(args)
    if args.config in wl.MOE:
        return moe_main(wl.MOE[args.config], args)
    cfg = wl.CONFIGS[args.config]
    if cfg.M > 16:
        return prefill_main(cfg, args)
    stack = build_stack(cfg, args.seed, variants=not args.no_precision_comparison)
    L = cfg.L
    B = cfg.alg_bytes()
    dt = stack.Y.dtype
    launches = q.layers_launches(stack.lay, cfg.M, dt)
    path = q.layers_path(stack.lay, cfg.M, dt)

    # the timed step: every block on its own input, back to back
    # timed in both launch modes; `value` is the one --mode names, the other is
    # reported beside it
    # the K timed steps back to back, bracketed by two events and a
    # synchronize on both sides; per-step events (a second pass) give the
    # spread of single steps
    eager_step = time_block(lambda: run_blocks_once(stack), args.steps, args.warmup, args.min_warm_s)
    eager_ms, _ = time_passes(lambda: run_blocks_once(stack), args.steps, 1, 0.0)
    g = capture(lambda: run_blocks_once(stack))
    graph_step = time_block(g.replay, args.steps, args.warmup, args.min_warm_s)
    graph_ms, wall = time_passes(g.replay, args.steps, 1, 0.0)
    head = graph_ms if args.mode == "graph" else eager_ms
    t_step = graph_step if args.mode == "graph" else eager_step
    gbs = L * B / (t_step * 1e-3) / 1e9
    us_layer = t_step * 1e3 / L
    err = parity_blocks(stack, args.seed, sample=(0, L // 2, L - 1))

    # context: the same blocks as a decoder stack on the residual stream, and
    # one qmlp_forward launch per block (graph replay)
    context = {}
    if stack.sws is not None:
        gs = capture(lambda: run_stack_once(stack))
        stack_ms, _ = time_passes(gs.replay, max(5, args.steps // 2), 2, args.min_warm_s)
        context["dependent_stack_us_per_mlp_step"] = round(sum(stack_ms) / len(stack_ms) * 1e3 / L, 3)
        context["dependent_stack_launches"] = q.stack_launches(stack.st, cfg.M, dt)
        if q.stack_launches(stack.st, cfg.M, dt) < L:
            err_bits = q.stack_errors(stack.st, stack.sws, cfg.M, dt)
            if err_bits:
                raise RuntimeError("stack kernel reported error bits %#x" % err_bits)
        context["dependent_stack_parity_max_rel_err"] = {
            str(k): float("%.3e" % v) for k, v in parity_sampled(stack, args.seed, sample=(0,)).items()}
    gl = capture(lambda: run_layers_once(stack))
    layer_ms, _ = time_passes(gl.replay, max(5, args.steps // 2), 2, args.min_warm_s)
    per_layer_us = sum(layer_ms) / len(layer_ms) * 1e3 / L
    context["per_layer_path_us_per_mlp_step"] = round(per_layer_us, 3)
    if stack.variants:
        context["precision_comparison"] = precision_comparison(stack, args.seed,
                                                               max(5, args.steps // 2),
                                                               args.min_warm_s, us_layer)
        if cfg.name in wl.DECODERS:
            context["decoder_model"] = decoder_model(
                stack, args.seed, max(5, args.steps // 2), args.min_warm_s,
                context["precision_comparison"]["mlp_us"])

    # The step (one qmlp_forward_layers call) is the unit: its launches --
    # LoRA-A (inside the gate/up launch on the streamed path), gate/up and
    # down over every block of a batch of up to 40 --
    # are internal to the call, so the timed region's events give the step;
    # the per-kernel split is in the committed kernel trace.
    if path not in ("streamed", "mfma", "batched"):
        raise RuntimeError("binary16 decode streams, runs on the matrix cores or runs batched; got path %s"
                           % path)
    dom_name = ("%s step (%s launches of qmlp_forward_layers)"
                % (path, "gate/up with LoRA-A, and down" if path == "streamed" else "LoRA-A, gate/up and down"))
    dom_us, dom_b = t_step * 1e3, L * B
    kernel_us = {"step": round(dom_us, 3), "launches_per_step": launches}
    traffic = read_traffic(os.path.join(ROOT, "profiles", "layers_%s_%s.md" % (path, cfg.name)),
                           STEP_KERNELS[path]) if path in STEP_KERNELS else None
    achieved = dom_b / (dom_us * 1e-6) / 1e9

    out = {
        "metric": METRIC,
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(t_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {
            "workload": "%s decode MLP: M=%d, d=%d, f=%d, group %d, LoRA rank %d, %d independently "
                        "seeded blocks (own weights, own input) run back to back"
                        % (cfg.name, cfg.M, cfg.d, cfg.f, cfg.g, cfg.r, L),
            "us_per_mlp_step": round(us_layer, 3),
            "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
            "alg_bytes_per_mlp_step": B,
            "mode": "hip_graph" if args.mode == "graph" else "eager",
            "path": {"streamed": "streamed launches (gate/up with LoRA-A, then down, over every block)",
                     "mfma": "matrix-core launches (LoRA-A, gate/up, down over every block)",
                     "batched": "batched stand-alone kernels"}[path],
            "eager_us_per_mlp_step": round(eager_step * 1e3 / L, 3),
            "graph_us_per_mlp_step": round(graph_step * 1e3 / L, 3),
            "median_ms_per_step_with_per_step_events": round(statistics.median(head), 4),
            "p10_p90_ms_per_step": [round(float(np.percentile(head, 10)), 4),
                                    round(float(np.percentile(head, 90)), 4)],
            "kernel_us": kernel_us,
            "parity_max_rel_err": {str(k): float("%.3e" % v) for k, v in err.items()},
            **context,
        },
        "roofline": {
            "bound": "hbm",
            "kernel": dom_name,
            "achieved": round(achieved, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": None if traffic is None else int(traffic),
        },
    }
    calibrations(args)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, args.seed)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
