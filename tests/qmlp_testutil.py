"""Helpers shared by the test modules: move seeded workloads to the device,
pack them with the HIP library, and quantize them with the oracle."""
import numpy as np
import torch

import oracle as orc
import workloads as wl


def act_tensor(bits: np.ndarray, act: str = "f16", device="cuda") -> torch.Tensor:
    """Activation bits (uint16 numpy) -> float16/bfloat16 device tensor, same bits."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    t = t.view(torch.bfloat16 if act == "bf16" else torch.float16)
    return t.to(device)


def bits_of(t: torch.Tensor) -> np.ndarray:
    """Device float16/bfloat16 tensor -> uint16 numpy bits."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def values_of(t: torch.Tensor, act: str = "f16") -> np.ndarray:
    return orc.act_to_f64(bits_of(t), act == "bf16")


def gpu_mlp(layer: wl.Layer, lora_scale=None, rank=True):
    import paper_2606_04238_amd as q
    cfg = layer.cfg
    g = q.pack_w2(torch.from_numpy(layer.W_gate).cuda(), cfg.g)
    u = q.pack_w2(torch.from_numpy(layer.W_up).cuda(), cfg.g)
    d = q.pack_w4(torch.from_numpy(layer.W_down).cuda(), cfg.g)
    ls = cfg.lora_scale if lora_scale is None else lora_scale
    if not rank:
        return q.MLP(g, u, d, lora_scale=ls)
    return q.MLP(g, u, d, act_tensor(layer.A_gate, cfg.act), act_tensor(layer.B_gate, cfg.act),
                 act_tensor(layer.A_up, cfg.act), act_tensor(layer.B_up, cfg.act), lora_scale=ls)


def oracle_q(layer: wl.Layer):
    cfg = layer.cfg
    return (orc.quantize(layer.W_gate, 2, cfg.g), orc.quantize(layer.W_up, 2, cfg.g),
            orc.quantize(layer.W_down, 4, cfg.g))


def oracle_forward(layer: wl.Layer, q3=None, lora_scale=None, rank=True, x=None):
    cfg = layer.cfg
    qg, qu, qd = q3 if q3 is not None else oracle_q(layer)
    ls = cfg.lora_scale if lora_scale is None else lora_scale
    lo = (layer.A_gate, layer.B_gate, layer.A_up, layer.B_up) if rank else (None,) * 4
    return orc.forward(qg, qu, qd, *lo, layer.x if x is None else x, lora_scale=ls,
                       bf16=cfg.bf16, return_h=True)
