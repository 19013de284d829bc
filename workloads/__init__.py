"""Seeded synthetic workloads for the W4/W2-GateUp decode MLP.

This module only draws random inputs; it holds none of the method's
arithmetic (no quantization, packing, dequantization or matvec), so both the
HIP path and the fp64 oracle can take their inputs from it.

The shapes stand in for the gated MLP blocks of the models whose decode
throughput the paper analyses (Sec. 5.1: Qwen3-4B, Qwen3-14B and the
20B-class GPT-OSS width); their real weights and trained Recover-LoRA
adapters are not used.  Value distributions:

* source weights fp32 N(0, 0.02) (``W = 0.02 * standard_normal``, computed in
  fp32); the 14B-class block additionally has exactly round(1e-3 * size)
  entries per weight matrix replaced by +-0.5 (positions uniform without
  replacement, sign +-1 with probability 1/2) to stress min-max groups;
* LoRA factors A ~ N(0, 0.02), B ~ N(0, 0.002), rounded to the activation type;
* activations x ~ N(0, 1) rounded to binary16 (bfloat16 for the prefill chunk),
  independent rows per token.

Every tensor has its own stream ``np.random.default_rng([seed, layer, id])``
with ids 0 W_gate, 1 W_up, 2 W_down, 3 A_gate, 4 B_gate, 5 A_up, 6 B_up, 7 x,
8/9/10 outlier positions and signs for gate/up/down; the linears outside the
MLP (whole-decoder throughput model) use 11 q/k/v, 12 o, 13 LM head and
14 + 16 * id for their inputs.
"""
from __future__ import annotations

import dataclasses

import numpy as np

TID_W_GATE, TID_W_UP, TID_W_DOWN = 0, 1, 2
TID_A_GATE, TID_B_GATE, TID_A_UP, TID_B_UP = 3, 4, 5, 6
TID_X = 7
TID_OUTLIER = {0: 8, 1: 9, 2: 10}


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    M: int          # tokens per step
    d: int          # hidden size
    f: int          # intermediate size
    g: int          # quantization group (gate/up and down)
    r: int          # LoRA rank
    L: int          # layers in the timed stack
    act: str = "f16"            # activation / LoRA / h / y type: "f16" or "bf16"
    outliers: bool = False
    lora_scale: float = 1.0

    @property
    def bf16(self) -> bool:
        return self.act == "bf16"

    def alg_bytes(self, M: int | None = None) -> int:
        """Bytes one MLP step must move (intermediate kept on-chip):
        2-bit gate+up codes and 4-bit down codes (f*d), fp16 scale+zero for the
        three matrices (12*f*d/g), LoRA A and B for gate and up (4*r*(d+f)),
        x in and y out (4*M*d)."""
        M = self.M if M is None else M
        f, d, g, r = self.f, self.d, self.g, self.r
        return f * d + 12 * f * d // g + 4 * r * (d + f) + 4 * M * d

    def alg_flops(self, M: int | None = None) -> int:
        M = self.M if M is None else M
        return 6 * M * self.f * self.d + 4 * M * self.r * (self.d + self.f)


CONFIGS = {
    "tiny": Config("tiny", M=1, d=512, f=1536, g=64, r=8, L=1),
    "qwen3_4b": Config("qwen3_4b", M=1, d=2560, f=9728, g=128, r=16, L=36),
    "qwen3_8b_m1": Config("qwen3_8b_m1", M=1, d=4096, f=12288, g=128, r=32, L=36),
    "qwen3_8b_m4": Config("qwen3_8b_m4", M=4, d=4096, f=12288, g=128, r=32, L=36),
    "qwen3_8b_m16": Config("qwen3_8b_m16", M=16, d=4096, f=12288, g=128, r=32, L=36),
    "dense14b_m8": Config("dense14b_m8", M=8, d=5120, f=17408, g=64, r=16, L=40, outliers=True),
    "prefill20b": Config("prefill20b", M=512, d=6144, f=16384, g=128, r=32, L=1, act="bf16"),
}


def rng_for(seed: int, layer: int, tensor_id: int) -> np.random.Generator:
    return np.random.default_rng([seed, layer, tensor_id])


def f32_to_f16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> binary16 bits, round to nearest even (numpy's cast)."""
    return np.ascontiguousarray(a, np.float32).astype(np.float16).view(np.uint16)


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> bfloat16 bits, round to nearest even on the fp32 bit pattern
    (inputs here are finite)."""
    u = np.ascontiguousarray(a, np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def to_act_bits(a: np.ndarray, act: str) -> np.ndarray:
    return f32_to_bf16_bits(a) if act == "bf16" else f32_to_f16_bits(a)


def weight(cfg: Config, layer: int, which: int, seed: int = 0) -> np.ndarray:
    """fp32 source weight: which = 0 gate [f][d], 1 up [f][d], 2 down [d][f]."""
    shape = (cfg.f, cfg.d) if which in (0, 1) else (cfg.d, cfg.f)
    w = rng_for(seed, layer, which).standard_normal(shape, dtype=np.float32)
    w *= np.float32(0.02)
    if cfg.outliers:
        ro = rng_for(seed, layer, TID_OUTLIER[which])
        n = int(round(1e-3 * w.size))
        pos = ro.choice(w.size, size=n, replace=False)
        sign = ro.integers(0, 2, size=n) * 2 - 1
        w.reshape(-1)[pos] = (np.float32(0.5) * sign).astype(np.float32)
    return w


def lora(cfg: Config, layer: int, seed: int = 0):
    """(A_gate [r][d], B_gate [f][r], A_up [r][d], B_up [f][r]) as activation bits."""
    out = []
    for tid, shape, sd in ((TID_A_GATE, (cfg.r, cfg.d), 0.02), (TID_B_GATE, (cfg.f, cfg.r), 0.002),
                           (TID_A_UP, (cfg.r, cfg.d), 0.02), (TID_B_UP, (cfg.f, cfg.r), 0.002)):
        a = rng_for(seed, layer, tid).standard_normal(shape, dtype=np.float32) * np.float32(sd)
        out.append(to_act_bits(a, cfg.act))
    return tuple(out)


def activations(cfg: Config, layer: int, seed: int = 0, M: int | None = None) -> np.ndarray:
    """x [M][d] as activation bits, N(0, 1)."""
    M = cfg.M if M is None else M
    a = rng_for(seed, layer, TID_X).standard_normal((M, cfg.d), dtype=np.float32)
    return to_act_bits(a, cfg.act)


@dataclasses.dataclass
class Layer:
    cfg: Config
    index: int
    W_gate: np.ndarray
    W_up: np.ndarray
    W_down: np.ndarray
    A_gate: np.ndarray
    B_gate: np.ndarray
    A_up: np.ndarray
    B_up: np.ndarray
    x: np.ndarray


def layer(cfg: Config, index: int, seed: int = 0, M: int | None = None) -> Layer:
    Ag, Bg, Au, Bu = lora(cfg, index, seed)
    return Layer(cfg, index,
                 weight(cfg, index, 0, seed), weight(cfg, index, 1, seed), weight(cfg, index, 2, seed),
                 Ag, Bg, Au, Bu, activations(cfg, index, seed, M))


def scaled(cfg: Config, **kw) -> Config:
    """A copy of cfg with some fields replaced (small parity shapes, other M)."""
    return dataclasses.replace(cfg, **kw)


# ------------------------------------------------------------------ the rest of a decoder layer
# Dimensions of the decoder around the MLP, for the whole-layer throughput
# model of the precision comparison.  The paper gives none (Sec. 5 names the
# models only); these are the public configuration of the model each MLP
# shape stands in for.  Weights stay synthetic (N(0, 0.02), as above).
@dataclasses.dataclass(frozen=True)
class DecoderDims:
    heads: int          # query heads
    kv_heads: int       # key/value heads (grouped-query attention)
    head_dim: int
    vocab: int          # LM head rows (tied embeddings)
    ctx: int            # context length of the KV cache the step reads

    def qkv_rows(self) -> int:
        return (self.heads + 2 * self.kv_heads) * self.head_dim

    def o_cols(self) -> int:
        return self.heads * self.head_dim

    def kv_bytes_per_layer(self) -> int:
        """BF16 K and V of ctx positions read by one decode step of one layer."""
        return 2 * self.kv_heads * self.head_dim * self.ctx * 2


DECODERS = {"qwen3_4b": DecoderDims(heads=32, kv_heads=8, head_dim=128, vocab=151936, ctx=1024)}

TID_QKV, TID_O, TID_LM_HEAD, TID_LIN_X = 11, 12, 13, 14


def linear_weight(n: int, k: int, layer: int, tensor_id: int, seed: int = 0) -> np.ndarray:
    """fp32 source weight [n][k] of a linear outside the MLP (ids 11 qkv,
    12 o, 13 LM head), N(0, 0.02)."""
    w = rng_for(seed, layer, tensor_id).standard_normal((n, k), dtype=np.float32)
    w *= np.float32(0.02)
    return w


def linear_input(M: int, k: int, layer: int, tensor_id: int, seed: int = 0) -> np.ndarray:
    """Binary16 input bits [M][k] of a linear, N(0, 1) (stream id 14 + 16 * which)."""
    a = rng_for(seed, layer, TID_LIN_X + 16 * tensor_id).standard_normal((M, k), dtype=np.float32)
    return f32_to_f16_bits(a)


# ------------------------------------------------------------------ mixture of experts
# The GPT-OSS-20B-class MoE layer (Sec. 5.1): 32 experts of hidden 2880 and
# expert width 2880, 4 routed per token, INT4 group 64 base (Sec. 5.2); the
# expert MLPs take the W4/W2-GateUp form with rank-16 adapters.
@dataclasses.dataclass(frozen=True)
class MoeConfig:
    name: str
    experts: int
    topk: int
    block: Config        # one expert's block (M = tokens per step, L = MoE layers timed)


MOE = {"gptoss20b_moe": MoeConfig("gptoss20b_moe", experts=32, topk=4,
                                  block=Config("gptoss20b_expert", M=1, d=2880, f=2880, g=64, r=16, L=24))}

TID_ROUTE = 15


def routing(M: int, experts: int, topk: int, layer: int, seed: int = 0):
    """Synthetic routing: per token topk distinct expert ids uniform without
    replacement (int32 [M][topk]) and weights = softmax of N(0, 1) logits
    (float32 [M][topk])."""
    rng = rng_for(seed, layer, TID_ROUTE)
    idx = np.stack([rng.choice(experts, size=topk, replace=False) for _ in range(M)]).astype(np.int32)
    logits = rng.standard_normal((M, topk))
    w = np.exp(logits - logits.max(axis=1, keepdims=True))
    return idx, (w / w.sum(axis=1, keepdims=True)).astype(np.float32)
