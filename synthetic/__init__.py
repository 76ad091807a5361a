"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module only draws random inputs of the shapes and distributions of the
paper's workloads; it holds none of the method's arithmetic (no quantization,
routing or expert math).  Each tensor comes from its own numpy PCG64 stream,
``default_rng([seed, stream])`` with ``seed = 20241006 + config_id``, so any
piece (one expert matrix, the logits, the mask) can be drawn on its own.

Workloads (the paper's Mixtral 8x7b and OLMoE shapes; no dataset is used):

* 1 ``tiny``:    d=256, ffn=512, E=4, top-2, bits [1,2,3,2], G=32, T=64,
                 logits N(0,1), tau=0.3.
* 2 ``mixtral``: d=4096, ffn=14336, E=8, top-2, bits [3,3,3,2,2,2,2,3]
                 (2.5 expert bits = the paper's 2.54-bit setting), G=128,
                 logits N(0,1) + per-expert bias N(0, 0.5^2), tau=0.3,
                 decode T in {1, 8, 32}.
* 3 ``mixtral_prefill``: as 2 with T=4096 and tau in {0, 0.2, 0.4}.
* 4 ``olmoe``:   d=2048, ffn=1024, E=64, top-8, bits iid {1,2,3} with
                 p {0.2,0.5,0.3}, G=64, logits N(0,1) + ln Zipf(1.1)
                 popularity over a seeded expert permutation, tau=0.05,
                 prefill T=2048, decode T=16.
* 5 ``mixtral_stack``: 32 layers of the shape of 2, each layer with the
                 widths [3,3,3,2,2,2,2,3] in its own seeded order, its own
                 weights, logits (N(0,1) + its own per-expert bias
                 N(0, 0.5^2)) and protected tokens; decode T in {1, 64},
                 prefill T=1024, tau=0.3.

Weights are N(0, 0.02^2) fp32, activations N(0,1) rounded once to bfloat16,
router weights [E][d] N(0, 1/d) rounded to bfloat16 (unit-variance logits on
such activations), calibration inputs for GPTQ [N][K] with correlated
channels (rank-8 N(0,1) factors plus N(0, 0.5^2) noise) and per-channel
scales exp(N(0, 0.5^2)), 1 % of channels x8 (outlier features), in bfloat16,
and round(0.1*T) tokens (a seeded permutation) are marked important.
Attention maps (the input of token importance) are causal row softmaxes of
scores N(0, 1.5^2) with +4 on the first key (an attention sink), rounded to
bfloat16.
"""
from __future__ import annotations

import numpy as np

BASE_SEED = 20241006

CONFIGS = {
    1: dict(name="tiny", d=256, ffn=512, E=4, k=2, bits=[1, 2, 3, 2], G=32,
            T=[64], tau=[0.3], bias_std=0.0, zipf=None),
    2: dict(name="mixtral", d=4096, ffn=14336, E=8, k=2, bits=[3, 3, 3, 2, 2, 2, 2, 3], G=128,
            T=[1, 8, 32], tau=[0.3], bias_std=0.5, zipf=None),
    3: dict(name="mixtral_prefill", d=4096, ffn=14336, E=8, k=2, bits=[3, 3, 3, 2, 2, 2, 2, 3],
            G=128, T=[4096], tau=[0.0, 0.2, 0.4], bias_std=0.5, zipf=None),
    4: dict(name="olmoe", d=2048, ffn=1024, E=64, k=8, bits=None, G=64,
            T=[2048, 16], tau=[0.05], bias_std=0.0, zipf=1.1),
    5: dict(name="mixtral_stack", d=4096, ffn=14336, E=8, k=2, bits=[3, 3, 3, 2, 2, 2, 2, 3],
            G=128, T=[1, 64, 1024], tau=[0.3], bias_std=0.5, zipf=None, layers=32),
}

# stream ids inside a config's seed
_S_X, _S_BIAS, _S_LOGITS, _S_MASK, _S_BITS, _S_ATTN, _S_ROUTER = 1, 2, 3, 4, 5, 6, 7
_S_CALIB = 500          # + tag: calibration inputs of one matrix
_S_WEIGHT = 1000
_S_LAYER = 100000       # stream offset per layer of a stack (config 5)


def rng(config_id: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([BASE_SEED + config_id, stream])


def config(config_id: int) -> dict:
    c = dict(CONFIGS[config_id])
    c["bits"] = expert_bits(config_id)
    return c


def expert_bits(config_id: int) -> list:
    c = CONFIGS[config_id]
    if c["bits"] is not None:
        return list(c["bits"])
    g = rng(config_id, _S_BITS)
    return [int(b) for b in g.choice([1, 2, 3], size=c["E"], p=[0.2, 0.5, 0.3])]


def weight(config_id: int, e: int, m: int, shape=None, std: float = 0.02) -> np.ndarray:
    """fp32 N(0, std^2) matrix m (0 gate [ffn][d], 1 up [ffn][d], 2 down [d][ffn])
    of expert e."""
    c = CONFIGS[config_id]
    if shape is None:
        shape = (c["ffn"], c["d"]) if m < 2 else (c["d"], c["ffn"])
    g = rng(config_id, _S_WEIGHT + 3 * e + m)
    w = g.standard_normal(size=shape, dtype=np.float32)
    w *= np.float32(std)
    return w


def layer_weights(config_id: int, E=None, d=None, ffn=None):
    c = CONFIGS[config_id]
    E = c["E"] if E is None else E
    d = c["d"] if d is None else d
    ffn = c["ffn"] if ffn is None else ffn
    return [tuple(weight(config_id, e, m, (ffn, d) if m < 2 else (d, ffn)) for m in range(3))
            for e in range(E)]


def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to bfloat16 (nearest, ties to even); returns uint16 bits.
    Input preparation only: finite inputs are assumed."""
    b = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return b.astype(np.uint16)


def activations(config_id: int, T: int, d=None) -> np.ndarray:
    """x ~ N(0,1) rounded to bfloat16: uint16 bits [T][d]."""
    c = CONFIGS[config_id]
    d = c["d"] if d is None else d
    g = rng(config_id, _S_X + 100 * T)
    return to_bf16_bits(g.standard_normal(size=(T, d), dtype=np.float32))


def logits(config_id: int, T: int, E=None) -> np.ndarray:
    """Router logits [T][E] fp32: N(0,1) plus a fixed per-expert offset
    (N(0, bias_std^2) or ln of a Zipf popularity over a seeded permutation)."""
    c = CONFIGS[config_id]
    E = c["E"] if E is None else E
    offset = np.zeros(E, np.float64)
    if c["bias_std"]:
        offset = rng(config_id, _S_BIAS).normal(0.0, c["bias_std"], size=E)
    elif c["zipf"]:
        gp = rng(config_id, _S_BIAS)
        perm = gp.permutation(E)
        ranks = np.arange(1, E + 1, dtype=np.float64)
        p = ranks ** (-c["zipf"])
        p /= p.sum()
        offset = np.log(p[perm])
    g = rng(config_id, _S_LOGITS + 100 * T)
    return (g.standard_normal(size=(T, E)) + offset[None, :]).astype(np.float32)


def router_weights(config_id: int, E=None, d=None) -> np.ndarray:
    """Router weight W_r [E][d] ~ N(0, 1/d) rounded to bfloat16: uint16 bits."""
    c = CONFIGS[config_id]
    E = c["E"] if E is None else E
    d = c["d"] if d is None else d
    g = rng(config_id, _S_ROUTER)
    return to_bf16_bits(g.standard_normal(size=(E, d), dtype=np.float32) / np.float32(np.sqrt(d)))


def calibration(config_id: int, N: int, K: int, tag: int = 0, rank: int = 8) -> np.ndarray:
    """Calibration inputs X [N][K] of one linear layer (bf16 bits): rank-`rank`
    correlated N(0,1) factors plus N(0, 0.5^2) noise, each channel scaled by
    exp(N(0, 0.5^2)) and 1 % of the channels by a further 8 (outliers)."""
    g = rng(config_id, _S_CALIB + tag)
    V = g.standard_normal((rank, K))
    c = g.standard_normal((N, rank))
    x = c @ V / np.sqrt(rank) + 0.5 * g.standard_normal((N, K))
    scale = np.exp(0.5 * g.standard_normal(K))
    scale[g.choice(K, max(1, K // 100), replace=False)] *= 8.0
    return to_bf16_bits((x * scale).astype(np.float32))


def important_mask(config_id: int, T: int, frac: float = 0.1) -> np.ndarray:
    """uint8 [T]: exactly floor(frac*T + 0.5) tokens set, chosen by a seeded permutation."""
    n = int(np.floor(frac * T + 0.5))
    g = rng(config_id, _S_MASK + 100 * T)
    m = np.zeros(T, np.uint8)
    m[g.permutation(T)[:n]] = 1
    return m


def attention(config_id: int, H: int, L: int) -> np.ndarray:
    """Causal attention probabilities [H][L][L] as bfloat16 bits, query-major:
    row i is a softmax over keys 0..i of N(0, 1.5^2) scores with +4 on key 0,
    zeros above the diagonal."""
    g = rng(config_id, _S_ATTN + 100 * L + 100000 * H)
    out = np.empty((H, L, L), np.uint16)
    above = np.triu(np.ones((L, L), bool), 1)
    for h in range(H):
        s = g.standard_normal(size=(L, L), dtype=np.float32)
        s *= np.float32(1.5)
        s[:, 0] += np.float32(4.0)
        s[above] = -np.inf
        s -= s.max(axis=1, keepdims=True)
        np.exp(s, out=s)
        s /= s.sum(axis=1, keepdims=True)
        out[h] = to_bf16_bits(s)
    return out


# ------------------------------------------------------------------ stacks --
# Layer l of a stack draws every tensor from the streams of a single layer
# shifted by _S_LAYER * (l + 1), so no two layers share a stream.

def stack_bits(config_id: int, layer: int) -> list:
    """Expert widths of one layer: the config's widths in a seeded order."""
    c = CONFIGS[config_id]
    g = rng(config_id, _S_LAYER * (layer + 1) + _S_BITS)
    return [int(b) for b in g.permutation(np.asarray(c["bits"]))]


def stack_expert_weights(config_id: int, layer: int, e: int, d=None, ffn=None, std: float = 0.02):
    """fp32 N(0, std^2) gate [ffn][d], up [ffn][d], down [d][ffn] of expert e of one layer."""
    c = CONFIGS[config_id]
    d = c["d"] if d is None else d
    ffn = c["ffn"] if ffn is None else ffn
    mats = []
    for m in range(3):
        g = rng(config_id, _S_LAYER * (layer + 1) + _S_WEIGHT + 3 * e + m)
        w = g.standard_normal(size=(ffn, d) if m < 2 else (d, ffn), dtype=np.float32)
        w *= np.float32(std)
        mats.append(w)
    return tuple(mats)


def stack_layer_weights(config_id: int, layer: int, E=None, d=None, ffn=None, std: float = 0.02):
    E = CONFIGS[config_id]["E"] if E is None else E
    return [stack_expert_weights(config_id, layer, e, d, ffn, std) for e in range(E)]


def stack_logits(config_id: int, layer: int, T: int, E=None) -> np.ndarray:
    """Router logits of one layer [T][E] fp32: N(0,1) + the layer's per-expert
    offset N(0, bias_std^2)."""
    c = CONFIGS[config_id]
    E = c["E"] if E is None else E
    base = _S_LAYER * (layer + 1)
    offset = rng(config_id, base + _S_BIAS).normal(0.0, c["bias_std"], size=E)
    g = rng(config_id, base + _S_LOGITS + 100 * T)
    return (g.standard_normal(size=(T, E)) + offset[None, :]).astype(np.float32)


def stack_mask(config_id: int, layer: int, T: int, frac: float = 0.1) -> np.ndarray:
    """Protected tokens of one layer: floor(frac*T + 0.5) of them, seeded."""
    n = int(np.floor(frac * T + 0.5))
    g = rng(config_id, _S_LAYER * (layer + 1) + _S_MASK + 100 * T)
    m = np.zeros(T, np.uint8)
    m[g.permutation(T)[:n]] = 1
    return m
