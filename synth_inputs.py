"""Seeded synthetic inputs shared by the oracle and the GPU path.

This module holds data only: the five transformer workload shapes and the
seeded generators for the graph input and the constants (weights, biases,
norm scales, rotary tables).  It performs none of the method's arithmetic
(no layout choice, no planning, no operator evaluation) and imports neither
the oracle nor the GPU package, so both sides can draw identical inputs from
it without sharing any compute code.

Recipe (same for every workload):
  * ``rng = numpy.random.default_rng(seed)`` with seed = workload index 1..5.
  * Draw order: first the input ``x = rng.standard_normal((B, S, H))``, then,
    walking the constants in graph order, every projection matrix of shape
    [K, N] as ``0.02 * rng.standard_normal((K, N))``.  Biases and LayerNorm
    shifts are 0, norm scales are 1.  All values are rounded to float32.
  * bf16 workloads: input and every constant except the rotary tables are
    then rounded to bfloat16 (round-to-nearest-even, done by torch's CPU
    cast); they are returned as float32 arrays holding bf16-exact values.
  * Rotary tables [S, D/2]: cos / sin of ``p * base**(-2i/D)`` evaluated in
    float64 and rounded to float32, p the sequence position, i < D/2.
  * Convolutional workload (VGG-shaped): the input is an image batch
    ``x = rng.standard_normal((B, C, H, W))``; every weight -- convolution
    kernels [Co, Ci, KH, KW] and classifier matrices [K, N] -- is
    ``sqrt(2 / fan_in) * rng.standard_normal(shape)`` with fan_in = Ci*KH*KW
    or K (scaled so that activations keep their size through the ReLU
    layers); biases are 0.
"""
from __future__ import annotations

import numpy as np

# Workload table: the post-LN encoder, pre-LN decoder and Llama-style
# decoder shapes that the benchmark and the parity tests run.
CONFIGS = {
    1: dict(name="bert-1layer-b1-s32-h64", arch="post_ln", layers=1, batch=1,
            seq=32, hidden=64, heads=2, ffn=256, dtype="f32"),
    2: dict(name="bert-base-12l-b1-s128-h768", arch="post_ln", layers=12,
            batch=1, seq=128, hidden=768, heads=12, ffn=3072, dtype="f32"),
    3: dict(name="gpt2-small-12l-b1-s512-h768-prefill", arch="pre_ln",
            layers=12, batch=1, seq=512, hidden=768, heads=12, ffn=3072,
            dtype="f32"),
    4: dict(name="bert-large-24l-b8-s512-h1024", arch="post_ln", layers=24,
            batch=8, seq=512, hidden=1024, heads=16, ffn=4096, dtype="f32"),
    5: dict(name="llama-8l-b1-s2048-h4096-prefill", arch="llama", layers=8,
            batch=1, seq=2048, hidden=4096, heads=32, ffn=11008,
            dtype="bf16"),
    # VGG-16-shaped convolutional network: five stages of 3x3 convolutions
    # (zero Pad then Conv with bias then ReLU), a 2x2 MaxPool after each
    # stage, then the classifier (two 4096-wide layers with ReLU, 1000
    # classes, Softmax)
    6: dict(name="vgg16-b1-224", arch="vgg", batch=1, channels=3, image=224,
            stages=((64, 2), (128, 2), (256, 3), (512, 3), (512, 3)), fc=4096,
            classes=1000, dtype="f32"),
}
EPS = 1e-5
ROPE_BASE = 10000.0
WEIGHT_STD = 0.02

ROLES = ("weight", "bias", "gamma", "beta", "rope_cos", "rope_sin")


def config(index: int, **overrides) -> dict:
    """A copy of workload ``index`` with optional field overrides."""
    c = dict(CONFIGS[index])
    c.update(overrides)
    c.setdefault("eps", EPS)
    c.setdefault("rope_base", ROPE_BASE)
    return c


def _to_bf16_exact(a: np.ndarray) -> np.ndarray:
    import torch  # CPU cast only; round-to-nearest-even
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def rope_tables(seq: int, head_dim: int, base: float = ROPE_BASE):
    pos = np.arange(seq, dtype=np.float64)[:, None]
    i = np.arange(head_dim // 2, dtype=np.float64)[None, :]
    ang = pos * np.power(base, -2.0 * i / head_dim)
    return np.cos(ang).astype(np.float32), np.sin(ang).astype(np.float32)


def make_inputs(cfg: dict, const_specs, seed: int, rope_head_dim=None):
    """Draw the graph input and all constants.

    ``const_specs`` is the graph's constant list in graph order, each item a
    ``(role, shape)`` pair with role in ``ROLES``.  Returns ``(x, consts)``:
    ``x`` float32 [B, S, H]; ``consts`` a list of float32 arrays.
    """
    rng = np.random.default_rng(seed)
    conv = cfg["arch"] == "vgg"
    if conv:
        x = rng.standard_normal((cfg["batch"], cfg["channels"], cfg["image"], cfg["image"])).astype(np.float32)
    else:
        x = rng.standard_normal((cfg["batch"], cfg["seq"], cfg["hidden"])).astype(np.float32)
    consts = []
    for role, shape in const_specs:
        shape = tuple(int(s) for s in shape)
        if role == "weight" and conv:
            fan_in = int(np.prod(shape[1:])) if len(shape) == 4 else shape[0]
            a = (np.sqrt(2.0 / fan_in) * rng.standard_normal(shape)).astype(np.float32)
        elif role == "weight":
            a = (WEIGHT_STD * rng.standard_normal(shape)).astype(np.float32)
        elif role in ("bias", "beta"):
            a = np.zeros(shape, np.float32)
        elif role == "gamma":
            a = np.ones(shape, np.float32)
        elif role in ("rope_cos", "rope_sin"):
            d = rope_head_dim if rope_head_dim is not None else 2 * shape[1]
            c, s = rope_tables(shape[0], d, cfg.get("rope_base", ROPE_BASE))
            a = c if role == "rope_cos" else s
        else:
            raise ValueError(f"unknown constant role {role!r}")
        consts.append(a)
    if cfg["dtype"] == "bf16":
        x = _to_bf16_exact(x)
        consts = [a if role in ("rope_cos", "rope_sin") else _to_bf16_exact(a)
                  for a, (role, _) in zip(consts, const_specs)]
    return x, consts


def random_tensor(shape, seed: int, scale: float = 1.0, dtype="f32"):
    """Seeded N(0, scale^2) tensor for single-operator parity tests."""
    rng = np.random.default_rng(seed)
    a = (scale * rng.standard_normal(tuple(shape))).astype(np.float32)
    return _to_bf16_exact(a) if dtype == "bf16" else a
