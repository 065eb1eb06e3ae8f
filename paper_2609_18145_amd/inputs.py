"""Seeded synthetic inputs for the mixing stack.

This module only draws numbers: it holds none of the layer's arithmetic, and
is the one piece of Python that both the GPU-path tests and the CPU oracle's
tests use.  Every array is produced by ``numpy.random.default_rng(seed)`` in a
fixed draw order (inputs/labels/tokens, embedding table, then for each layer
``W_self`` then ``W_off``, then ``dY``), as float32; for bf16 workloads every
value is rounded once to the nearest bf16 (ties to even) so the same numbers
are exactly representable on both sides.

Workloads (shapes and value distributions of the paper's experiments):
  tiny      n=16,   width 32,   batch 2,  4 layers,  fp32, bidirectional, N(0,1) inputs
  reach     n=256,  width 64,   batch 64, 8 layers,  bf16, bidirectional; per-position
            labels in [0,16) embedded through an N(0,1) table; target = sum of labels mod 16
            (the count-the-ones task of Section 4, widened to 16 classes)
  lm256     n=256,  width 512,  batch 64, 16 layers, bf16, causal; byte tokens with Zipf(1.1)
            frequencies over a shuffled byte ranking, embedded through an N(0,1) table
            (stand-in for the character-level corpora of Section 5, which are not used)
  long4096  n=4096, width 1024, batch 8,  24 layers, bf16, causal; N(0,1) inputs
  shared256 n=256, width 512, batch 64, 16 layers, bf16, causal; the lm256 inputs with the
            channel-shared layer: one n x n table per layer, entries N(0, 1/2)
Weights are N(0, 1/width); the upstream gradient dY is N(0,1).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

PRESETS = {
    "tiny": dict(batch=2, n=16, width=32, num_layers=4, causal=False, dtype="f32", kind="normal"),
    "reach": dict(batch=64, n=256, width=64, num_layers=8, causal=False, dtype="bf16", kind="labels16"),
    "lm256": dict(batch=64, n=256, width=512, num_layers=16, causal=True, dtype="bf16", kind="zipf_bytes"),
    "long4096": dict(batch=8, n=4096, width=1024, num_layers=24, causal=True, dtype="bf16", kind="normal"),
}


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 value (ties to even), kept as float32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def _finish(a: np.ndarray, dtype: str) -> np.ndarray:
    a = a.astype(np.float32)
    return round_bf16(a) if dtype == "bf16" else a


@dataclass
class StackInputs:
    x: np.ndarray                      # [batch, n, width] float32
    w_self: list = field(default_factory=list)   # per layer [width, width] float32
    w_off: list = field(default_factory=list)
    layers: list = field(default_factory=list)   # layer index handed to the layer
    dy: np.ndarray | None = None       # [batch, n, width] float32
    causal: bool = False
    dtype: str = "f32"
    tokens: np.ndarray | None = None   # integer inputs when the workload has them
    targets: np.ndarray | None = None


def zipf_byte_tokens(rng, shape, s: float = 1.1, vocab: int = 256) -> np.ndarray:
    """Token ids whose frequencies follow Zipf(s) over ranks 1..vocab, with the
    rank -> byte value assignment a seeded shuffle."""
    ranks = np.arange(1, vocab + 1, dtype=np.float64)
    p = ranks ** (-s)
    p /= p.sum()
    byte_of_rank = rng.permutation(vocab)
    r = rng.choice(vocab, size=shape, p=p)
    return byte_of_rank[r].astype(np.int64)


def make_stack(batch: int, n: int, width: int, num_layers: int, causal: bool,
               dtype: str = "bf16", kind: str = "normal", seed: int = 0,
               layers=None, with_dy: bool = True) -> StackInputs:
    """Draw one workload.  ``layers`` overrides the default schedule l = 0..L-1."""
    rng = np.random.default_rng(seed)
    tokens = targets = None
    if kind == "normal":
        x = rng.standard_normal((batch, n, width))
    elif kind == "labels16":
        tokens = rng.integers(0, 16, size=(batch, n))
        table = rng.standard_normal((16, width))
        x = table[tokens]
        targets = np.repeat(tokens.sum(axis=1, keepdims=True) % 16, n, axis=1)
    elif kind == "zipf_bytes":
        seq = zipf_byte_tokens(rng, (batch, n + 1))
        tokens, targets = seq[:, :n], seq[:, 1:]
        table = rng.standard_normal((256, width))
        x = table[tokens]
    else:
        raise ValueError(kind)
    std = 1.0 / np.sqrt(width)
    w_self, w_off = [], []
    for _ in range(num_layers):
        w_self.append(_finish(rng.standard_normal((width, width)) * std, dtype))
        w_off.append(_finish(rng.standard_normal((width, width)) * std, dtype))
    dy = _finish(rng.standard_normal((batch, n, width)), dtype) if with_dy else None
    if layers is None:
        layers = list(range(num_layers))
    return StackInputs(x=_finish(x, dtype), w_self=w_self, w_off=w_off, layers=list(layers),
                       dy=dy, causal=causal, dtype=dtype, tokens=tokens, targets=targets)


def make_preset(name: str, seed: int = 0, **overrides) -> StackInputs:
    cfg = dict(PRESETS[name])
    cfg.update(overrides)
    return make_stack(seed=seed, **cfg)


def make_layer(batch: int, n: int, width: int, dtype: str = "bf16", seed: int = 0):
    """One layer's operands: (x, w_self, w_off, dy), N(0,1) data, N(0,1/width) weights."""
    rng = np.random.default_rng(seed)
    x = _finish(rng.standard_normal((batch, n, width)), dtype)
    std = 1.0 / np.sqrt(width)
    ws = _finish(rng.standard_normal((width, width)) * std, dtype)
    wo = _finish(rng.standard_normal((width, width)) * std, dtype)
    dy = _finish(rng.standard_normal((batch, n, width)), dtype)
    return x, ws, wo, dy


@dataclass
class SharedInputs:
    x: np.ndarray                      # [batch, n, width] float32
    tables: list = field(default_factory=list)   # per layer [n, n] float32
    layers: list = field(default_factory=list)
    dy: np.ndarray | None = None
    causal: bool = True
    dtype: str = "bf16"


def make_shared_stack(batch: int, n: int, width: int, num_layers: int, causal: bool = True,
                      dtype: str = "bf16", kind: str = "normal", seed: int = 0,
                      layers=None) -> SharedInputs:
    """Inputs of the channel-shared stack: x (drawn as in make_stack), then one
    n x n table per layer with N(0, 1/2) entries (a position and its partner
    then keep the activations' scale on average), then dY.  Tables stay fp32."""
    rng = np.random.default_rng(seed)
    if kind == "normal":
        x = rng.standard_normal((batch, n, width))
    elif kind == "zipf_bytes":
        seq = zipf_byte_tokens(rng, (batch, n + 1))
        table = rng.standard_normal((256, width))
        x = table[seq[:, :n]]
    else:
        raise ValueError(kind)
    tables = [(rng.standard_normal((n, n)) * np.sqrt(0.5)).astype(np.float32)
              for _ in range(num_layers)]
    dy = _finish(rng.standard_normal((batch, n, width)), dtype)
    if layers is None:
        layers = list(range(num_layers))
    return SharedInputs(x=_finish(x, dtype), tables=tables, layers=list(layers), dy=dy,
                        causal=causal, dtype=dtype)


@dataclass
class FieldInputs:
    p: np.ndarray                      # [batch, n, coord_dim] float32 coordinates
    x: np.ndarray                      # [batch, n, width] float32 (bf16 values)
    dy: np.ndarray                     # [batch, n, width] float32 (bf16 values)
    tau: float = 1.0
    scaled: bool = True


def make_field(batch: int, n: int, width: int, coord_dim: int = 32, tau: float = 1.0,
               scaled: bool = True, mean_sq_dist: float = 100.0, kind: str = "normal",
               seed: int = 0) -> FieldInputs:
    """Inputs of the field coupling (Section 3.4's dynamics variant): x (drawn
    as in make_stack), then coordinates N(0, s^2) per component with s chosen so
    that the expected squared distance of two positions, 2 coord_dim s^2, is
    mean_sq_dist (about 100 is the regime Section 7 describes at
    initialisation), then dY N(0,1).  x and dY are rounded to bf16; the
    coordinates stay fp32."""
    rng = np.random.default_rng(seed)
    if kind == "normal":
        x = rng.standard_normal((batch, n, width))
    elif kind == "zipf_bytes":
        seq = zipf_byte_tokens(rng, (batch, n + 1))
        table = rng.standard_normal((256, width))
        x = table[seq[:, :n]]
    else:
        raise ValueError(kind)
    s = np.sqrt(mean_sq_dist / (2.0 * coord_dim))
    p = (rng.standard_normal((batch, n, coord_dim)) * s).astype(np.float32)
    dy = _finish(rng.standard_normal((batch, n, width)), "bf16")
    return FieldInputs(p=p, x=_finish(x, "bf16"), dy=dy, tau=tau, scaled=scaled)


def make_field_chain(batch: int, n: int, width: int, coord_dim: int = 32, steps: int = 8,
                     tau: float = 1.0, scaled: bool = True, mean_sq_dist: float = 100.0,
                     seed: int = 0):
    """Inputs of `steps` field applications in a chain: x (Zipf byte tokens
    through an N(0,1) table, as in make_stack), then one coordinate array per
    application drawn as in make_field, then dY.  Returns (x, [p_1..p_T], dy,
    tau, scaled)."""
    rng = np.random.default_rng(seed)
    seq = zipf_byte_tokens(rng, (batch, n + 1))
    table = rng.standard_normal((256, width))
    x = _finish(table[seq[:, :n]], "bf16")
    s = np.sqrt(mean_sq_dist / (2.0 * coord_dim))
    ps = [(rng.standard_normal((batch, n, coord_dim)) * s).astype(np.float32)
          for _ in range(steps)]
    dy = _finish(rng.standard_normal((batch, n, width)), "bf16")
    return x, ps, dy, tau, scaled
