"""Seeded random inputs for the workloads.

Every tensor is drawn from NumPy's PCG64 with a SeedSequence keyed by
(26140, workload id, stream, layer, tensor, chunk), so the same bits come
out regardless of how many threads draw them.  Streams: 0 weights,
1 hidden rows / embeddings, 2 token ids, 3 stale-cache perturbation and
donor context, 4 test-only arrays (scores, permutations).

bf16 tensors are returned as uint16 bit patterns, rounded to nearest-even
from float32, so the GPU path and the oracle consume identical bits.
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass
from typing import Optional

import numpy as np

from .configs import Workload

ROOT_SEED = 26140
_CHUNK = 1 << 22  # elements per independently seeded chunk


def rng_for(seed_id: int, stream: int, layer: int = 0, tensor: int = 0, chunk: int = 0) -> np.random.Generator:
    ss = np.random.SeedSequence([ROOT_SEED, seed_id, stream, layer, tensor, chunk])
    return np.random.Generator(np.random.PCG64(ss))


def bf16_bits_from_f32(a: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); return uint16 bits."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        r[nan] = np.uint16(0x7FC0)
    return r


def _normal_f32(shape, std: float, seed_id: int, stream: int, layer: int, tensor: int,
                threads: Optional[int] = None) -> np.ndarray:
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.float32)
    n_chunks = (n + _CHUNK - 1) // _CHUNK

    def fill(c):
        lo, hi = c * _CHUNK, min(n, (c + 1) * _CHUNK)
        g = rng_for(seed_id, stream, layer, tensor, c)
        g.standard_normal(hi - lo, dtype=np.float32, out=out[lo:hi])
        if std != 1.0:
            out[lo:hi] *= np.float32(std)

    if n_chunks == 1:
        fill(0)
    else:
        workers = threads or min(16, len(os.sched_getaffinity(0)))
        with ThreadPoolExecutor(max_workers=workers) as ex:
            list(ex.map(fill, range(n_chunks)))
    return out.reshape(shape)


def _store(a_f32: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return bf16_bits_from_f32(a_f32)
    if dtype == "f32":
        return np.ascontiguousarray(a_f32, dtype=np.float32)
    raise ValueError(dtype)


@dataclass
class LayerWeightsBits:
    """One transformer layer, in storage bits (uint16 for bf16, float32 for f32).

    Matrices use the [out_features, in_features] layout:
      w_qkv     [(H + 2*H_kv) * d_h, d]  rows: Q heads, then K heads, then V heads
      w_o       [d, H * d_h]
      w_gate_up [2 * F, d]               rows: F gate rows, then F up rows
      w_down    [d, F]
    attn_norm / mlp_norm are the RMSNorm gains [d].
    """

    attn_norm: np.ndarray
    w_qkv: np.ndarray
    w_o: np.ndarray
    mlp_norm: np.ndarray
    w_gate_up: np.ndarray
    w_down: np.ndarray


def _layer_shapes(w: Workload):
    d = w.dims
    return [
        (d.qkv_width, d.d_model),
        (d.d_model, d.n_heads * d.head_dim),
        (2 * d.d_ff, d.d_model),
        (d.d_model, d.d_ff),
    ]


def draw_layer_qkv(w: Workload, layer: int, std: float = 0.02) -> np.ndarray:
    """w_qkv of one layer alone: the same bits draw_layer_weights returns."""
    return _store(_normal_f32(_layer_shapes(w)[0], std, w.seed_id, 0, layer, 0), w.dims.dtype)


def draw_layer_weights(w: Workload, layer: int, std: float = 0.02) -> LayerWeightsBits:
    d = w.dims
    mats = [_store(_normal_f32(s, std, w.seed_id, 0, layer, i), d.dtype) for i, s in enumerate(_layer_shapes(w))]
    ones = layer_norm_gains(w)
    return LayerWeightsBits(attn_norm=ones, w_qkv=mats[0], w_o=mats[1], mlp_norm=ones.copy(),
                            w_gate_up=mats[2], w_down=mats[3])


def layer_norm_gains(w: Workload) -> np.ndarray:
    """The RMSNorm gains of every layer: ones."""
    return _store(np.ones(w.dims.d_model, dtype=np.float32), w.dims.dtype)


def draw_hidden_rows(w: Workload, n_req: Optional[int] = None) -> np.ndarray:
    """Layer-0 input rows [B, S, d] in storage bits, N(0, 1) per entry.

    With mask_rows == "shared", every masked row of every request holds one
    fixed mask vector (the embedding of the mask token)."""
    d, lay = w.dims, w.layout
    b = w.batch if n_req is None else n_req
    x = _normal_f32((b, lay.seq_len, d.d_model), 1.0, w.seed_id, 1, 0, 0)
    if w.mask_rows == "shared":
        m = _normal_f32((d.d_model,), 1.0, w.seed_id, 1, 0, 1)
        x[:, lay.mask_begin:lay.mask_begin + lay.mask_len, :] = m
    return _store(x, d.dtype)


def draw_noise(w: Workload, std: float = 0.1) -> np.ndarray:
    """Perturbation [L, d] (float32) added to the affix inputs to build the
    stale affix cache: the cache was materialised in a different context."""
    return _normal_f32((w.layout.affix_len, w.dims.d_model), std, w.seed_id, 3, 0, 0)


def draw_token_ids(w: Workload, n_req: Optional[int] = None):
    """Token ids [B, S] int32 for the stacks: shared affix ids, per-request
    unique ids uniform in the vocabulary, and the mask id at masked positions;
    plus the donor request [S] used to materialise the stale affix cache."""
    d, lay = w.dims, w.layout
    b = w.batch if n_req is None else n_req
    vocab = d.vocab
    mask_id = vocab - 1
    g = rng_for(w.seed_id, 2)
    affix = g.integers(0, vocab - 1, size=lay.affix_len, dtype=np.int64)
    ids = g.integers(0, vocab - 1, size=(b + 1, lay.seq_len), dtype=np.int64)
    ids[:, lay.affix_begin:lay.affix_end] = affix
    ids[:, lay.mask_begin:lay.mask_begin + lay.mask_len] = mask_id
    return ids[:b].astype(np.int32), ids[b].astype(np.int32)


def draw_embedding(w: Workload, std: float = 0.02) -> np.ndarray:
    d = w.dims
    return _store(_normal_f32((d.vocab, d.d_model), std, w.seed_id, 1, 0, 7), d.dtype)


def draw_lm_head(w: Workload, std: float = 0.02):
    """Final RMSNorm gain (ones) and LM head [vocab, d] N(0, std^2) of a stack
    for the serving schedule; weights stream, layer index n_layers."""
    d = w.dims
    head = _store(_normal_f32((d.vocab, d.d_model), std, w.seed_id, 0, d.n_layers, 0), d.dtype)
    return _store(np.ones(d.d_model, dtype=np.float32), d.dtype), head


def draw_scores(n_req: int, L: int, seed: int, kind: str = "normal") -> np.ndarray:
    """float32 score arrays [n_req, L] for selection tests.

    kinds: "normal" N(0,1); "ties" few distinct values; "signed_zero" mixes
    +0 and -0 with a few positives; "special" mixes inf, -inf, NaN,
    denormals and ties; "equal" all one value."""
    g = rng_for(99, 4, 0, seed)
    if kind == "normal":
        return g.standard_normal((n_req, L), dtype=np.float32)
    if kind == "ties":
        return g.integers(0, 5, size=(n_req, L)).astype(np.float32)
    if kind == "signed_zero":
        s = np.where(g.random((n_req, L)) < 0.5, np.float32(0.0), np.float32(-0.0)).astype(np.float32)
        pos = g.random((n_req, L)) < 0.05
        s[pos] = g.random(int(pos.sum())).astype(np.float32) + 1.0
        return s
    if kind == "special":
        s = g.integers(-3, 4, size=(n_req, L)).astype(np.float32)
        r = g.random((n_req, L))
        s[r < 0.05] = np.inf
        s[(r >= 0.05) & (r < 0.10)] = -np.inf
        s[(r >= 0.10) & (r < 0.15)] = np.nan
        s[(r >= 0.15) & (r < 0.20)] = np.float32(1e-40)
        s[(r >= 0.20) & (r < 0.25)] = np.float32(-1e-40)
        s[(r >= 0.25) & (r < 0.30)] = np.float32(-0.0)
        return s
    if kind == "equal":
        return np.full((n_req, L), 0.5, dtype=np.float32)
    raise ValueError(kind)


def draw_tensor(shape, dtype: str, std: float = 1.0, seed: int = 0, tag: int = 0) -> np.ndarray:
    """A test tensor N(0, std^2) in storage bits (stream 4)."""
    return _store(_normal_f32(tuple(shape), std, 98, 4, seed, tag), dtype)


def draw_ints(shape, low: int, high: int, seed: int = 0, tag: int = 0) -> np.ndarray:
    """Uniform int32 in [low, high) (stream 4)."""
    return rng_for(97, 4, seed, tag).integers(low, high, size=shape).astype(np.int32)


def draw_permutation(n: int, seed: int = 0, tag: int = 0) -> np.ndarray:
    return rng_for(96, 4, seed, tag).permutation(n).astype(np.int32)


def draw_donor_rows(w: Workload, hidden_bits: np.ndarray) -> np.ndarray:
    """Layer-0 inputs [L, d] of the context the shared affix cache was
    materialised in, for the "perturb" recipe: the affix rows of request 0
    plus N(0, 0.1^2) noise, stored in the workload's type.  (Input
    preparation only: a float add and a rounding.)"""
    lay = w.layout
    if w.dims.dtype == "bf16":
        base = (hidden_bits[0, lay.affix_begin:lay.affix_end].astype(np.uint32) << np.uint32(16)).view(np.float32)
    else:
        base = hidden_bits[0, lay.affix_begin:lay.affix_end].astype(np.float32)
    return _store(base + draw_noise(w), w.dims.dtype)
