"""Plain fp64 CPU oracle for ACache's selective affix-KV recompute.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only the tests, the smoke check and the benchmark's
CPU-baseline leg use it.  It shares no code with the GPU path; both read the
same seeded input bits from ``workloads``.

Everything is float64, with no intermediate rounding.  Each function names
the passage of "Affix Cache for Diffusion Large Language Models" it follows:

* Section 3.1: the affix F is a span of non-masked positions, L = |F|; the
  masked set M_T is the initially masked response region.
* Section 3.2, Eq. 4: a_{j,k} = [softmax(Q_mask K_affix^T / sqrt(d_h))]_{k,j},
  the weight from masked query k to affix key j at layer n, head h.
* Section 3.2, Eq. 5: s_j = sum over layers, heads and masked queries of a.
* Section 3.2, Eq. 6: the anchor set A = TopK(s, K); S = F minus A; K from
  the anchor ratio rho as the integer nearest to rho * L.
* Section 3.2 (probe): the request's non-affix positions are forwarded with
  the precomputed affix cache as fixed past KV; affix states are neither
  forwarded nor updated.
* Section 3.3: at a recomputation point, anchors and all request-specific
  positions are recomputed; non-anchor affix tokens keep the shared cache.
* Section 4.1: write-side recomputation map and read-slot map.
* Section 4.3 and Appendix C.1: queries are formed only for recomputed
  positions; their fresh KV is stored first, then attention reads the full
  logical view (store-then-attend).

The transformer block itself is not defined in the paper; it is the block of
the LLaDA / Dream model families the paper evaluates (Section 5, "Models"):
RMSNorm, Q/K/V projections without bias, rotary embedding (half-split pairs),
bidirectional softmax attention with grouped KV heads, output projection with
residual, RMSNorm, SwiGLU MLP with residual.

Readings where the paper is silent or ambiguous (each is listed in the
design notes):
* Eq. 4's softmax runs over the affix keys only ("affix" norm, the literal
  equation).  The other reading, the columns of the model's softmax over all
  keys ("full" norm), is available as norm="full".
* Scores are summed over all layers (Eq. 5) and one top-K is taken after the
  last layer.
* Ties in Eq. 6 go to the lowest affix index; -0 equals +0; NaN ranks below
  every other value (ties among NaNs again by index).  The anchor list is
  returned in ascending order.
* Anchors are recomputed from their layer-0 input through every layer, like
  request-specific rows.
"""

from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np


# ----------------------------------------------------------------------------
# storage bits -> float64
# ----------------------------------------------------------------------------

def from_bits(a: np.ndarray, dtype: str) -> np.ndarray:
    """bf16 bit patterns (uint16) or float32 values -> float64."""
    if dtype == "bf16":
        a = np.ascontiguousarray(a, dtype=np.uint16)
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return np.asarray(a, dtype=np.float32).astype(np.float64)


@dataclass
class Dims:
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    rms_eps: float = 1e-5
    rope_base: float = 10000.0


@dataclass
class Layer:
    """One block's weights in float64, [out_features, in_features]."""

    g1: np.ndarray
    wq: np.ndarray
    wk: np.ndarray
    wv: np.ndarray
    wo: np.ndarray
    g2: np.ndarray
    wg: np.ndarray
    wu: np.ndarray
    wd: np.ndarray


def layer_from_bits(bits, dims: Dims, dtype: str) -> Layer:
    """Split the fused storage matrices (Q|K|V rows, gate|up rows)."""
    hq = dims.n_heads * dims.head_dim
    hk = dims.n_kv_heads * dims.head_dim
    f = dims.d_ff
    qkv = from_bits(bits.w_qkv, dtype)
    gu = from_bits(bits.w_gate_up, dtype)
    return Layer(
        g1=from_bits(bits.attn_norm, dtype),
        wq=qkv[:hq], wk=qkv[hq:hq + hk], wv=qkv[hq + hk:hq + 2 * hk],
        wo=from_bits(bits.w_o, dtype),
        g2=from_bits(bits.mlp_norm, dtype),
        wg=gu[:f], wu=gu[f:2 * f],
        wd=from_bits(bits.w_down, dtype),
    )


# ----------------------------------------------------------------------------
# block pieces (model family of Section 5, "Models")
# ----------------------------------------------------------------------------

def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope(x: np.ndarray, pos: np.ndarray, base: float) -> np.ndarray:
    """Rotary embedding, half-split pairs (i, i + d_h/2) rotated by pos * theta_i,
    theta_i = base^(-2i/d_h).  x: [M, n_heads, d_h]; pos: [M]."""
    dh = x.shape[-1]
    half = dh // 2
    inv_freq = base ** (-(2.0 * np.arange(half, dtype=np.float64)) / dh)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray):
    """Bidirectional softmax attention, no mask, grouped KV heads.

    q: [M, H, d_h]; k, v: [S, H_kv, d_h].  Query head h reads KV head
    h // (H / H_kv).  Returns o [M, H, d_h] and the natural-log
    log-sum-exp of the scaled logits, lse [M, H]."""
    m, nh, dh = q.shape
    nkv = k.shape[1]
    group = nh // nkv
    scale = 1.0 / np.sqrt(dh)
    o = np.empty_like(q)
    lse = np.empty((m, nh))
    for h in range(nh):
        g = h // group
        logits = (q[:, h, :] @ k[:, g, :].T) * scale
        mx = logits.max(axis=1, keepdims=True)
        e = np.exp(logits - mx)
        z = e.sum(axis=1, keepdims=True)
        o[:, h, :] = (e / z) @ v[:, g, :]
        lse[:, h] = (mx + np.log(z))[:, 0]
    return o, lse


def silu(a: np.ndarray) -> np.ndarray:
    return a / (1.0 + np.exp(-a))


def layer_kv(w: Layer, dims: Dims, x: np.ndarray, pos: np.ndarray):
    """The K and V a block writes for rows x [R, d] at positions pos: RMSNorm,
    the K and V projections, rotation of K (Section 4.3).  Row-local, so
    layer 0's affix K/V depend only on the affix rows' own inputs.
    Returns (k, v), each [R, H_kv, d_h]."""
    r = x.shape[0]
    h = rms_norm(x, w.g1, dims.rms_eps)
    k = (h @ w.wk.T).reshape(r, dims.n_kv_heads, dims.head_dim)
    v = (h @ w.wv.T).reshape(r, dims.n_kv_heads, dims.head_dim)
    return rope(k, pos, dims.rope_base), v


def layer_queries(w: Layer, dims: Dims, x: np.ndarray, pos: np.ndarray) -> np.ndarray:
    """The queries a block forms for rows x [R, d] at positions pos: RMSNorm,
    the Q projection, rotation.  Returns q [R, H, d_h]."""
    h = rms_norm(x, w.g1, dims.rms_eps)
    q = (h @ w.wq.T).reshape(x.shape[0], dims.n_heads, dims.head_dim)
    return rope(q, pos, dims.rope_base)


def layer_forward(w: Layer, dims: Dims, x: np.ndarray, pos: np.ndarray,
                  rows: np.ndarray, view_k: np.ndarray, view_v: np.ndarray):
    """One block over the recomputed rows (Section 4.3, Appendix C.1).

    x: [R, d] inputs of the recomputed rows, whose logical indices are
    ``rows``; view_k / view_v: [S, H_kv, d_h] logical KV view of the request,
    updated in place with the fresh K/V of ``rows`` before attention reads the
    whole view.  Returns (x_out [R, d], q [R, H, d_h] post-rotation,
    lse [R, H])."""
    r = x.shape[0]
    nh, dh = dims.n_heads, dims.head_dim
    q = layer_queries(w, dims, x, pos)
    k, v = layer_kv(w, dims, x, pos)
    view_k[rows] = k
    view_v[rows] = v
    o, lse = attention(q, view_k, view_v)
    x = x + o.reshape(r, nh * dh) @ w.wo.T
    h2 = rms_norm(x, w.g2, dims.rms_eps)
    x = x + (silu(h2 @ w.wg.T) * (h2 @ w.wu.T)) @ w.wd.T
    return x, q, lse


# ----------------------------------------------------------------------------
# anchor importance (Section 3.2, Eq. 4-5) and selection (Eq. 6)
# ----------------------------------------------------------------------------

def affix_attention_mass(q_masked: np.ndarray, k_affix: np.ndarray, norm: str = "affix",
                         lse_full: Optional[np.ndarray] = None) -> np.ndarray:
    """One layer's contribution to s_j: sum over heads h and masked queries k
    of a_{j,k}^{(n,h)} (Eq. 4-5).

    q_masked: [G, H, d_h] masked-position queries (post-rotation);
    k_affix: [L, H_kv, d_h] affix keys; norm "affix" normalises over the
    affix keys (Eq. 4 as written), "full" uses the model's softmax over all
    keys, whose log-sum-exp lse_full [G, H] the caller supplies."""
    g_rows, nh, dh = q_masked.shape
    nkv = k_affix.shape[1]
    group = nh // nkv
    scale = 1.0 / np.sqrt(dh)
    s = np.zeros(k_affix.shape[0])
    for h in range(nh):
        logits = (q_masked[:, h, :] @ k_affix[:, h // group, :].T) * scale
        if norm == "affix":
            mx = logits.max(axis=1, keepdims=True)
            e = np.exp(logits - mx)
            a = e / e.sum(axis=1, keepdims=True)
        elif norm == "full":
            a = np.exp(logits - lse_full[:, h][:, None])
        else:
            raise ValueError(norm)
        s += a.sum(axis=0)
    return s


def anchor_count(ratio: float, affix_len: int) -> int:
    """Eq. 6 takes K tokens; the anchor ratio rho fixes K as the integer
    nearest to rho * L, halves rounded up (the paper gives no rounding rule;
    the tiny workload's "ratio 0.2 (26 tokens)" at L = 128 rules out the
    floor), clamped to [0, L].  Exact rational arithmetic on the binary value
    of rho, so no float rounding decides a half."""
    from fractions import Fraction
    r = Fraction(ratio)
    if r < 0 or r > 1:
        raise ValueError(f"anchor ratio {ratio} outside [0, 1]")
    k = math.floor(r * affix_len + Fraction(1, 2))
    return max(0, min(int(affix_len), int(k)))


def topk_anchors(s: np.ndarray, k: int) -> np.ndarray:
    """Eq. 6: indices of the k largest scores, ties to the lowest index,
    -0 == +0, NaN below everything; returned ascending (int64)."""
    s = np.asarray(s, dtype=np.float64)
    n = s.shape[0]
    nan = np.isnan(s)
    neg = np.where(nan, 0.0, -s)
    order = np.lexsort((np.arange(n), neg, nan))
    return np.sort(order[:k])


def greedy_commit(logits: np.ndarray) -> np.ndarray:
    """The commit step of the predict-then-commit loop (Section 3.1) in its
    greedy form, as the serving schedule uses it: per row of logits, the
    index of the largest value, -0 == +0, NaN below every value, the lowest
    index among equal values (int64)."""
    x = np.asarray(logits, dtype=np.float64)
    out = np.empty(x.shape[0], dtype=np.int64)
    for i, row in enumerate(x):
        nan = np.isnan(row)
        out[i] = np.lexsort((np.arange(row.size), -np.where(nan, 0.0, row), nan))[0]
    return out


def confidence(logits: np.ndarray) -> np.ndarray:
    """A row's confidence in the predict-then-commit loop (Section 3.1): the
    softmax probability of its largest finite logit, 1 / sum_j exp(x_j - max)
    over the finite values (0 for a row with none)."""
    x = np.asarray(logits, dtype=np.float64)
    out = np.zeros(x.shape[0])
    for i, row in enumerate(x):
        fin = row[np.isfinite(row) | (row == np.inf)]
        fin = fin[fin > -np.inf]
        if fin.size == 0:
            continue
        m = fin.max()
        top = fin == m  # equal maxima, +inf included, count exactly once each
        with np.errstate(invalid="ignore"):  # inf - inf where top; replaced by 0
            d = np.where(top, 0.0, fin - m)
        out[i] = 1.0 / np.sum(np.where(top, 1.0, np.exp(d)))
    return out


def threshold_commit(conf: np.ndarray, committed: np.ndarray, tau: float) -> np.ndarray:
    """One decode step's commit over a block (Sections 3.1, 5): the
    uncommitted rows with confidence >= tau, or, if there is none, the single
    most confident uncommitted row (the lowest row among equals).  Returns the
    boolean mask of rows committed by this step."""
    conf = np.asarray(conf, dtype=np.float64)
    free = ~np.asarray(committed, dtype=bool)
    take = free & (conf >= tau)
    if not take.any() and free.any():
        key = np.where(free, np.where(np.isnan(conf), -0.5, conf), -np.inf)
        take = np.zeros_like(free)
        take[int(np.argmax(key))] = True
    return take


def decode_step(layers: Sequence["Layer"], dims: "Dims", views_k, views_v, x_block: np.ndarray,
                block_pos: np.ndarray):
    """A block decoding step (Section 4.3): queries only for the block's rows,
    whose fresh K/V are written into the request's logical view before
    attention reads the whole view through every layer.  views_k/views_v:
    per layer [S, H_kv, d_h], updated in place.  Returns the block's outputs."""
    x = np.asarray(x_block, dtype=np.float64).copy()
    for n, w in enumerate(layers):
        x, _, _ = layer_forward(w, dims, x, block_pos, block_pos, views_k[n], views_v[n])
    return x


# ----------------------------------------------------------------------------
# requests: probe, selective refresh, full refresh, direct reuse
# ----------------------------------------------------------------------------

@dataclass
class Request:
    """One request: layer-0 inputs of all S logical rows, their positions,
    the affix rows (their order defines the affix-local index j) and the
    initially masked rows M_T."""

    x0: np.ndarray      # [S, d] float64
    pos: np.ndarray     # [S] int
    affix: np.ndarray   # [L] logical row indices
    masked: np.ndarray  # [G] logical row indices

    @property
    def nonaffix(self) -> np.ndarray:
        keep = np.ones(self.x0.shape[0], dtype=bool)
        keep[self.affix] = False
        return np.nonzero(keep)[0]


@dataclass
class Result:
    rows: np.ndarray                 # logical indices of the recomputed rows (ascending)
    x: np.ndarray                    # [R, d] outputs of the recomputed rows after the last layer
    views_k: List[np.ndarray]        # per layer [S, H_kv, d_h]
    views_v: List[np.ndarray]
    scores: Optional[np.ndarray]     # [L] (probe only)


def run_request(layers: Sequence[Layer], dims: Dims, req: Request, rows: np.ndarray,
                stale_k: Optional[Sequence[np.ndarray]] = None,
                stale_v: Optional[Sequence[np.ndarray]] = None,
                score_norm: Optional[str] = None) -> Result:
    """Forward the recomputed rows through every layer.  Affix rows that are
    not recomputed read the stale cache (stale_k[n], stale_v[n]: [L, H_kv, d_h]
    in affix-local order).  With score_norm set, accumulate Eq. 5 from the
    masked rows' queries against the affix keys of each layer's view."""
    s_len = req.x0.shape[0]
    rows = np.sort(np.asarray(rows))
    x = req.x0[rows].copy()
    pos = np.asarray(req.pos)[rows]
    nkv, dh = dims.n_kv_heads, dims.head_dim
    row_of = {int(r): i for i, r in enumerate(rows)}
    masked_in_rows = np.array([row_of[int(m)] for m in req.masked], dtype=np.int64) if score_norm else None
    scores = np.zeros(len(req.affix)) if score_norm else None
    vks, vvs = [], []
    for n, w in enumerate(layers):
        vk = np.full((s_len, nkv, dh), np.nan)
        vv = np.full((s_len, nkv, dh), np.nan)
        if stale_k is not None:
            vk[req.affix] = stale_k[n]
            vv[req.affix] = stale_v[n]
        x, q, lse = layer_forward(w, dims, x, pos, rows, vk, vv)
        if score_norm:
            scores += affix_attention_mass(q[masked_in_rows], vk[req.affix], score_norm,
                                           lse[masked_in_rows])
        vks.append(vk)
        vvs.append(vv)
    return Result(rows=rows, x=x, views_k=vks, views_v=vvs, scores=scores)


def probe(layers, dims, req: Request, stale_k, stale_v, norm: str = "affix") -> Result:
    """Section 3.2: forward the non-affix rows against the fixed stale affix
    cache and accumulate the masked-to-affix importance s."""
    return run_request(layers, dims, req, req.nonaffix, stale_k, stale_v, score_norm=norm)


def selective_rows(req: Request, anchors: np.ndarray) -> np.ndarray:
    """Section 3.3: anchors plus every request-specific position."""
    return np.sort(np.concatenate([req.nonaffix, np.asarray(req.affix)[np.asarray(anchors, dtype=np.int64)]]))


def selective_refresh(layers, dims, req: Request, anchors, stale_k, stale_v) -> Result:
    return run_request(layers, dims, req, selective_rows(req, anchors), stale_k, stale_v)


def hkvd_layer(n_layers: int) -> int:
    """Selection layer of the KV-deviation selector: the first layer whose
    affix K/V depend on the rest of the prompt (layer 0's are row-local)."""
    return min(1, n_layers - 1)


def hkvd_scores(layers, dims, req: Request, stale_k, stale_v) -> np.ndarray:
    """The CacheBlend-style selector the appendix compares against (HKVD): each affix token's
    KV deviation between the shared (affix-only) cache and the full-prompt
    cache, the squared difference of its K and V summed over all heads and
    dimensions at the selection layer.  The full-prompt cache is a full
    forward of the request through that layer.  Returns s [L]."""
    n = hkvd_layer(len(layers))
    full = full_refresh(layers[:n + 1], dims, req)
    return kv_deviation(full.views_k[n][req.affix], full.views_v[n][req.affix], stale_k[n], stale_v[n])


def kv_deviation(k_a, v_a, k_b, v_b) -> np.ndarray:
    """Per token, the squared difference of two caches' K and V summed over
    heads and dimensions (the HKVD selector's deviation).  Each [L, H_kv, d_h]."""
    dk = np.asarray(k_a) - np.asarray(k_b)
    dv = np.asarray(v_a) - np.asarray(v_b)
    return (dk * dk).sum(axis=(1, 2)) + (dv * dv).sum(axis=(1, 2))


def rerotate_keys(k: np.ndarray, delta: np.ndarray, base: float) -> np.ndarray:
    """Cached K moved by delta positions (reuse of a span at other positions;
    the cache holds K after rotation, Section 4): the half-split pairs of
    every head turn by delta * theta_i, i.e. the rotation at position delta
    applied to the cached K.  k [n, H_kv, d_h], delta [n]."""
    return rope(k, np.asarray(delta), base)


def drop_non_anchor_refresh(layers, dims, req: Request, anchors) -> Result:
    """DropNA, the ablation of Section 5.3: the same anchors and request rows
    are recomputed, but the non-anchor affix entries are discarded, so
    attention sees only the recomputed rows (at their original positions).
    That is a full recomputation of the request restricted to those rows."""
    rows = selective_rows(req, anchors)
    sub = Request(x0=req.x0[rows], pos=np.asarray(req.pos)[rows], affix=np.arange(0), masked=np.arange(0))
    res = full_refresh(layers, dims, sub)
    return Result(rows=rows, x=res.x, views_k=res.views_k, views_v=res.views_v, scores=None)


def full_refresh(layers, dims, req: Request) -> Result:
    """Periodic full recomputation (Section 2.2): every position."""
    return run_request(layers, dims, req, np.arange(req.x0.shape[0]))


def direct_reuse(layers, dims, req: Request, stale_k, stale_v) -> Result:
    """Anchor ratio 0: only request-specific rows, the whole affix stale."""
    return run_request(layers, dims, req, req.nonaffix, stale_k, stale_v)


def materialize_affix_cache(layers, dims, donor: Request):
    """The shared affix cache, computed once (Sections 3.3 and 4.2): a full
    forward of a donor sequence, keeping each layer's K/V of its affix rows
    ([L, H_kv, d_h] per layer, affix-local order)."""
    res = full_refresh(layers, dims, donor)
    return ([vk[donor.affix].copy() for vk in res.views_k],
            [vv[donor.affix].copy() for vv in res.views_v])


def select_anchors(layers, dims, req: Request, stale_k, stale_v, k: int, norm: str = "affix"):
    """One-shot selection: probe, then Eq. 6."""
    res = probe(layers, dims, req, stale_k, stale_v, norm)
    return topk_anchors(res.scores, k), res


# ----------------------------------------------------------------------------
# KV layout and the two maps (Section 4.1)
# ----------------------------------------------------------------------------

def build_maps(seq_len: int, affix_begin: int, affix_len: int, mask_begin: int, mask_len: int,
               anchors: np.ndarray, shared_base: int, private_base: int, private_stride: int):
    """Write-side recomputation map and read-slot map for a batch.

    anchors: [B, K] affix-local indices (ascending per request).  Request b's
    recomputed positions, ascending, take private slots
    private_base + b * private_stride + i; every logical position reads its
    private slot when recomputed, else the shared slot shared_base + (p -
    affix_begin).  Returns row_pos, row_src (b * seq_len + p), write_slots,
    read_slots [B * seq_len], q_rows (batch row index of each masked
    position)."""
    return _maps(seq_len, affix_begin, affix_len, mask_begin, mask_len, anchors,
                 lambda j: shared_base + j, lambda b, i: private_base + b * private_stride + i)


def build_maps_paged(seq_len: int, affix_begin: int, affix_len: int, mask_begin: int, mask_len: int,
                     anchors: np.ndarray, block_size: int, shared_blocks, private_blocks,
                     blocks_per_request: int):
    """The same maps over block-granular slots (Section 4.1: shared blocks
    for the affix cache, private blocks per request): affix-local index j
    lives in slot shared_blocks[j // bs] * bs + j % bs, request b's i-th
    recomputed position in private_blocks[b * blocks_per_request + i // bs]
    * bs + i % bs."""
    bs = block_size
    return _maps(seq_len, affix_begin, affix_len, mask_begin, mask_len, anchors,
                 lambda j: int(shared_blocks[j // bs]) * bs + j % bs,
                 lambda b, i: int(private_blocks[b * blocks_per_request + i // bs]) * bs + i % bs)


def _maps(seq_len, affix_begin, affix_len, mask_begin, mask_len, anchors, shared_slot, private_slot):
    anchors = np.asarray(anchors, dtype=np.int64).reshape(len(anchors), -1)
    n_req = anchors.shape[0]
    row_pos, row_src, write_slots, q_rows = [], [], [], []
    read_slots = np.empty(n_req * seq_len, dtype=np.int64)
    base_row = 0
    for b in range(n_req):
        anchor_pos = set(int(affix_begin + a) for a in anchors[b])
        recomputed = [p for p in range(seq_len)
                      if not (affix_begin <= p < affix_begin + affix_len) or p in anchor_pos]
        slot_of = {}
        for i, p in enumerate(recomputed):
            slot = private_slot(b, i)
            slot_of[p] = slot
            row_pos.append(p)
            row_src.append(b * seq_len + p)
            write_slots.append(slot)
        for p in range(seq_len):
            read_slots[b * seq_len + p] = slot_of[p] if p in slot_of else shared_slot(p - affix_begin)
        index_of = {p: i for i, p in enumerate(recomputed)}
        for p in range(mask_begin, mask_begin + mask_len):
            q_rows.append(base_row + index_of[p])
        base_row += len(recomputed)
    a = lambda v: np.asarray(v, dtype=np.int64)
    return a(row_pos), a(row_src), a(write_slots), read_slots, a(q_rows)


# ----------------------------------------------------------------------------
# single operations over physical KV pools (Appendix C.1 read-slot view)
# ----------------------------------------------------------------------------

def attention_via_slots(q: np.ndarray, k_pool: np.ndarray, v_pool: np.ndarray,
                        read_slots: np.ndarray, cu_rows: Sequence[int], cu_keys: Sequence[int]):
    """Read-slot attention (Appendix C.1): request b's queries are rows
    cu_rows[b]..cu_rows[b+1] of q [M, H, d_h]; its logical keys are the pool
    rows named by read_slots[cu_keys[b]..cu_keys[b+1]].  Pools are
    [n_slots, H_kv, d_h].  Returns o [M, H, d_h] and lse [M, H]."""
    o = np.empty_like(q)
    lse = np.empty(q.shape[:2])
    for b in range(len(cu_rows) - 1):
        r0, r1 = cu_rows[b], cu_rows[b + 1]
        if r1 == r0:
            continue
        slots = np.asarray(read_slots[cu_keys[b]:cu_keys[b + 1]])
        o[r0:r1], lse[r0:r1] = attention(q[r0:r1], k_pool[slots], v_pool[slots])
    return o, lse


def scores_via_slots(q: np.ndarray, q_rows: np.ndarray, cu_q: Sequence[int], k_pool: np.ndarray,
                     affix_slots: np.ndarray, norm: str = "affix",
                     row_lse: Optional[np.ndarray] = None) -> np.ndarray:
    """Eq. 4-5 for one layer over a batch: request b's masked queries are
    q[q_rows[cu_q[b]..cu_q[b+1]]]; the affix keys are k_pool[affix_slots].
    Returns s [B, L] (this layer's contribution)."""
    n_req = len(cu_q) - 1
    out = np.zeros((n_req, len(affix_slots)))
    k_aff = k_pool[np.asarray(affix_slots)]
    for b in range(n_req):
        rows = np.asarray(q_rows[cu_q[b]:cu_q[b + 1]])
        if len(rows) == 0:
            continue
        lse = None if row_lse is None else row_lse[rows]
        out[b] = affix_attention_mass(q[rows], k_aff, norm, lse)
    return out
