"""Planted mistakes in the oracle must each fail at least one pin.

Each case swaps one oracle function for a plausibly wrong variant (a sign,
a transposed operand, a dropped term, a wrong index), runs the pins that
should notice, and requires that one of them fails.  CPU only."""

import numpy as np
import pytest

from oracle import acache_oracle as O
from tests import test_oracle_ops as T_ops
from tests import test_oracle_request as T_req
from tests.oracle_fixtures import tiny_dims, tiny_layers, tiny_request, tiny_stale


def _rope_wrong_sign(x, pos, base):
    dh = x.shape[-1]
    half = dh // 2
    inv = base ** (-(2.0 * np.arange(half)) / dh)
    ang = np.asarray(pos, float)[:, None] * inv[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c + x2 * s, x2 * c - x1 * s], axis=-1)


def _rope_interleaved(x, pos, base):
    dh = x.shape[-1]
    half = dh // 2
    inv = base ** (-(2.0 * np.arange(half)) / dh)
    ang = np.asarray(pos, float)[:, None] * inv[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = x[..., 0::2], x[..., 1::2]
    out = np.empty_like(x)
    out[..., 0::2] = x1 * c - x2 * s
    out[..., 1::2] = x2 * c + x1 * s
    return out


def _rms_no_mean(x, g, eps):
    return x / np.sqrt(np.sum(x * x, axis=-1, keepdims=True) + eps) * g


def _attention_no_scale(q, k, v):
    return _orig_attention(q * np.sqrt(q.shape[-1]), k, v)


def _attention_gqa_modulo(q, k, v):
    m, nh, dh = q.shape
    nkv = k.shape[1]
    o = np.empty_like(q)
    lse = np.empty((m, nh))
    for h in range(nh):
        oh, lh = _orig_attention(q[:, h:h + 1], k[:, (h % nkv):(h % nkv) + 1], v[:, (h % nkv):(h % nkv) + 1])
        o[:, h], lse[:, h] = oh[:, 0], lh[:, 0]
    return o, lse


def _mass_wrong_axis(q_masked, k_affix, norm="affix", lse_full=None):
    g_rows, nh, dh = q_masked.shape
    grp = nh // k_affix.shape[1]
    s = np.zeros(k_affix.shape[0])
    for h in range(nh):
        lg = (q_masked[:, h] @ k_affix[:, h // grp].T) / np.sqrt(dh)
        e = np.exp(lg - lg.max(axis=0, keepdims=True))
        s += (e / e.sum(axis=0, keepdims=True)).sum(axis=0)
    return s


def _topk_ties_high(s, k):
    n = len(s)
    order = np.lexsort((-np.arange(n), -np.nan_to_num(s, nan=-np.inf)))
    return np.sort(order[:k])


def _silu_wrong(a):
    return a / (1.0 + np.exp(a))


_orig_attention = O.attention


def _anchor_count_ceil(ratio, L):
    return min(L, int(np.ceil(ratio * L)))


def _anchor_count_floor(ratio, L):
    return int(ratio * L)


def _anchor_count_half_down(ratio, L):
    return min(L, int(np.ceil(ratio * L - 0.5)))


def _layer_swapped_gate_up(w, dims, x, pos, rows, vk, vv):
    w2 = O.Layer(g1=w.g1, wq=w.wq, wk=w.wk, wv=w.wv, wo=w.wo, g2=w.g2, wg=w.wu, wu=w.wg, wd=w.wd)
    return _orig_layer(w2, dims, x, pos, rows, vk, vv)


def _layer_attend_before_store(w, dims, x, pos, rows, vk, vv):
    stale_k, stale_v = vk.copy(), vv.copy()
    r = x.shape[0]
    nh, nkv, dh = dims.n_heads, dims.n_kv_heads, dims.head_dim
    h = O.rms_norm(x, w.g1, dims.rms_eps)
    q = O.rope((h @ w.wq.T).reshape(r, nh, dh), pos, dims.rope_base)
    k = O.rope((h @ w.wk.T).reshape(r, nkv, dh), pos, dims.rope_base)
    v = (h @ w.wv.T).reshape(r, nkv, dh)
    sk = np.nan_to_num(stale_k)
    sv = np.nan_to_num(stale_v)
    o, lse = O.attention(q, sk, sv)
    vk[rows], vv[rows] = k, v
    x = x + o.reshape(r, nh * dh) @ w.wo.T
    h2 = O.rms_norm(x, w.g2, dims.rms_eps)
    return x + (O.silu(h2 @ w.wg.T) * (h2 @ w.wu.T)) @ w.wd.T, q, lse


_orig_layer = O.layer_forward


def _run_pins(pins):
    failed = []
    for name, fn in pins:
        try:
            fn()
        except (AssertionError, pytest.fail.Exception):
            failed.append(name)
    return failed


def _request_fixture():
    dims = tiny_dims(nkv=2)
    layers = tiny_layers(dims, 2, seed=30)
    req = tiny_request(dims, seed=31)
    sk, sv = tiny_stale(layers, dims, req, seed=32)
    return dims, layers, req, sk, sv


MUTATIONS = {
    "rope_sign": ("rope", _rope_wrong_sign),
    "rope_interleaved": ("rope", _rope_interleaved),
    "rms_sum_not_mean": ("rms_norm", _rms_no_mean),
    "attention_no_scale": ("attention", _attention_no_scale),
    "attention_gqa_modulo": ("attention", _attention_gqa_modulo),
    "scores_softmax_axis": ("affix_attention_mass", _mass_wrong_axis),
    "topk_ties_high": ("topk_anchors", _topk_ties_high),
    "silu_sign": ("silu", _silu_wrong),
    "gate_up_swapped": ("layer_forward", _layer_swapped_gate_up),
    "attend_before_store": ("layer_forward", _layer_attend_before_store),
    "anchor_count_ceil": ("anchor_count", _anchor_count_ceil),
    "anchor_count_floor": ("anchor_count", _anchor_count_floor),
    "anchor_count_half_down": ("anchor_count", _anchor_count_half_down),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, monkeypatch):
    attr, bad = MUTATIONS[name]
    monkeypatch.setattr(O, attr, bad)
    fx = _request_fixture()
    pins = [
        ("rms_example", T_ops.test_rmsnorm_worked_example),
        ("rms_torch", T_ops.test_rmsnorm_matches_torch),
        ("rope_complex", T_ops.test_rope_matches_complex_rotation),
        ("rope_plane", T_ops.test_rope_two_dims_is_plane_rotation),
        ("attn_brute", lambda: T_ops.test_attention_brute_force(4, 2)),
        ("attn_sdpa", T_ops.test_attention_matches_torch_sdpa_and_logsumexp),
        ("scores_brute", lambda: T_ops.test_scores_brute_force_affix_norm(2, 2)),
        ("scores_mass", T_ops.test_scores_mass_conservation_and_equal_keys),
        ("topk_brute", lambda: T_ops.test_topk_brute_force_subsets(1)),
        ("topk_argsort", T_ops.test_topk_matches_stable_argsort),
        ("layer_torch", lambda: T_req.test_layer_matches_torch_block(2)),
        ("poison", lambda: T_req.test_anchor_poison_does_not_reach_outputs(fx)),
        ("ratio_one", lambda: T_req.test_ratio_one_is_full_recompute_and_ignores_stale(fx)),
        ("k_workloads", T_ops.test_anchor_count_of_the_workloads),
        ("k_nearest", lambda: T_ops.test_anchor_count_is_nearest_integer(10)),
        ("k_halves", T_ops.test_anchor_count_halves_and_bounds),
    ]
    assert _run_pins(pins), f"planted mistake {name} passed every pin"
