"""Pins for the oracle's block, probe, selection, refresh and maps:
an independent torch re-derivation of the block, the paper's endpoint
invariants (ratio 1 = full recompute, ratio 0 = direct reuse), NaN poison,
permutation and shift invariance, and properties of the two maps.  CPU only."""

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import acache_oracle as O
from tests.oracle_fixtures import tiny_dims, tiny_layers, tiny_request, tiny_stale
from tests.test_oracle_ops import rope_complex


def layer_torch(w, dims, x, pos, k_view_fn):
    """The block from torch.nn.functional pieces; k_view_fn(k, v) returns the
    full logical K/V view after the rows' fresh K/V are stored."""
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))
    r = x.shape[0]
    nh, nkv, dh = dims.n_heads, dims.n_kv_heads, dims.head_dim
    h = F.rms_norm(t(x), (dims.d_model,), t(w.g1), eps=dims.rms_eps)
    q = F.linear(h, t(w.wq)).reshape(r, nh, dh).numpy()
    k = F.linear(h, t(w.wk)).reshape(r, nkv, dh).numpy()
    v = F.linear(h, t(w.wv)).reshape(r, nkv, dh).numpy()
    q = rope_complex(q, pos, dims.rope_base)
    k = rope_complex(k, pos, dims.rope_base)
    kv, vv = k_view_fn(k, v)
    tq = t(q).permute(1, 0, 2)
    tk = t(kv).permute(1, 0, 2).repeat_interleave(nh // nkv, dim=0)
    tv = t(vv).permute(1, 0, 2).repeat_interleave(nh // nkv, dim=0)
    o = F.scaled_dot_product_attention(tq, tk, tv).permute(1, 0, 2).reshape(r, nh * dh)
    xo = t(x) + F.linear(o, t(w.wo))
    h2 = F.rms_norm(xo, (dims.d_model,), t(w.g2), eps=dims.rms_eps)
    xo = xo + F.linear(F.silu(F.linear(h2, t(w.wg))) * F.linear(h2, t(w.wu)), t(w.wd))
    return xo.numpy()


@pytest.mark.parametrize("nkv", [4, 2, 1])
def test_layer_matches_torch_block(nkv):
    dims = tiny_dims(nkv=nkv)
    w = tiny_layers(dims, 1, seed=20 + nkv)[0]
    rng = np.random.default_rng(21)
    S = 15
    rows = np.array([0, 3, 4, 8, 14])
    x = rng.standard_normal((len(rows), dims.d_model))
    pos = rows + 100
    vk = rng.standard_normal((S, nkv, dims.head_dim))
    vv = rng.standard_normal((S, nkv, dims.head_dim))

    def view(k, v):
        a, b = vk.copy(), vv.copy()
        a[rows], b[rows] = k, v
        return a, b

    ref = layer_torch(w, dims, x, pos, view)
    out, _, _ = O.layer_forward(w, dims, x, pos, rows, vk.copy(), vv.copy())
    np.testing.assert_allclose(out, ref, rtol=1e-10, atol=1e-11)


def test_layer_with_zero_output_projections_is_identity():
    dims = tiny_dims()
    w = tiny_layers(dims, 1, seed=22)[0]
    w.wo[:] = 0.0
    w.wd[:] = 0.0
    x = np.random.default_rng(23).standard_normal((4, dims.d_model))
    vk = np.zeros((4, dims.n_kv_heads, dims.head_dim))
    out, _, _ = O.layer_forward(w, dims, x, np.arange(4), np.arange(4), vk, vk.copy())
    np.testing.assert_array_equal(out, x)


# ----------------------------------------------------------------------------- request setup

@pytest.fixture(scope="module")
def setup2():
    dims = tiny_dims(nkv=2)
    layers = tiny_layers(dims, 2, seed=30)
    req = tiny_request(dims, seed=31)
    sk, sv = tiny_stale(layers, dims, req, seed=32)
    return dims, layers, req, sk, sv


def test_ratio_one_is_full_recompute_and_ignores_stale(setup2):
    dims, layers, req, sk, sv = setup2
    L = len(req.affix)
    full = O.full_refresh(layers, dims, req)
    poison_k = [np.full_like(a, np.nan) for a in sk]
    poison_v = [np.full_like(a, np.nan) for a in sv]
    sel = O.selective_refresh(layers, dims, req, np.arange(L), poison_k, poison_v)
    assert np.all(np.isfinite(sel.x))
    np.testing.assert_array_equal(sel.rows, full.rows)
    np.testing.assert_allclose(sel.x, full.x, rtol=1e-13, atol=1e-13)
    for n in range(len(layers)):
        np.testing.assert_allclose(sel.views_k[n], full.views_k[n], rtol=1e-13, atol=1e-13)


def test_ratio_zero_is_direct_reuse(setup2):
    dims, layers, req, sk, sv = setup2
    sel = O.selective_refresh(layers, dims, req, np.array([], dtype=np.int64), sk, sv)
    dr = O.direct_reuse(layers, dims, req, sk, sv)
    np.testing.assert_array_equal(sel.rows, req.nonaffix)
    np.testing.assert_array_equal(sel.x, dr.x)
    # direct reuse reads the stale affix untouched at every layer
    for n in range(len(layers)):
        np.testing.assert_array_equal(dr.views_k[n][req.affix], sk[n])


def test_stale_cache_depends_on_context_beyond_layer_one(setup2):
    """The shared cache is stale: the affix K/V of layer 2 change with the
    rest of the sequence, while layer 1's are functions of the row alone."""
    dims, layers, req, sk, sv = setup2
    full = O.full_refresh(layers, dims, req)
    donor = O.Request(x0=req.x0[req.affix], pos=req.pos[req.affix],
                      affix=np.arange(len(req.affix)), masked=np.arange(0))
    ak, _ = O.materialize_affix_cache(layers, dims, donor)
    np.testing.assert_allclose(full.views_k[0][req.affix], ak[0], rtol=1e-12, atol=1e-13)
    assert np.max(np.abs(full.views_k[1][req.affix] - ak[1])) > 1e-3


def test_anchor_poison_does_not_reach_outputs(setup2):
    dims, layers, req, sk, sv = setup2
    anchors = np.array([1, 4, 7])
    base = O.selective_refresh(layers, dims, req, anchors, sk, sv)
    pk = [a.copy() for a in sk]
    pv = [a.copy() for a in sv]
    for n in range(len(layers)):
        pk[n][anchors] = np.nan
        pv[n][anchors] = np.nan
    pois = O.selective_refresh(layers, dims, req, anchors, pk, pv)
    np.testing.assert_array_equal(pois.x, base.x)
    # non-anchor affix entries of the view are the stale cache, bit for bit
    rest = np.setdiff1d(np.arange(len(req.affix)), anchors)
    for n in range(len(layers)):
        np.testing.assert_array_equal(base.views_k[n][req.affix[rest]], sk[n][rest])


def test_probe_mass_and_fixed_affix(setup2):
    dims, layers, req, sk, sv = setup2
    res = O.probe(layers, dims, req, sk, sv)
    G = len(req.masked)
    np.testing.assert_allclose(res.scores.sum(), len(layers) * dims.n_heads * G, rtol=1e-12)
    for n in range(len(layers)):
        np.testing.assert_array_equal(res.views_k[n][req.affix], sk[n])
    full = O.probe(layers, dims, req, sk, sv, norm="full")
    assert np.all(full.scores < res.scores)


def test_probe_scores_match_per_layer_recomputation(setup2):
    """Eq. 5 accumulated by the probe equals a fresh loop over layers that
    recomputes the masked queries from the probe's own layer inputs."""
    dims, layers, req, sk, sv = setup2
    res = O.probe(layers, dims, req, sk, sv)
    rows = req.nonaffix
    x = req.x0[rows].copy()
    total = np.zeros(len(req.affix))
    midx = np.searchsorted(rows, req.masked)
    for n, w in enumerate(layers):
        h = O.rms_norm(x, w.g1, dims.rms_eps)
        q = (h @ w.wq.T).reshape(len(rows), dims.n_heads, dims.head_dim)
        q = rope_complex(q, req.pos[rows], dims.rope_base)
        total += O.affix_attention_mass(q[midx], sk[n], "affix")
        vk = np.full((req.x0.shape[0], dims.n_kv_heads, dims.head_dim), np.nan)
        vv = vk.copy()
        vk[req.affix], vv[req.affix] = sk[n], sv[n]
        x, _, _ = O.layer_forward(w, dims, x, req.pos[rows], rows, vk, vv)
    np.testing.assert_allclose(res.scores, total, rtol=1e-12)


def test_affix_permutation_with_positions(setup2):
    """Permuting the affix tokens' storage order together with their
    positions and stale cache leaves the non-affix outputs unchanged and
    permutes s the same way."""
    dims, layers, req, sk, sv = setup2
    rng = np.random.default_rng(33)
    L = len(req.affix)
    perm = rng.permutation(L)
    x0 = req.x0.copy()
    pos = req.pos.copy()
    x0[req.affix] = req.x0[req.affix[perm]]
    pos[req.affix] = req.pos[req.affix[perm]]
    req_p = O.Request(x0=x0, pos=pos, affix=req.affix, masked=req.masked)
    sk_p = [a[perm] for a in sk]
    sv_p = [a[perm] for a in sv]
    a = O.probe(layers, dims, req, sk, sv)
    b = O.probe(layers, dims, req_p, sk_p, sv_p)
    np.testing.assert_allclose(b.scores, a.scores[perm], rtol=1e-11)
    np.testing.assert_allclose(b.x, a.x, rtol=1e-11, atol=1e-12)
    anchors = O.topk_anchors(a.scores, 4)
    inv = np.argsort(perm)
    r1 = O.selective_refresh(layers, dims, req, anchors, sk, sv)
    r2 = O.selective_refresh(layers, dims, req_p, np.sort(inv[anchors]), sk_p, sv_p)
    non = np.isin(r1.rows, req.nonaffix)
    np.testing.assert_allclose(r2.x[np.isin(r2.rows, req.nonaffix)], r1.x[non], rtol=1e-11, atol=1e-12)


def test_shift_invariance(setup2):
    dims, layers, req, sk, sv = setup2
    req_s = O.Request(x0=req.x0, pos=req.pos + 321, affix=req.affix, masked=req.masked)
    sk_s, sv_s = tiny_stale(layers, dims, req_s, seed=32)
    a = O.probe(layers, dims, req, sk, sv)
    b = O.probe(layers, dims, req_s, sk_s, sv_s)
    np.testing.assert_allclose(b.scores, a.scores, rtol=1e-10)
    np.testing.assert_allclose(b.x, a.x, rtol=1e-10, atol=1e-11)


# ----------------------------------------------------------------------------- maps (Section 4.1)

@pytest.mark.parametrize("layout", [(40, 0, 24, 32, 8), (40, 6, 20, 34, 6), (30, 10, 20, 0, 5)])
@pytest.mark.parametrize("k", [0, 5, "all"])
def test_maps_properties(layout, k):
    S, ab, L, mb, G = layout
    rng = np.random.default_rng(40)
    B = 3
    k = L if k == "all" else k
    anchors = np.stack([np.sort(rng.choice(L, size=k, replace=False)) for _ in range(B)]) if k else np.zeros((B, 0), int)
    stride = S
    row_pos, row_src, wslots, rslots, q_rows = O.build_maps(S, ab, L, mb, G, anchors, 0, L, stride)
    R = S - L + k
    assert len(row_pos) == B * R
    assert len(set(wslots.tolist())) == B * R and wslots.min() >= L  # private and unique
    for b in range(B):
        pos_b = row_pos[b * R:(b + 1) * R]
        assert np.all(np.diff(pos_b) > 0)
        expect = sorted(set(range(S)) - set(range(ab, ab + L)) | {ab + a for a in anchors[b]})
        np.testing.assert_array_equal(pos_b, expect)
        np.testing.assert_array_equal(row_src[b * R:(b + 1) * R], b * S + pos_b)
        for i, p in enumerate(pos_b):  # recomputed positions read what they wrote
            assert rslots[b * S + p] == wslots[b * R + i]
        for p in range(ab, ab + L):
            if p - ab not in set(anchors[b]):
                assert rslots[b * S + p] == p - ab  # shared region
        np.testing.assert_array_equal(row_pos[q_rows[b * G:(b + 1) * G]], np.arange(mb, mb + G))
        assert np.all((q_rows[b * G:(b + 1) * G] >= b * R) & (q_rows[b * G:(b + 1) * G] < (b + 1) * R))


# ----------------------------------------------------------------------------- DropNA (Section 5.3)

def test_dropna_equals_keepna_and_full_at_ratio_one(setup2):
    dims, layers, req, sk, sv = setup2
    L = len(req.affix)
    drop = O.drop_non_anchor_refresh(layers, dims, req, np.arange(L))
    keep = O.selective_refresh(layers, dims, req, np.arange(L), sk, sv)
    full = O.full_refresh(layers, dims, req)
    np.testing.assert_array_equal(drop.rows, full.rows)
    np.testing.assert_allclose(drop.x, keep.x, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(drop.x, full.x, rtol=1e-13, atol=1e-13)


def test_dropna_one_layer_matches_torch_block_over_recomputed_rows():
    """Attention sees exactly the recomputed rows' fresh K/V, nothing else."""
    dims = tiny_dims(nkv=2)
    layers = tiny_layers(dims, 1, seed=40)
    req = tiny_request(dims, seed=41)
    anchors = np.array([1, 4, 5, 9])
    drop = O.drop_non_anchor_refresh(layers, dims, req, anchors)
    rows = O.selective_rows(req, anchors)
    ref = layer_torch(layers[0], dims, req.x0[rows], req.pos[rows], lambda k, v: (k, v))
    np.testing.assert_allclose(drop.x, ref, rtol=1e-10, atol=1e-11)


def test_dropna_differs_from_keepna_below_ratio_one(setup2):
    dims, layers, req, sk, sv = setup2
    anchors = np.arange(0, len(req.affix), 5)
    drop = O.drop_non_anchor_refresh(layers, dims, req, anchors)
    keep = O.selective_refresh(layers, dims, req, anchors, sk, sv)
    np.testing.assert_array_equal(drop.rows, keep.rows)
    assert np.max(np.abs(drop.x - keep.x)) > 1e-3


# ----------------------------------------------------------------------------- shifted reuse (Section 4)

def test_rerotation_composes_with_rope():
    dims = tiny_dims(nkv=2)
    rng = np.random.default_rng(50)
    k = rng.standard_normal((9, dims.n_kv_heads, dims.head_dim))
    a = rng.integers(-500, 500, size=9)
    b = rng.integers(-5000, 5000, size=9)
    np.testing.assert_allclose(O.rerotate_keys(O.rope(k, a, dims.rope_base), b, dims.rope_base),
                               O.rope(k, a + b, dims.rope_base), rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(O.rerotate_keys(k, np.zeros(9, dtype=int), dims.rope_base), k, rtol=0, atol=0)


def test_shifted_donor_cache_is_the_rerotated_cache(setup2):
    """A donor materialised delta positions later has, at every layer, the
    same V and the K of the original donor turned by delta (attention sees
    only relative positions)."""
    dims, layers, req, sk, sv = setup2
    delta = 137
    donor = O.Request(x0=req.x0, pos=req.pos, affix=req.affix, masked=np.arange(0))
    moved = O.Request(x0=req.x0, pos=req.pos + delta, affix=req.affix, masked=np.arange(0))
    k0, v0 = O.materialize_affix_cache(layers, dims, donor)
    k1, v1 = O.materialize_affix_cache(layers, dims, moved)
    for n in range(len(layers)):
        d = np.full(len(req.affix), delta)
        np.testing.assert_allclose(k1[n], O.rerotate_keys(k0[n], d, dims.rope_base), rtol=1e-9, atol=1e-10)
        np.testing.assert_allclose(v1[n], v0[n], rtol=1e-9, atol=1e-10)


# ----------------------------------------------------------------------------- HKVD selector (appendix, CacheBlend-style selection)

def test_hkvd_scores_brute_force_and_zero_deviation(setup2):
    dims, layers, req, sk, sv = setup2
    s = O.hkvd_scores(layers, dims, req, sk, sv)
    n = O.hkvd_layer(len(layers))
    assert n == 1
    full = O.full_refresh(layers, dims, req)
    for j, row in enumerate(req.affix[:5]):
        want = 0.0
        for h in range(dims.n_kv_heads):
            for e in range(dims.head_dim):
                want += (full.views_k[n][row, h, e] - sk[n][j, h, e]) ** 2
                want += (full.views_v[n][row, h, e] - sv[n][j, h, e]) ** 2
        assert s[j] == pytest.approx(want, rel=1e-12)
    # a shared cache equal to the full-prompt cache deviates nowhere
    fk = [v[req.affix] for v in full.views_k]
    fv = [v[req.affix] for v in full.views_v]
    np.testing.assert_allclose(O.hkvd_scores(layers, dims, req, fk, fv), 0.0, atol=1e-20)


def test_hkvd_one_layer_uses_layer_zero():
    dims = tiny_dims(nkv=2)
    layers = tiny_layers(dims, 1, seed=70)
    req = tiny_request(dims, seed=71)
    sk, sv = tiny_stale(layers, dims, req, seed=72)
    assert O.hkvd_layer(1) == 0
    s = O.hkvd_scores(layers, dims, req, sk, sv)
    k0, v0 = O.layer_kv(layers[0], dims, req.x0[req.affix], req.pos[req.affix])
    np.testing.assert_allclose(s, ((k0 - sk[0]) ** 2).sum(axis=(1, 2)) + ((v0 - sv[0]) ** 2).sum(axis=(1, 2)),
                               rtol=1e-12)


@pytest.mark.parametrize("layout", [(40, 0, 24, 32, 8), (40, 6, 20, 34, 6)])
@pytest.mark.parametrize("k", [0, 5, "all"])
def test_paged_maps(layout, k):
    """Block-granular slots (Section 4.1).  With one slot per block and the
    flat plan's slots as the tables the paged maps are the flat maps; with
    larger blocks every request writes only inside its own blocks, every
    non-anchor affix position reads its shared block, and rows, positions
    and query rows do not depend on the slot plan."""
    S, ab, L, mb, G = layout
    rng = np.random.default_rng(41)
    B = 3
    k = L if k == "all" else k
    anchors = np.stack([np.sort(rng.choice(L, size=k, replace=False)) for _ in range(B)]) if k else np.zeros((B, 0), int)
    R = S - L + k
    flat = O.build_maps(S, ab, L, mb, G, anchors, 0, L, S)
    priv1 = np.array([L + b * S + i for b in range(B) for i in range(S)])
    paged1 = O.build_maps_paged(S, ab, L, mb, G, anchors, 1, np.arange(L), priv1, S)
    for a, p in zip(flat, paged1):
        np.testing.assert_array_equal(a, p)
    bs = 8
    nb_shared, nb = -(-L // bs), -(-R // bs)
    ids = rng.permutation(nb_shared + B * nb + 5)
    shared, private = ids[:nb_shared], ids[nb_shared:nb_shared + B * nb]
    row_pos, row_src, wslots, rslots, q_rows = O.build_maps_paged(S, ab, L, mb, G, anchors, bs, shared, private, nb)
    for a, p in zip((flat[0], flat[1], flat[4]), (row_pos, row_src, q_rows)):
        np.testing.assert_array_equal(a, p)
    assert len(set(wslots.tolist())) == B * R
    for b in range(B):
        own = set(int(i) for i in private[b * nb:(b + 1) * nb])
        assert all(int(s) // bs in own for s in wslots[b * R:(b + 1) * R])
        for i, p in enumerate(row_pos[b * R:(b + 1) * R]):
            assert rslots[b * S + p] == wslots[b * R + i]
        for j in sorted(set(range(L)) - set(int(a) for a in anchors[b])):
            s = rslots[b * S + ab + j]
            assert s // bs == shared[j // bs] and s % bs == j % bs
