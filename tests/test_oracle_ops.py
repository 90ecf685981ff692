"""Pins for the oracle's single operations: closed forms, brute force and
independent library routines.  CPU only."""

import itertools
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F
from scipy.special import logsumexp

from oracle import acache_oracle as O


# ----------------------------------------------------------------------------- RMSNorm

def test_rmsnorm_worked_example():
    # x = (3, 4): mean of squares 12.5, rms = 5/sqrt(2); unit gains, eps = 0
    y = O.rms_norm(np.array([[3.0, 4.0]]), np.ones(2), 0.0)
    np.testing.assert_allclose(y, [[3 * math.sqrt(2) / 5, 4 * math.sqrt(2) / 5]], rtol=1e-15)


def test_rmsnorm_scale_invariant_and_unit_rms():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 17))
    g = np.ones(17)
    y = O.rms_norm(x, g, 0.0)
    np.testing.assert_allclose(O.rms_norm(7.5 * x, g, 0.0), y, rtol=1e-13)
    np.testing.assert_allclose(np.sqrt(np.mean(y * y, axis=1)), 1.0, rtol=1e-13)


def test_rmsnorm_matches_torch():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((6, 33))
    g = rng.standard_normal(33)
    ref = F.rms_norm(torch.from_numpy(x), (33,), torch.from_numpy(g), eps=1e-5).numpy()
    np.testing.assert_allclose(O.rms_norm(x, g, 1e-5), ref, rtol=1e-12, atol=1e-14)


# ----------------------------------------------------------------------------- RoPE

def rope_complex(x, pos, base):
    """Rotary embedding written as complex multiplication: the pair
    (x_i, x_{i+d/2}) is the complex number x_i + 1j x_{i+d/2}, multiplied by
    exp(1j * pos * base^(-2i/d))."""
    dh = x.shape[-1]
    half = dh // 2
    z = x[..., :half] + 1j * x[..., half:]
    freqs = np.array([base ** (-(2 * i) / dh) for i in range(half)])
    rot = np.exp(1j * np.outer(pos, freqs))[:, None, :]
    w = z * rot
    return np.concatenate([w.real, w.imag], axis=-1)


def test_rope_matches_complex_rotation():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((9, 3, 16))
    pos = rng.integers(0, 5000, size=9)
    np.testing.assert_allclose(O.rope(x, pos, 10000.0), rope_complex(x, pos, 10000.0), rtol=1e-12, atol=1e-12)


def test_rope_two_dims_is_plane_rotation():
    # d_h = 2: one pair with theta_0 = 1, so position p rotates by p radians
    x = np.array([[[1.0, 0.0]], [[0.3, -2.0]]])
    pos = np.array([1, 3])
    y = O.rope(x, pos, 10000.0)
    for r in range(2):
        c, s = math.cos(pos[r]), math.sin(pos[r])
        rot = np.array([[c, -s], [s, c]])
        np.testing.assert_allclose(y[r, 0], rot @ x[r, 0], rtol=1e-14, atol=1e-15)


def test_rope_identity_at_zero_and_norm_preserving():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((4, 2, 8))
    np.testing.assert_array_equal(O.rope(x, np.zeros(4, dtype=int), 10000.0), x)
    y = O.rope(x, np.array([5, 77, 1000, 8000]), 10000.0)
    pair_norm = lambda t: t[..., :4] ** 2 + t[..., 4:] ** 2
    np.testing.assert_allclose(pair_norm(y), pair_norm(x), rtol=1e-12)


def test_rope_relative_position_property():
    # q_m . k_n depends only on m - n
    rng = np.random.default_rng(4)
    q = rng.standard_normal((1, 1, 16))
    k = rng.standard_normal((1, 1, 16))
    dots = []
    for shift in (0, 13, 400):
        qm = O.rope(q, np.array([50 + shift]), 10000.0)
        kn = O.rope(k, np.array([20 + shift]), 10000.0)
        dots.append(float((qm * kn).sum()))
    np.testing.assert_allclose(dots, dots[0], rtol=1e-11)


# ----------------------------------------------------------------------------- attention

def attention_loops(q, k, v):
    """Triple loop with math.exp (tiny inputs only)."""
    m, nh, dh = q.shape
    s, nkv, _ = k.shape
    grp = nh // nkv
    o = np.zeros_like(q)
    lse = np.zeros((m, nh))
    for i in range(m):
        for h in range(nh):
            g = h // grp
            logit = [sum(q[i, h, t] * k[j, g, t] for t in range(dh)) / math.sqrt(dh) for j in range(s)]
            mx = max(logit)
            w = [math.exp(l - mx) for l in logit]
            z = sum(w)
            lse[i, h] = mx + math.log(z)
            for t in range(dh):
                o[i, h, t] = sum(w[j] * v[j, g, t] for j in range(s)) / z
    return o, lse


@pytest.mark.parametrize("nh,nkv", [(2, 2), (4, 2), (3, 1)])
def test_attention_brute_force(nh, nkv):
    rng = np.random.default_rng(5 + nh)
    q = rng.standard_normal((3, nh, 4))
    k = rng.standard_normal((5, nkv, 4))
    v = rng.standard_normal((5, nkv, 4))
    o, lse = O.attention(q, k, v)
    o2, lse2 = attention_loops(q, k, v)
    np.testing.assert_allclose(o, o2, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(lse, lse2, rtol=1e-12)


def test_attention_matches_torch_sdpa_and_logsumexp():
    rng = np.random.default_rng(6)
    nh, nkv, dh = 8, 2, 16
    q = rng.standard_normal((11, nh, dh))
    k = rng.standard_normal((37, nkv, dh))
    v = rng.standard_normal((37, nkv, dh))
    o, lse = O.attention(q, k, v)
    tq = torch.from_numpy(q).permute(1, 0, 2)
    tk = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(nh // nkv, dim=0)
    tv = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(nh // nkv, dim=0)
    ref = F.scaled_dot_product_attention(tq, tk, tv).permute(1, 0, 2).numpy()
    np.testing.assert_allclose(o, ref, rtol=1e-11, atol=1e-12)
    for h in range(nh):
        logits = q[:, h] @ k[:, h // (nh // nkv)].T / math.sqrt(dh)
        np.testing.assert_allclose(lse[:, h], logsumexp(logits, axis=1), rtol=1e-13)


def test_attention_special_cases():
    rng = np.random.default_rng(7)
    q = rng.standard_normal((4, 2, 8))
    k = rng.standard_normal((6, 2, 8))
    # rows sum to one: V = 1 gives O = 1
    o, _ = O.attention(q, k, np.ones((6, 2, 8)))
    np.testing.assert_allclose(o, 1.0, rtol=1e-14)
    # one key: O = V
    v1 = rng.standard_normal((1, 2, 8))
    o, lse = O.attention(q, k[:1], v1)
    np.testing.assert_allclose(o, np.broadcast_to(v1, o.shape), rtol=1e-14)
    # equal keys: O = mean of V, lse = logit + log(S)
    kk = np.broadcast_to(k[:1], (6, 2, 8)).copy()
    v = rng.standard_normal((6, 2, 8))
    o, lse = O.attention(q, kk, v)
    np.testing.assert_allclose(o, np.broadcast_to(v.mean(axis=0), o.shape), rtol=1e-12, atol=1e-14)
    # permuting keys together with values leaves O unchanged
    perm = rng.permutation(6)
    o1, l1 = O.attention(q, k, v)
    o2, l2 = O.attention(q, k[perm], v[perm])
    np.testing.assert_allclose(o1, o2, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(l1, l2, rtol=1e-13)


def test_attention_via_slots_equals_gathered_view():
    rng = np.random.default_rng(8)
    pool_k = rng.standard_normal((20, 2, 8))
    pool_v = rng.standard_normal((20, 2, 8))
    q = rng.standard_normal((7, 4, 8))
    read = np.array([3, 9, 1, 0, 17, 5, 5, 12, 19])
    cu_rows, cu_keys = [0, 4, 7], [0, 5, 9]
    o, lse = O.attention_via_slots(q, pool_k, pool_v, read, cu_rows, cu_keys)
    o2, _ = attention_loops(q[:4], pool_k[read[:5]], pool_v[read[:5]])
    np.testing.assert_allclose(o[:4], o2, rtol=1e-12, atol=1e-13)
    o3, _ = attention_loops(q[4:], pool_k[read[5:]], pool_v[read[5:]])
    np.testing.assert_allclose(o[4:], o3, rtol=1e-12, atol=1e-13)


# ----------------------------------------------------------------------------- scores (Eq. 4-5)

def scores_loops(q, k, norm, lse_full=None):
    g_rows, nh, dh = q.shape
    L, nkv, _ = k.shape
    grp = nh // nkv
    s = [0.0] * L
    for h in range(nh):
        for r in range(g_rows):
            logit = [sum(q[r, h, t] * k[j, h // grp, t] for t in range(dh)) / math.sqrt(dh) for j in range(L)]
            if norm == "affix":
                z = sum(math.exp(l) for l in logit)
                for j in range(L):
                    s[j] += math.exp(logit[j]) / z
            else:
                for j in range(L):
                    s[j] += math.exp(logit[j] - lse_full[r, h])
    return np.array(s)


@pytest.mark.parametrize("nh,nkv", [(2, 2), (4, 1)])
def test_scores_brute_force_affix_norm(nh, nkv):
    rng = np.random.default_rng(9)
    q = rng.standard_normal((3, nh, 4))
    k = rng.standard_normal((6, nkv, 4))
    np.testing.assert_allclose(O.affix_attention_mass(q, k, "affix"), scores_loops(q, k, "affix"), rtol=1e-12)


def test_scores_full_norm_brute_force_and_bounds():
    rng = np.random.default_rng(10)
    nh, dh = 2, 4
    q = rng.standard_normal((3, nh, dh))
    k_all = rng.standard_normal((9, nh, dh))
    v_all = rng.standard_normal((9, nh, dh))
    affix = np.array([1, 2, 5, 7])
    _, lse = O.attention(q, k_all, v_all)
    full = O.affix_attention_mass(q, k_all[affix], "full", lse)
    np.testing.assert_allclose(full, scores_loops(q, k_all[affix], "full", lse), rtol=1e-12)
    aff = O.affix_attention_mass(q, k_all[affix], "affix")
    # a softmax over a superset of keys gives each affix key a smaller weight
    assert np.all(full <= aff + 1e-15)
    # affix columns plus the remaining columns of the full softmax sum to H * G
    rest = np.setdiff1d(np.arange(9), affix)
    other = O.affix_attention_mass(q, k_all[rest], "full", lse)
    np.testing.assert_allclose(full.sum() + other.sum(), nh * 3, rtol=1e-13)


def test_scores_mass_conservation_and_equal_keys():
    rng = np.random.default_rng(11)
    nh, g_rows, L = 4, 5, 9
    q = rng.standard_normal((g_rows, nh, 8))
    k = rng.standard_normal((L, 2, 8))
    s = O.affix_attention_mass(q, k, "affix")
    assert np.all(s >= 0)
    np.testing.assert_allclose(s.sum(), nh * g_rows, rtol=1e-13)
    keq = np.broadcast_to(k[:1], k.shape).copy()
    np.testing.assert_allclose(O.affix_attention_mass(q, keq, "affix"), nh * g_rows / L, rtol=1e-12)


def test_scores_gqa_equals_repeated_kv():
    rng = np.random.default_rng(12)
    q = rng.standard_normal((4, 6, 8))
    k = rng.standard_normal((7, 2, 8))
    s1 = O.affix_attention_mass(q, k, "affix")
    s2 = O.affix_attention_mass(q, np.repeat(k, 3, axis=1), "affix")
    np.testing.assert_allclose(s1, s2, rtol=1e-13)


def test_scores_via_slots_batches():
    rng = np.random.default_rng(13)
    pool = rng.standard_normal((30, 2, 8))
    q = rng.standard_normal((10, 2, 8))
    q_rows = np.array([1, 2, 3, 7, 9])
    cu_q = [0, 3, 5]
    aff = np.array([4, 5, 6, 10, 11])
    s = O.scores_via_slots(q, q_rows, cu_q, pool, aff)
    np.testing.assert_allclose(s[0], scores_loops(q[[1, 2, 3]], pool[aff], "affix"), rtol=1e-12)
    np.testing.assert_allclose(s[1], scores_loops(q[[7, 9]], pool[aff], "affix"), rtol=1e-12)


# ----------------------------------------------------------------------------- top-K (Eq. 6)

def topk_brute(s, k):
    """Among all k-subsets with the largest score sum, the lexicographically
    smallest ascending index tuple (finite scores only)."""
    best = None
    for comb in itertools.combinations(range(len(s)), k):
        key = (-sum(s[i] for i in comb), comb)
        if best is None or key < best:
            best = key
    return np.array(best[1] if best else [], dtype=np.int64)


@pytest.mark.parametrize("seed", range(6))
def test_topk_brute_force_subsets(seed):
    rng = np.random.default_rng(100 + seed)
    L = 9
    s = rng.integers(0, 4, size=L).astype(np.float64) if seed % 2 else rng.standard_normal(L)
    for k in range(L + 1):
        np.testing.assert_array_equal(O.topk_anchors(s, k), topk_brute(list(s), k))


def test_topk_matches_stable_argsort():
    rng = np.random.default_rng(14)
    s = rng.integers(0, 50, size=1000).astype(np.float64)
    for k in (0, 1, 200, 999, 1000):
        ref = np.sort(np.argsort(-s, kind="stable")[:k])
        np.testing.assert_array_equal(O.topk_anchors(s, k), ref)


def test_topk_signed_zero_nan_inf():
    assert list(O.topk_anchors(np.array([-0.0, 0.0]), 1)) == [0]
    assert list(O.topk_anchors(np.array([0.0, -0.0]), 1)) == [0]
    s = np.array([np.nan, -np.inf, 1.0, np.nan, np.inf, -0.0])
    assert list(O.topk_anchors(s, 1)) == [4]
    assert list(O.topk_anchors(s, 3)) == [2, 4, 5]
    assert list(O.topk_anchors(s, 4)) == [1, 2, 4, 5]
    assert list(O.topk_anchors(s, 5)) == [0, 1, 2, 4, 5]
    assert list(O.topk_anchors(s, 6)) == [0, 1, 2, 3, 4, 5]


# ----------------------------------------------------------------------------- greedy commit (Section 3.1)

def test_greedy_commit_special_rows():
    nan, inf = np.nan, np.inf
    rows = [
        [1.0, 3.0, 3.0, 2.0],      # tie: lowest index
        [-0.0, 0.0, -1.0, -2.0],   # -0 == +0: index 0
        [nan, -inf, nan, -5.0],    # NaN below everything
        [nan, nan, nan, nan],      # all NaN: lowest index
        [-inf, -inf, -inf, -inf],
        [inf, 1.0, inf, nan],
    ]
    np.testing.assert_array_equal(O.greedy_commit(np.array(rows)), [1, 0, 3, 0, 0, 0])


def test_greedy_commit_brute_force_and_numpy():
    rng = np.random.default_rng(7)
    x = rng.integers(-3, 4, size=(50, 37)).astype(np.float64)  # many ties
    got = O.greedy_commit(x)
    for i, row in enumerate(x):
        best = 0
        for j in range(1, row.size):
            if row[j] > row[best]:
                best = j
        assert got[i] == best
    np.testing.assert_array_equal(got, np.argmax(x, axis=1))  # first maximum, as numpy defines it


def test_confidence_and_threshold_commit():
    x = np.array([[0.0, np.log(3.0), -np.inf, np.nan],   # probs 1/4, 3/4 -> 0.75
                  [1.0, 1.0, 1.0, 1.0],                    # 0.25
                  [np.nan, -np.inf, np.nan, -np.inf]])     # no finite value -> 0
    np.testing.assert_allclose(O.confidence(x), [0.75, 0.25, 0.0], rtol=1e-12)
    conf = np.array([0.3, 0.95, 0.2, 0.97, np.nan])
    np.testing.assert_array_equal(O.threshold_commit(conf, np.zeros(5, bool), 0.9), [0, 1, 0, 1, 0])
    # none above tau: the single most confident free row, lowest row on ties
    np.testing.assert_array_equal(O.threshold_commit(np.array([0.3, 0.5, 0.5, 0.1]), np.array([0, 0, 0, 0], bool), 0.9),
                                  [0, 1, 0, 0])
    np.testing.assert_array_equal(O.threshold_commit(np.array([0.3, 0.5, 0.5, 0.1]), np.array([0, 1, 0, 0], bool), 0.9),
                                  [0, 0, 1, 0])
    # nothing left to commit
    assert not O.threshold_commit(np.array([0.9]), np.array([True]), 0.5).any()
    # brute force: random confidences
    rng = np.random.default_rng(5)
    for _ in range(50):
        c = rng.random(8)
        done = rng.random(8) < 0.3
        t = O.threshold_commit(c, done, 0.7)
        want = (~done) & (c >= 0.7)
        if not want.any() and (~done).any():
            want = np.zeros(8, bool)
            want[min(np.flatnonzero(~done), key=lambda i: (-c[i], i))] = True
        np.testing.assert_array_equal(t, want)


# ----------------------------------------------------------------------------- anchor count (Eq. 6's K)

def anchor_count_brute(ratio, L):
    """The integer K in [0, L] nearest to ratio * L, the larger one on a tie
    (distance compared exactly in rationals)."""
    from fractions import Fraction
    t = Fraction(ratio) * L
    best = None
    for k in range(L + 1):
        d = abs(Fraction(k) - t)
        if best is None or d < best[0] or (d == best[0] and k > best[1]):
            best = (d, k)
    return best[1]


def test_anchor_count_of_the_workloads():
    # ratio 0.2 at the workloads' affix lengths: rho * L = 25.6, 204.8,
    # 409.6, 819.2, 1638.4; the tiny workload states "26 tokens" for 0.2 x 128
    assert O.anchor_count(0.2, 128) == 26
    assert O.anchor_count(0.2, 1024) == 205
    assert O.anchor_count(0.2, 2048) == 410
    assert [O.anchor_count(r, 4096) for r in (0.1, 0.2, 0.4)] == [410, 819, 1638]
    assert O.anchor_count(0.2, 8192) == 1638
    # the readings it rules out: floor gives 25 at 25.6, ceil 820 at 819.2
    assert math.floor(0.2 * 128) == 25 and math.ceil(0.2 * 4096) == 820


@pytest.mark.parametrize("L", [0, 1, 2, 7, 10, 128, 250, 1000])
def test_anchor_count_is_nearest_integer(L):
    for ratio in (0.0, 0.05, 0.1, 0.125, 0.2, 0.25, 0.3, 1 / 3, 0.5, 0.75, 0.999, 1.0):
        assert O.anchor_count(ratio, L) == anchor_count_brute(ratio, L), (ratio, L)


def test_anchor_count_halves_and_bounds():
    assert O.anchor_count(0.5, 1) == 1      # 0.5 exactly: up
    assert O.anchor_count(0.25, 2) == 1     # 0.5 exactly: up
    assert O.anchor_count(0.375, 4) == 2    # 1.5 exactly: up
    assert O.anchor_count(0.0, 100) == 0 and O.anchor_count(1.0, 100) == 100
    with pytest.raises(ValueError):
        O.anchor_count(-0.1, 10)
    with pytest.raises(ValueError):
        O.anchor_count(1.5, 10)
