"""End-to-end GPU parity of the hot path on seeded workloads, through the
C ABI: stale affix cache, probe scores (Eq. 4-5), anchors (Eq. 6) and the
selective refresh (Section 3.3), each against the fp64 oracle computed
from the same input bits; plus the paper's invariants on the GPU path.

Workloads: the tiny fp32 layer and the LLaDA-shaped bf16 layer at their
full sizes, and small bf16 / fp32 stacks (prefix MHA, infix GQA)."""

import numpy as np
import pytest

import workloads as W
from oracle import acache_oracle as O
from tests.gpu_util import TOL, assert_close, down, down_bits, errors, up, up_i32
from tests.oracle_side import anchor_count, rows_selective, check_anchors, oracle_dims, oracle_layers, oracle_request, oracle_stale

pytestmark = pytest.mark.gpu

NAMES = ["tiny-f32", "llada-layer", "mini-stack", "mini-affix64", "mini-infix64", "mini-gqa-infix", "mini-f32-stack"]


def storage_round(a: np.ndarray, dtype: str) -> np.ndarray:
    """float64 -> storage bits of the KV cache type."""
    return W.bf16_bits_from_f32(a.astype(np.float32)) if dtype == "bf16" else a.astype(np.float32)


@pytest.fixture(scope="module", params=NAMES)
def case(request):
    """GPU setup plus the oracle.  The GPU first materialises its own stale
    affix cache (kept in ``materialized``); then both sides switch to one
    common stale cache, the oracle's rounded to the storage type, so the
    probe, selection and refresh are compared on identical inputs."""
    import torch
    assert torch.cuda.is_available()
    from paper_2608_26140_amd import workload as WL
    w = W.get_config(request.param)
    s = WL.build(w)
    torch.cuda.synchronize()
    dt = w.dims.dtype
    L = w.layout.affix_len
    layers = oracle_layers(w, s.host)
    sk64, sv64 = oracle_stale(w, s.host, layers)
    materialized = [(k[:L].clone(), v[:L].clone()) for k, v in zip(s.batch.k_pools, s.batch.v_pools)]
    sk, sv = [], []
    for n in range(len(layers)):
        kb, vb = storage_round(sk64[n], dt), storage_round(sv64[n], dt)
        s.batch.k_pools[n][:L] = up(kb.reshape(L, -1), dt)
        s.batch.v_pools[n][:L] = up(vb.reshape(L, -1), dt)
        sk.append(O.from_bits(kb, dt))
        sv.append(O.from_bits(vb, dt))
    torch.cuda.synchronize()
    s.host["materialized"] = materialized
    s.host["stale64"] = (sk64, sv64)
    return w, s, layers, sk, sv, OracleCache(w, s.host, layers, sk, sv)


class OracleCache:
    """Each oracle quantity is computed once per workload."""

    def __init__(self, w, host, layers, sk, sv):
        self.w, self.host, self.layers, self.sk, self.sv = w, host, layers, sk, sv
        self.dims = oracle_dims(w)
        self.memo = {}

    def _get(self, key, fn):
        if key not in self.memo:
            self.memo[key] = fn()
        return self.memo[key]

    def req(self, b):
        return self._get(("req", b), lambda: oracle_request(self.w, self.host, b))

    def probe(self, b, norm="affix"):
        return self._get(("probe", b, norm), lambda: O.probe(self.layers, self.dims, self.req(b), self.sk, self.sv, norm))

    def anchors(self, b):
        return self._get(("anchors", b), lambda: O.topk_anchors(self.probe(b).scores, anchor_count(self.w)))

    def selective(self, b):
        return self._get(("sel", b), lambda: O.selective_refresh(self.layers, self.dims, self.req(b), self.anchors(b),
                                                                   self.sk, self.sv))

    def drop(self, b):
        return self._get(("drop", b), lambda: O.drop_non_anchor_refresh(self.layers, self.dims, self.req(b),
                                                                          self.anchors(b)))

    def full(self, b):
        return self._get(("full", b), lambda: O.full_refresh(self.layers, self.dims, self.req(b)))


def _pool_rows(pool, slots, w):
    d = w.dims
    return down(pool)[np.asarray(slots)].reshape(len(slots), d.n_kv_heads, d.head_dim)


def test_stale_cache(case):
    """The GPU's own materialisation of the shared affix cache (a full
    forward of the donor context) against the oracle's."""
    w, s, layers, sk, sv, oc = case
    sk64, sv64 = s.host["stale64"]
    for n, (k, v) in enumerate(s.host["materialized"]):
        assert_close(_pool_rows(k, np.arange(k.shape[0]), w), sk64[n], w.dims.dtype, f"stale K layer {n}")
        assert_close(_pool_rows(v, np.arange(v.shape[0]), w), sv64[n], w.dims.dtype, f"stale V layer {n}")


@pytest.mark.parametrize("norm", ["affix", "full"])
def test_probe_scores_and_anchors(case, norm):
    from paper_2608_26140_amd import acache as A
    w, s, layers, sk, sv, oc = case
    dims = oracle_dims(w)
    dt = w.dims.dtype
    code = A.ACACHE_NORM_AFFIX if norm == "affix" else A.ACACHE_NORM_FULL
    scores, x_probe, m = s.batch.probe(code)
    anchors = A.acache_topk(scores, anchor_count(w))
    g_scores = down(scores)
    g_anchors = anchors.cpu().numpy()
    P = w.layout.n_nonaffix
    K = anchor_count(w)
    # anchors from the GPU scores are exactly the oracle's top-K of those scores
    for b in range(w.batch):
        np.testing.assert_array_equal(g_anchors[b], O.topk_anchors(g_scores[b], K))
    for b in range(w.batch):
        res = oc.probe(b, norm)
        e = assert_close(g_scores[b], res.scores, dt, f"scores request {b}")
        assert_close(down(x_probe)[b * P:(b + 1) * P], res.x, dt, f"probe rows request {b}")
        check_anchors(g_anchors[b], res.scores, K, e["max_abs"], f"{w.name} request {b} ({norm})")
        if norm == "affix":
            np.testing.assert_allclose(g_scores[b].sum(), len(layers) * w.dims.n_heads * w.layout.mask_len,
                                       rtol=1e-3 if dt == "bf16" else 1e-5)


@pytest.mark.parametrize("norm", ["affix", "full"])
def test_score_only_last_layer(case, norm):
    """The probe whose last layer stops at its score (acache_layer_score):
    scores and anchors against the oracle's full probe, scores close to the
    GPU's full probe, and under the affix-only normalisation the last
    layer's pools are not written."""
    import torch
    from paper_2608_26140_amd import acache as A
    w, s, layers, sk, sv, oc = case
    dt = w.dims.dtype
    code = A.ACACHE_NORM_AFFIX if norm == "affix" else A.ACACHE_NORM_FULL
    full_scores, _, _ = s.batch.probe(code)
    before = (s.batch.k_pools[-1].clone(), s.batch.v_pools[-1].clone())
    scores, x, _ = s.batch.probe(code, outputs=False)
    torch.cuda.synchronize()
    assert x is None
    if norm == "affix":
        assert torch.equal(s.batch.k_pools[-1], before[0]) and torch.equal(s.batch.v_pools[-1], before[1])
    g = down(scores)
    assert_close(g, down(full_scores), dt, "score-only against full probe")
    K = anchor_count(w)
    anchors = A.acache_topk(scores, K).cpu().numpy()
    for b in range(w.batch):
        res = oc.probe(b, norm)
        e = assert_close(g[b], res.scores, dt, f"scores request {b}")
        check_anchors(anchors[b], res.scores, K, e["max_abs"], f"{w.name} score-only request {b} ({norm})")


def test_probe_affix_lse_from_attention(case):
    """Affix-normalised probe scores whether the attention hands the score
    each row's log-sum-exp over the affix keys (the probe reads the affix
    keys first; taken where the affix is whole 64-key tiles: the LLaDA layer,
    mini-affix64 and the infix mini-infix64, whose small probe grids split
    the attention's keys, so the splits' shares go through the merge) or the
    score makes its own pass over them, keys in logical order: both against
    the oracle and close to each other."""
    from paper_2608_26140_amd import acache as A
    w, s, layers, sk, sv, oc = case
    dt = w.dims.dtype
    with_lse, _, _ = s.batch.probe(A.ACACHE_NORM_AFFIX, attention_lse=True)
    own, _, _ = s.batch.probe(A.ACACHE_NORM_AFFIX, attention_lse=False)
    g, h = down(with_lse), down(own)
    assert_close(g, h, dt, "attention log-sum-exp against the score's own")
    for b in range(w.batch):
        res = oc.probe(b, "affix")
        assert_close(g[b], res.scores, dt, f"scores request {b} (attention log-sum-exp)")
        assert_close(h[b], res.scores, dt, f"scores request {b} (score's own pass)")


def test_score_init_writes(case):
    """init on the probe's first layer writes the scores instead of adding:
    a buffer full of NaN ends with the same bits as the accumulating path on
    a cleared buffer."""
    import torch
    from paper_2608_26140_amd import acache as A
    w, s, layers, sk, sv, oc = case
    b = s.batch
    m = b.maps(None, 0)
    out = {}
    for init, fill in ((0, 0.0), (1, float("nan"))):
        x = b.gather_inputs(m)
        scores = torch.full((b.B, b.L), fill, dtype=torch.float32, device="cuda")
        score = dict(q_rows=m["q_rows"], cu_q=[i * b.G for i in range(b.B + 1)], affix_slots=b.affix_slots,
                     scores=scores, norm=A.ACACHE_NORM_AFFIX, init=init)
        b.run_layers(x, m, 0, score=score)
        torch.cuda.synchronize()
        out[init] = scores.clone()
    assert not torch.isnan(out[1]).any()
    assert torch.equal(out[0], out[1])


def test_selective_refresh_with_common_anchors(case):
    """Both sides refresh with the oracle's anchor set."""
    w, s, layers, sk, sv, oc = case
    dims = oracle_dims(w)
    dt = w.dims.dtype
    anchors = [oc.anchors(b) for b in range(w.batch)]
    refs = [oc.selective(b) for b in range(w.batch)]
    x, m = s.batch.refresh(up_i32(np.stack(anchors)), anchor_count(w))
    R = rows_selective(w)
    gx = down(x)
    wslots = m["write_slots"].cpu().numpy()
    for b in range(w.batch):
        assert_close(gx[b * R:(b + 1) * R], refs[b].x, dt, f"refresh rows request {b}")
        rows = refs[b].rows
        for n in range(len(layers)):
            assert_close(_pool_rows(s.batch.k_pools[n], wslots[b * R:(b + 1) * R], w), refs[b].views_k[n][rows], dt,
                         f"fresh K request {b} layer {n}")
            assert_close(_pool_rows(s.batch.v_pools[n], wslots[b * R:(b + 1) * R], w), refs[b].views_v[n][rows], dt,
                         f"fresh V request {b} layer {n}")


def test_end_to_end_own_anchors(case):
    """GPU probe -> GPU top-K -> GPU refresh, against the oracle's own chain;
    compared on the request-specific rows (present in both)."""
    from paper_2608_26140_amd import acache as A
    w, s, layers, sk, sv, oc = case
    dims = oracle_dims(w)
    dt = w.dims.dtype
    anchors, _ = s.batch.select_anchors(anchor_count(w))
    x, m = s.batch.refresh(anchors, anchor_count(w))
    R = rows_selective(w)
    gx = down(x)
    pos = m["row_pos"].cpu().numpy()
    for b in range(w.batch):
        req = oc.req(b)
        ref = oc.selective(b)
        pb = pos[b * R:(b + 1) * R]
        keep = np.isin(pb, req.nonaffix)
        keep_ref = np.isin(ref.rows, req.nonaffix)
        assert_close(gx[b * R:(b + 1) * R][keep], ref.x[keep_ref], dt, f"end-to-end request {b}")


def test_ratio_one_equals_full_and_ignores_stale(case):
    """Anchor ratio 1 is full recomputation: poisoning the whole shared
    affix cache with NaN leaves the output finite and unchanged."""
    import torch
    w, s, layers, sk, sv, oc = case
    L = w.layout.affix_len
    x_full, _ = s.batch.full_refresh()
    ref = down(x_full).copy()
    saved = [(k[:L].clone(), v[:L].clone()) for k, v in zip(s.batch.k_pools, s.batch.v_pools)]
    for k, v in zip(s.batch.k_pools, s.batch.v_pools):
        k[:L] = float("nan")
        v[:L] = float("nan")
    every = torch.arange(L, dtype=torch.int32, device="cuda").repeat(w.batch, 1).contiguous()
    x_sel, _ = s.batch.refresh(every, L)
    got = down(x_sel)
    for (k0, v0), k, v in zip(saved, s.batch.k_pools, s.batch.v_pools):
        k[:L] = k0
        v[:L] = v0
    assert np.all(np.isfinite(got))
    np.testing.assert_array_equal(got, ref)
    # and it matches the oracle's full recompute
    dims = oracle_dims(w)
    S = w.layout.seq_len
    for b in range(w.batch):
        r = oc.full(b)
        assert_close(got[b * S:(b + 1) * S], r.x, w.dims.dtype, f"full refresh request {b}")


def test_ratio_zero_equals_direct_reuse(case):
    """Anchor ratio 0 is direct reuse: the rows and outputs of the probe
    forward (scoring does not change them).  Bit for bit with the keys in
    logical order; the probe's own order (affix keys first) changes only the
    attention's summation order."""
    w, s, layers, sk, sv, oc = case
    x0, _ = s.batch.refresh(None, 0)
    g0 = down_bits(x0)
    _, x_probe, _ = s.batch.probe(attention_lse=False)
    np.testing.assert_array_equal(g0, down_bits(x_probe))
    _, x_first, _ = s.batch.probe()
    if w.layout.affix_begin == 0:
        np.testing.assert_array_equal(g0, down_bits(x_first))
    else:
        assert_close(down(x_first), down(x0), w.dims.dtype, "probe rows, affix keys first")
    x1, _ = s.batch.direct_reuse()
    np.testing.assert_array_equal(g0, down_bits(x1))


def test_dropna_against_oracle_and_never_reads_non_anchors(case):
    """DropNA (Section 5.3): the same anchors, attention over the recomputed
    rows only.  The shared affix region is poisoned with NaN: no non-anchor
    entry may be read."""
    w, s, layers, sk, sv, oc = case
    dt = w.dims.dtype
    L, R = w.layout.affix_len, rows_selective(w)
    anchors = np.stack([oc.anchors(b) for b in range(w.batch)])
    saved = [(k[:L].clone(), v[:L].clone()) for k, v in zip(s.batch.k_pools, s.batch.v_pools)]
    for k, v in zip(s.batch.k_pools, s.batch.v_pools):
        k[:L] = float("nan")
        v[:L] = float("nan")
    try:
        x, _ = s.batch.refresh(up_i32(anchors), anchor_count(w), drop_non_anchor=True)
        gx = down(x)
    finally:
        for (k0, v0), k, v in zip(saved, s.batch.k_pools, s.batch.v_pools):
            k[:L] = k0
            v[:L] = v0
    for b in range(w.batch):
        assert_close(gx[b * R:(b + 1) * R], oc.drop(b).x, dt, f"DropNA rows request {b}")


def test_keepna_equals_dropna_at_ratio_one(case):
    """With every affix token an anchor there is no non-anchor entry left:
    KeepNA and DropNA read the same keys in the same order."""
    import torch
    w, s, layers, sk, sv, oc = case
    L = w.layout.affix_len
    every = torch.arange(L, dtype=torch.int32, device="cuda").repeat(w.batch, 1).contiguous()
    keep, _ = s.batch.refresh(every, L)
    keep = down_bits(keep).copy()
    drop, _ = s.batch.refresh(every, L, drop_non_anchor=True)
    np.testing.assert_array_equal(down_bits(drop), keep)


def test_hkvd_selector_against_oracle(case):
    """The CacheBlend-style selector (KV deviation between the shared cache
    and the full-prompt cache at the selection layer) and its top-K.

    The deviation is a difference of two nearly equal caches, so the bf16
    storage of the fresh K/V moves it far more than it moves either cache.
    The fresh K/V are held to the fp64 oracle (the tolerance gates); the
    deviation kernel and the anchor gate are checked on the K/V the GPU
    stored (the oracle's deviation of those bits); the overlap with the
    all-fp64 selection is reported."""
    w, s, layers, sk, sv, oc = case
    dims = oracle_dims(w)
    dt = w.dims.dtype
    lay = w.layout
    K = anchor_count(w)
    n = O.hkvd_layer(len(layers))
    anchors, scores = s.batch.select_anchors_hkvd(K)
    g_scores, g_anchors = down(scores), anchors.cpu().numpy()
    aff = np.arange(lay.affix_begin, lay.affix_end)
    fresh_slots = s.batch.private_slots(lay.seq_len)[:, aff]
    for b in range(w.batch):
        np.testing.assert_array_equal(g_anchors[b], O.topk_anchors(g_scores[b], K))
        full = O.full_refresh(layers[:n + 1], dims, oc.req(b))
        gk = _pool_rows(s.batch.k_pools[n], fresh_slots[b], w)
        gv = _pool_rows(s.batch.v_pools[n], fresh_slots[b], w)
        assert_close(gk, full.views_k[n][aff], dt, f"HKVD full-prompt K layer {n} request {b}")
        assert_close(gv, full.views_v[n][aff], dt, f"HKVD full-prompt V layer {n} request {b}")
        ref = O.kv_deviation(gk, gv, sk[n], sv[n])
        # fp32 arithmetic on the same inputs: the fp32 bar
        e = assert_close(g_scores[b], ref, "f32", f"KV deviation request {b}")
        check_anchors(g_anchors[b], ref, K, e["max_abs"], f"{w.name} HKVD request {b}")
        exact = O.hkvd_scores(layers, dims, oc.req(b), sk, sv)
        ov = len(set(g_anchors[b].tolist()) & set(O.topk_anchors(exact, K).tolist())) / max(K, 1)
        print(f"[anchors] {w.name} HKVD request {b}: overlap with the all-fp64 selection {ov:.4f}", flush=True)


def test_anchor_stale_poison_and_determinism(case):
    """NaN in the stale KV of the anchor slots must not reach any output;
    repeated runs are bit-identical."""
    import torch
    w, s, layers, sk, sv, oc = case
    anchors, scores = s.batch.select_anchors(anchor_count(w))
    anchors2, scores2 = s.batch.select_anchors(anchor_count(w))
    assert torch.equal(scores, scores2) and torch.equal(anchors, anchors2)
    x_a, _ = s.batch.refresh(anchors, anchor_count(w))
    ref = down_bits(x_a).copy()
    if w.batch == 1:
        a = anchors[0].long()
        saved = [(k[a].clone(), v[a].clone()) for k, v in zip(s.batch.k_pools, s.batch.v_pools)]
        for k, v in zip(s.batch.k_pools, s.batch.v_pools):
            k[a] = float("nan")
            v[a] = float("nan")
        x_p, _ = s.batch.refresh(anchors, anchor_count(w))
        for (k0, v0), k, v in zip(saved, s.batch.k_pools, s.batch.v_pools):
            k[a] = k0
            v[a] = v0
        np.testing.assert_array_equal(down_bits(x_p), ref)
    x_b, _ = s.batch.refresh(anchors, anchor_count(w))
    np.testing.assert_array_equal(down_bits(x_b), ref)


def test_materialized_chain_against_oracle_chain(case):
    """Fully independent chains: the GPU materialises its own stale cache,
    probes, selects and refreshes; the oracle does the same in fp64.  With
    a bf16 KV cache the stale keys differ by their storage rounding, which
    moves near-tied scores at the K-th place: every anchor in the symmetric
    difference must lie in the tie band, and the overlap is recorded."""
    import torch
    w, s, layers, sk, sv, oc = case
    L = w.layout.affix_len
    dt = w.dims.dtype
    common = [(k[:L].clone(), v[:L].clone()) for k, v in zip(s.batch.k_pools, s.batch.v_pools)]
    for (k0, v0), k, v in zip(s.host["materialized"], s.batch.k_pools, s.batch.v_pools):
        k[:L] = k0
        v[:L] = v0
    try:
        anchors, scores = s.batch.select_anchors(anchor_count(w))
        x, m = s.batch.refresh(anchors, anchor_count(w))
        g_scores, g_anchors, gx = down(scores), anchors.cpu().numpy(), down(x)
        pos = m["row_pos"].cpu().numpy()
    finally:
        for (k0, v0), k, v in zip(common, s.batch.k_pools, s.batch.v_pools):
            k[:L] = k0
            v[:L] = v0
    sk64, sv64 = s.host["stale64"]
    dims = oracle_dims(w)
    R = rows_selective(w)
    K = anchor_count(w)
    overlaps = []
    for b in range(w.batch):
        req = oc.req(b)
        a_ref, pr = O.select_anchors(layers, dims, req, sk64, sv64, K)
        e = assert_close(g_scores[b], pr.scores, dt, f"scores request {b}")
        overlaps.append(check_anchors(g_anchors[b], pr.scores, K, e["max_abs"], f"{w.name} independent chain {b}"))
        # the refresh with the anchor set the GPU chose (the choice itself is
        # gated just above): a swapped anchor changes which keys the rows read
        ref = O.selective_refresh(layers, dims, req, g_anchors[b], sk64, sv64)
        keep = np.isin(pos[b * R:(b + 1) * R], req.nonaffix)
        assert_close(gx[b * R:(b + 1) * R][keep], ref.x[np.isin(ref.rows, req.nonaffix)], dt, f"rows request {b}")
    print(f"\n{w.name}: anchor overlap with the oracle chain {overlaps}")


def test_refresh_error_is_that_of_bf16_storage(case):
    """The GPU refresh loses no more accuracy than bf16 storage itself: exact
    arithmetic that rounds to bf16 where the GPU path stores a value
    (tests/bf16_reference.py), through every layer on the same inputs and
    anchors, has about the same error against the fp64 oracle."""
    from tests.bf16_reference import layer_forward_bf16
    w, s, layers, sk, sv, oc = case
    if w.dims.dtype != "bf16":
        pytest.skip("the bf16 storage model applies to the bf16 path")
    dims = oracle_dims(w)
    R = rows_selective(w)
    anchors = [oc.anchors(b) for b in range(w.batch)]
    x, _ = s.batch.refresh(up_i32(np.stack(anchors)), anchor_count(w))
    gx = down(x)
    S = w.layout.seq_len
    for b in range(w.batch):
        req = oc.req(b)
        ref = oc.selective(b)
        rows = ref.rows
        xe = req.x0[rows]
        for n, lw in enumerate(layers):
            vk = np.zeros((S, w.dims.n_kv_heads, w.dims.head_dim))
            vv = np.zeros_like(vk)
            vk[req.affix], vv[req.affix] = sk[n], sv[n]
            xe = layer_forward_bf16(lw, dims, xe, req.pos[rows], rows, vk, vv)
        e_gpu = errors(gx[b * R:(b + 1) * R], ref.x)
        e_emu = errors(xe, ref.x)
        print(f"[bf16 floor] {w.name} request {b}: GPU rms_rel {e_gpu['rms_rel']:.3e} elem_rel {e_gpu['elem_rel']:.3e}"
              f"  bf16 storage rms_rel {e_emu['rms_rel']:.3e} elem_rel {e_emu['elem_rel']:.3e}", flush=True)
        assert e_gpu["rms_rel"] <= 1.25 * e_emu["rms_rel"], (e_gpu, e_emu)
        assert e_gpu["max_rel"] <= 1.5 * e_emu["max_rel"] + 1e-4, (e_gpu, e_emu)
