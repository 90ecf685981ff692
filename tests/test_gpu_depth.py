"""Full-depth parity of the stack workloads at their real shapes, teacher
forced layer by layer.

The GPU materialises the shared affix cache (a full forward of the donor
context), probes the whole batch through every layer with scoring, takes
the top-K, and refreshes the whole batch through every layer with its own
anchors; the Dream-shaped stack does so at anchor ratios 0.1, 0.2 and 0.4.
A layer hook copies one sampled request's rows at the input of every layer.
The oracle then takes the GPU's bf16 input of a layer and its view of the
shared cache, runs that one layer in fp64 and compares (the stacks'
per-layer check; free-running drift over 28-32 layers is not a property of
one layer's arithmetic):

* every layer's Eq. 5 contribution (the score buffer's change across the
  layer) against the oracle's masked-to-affix mass of that layer's queries,
  then the sum over all N layers (Eq. 5) and the Eq. 6 anchor set;
* at layers 0, N/2 and N-2 of the probe (its last layer stops at the score),
  and 0, N/2 and N-1 of each refresh: the layer's output rows and the fresh
  K/V it wrote to the request's private slots.
"""

import numpy as np
import pytest

import workloads as W
from oracle import acache_oracle as O
from tests.gpu_util import assert_close, down_bits
from tests.oracle_side import anchor_count, check_anchors, oracle_dims, rows_selective

pytestmark = pytest.mark.gpu

NAMES = ["llada-stack-b8", "dream-stack-b4", "llada-serve-b32"]


def f64(bits, dt):
    return O.from_bits(bits, dt)


@pytest.fixture(scope="module", params=NAMES)
def run(request):
    import torch
    from paper_2608_26140_amd import acache as A
    from paper_2608_26140_amd import workload as WL
    w = W.get_config(request.param)
    ratios = w.ratios or (w.ratio,)
    d, lay, dt = w.dims, w.layout, w.dims.dtype
    N, B, S, L, P = d.n_layers, w.batch, lay.seq_len, lay.affix_len, lay.n_nonaffix
    print(f"\n[depth] {w.name}: {N} layers, batch {B}, S {S}, L {L}, ratios {ratios}", flush=True)
    s = WL.build(w, keep_host=False, max_rows=max(rows_selective(w, r) for r in ratios))
    batch = s.batch
    b = B - 1
    probe_keep = {0, 1, N // 2, N // 2 + 1, N - 2, N - 1}
    refresh_keep = {0, 1, N // 2, N // 2 + 1, N - 1, N}

    # probe: request b's masked rows at every layer input, all its rows at the
    # kept ones, and the score buffer at every layer input
    nonaffix = np.array(lay.nonaffix_positions())
    masked_local = torch.from_numpy(b * P + np.searchsorted(nonaffix, np.array(lay.masked_positions()))).cuda()
    px, pm, psc = {}, {}, {}

    def probe_hook(n, x, scores):
        if n < N:
            pm[n] = x[masked_local].clone()
        if n in probe_keep:
            px[n] = x[b * P:(b + 1) * P].clone()
        if n > 0:
            psc[n] = scores[b].clone()

    scores, _, m_probe = batch.probe(layer_hook=probe_hook, outputs=False)
    torch.cuda.synchronize()
    wslots = m_probe["write_slots"][b * P:(b + 1) * P].long()
    probe_kv = {n: (down_bits(batch.k_pools[n][wslots]), down_bits(batch.v_pools[n][wslots]))
                for n in probe_keep if n < N - 1}
    out = dict(w=w, b=b, ratios=ratios, scores=scores.cpu().numpy()[b].astype(np.float64),
               px={n: down_bits(t) for n, t in px.items()}, pm={n: down_bits(t) for n, t in pm.items()},
               psc={n: t.cpu().numpy().astype(np.float64) for n, t in psc.items()},
               probe_kv=probe_kv, refresh={})
    out["psc"][N] = out["scores"]

    for r in ratios:
        K = anchor_count(w, r)
        R = K + P
        anchors = A.acache_topk(scores, K)
        rx = {}

        def refresh_hook(n, x):
            if n in refresh_keep:
                rx[n] = x[b * R:(b + 1) * R].clone()

        _, m = batch.refresh(anchors, K, layer_hook=refresh_hook)
        torch.cuda.synchronize()
        ws = m["write_slots"][b * R:(b + 1) * R].long()
        out["refresh"][r] = dict(
            K=K, anchors=anchors.cpu().numpy()[b], rows=m["row_pos"][b * R:(b + 1) * R].cpu().numpy().astype(np.int64),
            x={n: down_bits(t) for n, t in rx.items()},
            kv={n: (down_bits(batch.k_pools[n][ws]), down_bits(batch.v_pools[n][ws])) for n in refresh_keep if n < N})
    # the shared affix cache every view reads (affix-local order): K of every
    # layer (scores), V of the layers checked in full
    aslots = batch.affix_slots.long()
    out["stale"] = {n: (down_bits(batch.k_pools[n][aslots]),
                        down_bits(batch.v_pools[n][aslots]) if n in probe_keep | refresh_keep else None)
                    for n in range(N)}
    del s, batch
    torch.cuda.empty_cache()
    out["layers"] = {}
    return out


def _layer(run, n):
    if n not in run["layers"]:
        w = run["w"]
        run["layers"][n] = O.layer_from_bits(W.draw_layer_weights(w, n), oracle_dims(w), w.dims.dtype)
    return run["layers"][n]


def _view(run, n):
    w = run["w"]
    lay, d, dt = w.layout, w.dims, w.dims.dtype
    vk = np.full((lay.seq_len, d.n_kv_heads, d.head_dim), np.nan)
    vv = np.full_like(vk, np.nan)
    aff = np.arange(lay.affix_begin, lay.affix_end)
    sk, sv = run["stale"][n]
    vk[aff] = f64(sk, dt).reshape(len(aff), d.n_kv_heads, d.head_dim)
    vv[aff] = f64(sv, dt).reshape(len(aff), d.n_kv_heads, d.head_dim)
    return vk, vv


def test_probe_scores_every_layer_and_anchors(run):
    """Eq. 5 layer by layer, each from the GPU's input to that layer; the sum
    over all N layers against the GPU's accumulated scores; the Eq. 6 anchor
    set of every ratio against the top-K of that sum."""
    w = run["w"]
    d, lay, dt = w.dims, w.layout, w.dims.dtype
    N = d.n_layers
    dims = oracle_dims(w)
    hq = d.n_heads * d.head_dim
    g1 = f64(W.layer_norm_gains(w), dt)
    masked = np.array(lay.masked_positions())
    total = np.zeros(lay.affix_len)
    for n in range(N):
        sk, _ = run["stale"][n]
        k_aff = f64(sk, dt).reshape(lay.affix_len, d.n_kv_heads, d.head_dim)
        lw = O.Layer(g1=g1, wq=f64(W.draw_layer_qkv(w, n)[:hq], dt), wk=None, wv=None, wo=None, g2=None,
                     wg=None, wu=None, wd=None)
        q = O.layer_queries(lw, dims, f64(run["pm"][n], dt), masked)
        ref = O.affix_attention_mass(q, k_aff, "affix")
        got = run["psc"][n + 1] - (run["psc"][n] if n > 0 else 0.0)
        assert_close(got, ref, dt, f"{w.name} probe layer {n} Eq. 5 contribution")
        # a layer's contribution is H * G units of probability mass
        np.testing.assert_allclose(got.sum(), d.n_heads * lay.mask_len, rtol=2e-3)
        total += ref
    e = assert_close(run["scores"], total, dt, f"{w.name} Eq. 5 over {N} layers")
    for r in run["ratios"]:
        rr = run["refresh"][r]
        np.testing.assert_array_equal(rr["anchors"], O.topk_anchors(run["scores"], rr["K"]))
        check_anchors(rr["anchors"], total, rr["K"], e["max_abs"], f"{w.name} ratio {r} anchors")


def test_probe_layers(run):
    """Probe layers 0, N/2 and N-2: output rows and fresh K/V of the request's
    non-affix rows; plus each sampled layer's score contribution."""
    w = run["w"]
    d, lay, dt = w.dims, w.layout, w.dims.dtype
    N = d.n_layers
    dims = oracle_dims(w)
    nonaffix = np.array(lay.nonaffix_positions())
    masked_local = np.searchsorted(nonaffix, np.array(lay.masked_positions()))
    for n in sorted({0, N // 2, N - 2}):
        lw = _layer(run, n)
        vk, vv = _view(run, n)
        x_in = f64(run["px"][n], dt)
        x_out, q, _ = O.layer_forward(lw, dims, x_in, nonaffix, nonaffix, vk, vv)
        assert_close(f64(run["px"][n + 1], dt), x_out, dt, f"{w.name} probe layer {n} rows")
        gk, gv = run["probe_kv"][n]
        kv = (len(nonaffix), d.n_kv_heads, d.head_dim)
        assert_close(f64(gk, dt).reshape(kv), vk[nonaffix], dt, f"{w.name} probe layer {n} fresh K")
        assert_close(f64(gv, dt).reshape(kv), vv[nonaffix], dt, f"{w.name} probe layer {n} fresh V")
        ref = O.affix_attention_mass(q[masked_local], vk[np.arange(lay.affix_begin, lay.affix_end)], "affix")
        got = run["psc"][n + 1] - (run["psc"][n] if n > 0 else 0.0)
        assert_close(got, ref, dt, f"{w.name} probe layer {n} Eq. 5 contribution (full layer)")


@pytest.mark.parametrize("ri", [0, 1, 2])
def test_refresh_layers(run, ri):
    """Selective refresh with the GPU's anchors, layers 0, N/2 and N-1: output
    rows and the fresh K/V of the anchors and request rows."""
    w = run["w"]
    if ri >= len(run["ratios"]):
        pytest.skip(f"{w.name} runs one anchor ratio")
    r = run["ratios"][ri]
    rr = run["refresh"][r]
    d, lay, dt = w.dims, w.layout, w.dims.dtype
    N = d.n_layers
    dims = oracle_dims(w)
    rows = rr["rows"]
    aff = np.arange(lay.affix_begin, lay.affix_end)
    np.testing.assert_array_equal(rows, np.sort(np.concatenate([aff[rr["anchors"]], lay.nonaffix_positions()])))
    for n in sorted({0, N // 2, N - 1}):
        lw = _layer(run, n)
        vk, vv = _view(run, n)
        x_out, _, _ = O.layer_forward(lw, dims, f64(rr["x"][n], dt), rows, rows, vk, vv)
        assert_close(f64(rr["x"][n + 1], dt), x_out, dt, f"{w.name} ratio {r} refresh layer {n} rows")
        gk, gv = rr["kv"][n]
        kv = (len(rows), d.n_kv_heads, d.head_dim)
        assert_close(f64(gk, dt).reshape(kv), vk[rows], dt, f"{w.name} ratio {r} refresh layer {n} fresh K")
        assert_close(f64(gv, dt).reshape(kv), vv[rows], dt, f"{w.name} ratio {r} refresh layer {n} fresh V")
        assert not np.isnan(x_out).any()  # no NaN of the view reached the rows: every key they read exists
