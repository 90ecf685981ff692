"""bench.py's algorithmic work model (host arithmetic, no GPU): the linear
layers' FLOPs per row and the probe's scoring sweeps.  The score counts one
sweep over the affix keys per layer for the column sums, and one more for
the log-sum-exp in every layer whose attention does not hand it over: with
the probe reading the affix keys first in whole 64-key tiles, only the last
probe layer (which runs no attention) makes that sweep on bf16."""

import bench
import workloads as W


def _probe(name):
    w = W.get_config(name)
    out, rows = bench.flops_model(w, 0)  # the anchor count sizes only the refresh rows
    return w, out, rows


def _sweep(w):
    d, lay = w.dims, w.layout
    return 2 * lay.mask_len * lay.affix_len * d.n_heads * d.head_dim * w.batch


def test_score_sweeps_whole_tile_affix():
    # prefix (C5) and infix (C4) affixes of whole 64-key tiles: N + 1 sweeps
    for name in ("llada-serve-b32", "dream-stack-b4", "mini-affix64", "mini-infix64"):
        w, out, _ = _probe(name)
        assert w.layout.affix_len % 64 == 0
        assert out["probe"]["score_colsum"] == _sweep(w) * (w.dims.n_layers + 1), name


def test_score_sweeps_ragged_affix_and_f32():
    # an affix of 250 keys: both sweeps in every layer
    w, out, _ = _probe("mini-stack")
    assert out["probe"]["score_colsum"] == _sweep(w) * 2 * w.dims.n_layers
    # the fp32 path: one kernel per sweep, each in every layer
    w, out, _ = _probe("tiny-f32")
    assert out["probe"]["score_lse"] == out["probe"]["score_colsum"] == _sweep(w) * w.dims.n_layers


def test_linear_flops_per_row():
    w, out, rows = _probe("llada-layer")
    d = w.dims
    hq, hkv = d.n_heads * d.head_dim, d.n_kv_heads * d.head_dim
    n = d.n_layers
    assert out["full"]["gemm_gate_up"] == 2 * d.d_model * 2 * d.d_ff * rows["full"] * n
    assert out["full"]["gemm_qkv"] == 2 * d.d_model * (hq + 2 * hkv) * rows["full"] * n
    assert out["full"]["attention"] == 4 * w.layout.seq_len * hq * rows["full"] * n
