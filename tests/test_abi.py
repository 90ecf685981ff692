"""The C ABI library loads and exports every entry point include/acache.h
declares; host-side validation returns the documented status codes without
touching a GPU.  CPU only."""

import ctypes
import os
import re

import pytest

from tests.conftest import ROOT

HEADER = os.path.join(ROOT, "include", "acache.h")


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(acache_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def A():
    from paper_2608_26140_amd import acache
    return acache


def test_every_declared_symbol_is_exported(A):
    names = declared_symbols()
    assert len(names) >= 12
    for n in names:
        assert hasattr(A.lib, n), f"{n} declared in acache.h but not exported"


def test_five_paper_calls_present():
    names = declared_symbols()
    for n in ("acache_score", "acache_topk", "acache_gather_rows", "acache_layer_recompute", "acache_kv_scatter"):
        assert n in names


def test_status_strings(A):
    for st in range(7):
        assert A.lib.acache_status_string(st)


def test_workspace_size_validation(A):
    good = A.make_dims(4096, 32, 32, 128, 12288, "bf16")
    assert A.acache_workspace_size(good, 717, 1, 1024) > 717 * 4096 * 2
    bad = A.make_dims(4096, 32, 32, 64, 12288, "bf16")  # bf16 needs head_dim 128
    assert A.lib.acache_workspace_size(ctypes.byref(bad), 10, 1, 0) == 0
    gqa_bad = A.make_dims(4096, 30, 4, 128, 12288, "bf16")  # 30 % 4 != 0
    assert A.lib.acache_workspace_size(ctypes.byref(gqa_bad), 10, 1, 0) == 0


def test_host_validation_enqueues_nothing(A):
    """Invalid arguments return their status before any device work (these
    calls pass NULL or bogus pointers that a launch would fault on)."""
    lib = A.lib
    # k > L
    assert lib.acache_topk(None, 1, 10, 11, None, None) == 2
    # k == 0 and batch == 0 are no-ops even with NULL pointers
    assert lib.acache_topk(None, 1, 10, 0, None, None) == 0
    assert lib.acache_topk(None, 0, 10, 3, None, None) == 0
    # NULL scores with work to do
    assert lib.acache_topk(None, 1, 10, 3, None, None) == 1
    # L beyond the LDS capacity of one workgroup
    assert lib.acache_topk(ctypes.c_void_p(16), 1, 20000, 3, ctypes.c_void_p(16), None) == 4
    # gather: row bytes not a multiple of 16
    assert lib.acache_gather_rows(ctypes.c_void_p(16), 24, 5, ctypes.c_void_p(16), None, 0, 3, 24,
                                  ctypes.c_void_p(16), 24, None) == 2
    # gather: misaligned destination
    assert lib.acache_gather_rows(ctypes.c_void_p(16), 32, 5, ctypes.c_void_p(16), None, 0, 3, 32,
                                  ctypes.c_void_p(20), 32, None) == 3
    # scatter: unsupported dtype code
    assert lib.acache_kv_scatter(None, None, 8, 1, None, None, None, 8, 1, 8, 7, None) == 4
    # maps: anchors missing when k > 0; private stride too small
    lay = A.Layout(100, 0, 60, 80, 20, 0, 60, 100)
    assert lib.acache_build_maps(ctypes.byref(lay), 1, None, 5, ctypes.c_void_p(16), ctypes.c_void_p(16),
                                 ctypes.c_void_p(16), ctypes.c_void_p(16), None, None) == 1
    lay_small = A.Layout(100, 0, 60, 80, 20, 0, 60, 30)
    assert lib.acache_build_maps(ctypes.byref(lay_small), 1, ctypes.c_void_p(16), 5, ctypes.c_void_p(16),
                                 ctypes.c_void_p(16), ctypes.c_void_p(16), ctypes.c_void_p(16), None, None) == 2
    # maps: masked span overlapping the affix
    lay_ovl = A.Layout(100, 0, 60, 50, 20, 0, 60, 100)
    assert lib.acache_build_maps(ctypes.byref(lay_ovl), 1, None, 0, ctypes.c_void_p(16), ctypes.c_void_p(16),
                                 ctypes.c_void_p(16), ctypes.c_void_p(16), None, None) == 2
    # maps: unknown key order
    lay_ord = A.Layout(100, 0, 60, 80, 20, 0, 60, 100, 2)
    assert lib.acache_build_maps(ctypes.byref(lay_ord), 1, None, 0, ctypes.c_void_p(16), ctypes.c_void_p(16),
                                 ctypes.c_void_p(16), ctypes.c_void_p(16), None, None) == 4


def test_layer_recompute_validation(A):
    lib = A.lib
    dims = A.make_dims(4096, 32, 32, 128, 12288, "bf16")
    cu_rows = (ctypes.c_int32 * 2)(0, 10)
    cu_keys = (ctypes.c_int32 * 2)(0, 0)  # rows without keys
    rg = A.Ragged(1, cu_rows, cu_keys)
    w = A.LayerWeights(16, 16, 16, 16, 16, 16)
    p = ctypes.c_void_p(16)
    assert lib.acache_layer_recompute(ctypes.byref(dims), ctypes.byref(w), ctypes.byref(rg), p, p, p, p, p, p,
                                      4096, 100, None, p, 1 << 30, None) == 2
    cu_keys2 = (ctypes.c_int32 * 2)(0, 20)
    rg2 = A.Ragged(1, cu_rows, cu_keys2)
    # workspace too small
    assert lib.acache_layer_recompute(ctypes.byref(dims), ctypes.byref(w), ctypes.byref(rg2), p, p, p, p, p, p,
                                      4096, 100, None, p, 100, None) == 5
    # bf16 d_ff not a multiple of 128
    dims_bad = A.make_dims(4096, 32, 32, 128, 12200, "bf16")
    assert lib.acache_layer_recompute(ctypes.byref(dims_bad), ctypes.byref(w), ctypes.byref(rg2), p, p, p, p, p,
                                      p, 4096, 100, None, p, 1 << 30, None) == 4
    # batch above 64
    big = A.Ragged(65, cu_rows, cu_keys2)
    assert lib.acache_layer_recompute(ctypes.byref(dims), ctypes.byref(w), ctypes.byref(big), p, p, p, p, p, p,
                                      4096, 100, None, p, 1 << 30, None) == 2


def test_layer_decode_validation(A):
    lib = A.lib
    dims = A.make_dims(4096, 32, 32, 128, 12288, "bf16")
    w = A.LayerWeights(16, 16, 16, 16, 16, 16)
    p = ctypes.c_void_p(16)

    def call(dims=dims, batch=2, rows=8, L=64, k=8, plen=20, ws_bytes=1 << 30, anchors=p, priv=p):
        return lib.acache_layer_decode(ctypes.byref(dims), ctypes.byref(w), batch, rows, p, p, p, p, L, anchors, k,
                                       priv, plen, p, p, 4096, 1000, p, ws_bytes, None)
    # fp32 is not implemented by this entry point
    assert call(dims=A.make_dims(256, 4, 4, 64, 688, "f32")) == 4
    assert call(batch=65) == 2                 # batch above 64
    assert call(k=65) == 2                     # more anchors than affix positions
    assert call(L=70000, k=8) == 2             # affix beyond 65536
    assert call(L=8, k=8, plen=0) == 2         # a request without any key
    assert call(anchors=None) == 1             # anchors needed when 0 < k < L
    assert call(priv=None) == 1                # private slots needed when private_len > 0
    assert call(ws_bytes=100) == 5             # workspace too small
    assert call(batch=0) == 0 and call(rows=0) == 0   # nothing to do


def test_layer_score_validation(A):
    """acache_layer_score rejects bad arguments before any launch."""
    lib = A.lib
    dims = A.make_dims(4096, 32, 32, 128, 12288, "bf16")
    w = A.LayerWeights(16, 16, 0, 0, 0, 0)  # only attn_norm and w_qkv are read
    p = ctypes.c_void_p(16)
    cu_rows = (ctypes.c_int32 * 3)(0, 512, 1024)
    cu_keys = (ctypes.c_int32 * 3)(0, 1536, 3072)
    rg = A.Ragged(2, cu_rows, cu_keys)

    def call(cu_q=(0, 256, 512), L=1024, norm=A.ACACHE_NORM_AFFIX, score=True, wslots=None, rslots=None, vpool=None,
             ws_bytes=1 << 40):
        cq = (ctypes.c_int32 * 3)(*cu_q)
        sa = A.ScoreArgs(16, cq, 16, L, norm, 16)
        return lib.acache_layer_score(ctypes.byref(dims), ctypes.byref(w), ctypes.byref(rg), p, p, wslots, rslots, p,
                                      vpool, 4096, 100000, ctypes.byref(sa) if score else None, p, ws_bytes, None)
    assert call(score=False) == 1                      # score is required
    assert call(norm=7) == 4                           # unknown normalisation
    assert call(cu_q=(0, 256, 1025)) == 2              # more masked rows than rows
    assert call(cu_q=(0, 300, 200)) == 2               # decreasing offsets
    assert call(L=70000) == 2                          # affix beyond 65536
    assert call(norm=A.ACACHE_NORM_FULL) == 1          # the full softmax needs the slot lists and V
    assert call(ws_bytes=100) == 5                     # workspace too small
    assert call(cu_q=(0, 0, 0)) == 0 and call(L=0) == 0  # nothing to add


def test_offset_limits(A):
    """Operands whose element offsets would not fit 32 bits are rejected
    before any launch."""
    lib = A.lib
    dims = A.make_dims(4096, 32, 32, 128, 12288, "bf16")
    p = ctypes.c_void_p(16)
    # acache_linear: M * K >= 2^31
    assert lib.acache_linear(ctypes.byref(dims), p, p, p, 1 << 20, 256, 4096, 0, None, 0, None) == 4
    # acache_layer_recompute: rows * d_ff >= 2^31 (200000 rows of a 12288-wide MLP)
    cu_rows = (ctypes.c_int32 * 2)(0, 200000)
    cu_keys = (ctypes.c_int32 * 2)(0, 200000)
    rg = A.Ragged(1, cu_rows, cu_keys)
    w = A.LayerWeights(16, 16, 16, 16, 16, 16)
    assert lib.acache_layer_recompute(ctypes.byref(dims), ctypes.byref(w), ctypes.byref(rg), p, p, p, p, p, p,
                                      4096, 100, None, p, 1 << 62, None) == 4


def test_anchor_count_matches_the_oracle(A):
    """acache_anchor_count (host arithmetic in the library) against the
    oracle's exact-rational count, over the workloads' ratios and a grid of
    ratios and affix lengths with exact halves."""
    from oracle import acache_oracle as O
    for L in (0, 1, 2, 3, 4, 7, 10, 100, 128, 200, 250, 1024, 2048, 4096, 8192, 65536):
        for r in (0.0, 0.05, 0.1, 0.125, 0.2, 0.25, 0.3, 0.375, 0.4, 0.5, 0.6, 0.75, 0.9, 0.999, 1.0):
            assert A.acache_anchor_count(r, L) == O.anchor_count(r, L), (r, L)
    assert A.lib.acache_anchor_count(-0.1, 10) == -1
    assert A.lib.acache_anchor_count(1.5, 10) == -1
    assert A.lib.acache_anchor_count(float("nan"), 10) == -1
    assert A.lib.acache_anchor_count(0.5, -1) == -1


def test_workload_anchor_counts():
    import workloads as W
    from tests.oracle_side import anchor_count
    want = {"tiny-f32": 26, "llada-layer": 205, "llada-stack-b8": 410, "dream-stack-b4": 819, "llada-serve-b32": 1638}
    for name, k in want.items():
        assert anchor_count(W.get_config(name)) == k
    dream = W.get_config("dream-stack-b4")
    assert [anchor_count(dream, r) for r in dream.ratios] == [410, 819, 1638]
