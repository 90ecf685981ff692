"""Builds the oracle's model, requests and stale affix cache from the same
seeded host bits the GPU setup uploaded (test infrastructure)."""

import numpy as np

from oracle import acache_oracle as O


def anchor_count(w, ratio=None):
    """Eq. 6's K for the workload's anchor ratio: the library's count, which
    must equal the oracle's (each side derives it on its own)."""
    from paper_2608_26140_amd import acache as A
    r = w.ratio if ratio is None else ratio
    k = A.acache_anchor_count(r, w.layout.affix_len)
    ref = O.anchor_count(r, w.layout.affix_len)
    assert k == ref, f"{w.name}: library K {k} != oracle K {ref} at ratio {r}"
    return k


def rows_selective(w, ratio=None):
    """Recomputed rows per request: the K anchors plus every non-affix row."""
    return anchor_count(w, ratio) + w.layout.n_nonaffix


def oracle_dims(w):
    d = w.dims
    return O.Dims(d_model=d.d_model, n_heads=d.n_heads, n_kv_heads=d.n_kv_heads, head_dim=d.head_dim,
                  d_ff=d.d_ff, rms_eps=d.rms_eps, rope_base=d.rope_base)


def oracle_layers(w, host):
    dims = oracle_dims(w)
    return [O.layer_from_bits(b, dims, w.dims.dtype) for b in host["layers"]]


def layer0_inputs(w, host, b):
    """[S, d] float64 layer-0 inputs of request b."""
    if w.dims.vocab:
        return O.from_bits(host["embedding"][host["ids"][b]], w.dims.dtype)
    return O.from_bits(host["hidden"][b], w.dims.dtype)


def oracle_request(w, host, b):
    lay = w.layout
    return O.Request(x0=layer0_inputs(w, host, b), pos=np.arange(lay.seq_len),
                     affix=np.arange(lay.affix_begin, lay.affix_end),
                     masked=np.arange(lay.mask_begin, lay.mask_begin + lay.mask_len))


def oracle_stale(w, host, layers):
    dims = oracle_dims(w)
    lay = w.layout
    if w.stale == "perturb":
        donor = O.Request(x0=O.from_bits(host["donor"], w.dims.dtype), pos=np.arange(lay.affix_begin, lay.affix_end),
                          affix=np.arange(lay.affix_len), masked=np.arange(0))
    else:
        donor = O.Request(x0=O.from_bits(host["embedding"][host["donor_ids"]], w.dims.dtype),
                          pos=np.arange(lay.seq_len), affix=np.arange(lay.affix_begin, lay.affix_end),
                          masked=np.arange(0))
    return O.materialize_affix_cache(layers, dims, donor)


def check_anchors(got, scores_ref, k, score_err, what=""):
    """The anchor-set gate for Eq. 6 when the scores carry rounding.

    got: an anchor set chosen as the exact top-K of the GPU's scores;
    scores_ref: the oracle's scores; score_err: max_j |g_j - r_j| of the GPU's
    scores against them, measured by the calling test.  The oracle's set is
    the top-K of scores_ref.  An anchor can change sides only where the two
    scores' rounding reorders it with the K-th place: with every score within
    e of the oracle's, each element of the symmetric difference lies within
    2e of the oracle's K-th score.  The band is 3e.  Besides, when K >= 100
    (one swap is at most 1% of K) the sets must overlap by at least 99%;
    below that, any swap must still lie in the band.  Returns the overlap."""
    got = set(int(v) for v in got)
    ref_idx = O.topk_anchors(scores_ref, k)
    ref = set(int(v) for v in ref_idx)
    assert len(got) == k, f"{what}: {len(got)} distinct anchors, expected {k}"
    if k == 0:
        return 1.0
    overlap = len(got & ref) / k
    kth = np.sort(np.asarray(scores_ref, dtype=np.float64))[::-1][k - 1]
    band = 3.0 * float(score_err)
    for j in sorted(got ^ ref):
        assert abs(scores_ref[j] - kth) <= band, (
            f"{what}: anchor {j} changes sides outside the tie band (score {scores_ref[j]:.9g}, K-th {kth:.9g}, "
            f"band {band:.3e})")
    if k >= 100:
        assert overlap >= 0.99, f"{what}: anchor overlap {overlap:.4f} < 0.99 (K = {k})"
    print(f"[anchors] {what}: K {k} overlap {overlap:.4f} swaps {len(got - ref)} band {band:.3e}", flush=True)
    return overlap
