"""Builds the oracle's model, requests and stale affix cache from the same
seeded host bits the GPU setup uploaded (test infrastructure)."""

import numpy as np

from oracle import acache_oracle as O


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


def anchors_agree(got, ref, scores_ref, k, tol_rel):
    """Overlap >= 99% of K, and every anchor in the symmetric difference has
    an oracle score within tol_rel (relative to the K-th score) of the
    oracle's K-th largest score (the tie band).  Returns the overlap."""
    got, ref = set(int(v) for v in got), set(int(v) for v in ref)
    if k == 0:
        return 1.0
    overlap = len(got & ref) / k
    kth = np.sort(scores_ref)[::-1][k - 1]
    band = tol_rel * abs(kth)
    for j in got ^ ref:
        assert abs(scores_ref[j] - kth) <= band, f"anchor {j} outside the tie band ({scores_ref[j]} vs {kth})"
    return overlap


def assert_overlap(overlap, scores_ref, k, tol_rel, what=""):
    """The anchor-set overlap must reach 99%, except where the oracle's own
    K-th and (K+1)-th scores are closer than the tie band: then swapping
    them is within the scores' tolerance and anchors_agree has already
    checked that every swap lies in the band."""
    if overlap >= 0.99 or k == 0 or k >= len(scores_ref):
        return
    s = np.sort(np.asarray(scores_ref, dtype=np.float64))[::-1]
    gap = s[k - 1] - s[k]
    assert gap <= tol_rel * abs(s[k - 1]), (
        f"{what}: anchor overlap {overlap:.3f} < 0.99 with a clear boundary (K-th/K+1-th gap {gap:.3e})")
