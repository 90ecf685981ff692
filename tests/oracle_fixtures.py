"""Tiny random models and requests for the oracle pin tests (CPU only)."""

import numpy as np

from oracle import acache_oracle as O


def tiny_dims(d=32, nh=4, nkv=4, dh=8, ff=48):
    return O.Dims(d_model=d, n_heads=nh, n_kv_heads=nkv, head_dim=dh, d_ff=ff)


def tiny_layers(dims, n_layers, seed, std=0.3):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n_layers):
        d, f = dims.d_model, dims.d_ff
        hq, hk = dims.n_heads * dims.head_dim, dims.n_kv_heads * dims.head_dim
        out.append(O.Layer(
            g1=1.0 + 0.1 * rng.standard_normal(d),
            wq=std * rng.standard_normal((hq, d)),
            wk=std * rng.standard_normal((hk, d)),
            wv=std * rng.standard_normal((hk, d)),
            wo=std * rng.standard_normal((d, hq)),
            g2=1.0 + 0.1 * rng.standard_normal(d),
            wg=std * rng.standard_normal((f, d)),
            wu=std * rng.standard_normal((f, d)),
            wd=std * rng.standard_normal((d, f)),
        ))
    return out


def tiny_request(dims, seed, S=24, affix=(0, 12), masked=(18, 24), pos_offset=0):
    rng = np.random.default_rng(seed)
    x0 = rng.standard_normal((S, dims.d_model))
    return O.Request(x0=x0, pos=np.arange(S) + pos_offset,
                     affix=np.arange(*affix), masked=np.arange(*masked))


def tiny_stale(layers, dims, req, seed, noise=0.5):
    """Stale affix cache: materialised from the affix inputs plus noise."""
    rng = np.random.default_rng(seed)
    x_aff = req.x0[req.affix] + noise * rng.standard_normal((len(req.affix), dims.d_model))
    donor = O.Request(x0=x_aff, pos=np.asarray(req.pos)[req.affix],
                      affix=np.arange(len(req.affix)), masked=np.arange(0))
    return O.materialize_affix_cache(layers, dims, donor)
