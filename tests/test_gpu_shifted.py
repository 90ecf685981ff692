"""Reuse of the shared affix cache at shifted positions (the runtime piece
Section 4 leaves open): a cache materialised with the donor context placed
delta positions earlier, then re-rotated by delta, equals the cache
materialised in place, at every layer, against the oracle's."""

import numpy as np
import pytest

import workloads as W
from tests.gpu_util import assert_close, down, up_i32
from tests.oracle_side import oracle_layers, oracle_stale

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["mini-gqa-infix", "mini-stack"])
def test_shifted_materialisation_then_rerotation(name):
    import torch
    from paper_2608_26140_amd import acache as A
    from paper_2608_26140_amd import workload as WL
    w = W.get_config(name)
    s = WL.build(w)
    lay, dt = w.layout, w.dims.dtype
    S, L = lay.seq_len, lay.affix_len
    delta = 40 if lay.affix_begin == 0 else lay.affix_begin
    # donor context placed delta positions earlier (the affix moves by -delta)
    p = np.arange(S)
    in_affix = (p >= lay.affix_begin) & (p < lay.affix_end)
    wslots = np.where(in_affix, p - lay.affix_begin, L + p).astype(np.int32)
    dx = A.acache_gather_rows(s.batch.x_src, up_i32(np.arange(S)), up_i32(s.host["donor_ids"]))
    for k, v in zip(s.batch.k_pools, s.batch.v_pools):
        k.zero_()
        v.zero_()
    s.batch.materialize_affix(dx, up_i32(p - delta), up_i32(wslots), up_i32(wslots))
    s.batch.shift_affix(delta)
    torch.cuda.synchronize()
    layers = oracle_layers(w, s.host)
    sk, sv = oracle_stale(w, s.host, layers)  # materialised at the true positions
    kv = (L, w.dims.n_kv_heads, w.dims.head_dim)
    for n in range(len(layers)):
        assert_close(down(s.batch.k_pools[n][:L]).reshape(kv), sk[n], dt, f"shifted K layer {n}")
        assert_close(down(s.batch.v_pools[n][:L]).reshape(kv), sv[n], dt, f"shifted V layer {n}")
