"""The stack workloads at their full launch shapes: the batch, rows per
request, keys, affix length and model widths of the benchmarked
configurations, with one layer (layer 0) so that the oracle can follow.

At layer 0 a block's K and V are row-local, so the shared affix cache of
the donor context is the oracle's ``layer_kv`` of the affix rows; both sides
use that cache (rounded to storage) as the common input.  For a sampled
request the oracle then checks, against the GPU run over the whole batch:
the probe's Eq. 4-5 scores, the Eq. 6 anchor set (overlap and tie band), and
the selective refresh (output rows and the fresh K/V in the request's
private slots) with the oracle's anchors.  The serving workload also runs a
decode step of its first block for the whole batch (the shared affix for all
requests together, anchors masked, then the private slots), checked for a
sampled request against the oracle's step over the same view.
"""

import numpy as np
import pytest

import workloads as W
from oracle import acache_oracle as O
from tests.gpu_util import assert_close, down, up, up_i32
from tests.oracle_side import anchors_agree, assert_overlap, oracle_dims, oracle_request

pytestmark = pytest.mark.gpu

NAMES = ["llada-stack-b8", "dream-stack-b4", "llada-serve-b32"]


def storage_round(a: np.ndarray, dtype: str) -> np.ndarray:
    return W.bf16_bits_from_f32(a.astype(np.float32)) if dtype == "bf16" else a.astype(np.float32)


@pytest.fixture(scope="module", params=NAMES)
def case(request):
    import torch
    from paper_2608_26140_amd import workload as WL
    w = W.get_config(request.param)
    print(f"\n[full-size] {w.name}: batch {w.batch} S {w.layout.seq_len} L {w.layout.affix_len} "
          f"K {w.n_anchors} R {w.rows_selective}", flush=True)
    s = WL.build(w, n_layers=1, max_rows=w.rows_selective)
    torch.cuda.synchronize()
    dt, lay = w.dims.dtype, w.layout
    L = lay.affix_len
    dims = oracle_dims(w)
    layer0 = O.layer_from_bits(s.host["layers"][0], dims, dt)
    affix = np.arange(lay.affix_begin, lay.affix_end)
    donor_x = O.from_bits(s.host["embedding"][s.host["donor_ids"][affix]], dt)
    sk64, sv64 = O.layer_kv(layer0, dims, donor_x, affix)
    kb, vb = storage_round(sk64, dt), storage_round(sv64, dt)
    s.batch.k_pools[0][:L] = up(kb.reshape(L, -1), dt)
    s.batch.v_pools[0][:L] = up(vb.reshape(L, -1), dt)
    torch.cuda.synchronize()
    sk, sv = [O.from_bits(kb, dt)], [O.from_bits(vb, dt)]
    return w, s, layer0, dims, sk, sv


def test_layer0_full_size(case):
    w, s, layer0, dims, sk, sv = case
    dt = w.dims.dtype
    B, K, R = w.batch, w.n_anchors, w.rows_selective
    b = B - 1
    req = oracle_request(w, s.host, b)

    anchors, scores = s.batch.select_anchors(K)
    probe = O.probe([layer0], dims, req, sk, sv)
    assert_close(down(scores)[b], probe.scores, "f32" if dt == "f32" else "bf16", f"scores request {b}")
    ref_anchors = O.topk_anchors(probe.scores, K)
    overlap = anchors_agree(down(anchors)[b], ref_anchors, probe.scores, K, 2e-2)
    assert_overlap(overlap, probe.scores, K, 2e-2, f"request {b}")

    a = down(anchors).astype(np.int32)
    a[b] = ref_anchors
    x, m = s.batch.refresh(up_i32(a), K)
    ref = O.selective_refresh([layer0], dims, req, ref_anchors, sk, sv)
    # slice on the device: the whole batch's rows and pools are gigabytes in fp64
    assert_close(down(x[b * R:(b + 1) * R]), ref.x, dt, f"refresh rows request {b}")
    wslots = m["write_slots"][b * R:(b + 1) * R].long()
    kv = w.dims.n_kv_heads, w.dims.head_dim
    assert_close(down(s.batch.k_pools[0][wslots]).reshape(R, *kv), ref.views_k[0][ref.rows], dt, "fresh K")
    assert_close(down(s.batch.v_pools[0][wslots]).reshape(R, *kv), ref.views_v[0][ref.rows], dt, "fresh V")


def test_decode_step_full_size(case):
    w, s, layer0, dims, sk, sv = case
    if not w.decode_block:
        pytest.skip("no decode schedule for this workload")
    from paper_2608_26140_amd import driver as D
    dt, lay = w.dims.dtype, w.layout
    B, K, blen = w.batch, w.n_anchors, w.decode_block
    b = B // 2
    req = oracle_request(w, s.host, b)
    ref_anchors = O.topk_anchors(O.probe([layer0], dims, req, sk, sv).scores, K)
    anchors, _ = s.batch.select_anchors(K)
    a = down(anchors).astype(np.int32)
    a[b] = ref_anchors
    a_dev = up_i32(a)
    x, m = s.batch.refresh(a_dev, K)
    plan = D.DecodePlan(s.batch, K, blen, lay.mask_len // blen, full=False)
    h = D.decode_step(s.batch, plan, 0, m, a_dev)
    # the oracle's view after the refresh, layer 0: K/V are row-local there, so
    # the recomputed rows' entries are layer_kv of their inputs and the other
    # affix positions keep the shared cache
    rows = O.selective_rows(req, ref_anchors)
    vk = np.empty((lay.seq_len, w.dims.n_kv_heads, w.dims.head_dim))
    vv = np.empty_like(vk)
    vk[req.affix], vv[req.affix] = sk[0], sv[0]
    vk[rows], vv[rows] = O.layer_kv(layer0, dims, req.x0[rows], req.pos[rows])
    positions = np.arange(lay.mask_begin, lay.mask_begin + blen)
    xb = O.decode_step([layer0], dims, [vk], [vv], req.x0[positions], positions)
    assert_close(down(h[b * blen:(b + 1) * blen]), xb, dt, f"decode step rows request {b}")
