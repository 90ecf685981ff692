"""A decode step of the serving workload at its full launch shape: batch
32, 32 block rows per request against 8704 keys, the LLaDA-shaped layer,
with one layer (layer 0) so that the oracle can follow.  (Probe, scores,
anchors and refresh of the stacks at full depth: tests/test_gpu_depth.py.)

At layer 0 a block's K and V are row-local, so the shared affix cache of
the donor context is the oracle's ``layer_kv`` of the affix rows; both sides
use that cache (rounded to storage) as the common input.  After a refresh
with the oracle's anchors for a sampled request, the decode step of the
first block runs for the whole batch (the shared affix for all requests
together, anchors masked, then the private slots) and is checked for that
request against the oracle's step over the same view.
"""

import numpy as np
import pytest

import workloads as W
from oracle import acache_oracle as O
from tests.gpu_util import assert_close, down, up, up_i32
from tests.oracle_side import anchor_count, oracle_dims, oracle_request, rows_selective

pytestmark = pytest.mark.gpu

NAMES = ["llada-serve-b32"]


def storage_round(a: np.ndarray, dtype: str) -> np.ndarray:
    return W.bf16_bits_from_f32(a.astype(np.float32)) if dtype == "bf16" else a.astype(np.float32)


@pytest.fixture(scope="module", params=NAMES)
def case(request):
    import torch
    from paper_2608_26140_amd import workload as WL
    w = W.get_config(request.param)
    print(f"\n[full-size] {w.name}: batch {w.batch} S {w.layout.seq_len} L {w.layout.affix_len} "
          f"K {anchor_count(w)} R {rows_selective(w)}", flush=True)
    s = WL.build(w, n_layers=1, max_rows=rows_selective(w))
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


def test_decode_step_full_size(case):
    w, s, layer0, dims, sk, sv = case
    from paper_2608_26140_amd import driver as D
    dt, lay = w.dims.dtype, w.layout
    B, K, blen = w.batch, anchor_count(w), w.decode_block
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
