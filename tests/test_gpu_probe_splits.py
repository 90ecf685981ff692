"""The probe's affix log-sum-exp taken by the 256-query attention kernel
under key splits, each split's share combined by the merge kernel: four
LLaDA-shaped requests of 256 probe rows over 4352 keys (affix 4096 first),
where the launch's cost model picks that kernel with two key splits.  The
scores must match those of the probe whose score makes its own pass over
the affix keys (checked against the oracle on the other workloads), and so
must the anchors."""

import numpy as np
import pytest

import workloads as W
from tests.gpu_util import assert_close, down

pytestmark = pytest.mark.gpu


def test_probe_scores_with_split_wide_attention():
    import torch
    from paper_2608_26140_amd import acache as A
    from paper_2608_26140_amd import workload as WL
    w = W.get_config("probe-wide-split")
    print(f"\n[probe-split] {w.name}: batch {w.batch} S {w.layout.seq_len} L {w.layout.affix_len}", flush=True)
    s = WL.build(w, keep_host=False)
    torch.cuda.synchronize()
    with_lse, _, _ = s.batch.probe(A.ACACHE_NORM_AFFIX, attention_lse=True)
    own, _, _ = s.batch.probe(A.ACACHE_NORM_AFFIX, attention_lse=False)
    g, h = down(with_lse), down(own)
    assert_close(g, h, "bf16", "probe scores, attention log-sum-exp under key splits")
    # Eq. 5 under the affix-only normaliser: each layer, head and masked row adds 1
    np.testing.assert_allclose(g.sum(axis=1), w.dims.n_layers * w.dims.n_heads * w.layout.mask_len, rtol=1e-3)
    K = A.acache_anchor_count(w.ratio, w.layout.affix_len)
    a = A.acache_topk(with_lse, K).cpu().numpy()
    b = A.acache_topk(own, K).cpu().numpy()
    overlap = min(len(set(a[r]) & set(b[r])) / K for r in range(w.batch))
    print(f"[probe-split] anchor overlap {overlap:.4f}", flush=True)
    assert overlap >= 0.99
