"""Host-side logic of the stack driver (no GPU)."""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2608_26140_amd import acache as A  # noqa: E402
from paper_2608_26140_amd.driver import AffixBatch  # noqa: E402


class _Model:
    def __init__(self, dims):
        self.dims = dims


@pytest.mark.parametrize("B,R,dims", [
    (32, 8704, A.make_dims(4096, 32, 32, 128, 12288, "bf16")),   # full refresh, serving-scale stack
    (32, 2150, A.make_dims(4096, 32, 32, 128, 12288, "bf16")),   # its selective refresh
    (4, 5120, A.make_dims(3584, 28, 4, 128, 18944, "bf16")),
    (1, 1, A.make_dims(256, 4, 4, 64, 688, "f32")),
])
def test_request_groups_cover_batch_within_offset_limit(B, R, dims):
    ab = AffixBatch.__new__(AffixBatch)
    ab.model, ab.B = _Model(dims), B
    groups = ab.request_groups(R)
    assert groups[0][0] == 0 and groups[-1][1] == B
    assert all(g0[1] == g1[0] for g0, g1 in zip(groups, groups[1:]))
    widest = max(dims.d_model, dims.n_heads * dims.head_dim, dims.d_ff)
    for b0, b1 in groups:
        assert b1 > b0 and (b1 - b0) * R * widest < 2 ** 31
    # as few calls as the limit allows
    per = groups[0][1] - groups[0][0]
    assert per == B or (per + 1) * R * widest >= 2 ** 31


# ----------------------------------------------------------------------------- KV block pool (host)

def test_block_pool_against_model():
    """The library's block allocator against a set model: lowest free ids
    first, all-or-nothing allocation and frees, in-use and peak counts."""
    from paper_2608_26140_amd import acache as A
    rng = np.random.default_rng(8)
    cap = 50
    pool = A.BlockPool(cap)
    free, held, peak = set(range(cap)), [], 0
    for _ in range(400):
        if rng.random() < 0.55:
            n = int(rng.integers(0, 12))
            if n > len(free):
                with pytest.raises(A.AcacheError) as e:
                    pool.alloc(n)
                assert e.value.status == 7
                continue
            want = sorted(free)[:n]
            assert pool.alloc(n) == want
            free -= set(want)
            held += want
        elif held:
            n = int(rng.integers(1, len(held) + 1))
            pick = [held[i] for i in rng.choice(len(held), size=n, replace=False)]
            if rng.random() < 0.2:  # a bad list frees nothing
                bad = pick + [pick[0]] if rng.random() < 0.5 else pick + [cap]
                with pytest.raises(A.AcacheError):
                    pool.free(bad)
            pool.free(pick)
            for i in pick:
                held.remove(i)
            free |= set(pick)
        peak = max(peak, cap - len(free))
        st = pool.stats()
        assert st == dict(capacity=cap, in_use=cap - len(free), peak=peak)
    pool.reset_peak()
    assert pool.stats()["peak"] == cap - len(free)
    with pytest.raises(A.AcacheError):
        pool.free([next(iter(free))]) if free else pool.free([cap + 1])
    pool.close()
    with pytest.raises(A.AcacheError):
        A.BlockPool(-1)
