"""Host-side logic of the stack driver (no GPU)."""

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
