"""acache_score_noalloc (the library's fixed scratch instead of a caller's
workspace) against acache_score through the C ABI: identical bits, on two
calls in a row (the second smaller than the first, so it runs on what the
first left in the scratch), both normalisations and both storage types; the
result is also held to the oracle's scores.  A call past the scratch limit
is refused with nothing enqueued."""

import numpy as np
import pytest

import workloads as W
from oracle import acache_oracle as O
from tests.gpu_util import assert_close, down, up, up_i32

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def A():
    import torch
    assert torch.cuda.is_available()
    from paper_2608_26140_amd import acache
    return acache


def _case(dtype, H, Hkv, rows, nq, L, seed):
    dh = 128 if dtype == "bf16" else 64
    q = W.draw_tensor((rows, H * dh), dtype, seed=seed)
    n_slots = L + 300
    kp = W.draw_tensor((n_slots, Hkv * dh), dtype, seed=seed + 1)
    q_rows = W.draw_permutation(rows, seed=seed + 2)[:sum(nq)]
    cu_q = list(np.concatenate([[0], np.cumsum(nq)]).astype(int))
    affix_slots = W.draw_permutation(n_slots, seed=seed + 3)[:L]
    return dh, q, kp, q_rows, cu_q, affix_slots


@pytest.mark.parametrize("dtype,H,Hkv", [("bf16", 32, 32), ("bf16", 28, 4), ("f32", 4, 2)])
@pytest.mark.parametrize("norm", ["affix", "full"])
def test_noalloc_matches_workspace_call_twice(A, dtype, H, Hkv, norm):
    import torch
    code = A.ACACHE_NORM_AFFIX if norm == "affix" else A.ACACHE_NORM_FULL
    # the second call is smaller (fewer requests, rows and keys)
    for call, (rows, nq, L, seed) in enumerate([(700, [256, 200, 130], 3000, 40), (200, [57], 900, 50)]):
        dh, q, kp, q_rows, cu_q, affix_slots = _case(dtype, H, Hkv, rows, nq, L, seed)
        dims = A.make_dims(256 if dtype == "f32" else 4096, H, Hkv, dh, 512, dtype)
        qd, kd = up(q, dtype), up(kp, dtype)
        qr, asl = up_i32(q_rows), up_i32(affix_slots)
        row_lse, lse_np = None, None
        if norm == "full":
            qf = O.from_bits(q, dtype).reshape(rows, H, dh)
            kf = O.from_bits(kp, dtype).reshape(-1, Hkv, dh)
            lse_np = np.empty((rows, H))
            for h in range(H):
                lg = qf[:, h] @ kf[affix_slots, h // (H // Hkv)].T / np.sqrt(dh)
                lse_np[:, h] = np.log(np.exp(lg - lg.max(1, keepdims=True)).sum(1)) + lg.max(1) + 0.25
            row_lse = torch.from_numpy(lse_np.astype(np.float32)).cuda()
            lse_np = lse_np.astype(np.float32).astype(np.float64)
        ref = torch.full((len(nq), L), 0.5, dtype=torch.float32, device="cuda")
        got = ref.clone()
        A.acache_score(dims, qd, qr, cu_q, kd, asl, ref, norm=code, row_lse=row_lse)
        A.acache_score_noalloc(dims, qd, qr, cu_q, kd, asl, got, norm=code, row_lse=row_lse)
        torch.cuda.synchronize()
        print(f"call {call}: {dtype} H {H}/{Hkv} rows {rows} requests {len(nq)} L {L} {norm}", flush=True)
        assert torch.equal(got, ref), f"call {call}: noalloc scores differ from the workspace call"
        oracle = O.scores_via_slots(O.from_bits(q, dtype).reshape(rows, H, dh), q_rows, cu_q,
                                    O.from_bits(kp, dtype).reshape(-1, Hkv, dh), affix_slots, norm, lse_np)
        assert_close(down(got) - 0.5, oracle, dtype, f"call {call} scores against the oracle")


def test_noalloc_refuses_beyond_its_scratch(A):
    import torch
    limit = A.lib.acache_score_noalloc_max_bytes()
    assert limit == 64 << 20
    # 64 requests x 32 heads x 8200 keys x 4 B = 67 MB of column sums > 64 MiB
    B, H, L = 64, 32, 8200
    dims = A.make_dims(4096, H, H, 128, 512, "bf16")
    q = torch.zeros((B, H * 128), dtype=torch.bfloat16, device="cuda")
    kp = torch.zeros((L, H * 128), dtype=torch.bfloat16, device="cuda")
    scores = torch.zeros((B, L), dtype=torch.float32, device="cuda")
    with pytest.raises(A.AcacheError) as e:
        A.acache_score_noalloc(dims, q, torch.arange(B, dtype=torch.int32, device="cuda"), list(range(B + 1)), kp,
                               torch.arange(L, dtype=torch.int32, device="cuda"), scores)
    assert e.value.status == 5  # ACACHE_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert not scores.any()
