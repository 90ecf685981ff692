"""GPU parity of each kernel against the fp64 oracle, through the C ABI.

Sizes span several tiles with ragged tails; every case is seeded."""

import numpy as np
import pytest

import workloads as W
from oracle import acache_oracle as O
from tests.gpu_util import TOL, assert_close, down, down_bits, up, up_i32

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def A():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2608_26140_amd import acache
    return acache


def _torch():
    import torch
    return torch


# ----------------------------------------------------------------------------- top-K (Eq. 6)

@pytest.mark.parametrize("kind", ["normal", "ties", "signed_zero", "special", "equal"])
@pytest.mark.parametrize("B,L,k", [(1, 128, 26), (3, 1024, 205), (2, 8192, 1638), (1, 1, 1), (2, 300, 300),
                                   (1, 16384, 1), (4, 2048, 2047)])
def test_topk_bit_exact(A, kind, B, L, k):
    s = W.draw_scores(B, L, seed=L + k, kind=kind)
    out = A.acache_topk(up(s, "f32"), k)
    got = out.cpu().numpy()
    for b in range(B):
        ref = O.topk_anchors(s[b].astype(np.float64), k)
        np.testing.assert_array_equal(got[b], ref, err_msg=f"request {b}")


def test_topk_k_zero_is_noop(A):
    torch = _torch()
    s = up(W.draw_scores(1, 64, 0), "f32")
    out = torch.full((1, 0), 7, dtype=torch.int32, device="cuda")
    A.acache_topk(s, 0, out)


# ----------------------------------------------------------------------------- gather / scatter

@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_gather_rows_with_remap(A, dtype):
    src = W.draw_tensor((500, 384), dtype, seed=1)
    idx = W.draw_ints(777, 0, 300, seed=2)
    remap = W.draw_ints(300, 0, 500, seed=3)
    g = A.acache_gather_rows(up(src, dtype), up_i32(idx))
    np.testing.assert_array_equal(down_bits(g), src[idx])
    g2 = A.acache_gather_rows(up(src, dtype), up_i32(idx), up_i32(remap))
    np.testing.assert_array_equal(down_bits(g2), src[remap[idx]])


def test_gather_out_of_range_reads_zero(A):
    src = W.draw_tensor((10, 64), "f32", seed=4)
    idx = np.array([0, 9, 10, -1, 3], dtype=np.int32)
    g = down_bits(A.acache_gather_rows(up(src, "f32"), up_i32(idx)))
    np.testing.assert_array_equal(g[[0, 1, 4]], src[[0, 9, 3]])
    assert np.all(g[[2, 3]] == 0)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_kv_scatter(A, dtype):
    torch = _torch()
    n_slots, row = 900, 4 * 128
    kp0 = W.draw_tensor((n_slots, row), dtype, seed=5)
    vp0 = W.draw_tensor((n_slots, row), dtype, seed=6)
    ks = W.draw_tensor((300, row), dtype, seed=7)
    vs = W.draw_tensor((300, row), dtype, seed=8)
    slots = W.draw_permutation(n_slots, seed=9)[:300]
    slots[5] = n_slots + 3  # out of range: dropped
    kp, vp = up(kp0, dtype), up(vp0, dtype)
    A.acache_kv_scatter(up(ks, dtype), up(vs, dtype), up_i32(slots), kp, vp)
    ek, ev = kp0.copy(), vp0.copy()
    ok = slots < n_slots
    ek[slots[ok]] = ks[ok]
    ev[slots[ok]] = vs[ok]
    np.testing.assert_array_equal(down_bits(kp), ek)
    np.testing.assert_array_equal(down_bits(vp), ev)


# ----------------------------------------------------------------------------- maps (Section 4.1)

def affix_first(read_slots, B, S, ab, L):
    """Read slots in logical order -> the affix keys first (key_order 1)."""
    order = np.concatenate([np.arange(ab, ab + L), np.arange(ab), np.arange(ab + L, S)])
    return np.asarray(read_slots).reshape(B, S)[:, order].reshape(-1)


@pytest.mark.parametrize("layout,B,k", [((1536, 0, 1024, 1280, 256), 1, 205), ((192, 0, 128, 160, 32), 1, 26),
                                        ((5120, 512, 4096, 4864, 256), 4, 819), ((2432, 0, 2048, 2176, 256), 8, 0),
                                        ((2432, 0, 2048, 2176, 256), 3, 2048)])
@pytest.mark.parametrize("key_order", [0, 1])
def test_build_maps(A, layout, B, k, key_order):
    S, ab, L, mb, G = layout
    anchors = np.stack([np.sort(W.draw_permutation(L, seed=b)[:k]) for b in range(B)]).astype(np.int32)
    R = k + S - L
    lay = A.Layout(S, ab, L, mb, G, 0, L, S, key_order)
    got = A.acache_build_maps(lay, B, up_i32(anchors) if k else None, k)
    ref = list(O.build_maps(S, ab, L, mb, G, anchors, 0, L, S))
    if key_order:
        ref[3] = affix_first(ref[3], B, S, ab, L)
    for name, r in zip(["row_pos", "row_src", "write_slots", "read_slots", "q_rows"], ref):
        np.testing.assert_array_equal(got[name].cpu().numpy(), r, err_msg=name)
    assert got["row_pos"].numel() == B * R


@pytest.mark.parametrize("layout,B,k,bs", [((192, 0, 128, 160, 32), 3, 26, 16), ((5120, 512, 4096, 4864, 256), 4, 819, 256),
                                           ((2432, 0, 2048, 2176, 256), 2, 0, 100), ((300, 40, 200, 260, 40), 2, 200, 1)])
@pytest.mark.parametrize("key_order", [0, 1])
def test_build_maps_paged(A, layout, B, k, bs, key_order):
    S, ab, L, mb, G = layout
    anchors = np.stack([np.sort(W.draw_permutation(L, seed=b)[:k]) for b in range(B)]).astype(np.int32)
    R = k + S - L
    n_sh, nb = -(-L // bs), -(-R // bs) + 1          # one spare block per request
    ids = W.draw_permutation(n_sh + B * nb, seed=30 + bs)
    shared, private = ids[:n_sh], ids[n_sh:]
    lay = A.Layout(S, ab, L, mb, G, 0, 0, 0, key_order)
    got = A.acache_build_maps_paged(lay, B, up_i32(anchors) if k else None, k, bs, up_i32(shared), up_i32(private), nb)
    ref = list(O.build_maps_paged(S, ab, L, mb, G, anchors, bs, shared, private, nb))
    if key_order:
        ref[3] = affix_first(ref[3], B, S, ab, L)
    for name, r in zip(["row_pos", "row_src", "write_slots", "read_slots", "q_rows"], ref):
        np.testing.assert_array_equal(got[name].cpu().numpy(), r, err_msg=name)


# ----------------------------------------------------------------------------- RMSNorm, linear

@pytest.mark.parametrize("dtype,d", [("bf16", 4096), ("f32", 256), ("bf16", 3584)])
def test_rmsnorm(A, dtype, d):
    x = W.draw_tensor((77, d), dtype, seed=10)
    g = W.draw_tensor((d,), dtype, std=0.5, seed=11)
    dims = A.make_dims(d, 32, 32, 128, 128, dtype)
    y = A.acache_rmsnorm(dims, up(x, dtype), up(g, dtype))
    ref = O.rms_norm(O.from_bits(x, dtype), O.from_bits(g, dtype), 1e-5)
    assert_close(down(y), ref, dtype, "rmsnorm")


# Shapes and the schedule they take with a workspace on 256 CUs with
# 256 x 256 tiles (T tiles, nk K steps of 64): (256, 3072, 4096) T = 12,
# stream-K only; (520, 24576, 2048) T = 288, one data-parallel round +
# stream-K over 32 tiles; (512, 32768, 256) T = 256, data-parallel;
# (300, 4096, 128) nk = 2, too short for stream-K; (1280, 16384, 64) T = 320
# and (2304, 8192, 128) T = 288, two data-parallel rounds of one or two K
# steps, the second partial, on 256 persistent workgroups, so a workgroup's
# second tile starts right behind its first tile's stores (so does
# (520, 24576, 2048) without a workspace); the rest run data-parallel by the
# cost model.
@pytest.mark.parametrize("schedule", ["dp", "sk"])
@pytest.mark.parametrize("M,N,K", [(1, 256, 64), (77, 512, 256), (128, 256, 4096), (717, 768, 1024), (300, 4096, 128),
                                   (256, 3072, 4096), (520, 24576, 2048), (512, 32768, 256), (1280, 16384, 64),
                                   (2304, 8192, 128)])
def test_linear_bf16(A, M, N, K, schedule):
    a = W.draw_tensor((M, K), "bf16", seed=M)
    w = W.draw_tensor((N, K), "bf16", std=0.05, seed=N + K)
    dims = A.make_dims(256, 2, 2, 128, 128, "bf16")
    ws = A.workspace(dims, M, 1, 0) if schedule == "sk" else None
    c = A.acache_linear(dims, up(a, "bf16"), up(w, "bf16"), ws=ws)
    ref = O.from_bits(a, "bf16") @ O.from_bits(w, "bf16").T
    assert_close(down(c), ref, "bf16", "linear")
    c2 = A.acache_linear(dims, up(a, "bf16"), up(w, "bf16"), out=c.clone(), accumulate=True, ws=ws)
    assert_close(down(c2), 2 * ref, "bf16", "linear accumulate")
    if schedule == "sk":
        # the pieces are summed in a fixed order: repeat calls agree bit for bit,
        # and the data-parallel schedule differs by fp32 summation order only
        again = A.acache_linear(dims, up(a, "bf16"), up(w, "bf16"), ws=ws)
        assert _torch().equal(again, c)
        dp = down(A.acache_linear(dims, up(a, "bf16"), up(w, "bf16")))
        sk = down(c)
        # one bf16 ulp, plus fp32 reordering error on outputs near zero
        bound = 2.0 ** -7 * np.maximum(np.abs(dp), np.abs(sk)) + 1e-6 * np.abs(ref).max()
        assert np.all(np.abs(sk - dp) <= bound)


@pytest.mark.parametrize("M,N,K", [(90, 688, 256), (1, 5, 3), (65, 130, 77)])
def test_linear_f32(A, M, N, K):
    a = W.draw_tensor((M, K), "f32", seed=M)
    w = W.draw_tensor((N, K), "f32", std=0.05, seed=N + K)
    dims = A.make_dims(256, 4, 4, 64, 688, "f32")
    c = A.acache_linear(dims, up(a, "f32"), up(w, "f32"))
    ref = O.from_bits(a, "f32") @ O.from_bits(w, "f32").T
    assert_close(down(c), ref, "f32", "linear")


# ----------------------------------------------------------------------------- attention (Appendix C.1)

def _attn_case(dtype, H, Hkv, dh, rows, keys, seed):
    n_slots = sum(keys) + 37
    q = W.draw_tensor((sum(rows), H * dh), dtype, std=1.0, seed=seed)
    kp = W.draw_tensor((n_slots, Hkv * dh), dtype, std=1.0, seed=seed + 1)
    vp = W.draw_tensor((n_slots, Hkv * dh), dtype, std=1.0, seed=seed + 2)
    slots = W.draw_permutation(n_slots, seed=seed + 3)[:sum(keys)]
    cu_rows = np.concatenate([[0], np.cumsum(rows)]).astype(int).tolist()
    cu_keys = np.concatenate([[0], np.cumsum(keys)]).astype(int).tolist()
    return q, kp, vp, slots, cu_rows, cu_keys, n_slots


@pytest.mark.parametrize("dtype,H,Hkv,dh,rows,keys", [
    ("bf16", 4, 4, 128, [717], [1536]),
    ("bf16", 8, 2, 128, [65, 1, 130], [200, 64, 1]),
    ("bf16", 7, 1, 128, [33, 100], [5000, 333]),
    ("f32", 4, 4, 64, [90], [192]),
    ("f32", 4, 2, 64, [3, 70], [1, 100]),
])
def test_attention(A, dtype, H, Hkv, dh, rows, keys):
    torch = _torch()
    q, kp, vp, slots, cu_rows, cu_keys, n_slots = _attn_case(dtype, H, Hkv, dh, rows, keys, seed=sum(rows))
    dims = A.make_dims(256, H, Hkv, dh, 128, dtype)
    lse = torch.empty((sum(rows), H), dtype=torch.float32, device="cuda")
    out = A.acache_attention(dims, cu_rows, cu_keys, up(q, dtype), up_i32(slots), up(kp, dtype), up(vp, dtype),
                             lse=lse)
    f = lambda a: O.from_bits(a, dtype)
    o_ref, lse_ref = O.attention_via_slots(f(q).reshape(-1, H, dh), f(kp).reshape(-1, Hkv, dh),
                                           f(vp).reshape(-1, Hkv, dh), slots, cu_rows, cu_keys)
    assert_close(down(out), o_ref.reshape(sum(rows), H * dh), dtype, "attention out")
    assert_close(down(lse), lse_ref, dtype, "attention lse")


@pytest.mark.parametrize("H,Hkv,rows,keys", [
    (32, 32, [1000, 700, 300], [900, 650, 130]),   # grids that pick the wide-tile kernel
    (28, 4, [2304, 2560], [1300, 77]),
])
def test_attention_wide_tiles_and_absent_slots(A, H, Hkv, rows, keys):
    """Launch shapes whose grid fills whole rounds of CUs (the launcher's
    wide-tile kernel), ragged rows and keys, and some out-of-range slots:
    those keys read zeros (logit 0, value 0)."""
    torch = _torch()
    dtype, dh = "bf16", 128
    q, kp, vp, slots, cu_rows, cu_keys, n_slots = _attn_case(dtype, H, Hkv, dh, rows, keys, seed=sum(rows) + H)
    bad = W.draw_permutation(len(slots), seed=7)[:9]
    slots = slots.copy()
    slots[bad[:5]] = -1
    slots[bad[5:]] = n_slots + 3
    dims = A.make_dims(4096, H, Hkv, dh, 128, dtype)
    lse = torch.empty((sum(rows), H), dtype=torch.float32, device="cuda")
    out = A.acache_attention(dims, cu_rows, cu_keys, up(q, dtype), up_i32(slots), up(kp, dtype), up(vp, dtype),
                             lse=lse)
    f = lambda a: O.from_bits(a, dtype)
    # the oracle's view: an absent key is a zero row of the pools
    kz = np.concatenate([f(kp).reshape(-1, Hkv, dh), np.zeros((1, Hkv, dh))])
    vz = np.concatenate([f(vp).reshape(-1, Hkv, dh), np.zeros((1, Hkv, dh))])
    sl = np.where((slots < 0) | (slots >= n_slots), n_slots, slots)
    o_ref, lse_ref = O.attention_via_slots(f(q).reshape(-1, H, dh), kz, vz, sl, cu_rows, cu_keys)
    assert_close(down(out), o_ref.reshape(sum(rows), H * dh), dtype, "attention out")
    assert_close(down(lse), lse_ref, dtype, "attention lse")


def test_attention_whole_tiles_and_remainders(A):
    """Serving-like launch (16 requests of 2150 rows, 32 heads): the launcher
    runs each request's whole 256-row tiles on the wide kernel and its last
    102 rows, in a second launch, on the 128-row kernel.  Sampled rows of
    both launches (first and last rows of each part) are checked against the
    oracle; every output row must be written (finite)."""
    torch = _torch()
    dtype, H, Hkv, dh = "bf16", 32, 32, 128
    B, R, S = 16, 2150, 160
    rows, keys = [R] * B, [S + 7 * b for b in range(B)]
    q, kp, vp, slots, cu_rows, cu_keys, n_slots = _attn_case(dtype, H, Hkv, dh, rows, keys, seed=2150)
    dims = A.make_dims(4096, H, Hkv, dh, 128, dtype)
    lse = torch.full((sum(rows), H), float("nan"), dtype=torch.float32, device="cuda")
    out = torch.full((sum(rows), H * dh), float("nan"), dtype=torch.bfloat16, device="cuda")
    A.acache_attention(dims, cu_rows, cu_keys, up(q, dtype), up_i32(slots), up(kp, dtype), up(vp, dtype),
                       out=out, lse=lse)
    g_out, g_lse = down(out), down(lse)
    assert np.all(np.isfinite(g_out)) and np.all(np.isfinite(g_lse)), "a row was not written"
    f = lambda a: O.from_bits(a, dtype)
    pick = [0, 1, 255, 1023, 2047, 2048, 2049, 2100, R - 2, R - 1]
    sel, sub_rows = [], []
    for b in range(B):
        sel += [cu_rows[b] + i for i in pick]
        sub_rows.append(len(pick))
    sel = np.array(sel)
    sub_cu = np.concatenate([[0], np.cumsum(sub_rows)]).astype(int).tolist()
    o_ref, lse_ref = O.attention_via_slots(f(q)[sel].reshape(-1, H, dh), f(kp).reshape(-1, Hkv, dh),
                                           f(vp).reshape(-1, Hkv, dh), slots, sub_cu, cu_keys)
    assert_close(g_out[sel], o_ref.reshape(len(sel), H * dh), dtype, "attention out (sampled rows)")
    assert_close(g_lse[sel], lse_ref, dtype, "attention lse (sampled rows)")


def test_attention_rows_sum_to_one(A):
    """V = 1 gives O = 1 exactly up to rounding: attention rows sum to one."""
    torch = _torch()
    dtype, H, Hkv, dh = "bf16", 4, 2, 128
    q, kp, vp, slots, cu_rows, cu_keys, n_slots = _attn_case(dtype, H, Hkv, dh, [100, 64], [777, 65], seed=5)
    ones = torch.ones((n_slots, Hkv * dh), dtype=torch.bfloat16, device="cuda")
    dims = A.make_dims(256, H, Hkv, dh, 128, dtype)
    out = A.acache_attention(dims, cu_rows, cu_keys, up(q, dtype), up_i32(slots), up(kp, dtype), ones)
    np.testing.assert_allclose(down(out), 1.0, rtol=0, atol=2 ** -7)


# ----------------------------------------------------------------------------- scores (Eq. 4-5)

@pytest.mark.parametrize("dtype,H,Hkv,dh", [("bf16", 4, 4, 128), ("bf16", 8, 2, 128), ("f32", 4, 4, 64)])
@pytest.mark.parametrize("norm", ["affix", "full"])
def test_score(A, dtype, H, Hkv, dh, norm):
    torch = _torch()
    rows, nq, L = 300, [70, 33], 1000
    q = W.draw_tensor((rows, H * dh), dtype, seed=20)
    n_slots = L + 500
    kp = W.draw_tensor((n_slots, Hkv * dh), dtype, seed=21)
    q_rows = W.draw_permutation(rows, seed=22)[:sum(nq)]
    cu_q = [0, nq[0], nq[0] + nq[1]]
    affix_slots = W.draw_permutation(n_slots, seed=23)[:L]
    f = lambda a: O.from_bits(a, dtype)
    qf = f(q).reshape(rows, H, dh)
    kf = f(kp).reshape(n_slots, Hkv, dh)
    dims = A.make_dims(256, H, Hkv, dh, 128, dtype)
    scores = torch.zeros((2, L), dtype=torch.float32, device="cuda")
    row_lse = None
    lse_np = None
    if norm == "full":
        # any per-row log-normaliser works; use the affix LSE plus a positive offset
        lse_np = np.empty((rows, H))
        for h in range(H):
            lg = qf[:, h] @ kf[affix_slots, h // (H // Hkv)].T / np.sqrt(dh)
            lse_np[:, h] = np.log(np.exp(lg - lg.max(1, keepdims=True)).sum(1)) + lg.max(1) + 0.3
        row_lse = torch.from_numpy(lse_np.astype(np.float32)).cuda()
        lse_np = lse_np.astype(np.float32).astype(np.float64)
    A.acache_score(dims, up(q, dtype), up_i32(q_rows), cu_q, up(kp, dtype), up_i32(affix_slots), scores,
                   norm=A.ACACHE_NORM_AFFIX if norm == "affix" else A.ACACHE_NORM_FULL, row_lse=row_lse)
    ref = O.scores_via_slots(qf, q_rows, cu_q, kf, affix_slots, norm, lse_np)
    assert_close(down(scores), ref, dtype, "scores")
    if norm == "affix":
        np.testing.assert_allclose(down(scores).sum(1), H * np.array(nq), rtol=2e-3)
    # bit-reproducible: a second accumulation adds exactly the same values
    s1 = scores.clone()
    A.acache_score(dims, up(q, dtype), up_i32(q_rows), cu_q, up(kp, dtype), up_i32(affix_slots), scores,
                   norm=A.ACACHE_NORM_AFFIX if norm == "affix" else A.ACACHE_NORM_FULL, row_lse=row_lse)
    s2 = torch.zeros_like(scores)
    A.acache_score(dims, up(q, dtype), up_i32(q_rows), cu_q, up(kp, dtype), up_i32(affix_slots), s2,
                   norm=A.ACACHE_NORM_AFFIX if norm == "affix" else A.ACACHE_NORM_FULL, row_lse=row_lse)
    assert torch.equal(s2, s1)


# ----------------------------------------------------------------------------- greedy commit (Section 3.1)

@pytest.mark.parametrize("dtype,rows,n,ld", [
    ("bf16", 64, 126464, 126464),   # the serving workload's vocabulary
    ("bf16", 33, 1001, 1008),       # ragged width (scalar tail), padded rows
    ("bf16", 5, 7, 7),              # unaligned rows: scalar path only
    ("f32", 17, 4099, 4100),
])
def test_argmax_commit(A, dtype, rows, n, ld):
    torch = _torch()
    rng = np.random.default_rng(rows + n)
    vals = rng.integers(-20, 20, size=(rows, ld)).astype(np.float32) / 4  # many exact ties
    vals[0, :] = -np.inf
    vals[1, :5] = [np.nan, -0.0, 0.0, np.nan, -1.0]
    if n > 8:
        vals[1, 5:] = -2.0
        vals[2, n // 2] = np.inf
    vals[3, :] = np.nan
    bits = W.bf16_bits_from_f32(vals) if dtype == "bf16" else vals
    x = up(bits, dtype)
    ref = O.greedy_commit(O.from_bits(bits, dtype)[:, :n])
    ids = torch.full((3 * rows,), -7, dtype=torch.int32, device="cuda")
    pos = np.arange(rows, dtype=np.int32) * 2
    pos[1] = -1            # skipped
    pos[2] = 3 * rows      # skipped
    out = A.acache_argmax_commit(x[:, :n] if ld == n else x.narrow(1, 0, n), commit_pos=up_i32(pos), ids=ids)
    np.testing.assert_array_equal(out.cpu().numpy(), ref)
    want = np.full(3 * rows, -7)
    ok = (pos >= 0) & (pos < 3 * rows)
    want[pos[ok]] = ref[ok]
    np.testing.assert_array_equal(ids.cpu().numpy(), want)


# ----------------------------------------------------------------------------- shifted reuse (Section 4)

@pytest.mark.parametrize("dtype,hkv,dh,inplace", [("bf16", 4, 128, False), ("bf16", 1, 128, True),
                                                    ("f32", 2, 64, False), ("f32", 4, 64, True)])
def test_rerotate_k(A, dtype, hkv, dh, inplace):
    torch = _torch()
    n, n_slots = 300, 700
    k = W.draw_tensor((n_slots, hkv * dh), dtype, std=1.0, seed=60 + hkv)
    src = W.draw_permutation(n_slots, seed=61)[:n]
    dst = src if inplace else W.draw_permutation(n_slots, seed=62)[:n]
    delta = W.draw_ints((n,), -100000, 100000, seed=63)
    delta[:3] = [0, 1, -1]
    dims = A.make_dims(256, 4 * hkv, hkv, dh, 128, dtype)
    kp = up(k, dtype)
    out = kp if inplace else torch.zeros_like(kp)
    A.acache_rerotate_k(dims, kp, up_i32(src), out, up_i32(dst), up_i32(delta))
    ref = O.rerotate_keys(O.from_bits(k, dtype)[src].reshape(n, hkv, dh), delta, 10000.0)
    assert_close(down(out)[dst].reshape(n, hkv, dh), ref, dtype, "re-rotated K")
    if not inplace:  # untouched slots stay zero
        rest = np.setdiff1d(np.arange(n_slots), dst)
        assert not np.any(down(out)[rest])
