"""Python binding of libacache.so (ctypes).

Argument marshalling only: every function here checks Python-side shapes
and dtypes, passes raw device pointers and the current HIP stream to the C
entry point of the same name, and raises AcacheError on a non-zero status.
All computation runs in the library's HIP kernels.  Tensors are torch
tensors used as device memory.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libacache.so")

ACACHE_F32, ACACHE_BF16 = 0, 1
ACACHE_NORM_AFFIX, ACACHE_NORM_FULL = 0, 1


class AcacheError(RuntimeError):
    def __init__(self, fn: str, status: int, msg: str):
        super().__init__(f"{fn}: status {status}: {msg}")
        self.status = status


class Dims(ctypes.Structure):
    _fields_ = [("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("d_ff", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("rope_base", ctypes.c_float), ("dtype", ctypes.c_int32)]


class LayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")]


class Ragged(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("cu_rows", ctypes.POINTER(ctypes.c_int32)),
                ("cu_keys", ctypes.POINTER(ctypes.c_int32))]


class ScoreArgs(ctypes.Structure):
    _fields_ = [("q_rows", ctypes.c_void_p), ("cu_q", ctypes.POINTER(ctypes.c_int32)),
                ("affix_slots", ctypes.c_void_p), ("affix_len", ctypes.c_int32), ("norm", ctypes.c_int32),
                ("scores", ctypes.c_void_p), ("init", ctypes.c_int32), ("affix_keys_known", ctypes.c_int32),
                ("affix_key_begin", ctypes.c_int32)]


class Layout(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("seq_len", "affix_begin", "affix_len", "mask_begin", "mask_len",
                                              "shared_base", "private_base", "private_stride", "key_order")]


class Paging(ctypes.Structure):
    _fields_ = [("block_size", ctypes.c_int32), ("blocks_per_request", ctypes.c_int32),
                ("shared_blocks", ctypes.c_void_p), ("private_blocks", ctypes.c_void_p)]


def _load():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is not built; run `python -m paper_2608_26140_amd.build`")
    lib = ctypes.CDLL(_LIB_PATH)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    PI = ctypes.POINTER(ctypes.c_int32)
    sig = {
        "acache_score": [ctypes.POINTER(Dims), I32, P, I64, I64, P, PI, P, I64, I64, P, I32, P, I32, P, P, SZ, P],
        "acache_score_noalloc": [ctypes.POINTER(Dims), I32, P, I64, I64, P, PI, P, I64, I64, P, I32, P, I32, P, P],
        "acache_topk": [P, I32, I32, I32, P, P],
        "acache_gather_rows": [P, I64, I64, P, P, I64, I32, I32, P, I64, P],
        "acache_kv_scatter": [P, P, I64, I32, P, P, P, I64, I64, I32, I32, P],
        "acache_argmax_commit": [I32, P, I64, I32, I32, P, P, P, P, I64, P],
        "acache_threshold_commit": [I32, I32, P, P, ctypes.c_float, P, P, P, I64, P, P],
        "acache_rerotate_k": [ctypes.POINTER(Dims), P, P, P, P, P, I32, I64, I64, P],
        "acache_kv_deviation": [ctypes.POINTER(Dims), I32, I32, P, P, I64, I64, P, I64, P, P, P],
        "acache_build_maps": [ctypes.POINTER(Layout), I32, P, I32, P, P, P, P, P, P],
        "acache_build_maps_paged": [ctypes.POINTER(Layout), ctypes.POINTER(Paging), I32, P, I32, P, P, P, P, P, P],
        "acache_block_pool_create": [I32, ctypes.POINTER(P)],
        "acache_block_pool_destroy": [P],
        "acache_block_pool_alloc": [P, I32, PI],
        "acache_block_pool_free": [P, I32, PI],
        "acache_block_pool_stats": [P, PI, PI, PI],
        "acache_block_pool_reset_peak": [P],
        "acache_attention": [ctypes.POINTER(Dims), ctypes.POINTER(Ragged), P, P, P, P, I64, I64, P, P, P],
        "acache_layer_recompute": [ctypes.POINTER(Dims), ctypes.POINTER(LayerWeights), ctypes.POINTER(Ragged),
                                   P, P, P, P, P, P, I64, I64, ctypes.POINTER(ScoreArgs), P, SZ, P],
        "acache_layer_score": [ctypes.POINTER(Dims), ctypes.POINTER(LayerWeights), ctypes.POINTER(Ragged),
                               P, P, P, P, P, P, I64, I64, ctypes.POINTER(ScoreArgs), P, SZ, P],
        "acache_layer_decode": [ctypes.POINTER(Dims), ctypes.POINTER(LayerWeights), I32, I32, P, P, P, P, I32, P, I32,
                                P, I32, P, P, I64, I64, P, SZ, P],
        "acache_rmsnorm": [ctypes.POINTER(Dims), P, P, P, I32, P],
        "acache_layer_schedule": [ctypes.POINTER(Dims), I32, PI, PI],
        "acache_linear": [ctypes.POINTER(Dims), P, P, P, I32, I32, I32, I32, P, SZ, P],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int32
    lib.acache_workspace_size.argtypes = [ctypes.POINTER(Dims), I32, I32, I32]
    lib.acache_workspace_size.restype = ctypes.c_size_t
    lib.acache_status_string.argtypes = [ctypes.c_int32]
    lib.acache_status_string.restype = ctypes.c_char_p
    lib.acache_version.restype = ctypes.c_int32
    lib.acache_score_noalloc_max_bytes.argtypes = []
    lib.acache_score_noalloc_max_bytes.restype = ctypes.c_size_t
    lib.acache_anchor_count.argtypes = [ctypes.c_double, I32]
    lib.acache_anchor_count.restype = ctypes.c_int32
    return lib


lib = _load()
LIB_PATH = _LIB_PATH


def _check(name: str, st: int):
    if st != 0:
        raise AcacheError(name, st, lib.acache_status_string(st).decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _i32(values: Sequence[int]):
    arr = (ctypes.c_int32 * len(values))(*[int(v) for v in values])
    return arr


def _dev_i32(t: torch.Tensor, name: str):
    if t.dtype != torch.int32 or not t.is_cuda or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous int32 device tensor")


def make_dims(d_model, n_heads, n_kv_heads, head_dim, d_ff, dtype: str, rms_eps=1e-5, rope_base=10000.0) -> Dims:
    return Dims(d_model, n_heads, n_kv_heads, head_dim, d_ff, rms_eps, rope_base,
                ACACHE_BF16 if dtype == "bf16" else ACACHE_F32)


def torch_dtype(dims: Dims):
    return torch.bfloat16 if dims.dtype == ACACHE_BF16 else torch.float32


def acache_workspace_size(dims: Dims, max_rows: int, batch: int, affix_len: int) -> int:
    n = lib.acache_workspace_size(ctypes.byref(dims), max_rows, batch, affix_len)
    if n == 0:
        raise AcacheError("acache_workspace_size", 2, "invalid dims")
    return n


def workspace(dims: Dims, max_rows: int, batch: int, affix_len: int, device="cuda") -> torch.Tensor:
    return torch.empty(acache_workspace_size(dims, max_rows, batch, affix_len), dtype=torch.uint8, device=device)


def acache_layer_schedule(dims: Dims, rows: int):
    """(o_splits, down_splits) acache_layer_recompute uses for `rows` rows."""
    o, dn = ctypes.c_int32(0), ctypes.c_int32(0)
    _check("acache_layer_schedule", lib.acache_layer_schedule(ctypes.byref(dims), rows, ctypes.byref(o),
                                                              ctypes.byref(dn)))
    return o.value, dn.value


def acache_anchor_count(ratio: float, affix_len: int) -> int:
    k = lib.acache_anchor_count(float(ratio), int(affix_len))
    if k < 0:
        raise AcacheError("acache_anchor_count", 2, f"ratio {ratio} / affix length {affix_len} out of range")
    return k


def acache_topk(scores: torch.Tensor, k: int, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    if scores.dtype != torch.float32 or scores.dim() != 2 or not scores.is_contiguous():
        raise TypeError("scores must be a contiguous float32 [batch, L] tensor")
    b, L = scores.shape
    if out is None:
        out = torch.empty((b, k), dtype=torch.int32, device=scores.device)
    _check("acache_topk", lib.acache_topk(_ptr(scores), b, L, k, _ptr(out), _stream(stream)))
    return out


def acache_gather_rows(src: torch.Tensor, idx: torch.Tensor, remap: Optional[torch.Tensor] = None,
                       out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    _dev_i32(idx, "idx")
    if remap is not None:
        _dev_i32(remap, "remap")
    src2 = src.reshape(src.shape[0], -1)
    n = idx.numel()
    if out is None:
        out = torch.empty((n,) + tuple(src.shape[1:]), dtype=src.dtype, device=src.device)
    row_bytes = src2.shape[1] * src2.element_size()
    _check("acache_gather_rows", lib.acache_gather_rows(
        _ptr(src2), src2.stride(0) * src2.element_size(), src2.shape[0], _ptr(idx), _ptr(remap),
        0 if remap is None else remap.numel(), n, row_bytes, _ptr(out), row_bytes, _stream(stream)))
    return out


def acache_kv_scatter(k_src: torch.Tensor, v_src: torch.Tensor, dst_slots: torch.Tensor,
                      k_pool: torch.Tensor, v_pool: torch.Tensor, stream=None):
    _dev_i32(dst_slots, "dst_slots")
    dt = ACACHE_BF16 if k_src.dtype == torch.bfloat16 else ACACHE_F32
    n, row = k_src.shape
    _check("acache_kv_scatter", lib.acache_kv_scatter(
        _ptr(k_src), _ptr(v_src), k_src.stride(0), n, _ptr(dst_slots), _ptr(k_pool), _ptr(v_pool),
        k_pool.stride(0), k_pool.shape[0], row, dt, _stream(stream)))


def acache_build_maps(layout: Layout, batch: int, anchors: Optional[torch.Tensor], k: int, device="cuda",
                      stream=None):
    """Returns dict(row_pos, row_src, write_slots, read_slots, q_rows) of int32 device tensors."""
    if anchors is not None:
        _dev_i32(anchors, "anchors")
    R = k + layout.seq_len - layout.affix_len
    t = lambda n: torch.empty(n, dtype=torch.int32, device=device)
    out = dict(row_pos=t(batch * R), row_src=t(batch * R), write_slots=t(batch * R),
               read_slots=t(batch * layout.seq_len), q_rows=t(batch * layout.mask_len))
    _check("acache_build_maps", lib.acache_build_maps(
        ctypes.byref(layout), batch, _ptr(anchors) if k > 0 else None, k, _ptr(out["row_pos"]),
        _ptr(out["row_src"]), _ptr(out["write_slots"]), _ptr(out["read_slots"]), _ptr(out["q_rows"]),
        _stream(stream)))
    return out


def acache_build_maps_paged(layout: Layout, batch: int, anchors: Optional[torch.Tensor], k: int, block_size: int,
                            shared_blocks: Optional[torch.Tensor], private_blocks: torch.Tensor,
                            blocks_per_request: int, device="cuda", stream=None) -> dict:
    """acache_build_maps with slots from block tables (device int32)."""
    if anchors is not None:
        _dev_i32(anchors, "anchors")
    for t, n in ((shared_blocks, "shared_blocks"), (private_blocks, "private_blocks")):
        if t is not None:
            _dev_i32(t, n)
    R = k + layout.seq_len - layout.affix_len
    t = lambda n: torch.empty(n, dtype=torch.int32, device=device)
    out = dict(row_pos=t(batch * R), row_src=t(batch * R), write_slots=t(batch * R),
               read_slots=t(batch * layout.seq_len), q_rows=t(batch * layout.mask_len))
    pg = Paging(block_size, blocks_per_request, None if shared_blocks is None else shared_blocks.data_ptr(),
                None if private_blocks is None else private_blocks.data_ptr())
    _check("acache_build_maps_paged", lib.acache_build_maps_paged(
        ctypes.byref(layout), ctypes.byref(pg), batch, _ptr(anchors) if k > 0 else None, k, _ptr(out["row_pos"]),
        _ptr(out["row_src"]), _ptr(out["write_slots"]), _ptr(out["read_slots"]), _ptr(out["q_rows"]),
        _stream(stream)))
    return out


class BlockPool:
    """The library's host-side KV block allocator (acache_block_pool)."""

    def __init__(self, capacity: int):
        h = ctypes.c_void_p()
        _check("acache_block_pool_create", lib.acache_block_pool_create(int(capacity), ctypes.byref(h)))
        self._h = h

    def alloc(self, n: int) -> list:
        ids = (ctypes.c_int32 * max(n, 1))()
        _check("acache_block_pool_alloc", lib.acache_block_pool_alloc(self._h, int(n), ids))
        return list(ids[:n])

    def free(self, ids: Sequence[int]):
        arr = _i32(list(ids)) if len(ids) else (ctypes.c_int32 * 1)()
        _check("acache_block_pool_free", lib.acache_block_pool_free(self._h, len(ids), arr))

    def stats(self) -> dict:
        c, u, p = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        _check("acache_block_pool_stats", lib.acache_block_pool_stats(self._h, ctypes.byref(c), ctypes.byref(u),
                                                                      ctypes.byref(p)))
        return dict(capacity=c.value, in_use=u.value, peak=p.value)

    def reset_peak(self):
        _check("acache_block_pool_reset_peak", lib.acache_block_pool_reset_peak(self._h))

    def close(self):
        if self._h:
            lib.acache_block_pool_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _ragged(cu_rows: Sequence[int], cu_keys: Sequence[int]):
    r = _i32(cu_rows)
    k = _i32(cu_keys)
    return Ragged(len(cu_rows) - 1, r, k), (r, k)


def acache_attention(dims: Dims, cu_rows, cu_keys, q: torch.Tensor, read_slots: torch.Tensor,
                     k_pool: torch.Tensor, v_pool: torch.Tensor, out: Optional[torch.Tensor] = None,
                     lse: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    _dev_i32(read_slots, "read_slots")
    rg, keep = _ragged(cu_rows, cu_keys)
    if out is None:
        out = torch.empty_like(q)
    _check("acache_attention", lib.acache_attention(
        ctypes.byref(dims), ctypes.byref(rg), _ptr(q), _ptr(read_slots), _ptr(k_pool), _ptr(v_pool),
        k_pool.stride(0), k_pool.shape[0], _ptr(out), _ptr(lse), _stream(stream)))
    return out


def acache_score(dims: Dims, q: torch.Tensor, q_rows: torch.Tensor, cu_q, k_pool: torch.Tensor,
                 affix_slots: torch.Tensor, scores: torch.Tensor, norm: int = ACACHE_NORM_AFFIX,
                 row_lse: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None, stream=None):
    _dev_i32(q_rows, "q_rows")
    _dev_i32(affix_slots, "affix_slots")
    batch = len(cu_q) - 1
    L = affix_slots.numel()
    if ws is None:
        ws = workspace(dims, max(1, int(cu_q[-1])), batch, L, q.device)
    cq = _i32(cu_q)
    _check("acache_score", lib.acache_score(
        ctypes.byref(dims), batch, _ptr(q), q.stride(0), q.shape[0], _ptr(q_rows), cq, _ptr(k_pool),
        k_pool.stride(0), k_pool.shape[0], _ptr(affix_slots), L, _ptr(row_lse), norm, _ptr(scores),
        _ptr(ws), ws.numel(), _stream(stream)))
    return scores


def acache_score_noalloc(dims: Dims, q: torch.Tensor, q_rows: torch.Tensor, cu_q, k_pool: torch.Tensor,
                         affix_slots: torch.Tensor, scores: torch.Tensor, norm: int = ACACHE_NORM_AFFIX,
                         row_lse: Optional[torch.Tensor] = None, stream=None):
    """acache_score with the library's fixed scratch instead of a workspace."""
    _dev_i32(q_rows, "q_rows")
    _dev_i32(affix_slots, "affix_slots")
    batch = len(cu_q) - 1
    L = affix_slots.numel()
    cq = _i32(cu_q)
    _check("acache_score_noalloc", lib.acache_score_noalloc(
        ctypes.byref(dims), batch, _ptr(q), q.stride(0), q.shape[0], _ptr(q_rows), cq, _ptr(k_pool),
        k_pool.stride(0), k_pool.shape[0], _ptr(affix_slots), L, _ptr(row_lse), norm, _ptr(scores),
        _stream(stream)))
    return scores


def layer_weights(w: dict) -> LayerWeights:
    return LayerWeights(*[w[n].data_ptr() for n in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")])


def acache_layer_recompute(dims: Dims, weights, cu_rows, cu_keys, x: torch.Tensor, pos: torch.Tensor,
                           write_slots: torch.Tensor, read_slots: torch.Tensor, k_pool: torch.Tensor,
                           v_pool: torch.Tensor, ws: torch.Tensor, score: Optional[dict] = None, stream=None):
    """One block in place on x.  weights: LayerWeights or dict of tensors.
    score: dict(q_rows, cu_q, affix_slots, scores, norm, init, and optionally
    affix_key_begin: the key index at which every request's read slots hold
    the affix slots in order) for the probe."""
    for t, n in ((pos, "pos"), (write_slots, "write_slots"), (read_slots, "read_slots")):
        _dev_i32(t, n)
    lw = weights if isinstance(weights, LayerWeights) else layer_weights(weights)
    rg, keep = _ragged(cu_rows, cu_keys)
    sa = None
    cq = None
    if score is not None:
        cq = _i32(score["cu_q"])
        akb = score.get("affix_key_begin")
        sa = ScoreArgs(score["q_rows"].data_ptr(), cq, score["affix_slots"].data_ptr(),
                       score["affix_slots"].numel(), score.get("norm", ACACHE_NORM_AFFIX),
                       score["scores"].data_ptr(), int(score.get("init", 0)), int(akb is not None),
                       int(akb or 0))
    _check("acache_layer_recompute", lib.acache_layer_recompute(
        ctypes.byref(dims), ctypes.byref(lw), ctypes.byref(rg), _ptr(x), _ptr(pos), _ptr(write_slots),
        _ptr(read_slots), _ptr(k_pool), _ptr(v_pool), k_pool.stride(0), k_pool.shape[0],
        ctypes.byref(sa) if sa is not None else None, _ptr(ws), ws.numel(), _stream(stream)))


def acache_layer_score(dims: Dims, weights, cu_rows, cu_keys, x: torch.Tensor, pos: torch.Tensor,
                       write_slots: Optional[torch.Tensor], read_slots: Optional[torch.Tensor], k_pool: torch.Tensor,
                       v_pool: Optional[torch.Tensor], ws: torch.Tensor, score: dict, stream=None):
    """The probe's last layer reduced to its score: adds this layer's Eq. 4-5
    contribution into score["scores"]; x is not modified.  write_slots,
    read_slots and v_pool are needed only under ACACHE_NORM_FULL."""
    _dev_i32(pos, "pos")
    for t, n in ((write_slots, "write_slots"), (read_slots, "read_slots")):
        if t is not None:
            _dev_i32(t, n)
    lw = weights if isinstance(weights, LayerWeights) else layer_weights(weights)
    rg, keep = _ragged(cu_rows, cu_keys)
    cq = _i32(score["cu_q"])
    sa = ScoreArgs(score["q_rows"].data_ptr(), cq, score["affix_slots"].data_ptr(), score["affix_slots"].numel(),
                   score.get("norm", ACACHE_NORM_AFFIX), score["scores"].data_ptr(), int(score.get("init", 0)))
    _check("acache_layer_score", lib.acache_layer_score(
        ctypes.byref(dims), ctypes.byref(lw), ctypes.byref(rg), _ptr(x), _ptr(pos), _ptr(write_slots),
        _ptr(read_slots), _ptr(k_pool), _ptr(v_pool), k_pool.stride(0), k_pool.shape[0], ctypes.byref(sa), _ptr(ws),
        ws.numel(), _stream(stream)))


def acache_layer_decode(dims: Dims, weights, batch: int, rows_per_request: int, x: torch.Tensor, pos: torch.Tensor,
                        write_slots: torch.Tensor, affix_slots: torch.Tensor, anchors: Optional[torch.Tensor], k: int,
                        private_slots: torch.Tensor, private_len: int, k_pool: torch.Tensor, v_pool: torch.Tensor,
                        ws: torch.Tensor, stream=None):
    """One block of a decode step, in place on x [batch * rows_per_request, d]:
    the shared affix keys (minus each request's anchors) and each request's
    private slots [batch, private_len] form its view."""
    for t, n in ((pos, "pos"), (write_slots, "write_slots"), (affix_slots, "affix_slots"),
                 (private_slots, "private_slots")):
        _dev_i32(t, n)
    if anchors is not None:
        _dev_i32(anchors, "anchors")
    lw = weights if isinstance(weights, LayerWeights) else layer_weights(weights)
    _check("acache_layer_decode", lib.acache_layer_decode(
        ctypes.byref(dims), ctypes.byref(lw), batch, rows_per_request, _ptr(x), _ptr(pos), _ptr(write_slots),
        _ptr(affix_slots), affix_slots.numel(), _ptr(anchors) if k > 0 else None, k, _ptr(private_slots), private_len,
        _ptr(k_pool), _ptr(v_pool), k_pool.stride(0), k_pool.shape[0], _ptr(ws), ws.numel(), _stream(stream)))


def acache_rmsnorm(dims: Dims, x: torch.Tensor, g: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None):
    if out is None:
        out = torch.empty_like(x)
    _check("acache_rmsnorm", lib.acache_rmsnorm(ctypes.byref(dims), _ptr(x), _ptr(g), _ptr(out), x.shape[0],
                                                _stream(stream)))
    return out


def acache_linear(dims: Dims, a: torch.Tensor, w: torch.Tensor, out: Optional[torch.Tensor] = None,
                  accumulate: bool = False, ws: Optional[torch.Tensor] = None, stream=None):
    """ws (optional, from `workspace`): lets bf16 balance small row counts by
    splitting K across workgroups."""
    M, K = a.shape
    N = w.shape[0]
    if out is None:
        out = torch.empty((M, N), dtype=a.dtype, device=a.device)
    _check("acache_linear", lib.acache_linear(ctypes.byref(dims), _ptr(a), _ptr(w), _ptr(out), M, N, K,
                                              int(accumulate), _ptr(ws), 0 if ws is None else ws.numel(),
                                              _stream(stream)))
    return out


def acache_kv_deviation(dims: Dims, k_pool: torch.Tensor, v_pool: torch.Tensor, fresh_slots: torch.Tensor,
                        stale_slots: torch.Tensor, scores: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """fresh_slots [B, L] (any row stride), stale_slots [L] -> scores [B, L]."""
    B, L = fresh_slots.shape
    assert fresh_slots.dtype == torch.int32 and fresh_slots.stride(1) == 1
    _dev_i32(stale_slots, "stale_slots")
    if scores is None:
        scores = torch.empty((B, L), dtype=torch.float32, device=k_pool.device)
    _check("acache_kv_deviation", lib.acache_kv_deviation(
        ctypes.byref(dims), B, L, _ptr(k_pool), _ptr(v_pool), k_pool.stride(0), k_pool.shape[0],
        _ptr(fresh_slots), fresh_slots.stride(0), _ptr(stale_slots), _ptr(scores), _stream(stream)))
    return scores


def acache_rerotate_k(dims: Dims, k_src: torch.Tensor, src_slots: torch.Tensor, k_dst: torch.Tensor,
                      dst_slots: torch.Tensor, delta: torch.Tensor, stream=None):
    """k_dst[dst_slots[i]] = k_src[src_slots[i]] rotated by delta[i] positions."""
    for t, n in ((src_slots, "src_slots"), (dst_slots, "dst_slots"), (delta, "delta")):
        _dev_i32(t, n)
    assert k_src.stride(0) == k_dst.stride(0) and k_src.shape[0] == k_dst.shape[0]
    _check("acache_rerotate_k", lib.acache_rerotate_k(
        ctypes.byref(dims), _ptr(k_src), _ptr(src_slots), _ptr(k_dst), _ptr(dst_slots), _ptr(delta),
        src_slots.numel(), k_src.stride(0), k_src.shape[0], _stream(stream)))


def acache_argmax_commit(x: torch.Tensor, out: Optional[torch.Tensor] = None,
                         commit_pos: Optional[torch.Tensor] = None, ids: Optional[torch.Tensor] = None,
                         conf: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Row argmax of x [rows, n] (lowest index on ties, NaN lowest); with
    commit_pos, also ids[commit_pos[i]] = argmax of row i; conf (fp32 [rows],
    optional) receives each row's largest softmax probability."""
    rows, n = x.shape
    if out is None:
        out = torch.empty(rows, dtype=torch.int32, device=x.device)
    if commit_pos is not None:
        _dev_i32(commit_pos, "commit_pos")
        _dev_i32(ids, "ids")
    if conf is not None and (conf.dtype != torch.float32 or not conf.is_contiguous() or conf.numel() < rows):
        raise ValueError("conf must be a contiguous float32 tensor of at least `rows` values")
    dt = ACACHE_BF16 if x.dtype == torch.bfloat16 else ACACHE_F32
    _check("acache_argmax_commit", lib.acache_argmax_commit(
        dt, _ptr(x), x.stride(0), rows, n, _ptr(out), _ptr(conf), _ptr(commit_pos), _ptr(ids),
        0 if ids is None else ids.numel(), _stream(stream)))
    return out


def acache_threshold_commit(block: int, pick: torch.Tensor, conf: torch.Tensor, tau: float, committed: torch.Tensor,
                            commit_pos: torch.Tensor, ids: torch.Tensor, count: torch.Tensor, stream=None):
    """One decode step's commit over B requests x `block` rows (see the header)."""
    for t, n in ((pick, "pick"), (committed, "committed"), (commit_pos, "commit_pos"), (ids, "ids"),
                 (count, "count")):
        _dev_i32(t, n)
    if conf.dtype != torch.float32 or not conf.is_contiguous() or conf.numel() != pick.numel():
        raise ValueError("conf must be a contiguous float32 tensor shaped like pick")
    if block <= 0 or pick.numel() % block or committed.numel() != pick.numel() or commit_pos.numel() != pick.numel():
        raise ValueError("pick, committed and commit_pos hold batch * block values")
    batch = pick.numel() // block
    _check("acache_threshold_commit", lib.acache_threshold_commit(
        batch, block, _ptr(pick), _ptr(conf), float(tau), _ptr(committed), _ptr(commit_pos), _ptr(ids),
        ids.numel(), _ptr(count), _stream(stream)))


# ---------------------------------------------------------------------------- measurement hook
KERNEL_IDS = {"gemm_qkv": 0, "gemm_o": 1, "gemm_gate_up": 2, "gemm_down": 3, "attention": 4, "score_lse": 5,
              "score_colsum": 6, "score_reduce": 7, "rmsnorm": 8, "residual": 9, "topk": 10, "gather": 11,
              "maps": 12, "scatter": 13, "argmax": 14}
lib.acache_time_kernel.argtypes = [ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                   ctypes.POINTER(ctypes.c_int32)]
lib.acache_time_kernel.restype = ctypes.c_int32


def _hip_runtime():
    """The HIP runtime already loaded in this process (the one torch and the
    library share)."""
    for line in open("/proc/self/maps"):
        if "libamdhip64" in line:
            path = line.split()[-1]
            rt = ctypes.CDLL(path)
            rt.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
            rt.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
            rt.hipEventSynchronize.argtypes = [ctypes.c_void_p]
            rt.hipEventDestroy.argtypes = [ctypes.c_void_p]
            return rt
    raise RuntimeError("HIP runtime not loaded")


class KernelTimer:
    """Arms acache_time_kernel for one kernel id with `capacity` event pairs;
    durations() returns the recorded launch durations in milliseconds."""

    def __init__(self, kernel: str, capacity: int):
        self.rt = _hip_runtime()
        self.kernel = KERNEL_IDS[kernel]
        self.capacity = capacity
        self.starts = (ctypes.c_void_p * capacity)()
        self.stops = (ctypes.c_void_p * capacity)()
        for i in range(capacity):
            for arr in (self.starts, self.stops):
                ev = ctypes.c_void_p()
                if self.rt.hipEventCreate(ctypes.byref(ev)) != 0:
                    raise RuntimeError("hipEventCreate failed")
                arr[i] = ev
        self.count = ctypes.c_int32(0)

    def __enter__(self):
        self.count.value = 0
        _check("acache_time_kernel", lib.acache_time_kernel(self.kernel, self.starts, self.stops, self.capacity,
                                                             ctypes.byref(self.count)))
        return self

    def __exit__(self, *exc):
        lib.acache_time_kernel(-1, None, None, 0, None)

    def durations(self):
        out = []
        for i in range(self.count.value):
            self.rt.hipEventSynchronize(self.stops[i])
            ms = ctypes.c_float()
            if self.rt.hipEventElapsedTime(ctypes.byref(ms), self.starts[i], self.stops[i]) != 0:
                raise RuntimeError("hipEventElapsedTime failed")
            out.append(ms.value)
        return out

    def close(self):
        for arr in (self.starts, self.stops):
            for ev in arr:
                self.rt.hipEventDestroy(ev)
