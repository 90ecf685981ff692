"""Exact arithmetic with bfloat16 storage at the points where the bf16 GPU
path stores a value (test infrastructure, CPU, float64 between roundings).

It sizes the error that bf16 storage alone causes, against which the GPU's
error is judged: a kernel may lose no more than this.  The storage points of
one block over the recomputed rows are:
  h   = RMSNorm(x)                       (the GEMM operand)
  q,k = rotary(h W_q), rotary(h W_k);  v = h W_v   (q operand, K/V cache)
  P   = exp(logits - running max)        (the operand of P V)
  o   = P V / l                          (the O projection's operand)
  x1  = x + o W_o                        (the residual stream)
  h2  = RMSNorm(x1)
  a   = SiLU(h2 W_g) * (h2 W_u)          (the down projection's operand)
  out = x1 + a W_d
Accumulations and the softmax statistics are exact here.  The pieces are
the oracle's functions; only the roundings are added."""

import numpy as np

from oracle import acache_oracle as O


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 (ties to even), returned as float64."""
    a32 = np.ascontiguousarray(a, dtype=np.float32)
    u = a32.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = (((u + 0x7FFF + lsb) >> 16) << 16).astype(np.uint32)
    return r.view(np.float32).astype(np.float64)


def layer_forward_bf16(w: O.Layer, dims: O.Dims, x, pos, rows, view_k, view_v, points=None):
    """O.layer_forward with bf16 storage at `points` (default: all of them).
    view_k / view_v receive the rounded fresh K/V.  Returns x_out."""
    pts = {"h", "q", "k", "v", "p", "o", "x1", "h2", "a", "out"} if points is None else set(points)
    rd = (lambda name, t: bf16_round(t) if name in pts else t)
    r = x.shape[0]
    nh, nkv, dh = dims.n_heads, dims.n_kv_heads, dims.head_dim
    h = rd("h", O.rms_norm(x, w.g1, dims.rms_eps))
    q = rd("q", O.rope((h @ w.wq.T).reshape(r, nh, dh), pos, dims.rope_base))
    k = rd("k", O.rope((h @ w.wk.T).reshape(r, nkv, dh), pos, dims.rope_base))
    v = rd("v", (h @ w.wv.T).reshape(r, nkv, dh))
    view_k[rows] = k
    view_v[rows] = v
    group = nh // nkv
    o = np.empty((r, nh, dh))
    for hh in range(nh):
        lg = q[:, hh] @ view_k[:, hh // group].T / np.sqrt(dh)
        p = np.exp(lg - lg.max(axis=1, keepdims=True))
        l_sum = p.sum(axis=1, keepdims=True)
        o[:, hh] = (rd("p", p) @ view_v[:, hh // group]) / l_sum
    o = rd("o", o.reshape(r, nh * dh))
    x1 = rd("x1", x + o @ w.wo.T)
    h2 = rd("h2", O.rms_norm(x1, w.g2, dims.rms_eps))
    a = rd("a", O.silu(h2 @ w.wg.T) * (h2 @ w.wu.T))
    return rd("out", x1 + a @ w.wd.T)
