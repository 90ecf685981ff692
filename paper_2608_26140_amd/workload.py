"""Device setup of a synthetic workload: upload the seeded weights and
inputs, and materialise the stale shared affix cache by the workload's
recipe (the affix cache is computed once, in a context other than the
request's; Sections 3.3 and 4.2).

Recipes:
  "perturb"  the donor context is the affix rows' own inputs plus N(0, 0.1^2)
             noise, at the affix positions (one-layer workloads);
  "donor"    a full forward of a donor request with its own unique ids; its
             affix rows write the shared slots, its other rows a scratch
             private region.
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

import workloads as W

from . import acache as A
from .driver import AffixBatch, Model


def upload(bits: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(bits, dtype=np.float32)).to(device)


def upload_i32(a, device="cuda") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a), dtype=np.int32)).to(device)


def dims_of(w: W.Workload) -> A.Dims:
    d = w.dims
    return A.make_dims(d.d_model, d.n_heads, d.n_kv_heads, d.head_dim, d.d_ff, d.dtype, d.rms_eps, d.rope_base)


@dataclass
class Setup:
    workload: W.Workload
    model: Model
    batch: AffixBatch
    host: dict  # host copies of the inputs the oracle needs (bits)


def build(w: W.Workload, device="cuda", n_layers: Optional[int] = None, keep_host: bool = True,
          max_rows: Optional[int] = None, block_size: Optional[int] = None) -> Setup:
    d, lay = w.dims, w.layout
    nl = d.n_layers if n_layers is None else n_layers
    host = {"layers": []}
    layers = []
    for i in range(nl):
        bits = W.draw_layer_weights(w, i)
        if keep_host:
            host["layers"].append(bits)
        layers.append({name: upload(getattr(bits, name), d.dtype, device)
                       for name in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")})
    model = Model(dims_of(w), layers)
    S, B = lay.seq_len, w.batch
    if d.vocab:
        ids, donor_ids = W.draw_token_ids(w)
        emb = W.draw_embedding(w)
        if keep_host:
            host.update(ids=ids, donor_ids=donor_ids, embedding=emb)
        x_src = upload(emb, d.dtype, device)
        remap = upload_i32(ids.reshape(-1), device)
    else:
        hidden = W.draw_hidden_rows(w)
        if keep_host:
            host.update(hidden=hidden)
        x_src = upload(hidden.reshape(B * S, d.d_model), d.dtype, device)
        remap = None
    batch = AffixBatch(model, S, lay.affix_begin, lay.affix_len, lay.mask_begin, lay.mask_len, B, x_src,
                       remap, device=device, max_rows=max_rows, block_size=block_size)

    L = lay.affix_len
    if w.stale == "perturb":
        donor = W.draw_donor_rows(w, hidden)
        if keep_host:
            host.update(donor=donor)
        dx = upload(donor, d.dtype, device)
        pos = upload_i32(np.arange(lay.affix_begin, lay.affix_end))
        batch.materialize_affix(dx, pos, batch.affix_slots, batch.affix_slots)
    elif w.stale == "donor":
        # donor request: all S positions; affix rows -> the shared affix
        # slots, the rest -> request 0's private slots (overwritten later)
        p = np.arange(S)
        in_affix = (p >= lay.affix_begin) & (p < lay.affix_end)
        wslots = np.empty(S, dtype=np.int64)
        wslots[in_affix] = batch.affix_slots.cpu().numpy()
        wslots[~in_affix] = batch.private_slots(S - L)[0]
        dx = A.acache_gather_rows(x_src, upload_i32(np.arange(S)), upload_i32(donor_ids))
        batch.materialize_affix(dx, upload_i32(p), upload_i32(wslots), upload_i32(wslots))
    else:
        raise ValueError(w.stale)
    return Setup(workload=w, model=model, batch=batch, host=host)
