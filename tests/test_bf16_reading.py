"""Pins the reading of the bf16 tolerance (CPU, one LLaDA-shaped layer).

The stated bar is a maximum relative error of 2e-2 for bf16.  Exact
arithmetic that merely stores values in bf16 where the GPU path does
(tests/bf16_reference.py) is the best any bf16 implementation can do.  On
the one-layer LLaDA-shaped workload's 512 non-affix rows (2.1M outputs) its
per-element error max_i |g_i - r_i| / max(|r_i|, rms(r)) already exceeds
2e-2: the per-element form is out of reach of bf16 storage, so the bar is
read tensor-wise, max_i |g_i - r_i| / max_i |r_i| <= 2e-2, with the RMS
error <= 1e-2 and no element beyond 8x the RMS error (rounding noise has no
such outliers).  Those gates hold for the bf16-storage result."""

import numpy as np
import pytest

import workloads as W
from oracle import acache_oracle as O
from tests.bf16_reference import bf16_round, layer_forward_bf16
from tests.gpu_util import errors

pytestmark = pytest.mark.slow


def test_bf16_storage_exceeds_the_per_element_bar_but_meets_the_tensor_gates():
    w = W.get_config("llada-layer")
    d = w.dims
    dims = O.Dims(d_model=d.d_model, n_heads=d.n_heads, n_kv_heads=d.n_kv_heads, head_dim=d.head_dim,
                  d_ff=d.d_ff, rms_eps=d.rms_eps, rope_base=d.rope_base)
    layer = O.layer_from_bits(W.draw_layer_weights(w, 0), dims, "bf16")
    x0 = O.from_bits(W.draw_hidden_rows(w)[0], "bf16")
    lay = w.layout
    S = lay.seq_len
    pos = np.arange(S)
    rows = np.arange(lay.affix_end, S)              # the 512 unique + masked rows
    k_all, v_all = O.layer_kv(layer, dims, x0, pos)  # every key fresh: one block over the request
    vk, vv = k_all.copy(), v_all.copy()
    exact, _, _ = O.layer_forward(layer, dims, x0[rows], pos[rows], rows, vk, vv)
    bk, bv = bf16_round(k_all), bf16_round(v_all)
    emu = layer_forward_bf16(layer, dims, x0[rows], pos[rows], rows, bk, bv)
    e = errors(emu, exact)
    print(f"bf16 storage vs exact: {e}")
    assert e["elem_rel"] > 2e-2          # the per-element form fails for bf16 storage itself
    assert e["max_rel"] <= 2e-2          # the tensor-wise reading holds
    assert e["rms_rel"] <= 1e-2
    assert e["elem_rel"] <= 8 * e["rms_rel"]
