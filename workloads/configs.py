"""Workload shapes for the selective affix-KV recompute path.

Five synthetic workloads stand in for the paper's few-shot prompts (its
datasets and trained weights are not available): a tiny fp32 layer, one
LLaDA-8B-shaped bf16 layer, a 32-layer LLaDA-shaped stack, a 28-layer
Dream-7B-shaped GQA stack with an infix affix, and a serving-scale LLaDA
stack.  Generation length 256 and block length 32 follow the paper's
default settings (Section 5, "Default Settings"); affix lengths are chosen
per workload because the paper does not report token counts.

A workload names its anchor ratio rho; the anchor count K it implies is the
method's arithmetic and lives on each side (the library and the oracle),
not here.
"""

from __future__ import annotations

from dataclasses import dataclass, field, replace
from typing import Dict, Tuple


@dataclass(frozen=True)
class ModelDims:
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    n_layers: int
    dtype: str  # "f32" or "bf16": storage type of weights, activations and KV
    rms_eps: float = 1e-5
    rope_base: float = 10000.0
    vocab: int = 0  # 0: layer-0 inputs are given hidden rows, not token ids

    @property
    def qkv_width(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim


@dataclass(frozen=True)
class SeqLayout:
    """Logical positions of one request: a shared affix span, a masked
    generation span, and unique (request-specific, unmasked) positions for
    the rest.  Positions are 0-based and identical for every request."""

    seq_len: int
    affix_begin: int
    affix_len: int
    mask_begin: int
    mask_len: int

    @property
    def affix_end(self) -> int:
        return self.affix_begin + self.affix_len

    @property
    def n_nonaffix(self) -> int:
        return self.seq_len - self.affix_len

    def affix_positions(self):
        return list(range(self.affix_begin, self.affix_end))

    def masked_positions(self):
        return list(range(self.mask_begin, self.mask_begin + self.mask_len))

    def nonaffix_positions(self):
        return [p for p in range(self.seq_len) if not (self.affix_begin <= p < self.affix_end)]


@dataclass(frozen=True)
class Workload:
    name: str
    seed_id: int
    dims: ModelDims
    layout: SeqLayout
    batch: int
    ratio: float
    stale: str  # "perturb": stale KV from affix inputs + N(0, 0.1^2); "donor": from a donor request
    mask_rows: str = "random"  # "random": N(0,1) per masked row; "shared": one mask vector
    ratios: Tuple[float, ...] = field(default=())
    decode_block: int = 0  # serving schedule: commit the masked span in blocks of this many tokens (0: none)

    def with_ratio(self, ratio: float) -> "Workload":
        return replace(self, ratio=ratio)


LLADA = dict(d_model=4096, n_heads=32, n_kv_heads=32, head_dim=128, d_ff=12288)
DREAM = dict(d_model=3584, n_heads=28, n_kv_heads=4, head_dim=128, d_ff=18944)

CONFIGS: Dict[str, Workload] = {
    # one fp32 layer: 128 affix + 32 unique + 32 masked (one shared mask vector)
    "tiny-f32": Workload(
        name="tiny-f32", seed_id=1,
        dims=ModelDims(d_model=256, n_heads=4, n_kv_heads=4, head_dim=64, d_ff=688,
                       n_layers=1, dtype="f32"),
        layout=SeqLayout(seq_len=192, affix_begin=0, affix_len=128, mask_begin=160, mask_len=32),
        batch=1, ratio=0.2, stale="perturb", mask_rows="shared"),
    # one LLaDA-8B-shaped bf16 layer: 1024 affix + 256 unique + 256 masked, N(0,1) rows
    "llada-layer": Workload(
        name="llada-layer", seed_id=2,
        dims=ModelDims(n_layers=1, dtype="bf16", **LLADA),
        layout=SeqLayout(seq_len=1536, affix_begin=0, affix_len=1024, mask_begin=1280, mask_len=256),
        batch=1, ratio=0.2, stale="perturb"),
    # 32-layer LLaDA-shaped stack, 8 requests share a 2048-token prefix affix
    "llada-stack-b8": Workload(
        name="llada-stack-b8", seed_id=3,
        dims=ModelDims(n_layers=32, dtype="bf16", vocab=126464, **LLADA),
        layout=SeqLayout(seq_len=2432, affix_begin=0, affix_len=2048, mask_begin=2176, mask_len=256),
        batch=8, ratio=0.2, stale="donor"),
    # 28-layer Dream-shaped GQA stack, infix affix between two unique spans
    "dream-stack-b4": Workload(
        name="dream-stack-b4", seed_id=4,
        dims=ModelDims(n_layers=28, dtype="bf16", vocab=126464, **DREAM),
        layout=SeqLayout(seq_len=5120, affix_begin=512, affix_len=4096, mask_begin=4864, mask_len=256),
        batch=4, ratio=0.2, stale="donor", ratios=(0.1, 0.2, 0.4)),
    # serving-scale LLaDA stack: 32 requests share an 8192-token prefix affix
    "llada-serve-b32": Workload(
        name="llada-serve-b32", seed_id=5,
        dims=ModelDims(n_layers=32, dtype="bf16", vocab=126464, **LLADA),
        layout=SeqLayout(seq_len=8704, affix_begin=0, affix_len=8192, mask_begin=8448, mask_len=256),
        batch=32, ratio=0.2, stale="donor", decode_block=32),
}


# Small stacks for parity tests at sizes the oracle finishes in seconds.
TEST_CONFIGS: Dict[str, Workload] = {
    "mini-serve": Workload(
        name="mini-serve", seed_id=14,
        dims=ModelDims(d_model=512, n_heads=4, n_kv_heads=4, head_dim=128, d_ff=1024, n_layers=3,
                       dtype="bf16", vocab=1024),  # the LM head needs a multiple of 256 rows
        layout=SeqLayout(seq_len=330, affix_begin=0, affix_len=250, mask_begin=298, mask_len=32),
        batch=3, ratio=0.2, stale="donor", decode_block=8),
    "mini-stack": Workload(
        name="mini-stack", seed_id=11,
        dims=ModelDims(d_model=512, n_heads=4, n_kv_heads=4, head_dim=128, d_ff=1024, n_layers=3,
                       dtype="bf16", vocab=1000),
        layout=SeqLayout(seq_len=330, affix_begin=0, affix_len=250, mask_begin=298, mask_len=32),
        batch=3, ratio=0.2, stale="donor"),
    # prefix affix of whole 64-key tiles (the probe's attention hands the
    # score its affix log-sum-exp, here under key splits)
    "mini-affix64": Workload(
        name="mini-affix64", seed_id=15,
        dims=ModelDims(d_model=512, n_heads=4, n_kv_heads=2, head_dim=128, d_ff=1024, n_layers=3,
                       dtype="bf16", vocab=1000),
        layout=SeqLayout(seq_len=336, affix_begin=0, affix_len=256, mask_begin=304, mask_len=32),
        batch=3, ratio=0.2, stale="donor"),
    # infix affix of whole 64-key tiles (the probe reads the affix keys first)
    "mini-infix64": Workload(
        name="mini-infix64", seed_id=16,
        dims=ModelDims(d_model=512, n_heads=4, n_kv_heads=1, head_dim=128, d_ff=768, n_layers=3,
                       dtype="bf16", vocab=1000),
        layout=SeqLayout(seq_len=320, affix_begin=64, affix_len=192, mask_begin=288, mask_len=32),
        batch=2, ratio=0.25, stale="donor"),
    # four requests of 256 probe rows over 4352 keys, LLaDA-shaped: the probe's
    # attention takes the 256-query kernel with two key splits
    "probe-wide-split": Workload(
        name="probe-wide-split", seed_id=17,
        dims=ModelDims(n_layers=2, dtype="bf16", vocab=1024, **LLADA),
        layout=SeqLayout(seq_len=4352, affix_begin=0, affix_len=4096, mask_begin=4224, mask_len=128),
        batch=4, ratio=0.2, stale="donor"),
    "mini-gqa-infix": Workload(
        name="mini-gqa-infix", seed_id=12,
        dims=ModelDims(d_model=512, n_heads=4, n_kv_heads=1, head_dim=128, d_ff=768, n_layers=2,
                       dtype="bf16", vocab=1000),
        layout=SeqLayout(seq_len=300, affix_begin=40, affix_len=200, mask_begin=260, mask_len=40),
        batch=2, ratio=0.3, stale="donor"),
    "mini-f32-stack": Workload(
        name="mini-f32-stack", seed_id=13,
        dims=ModelDims(d_model=128, n_heads=4, n_kv_heads=2, head_dim=32, d_ff=256, n_layers=2,
                       dtype="f32", vocab=500),
        layout=SeqLayout(seq_len=150, affix_begin=20, affix_len=100, mask_begin=130, mask_len=20),
        batch=2, ratio=0.2, stale="donor"),
}


def get_config(name: str) -> Workload:
    if name in TEST_CONFIGS:
        return TEST_CONFIGS[name]
    return CONFIGS[name]
