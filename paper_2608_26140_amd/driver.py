"""Stack driver: sequences the C-ABI calls for a batch of requests that share
one affix (Sections 3.2, 3.3 and 4.1-4.3).

    probe      build_maps(k=0) -> gather_rows -> layer_recompute with scoring
               (every layer) -> topk                                 [Eq. 4-6]
    refresh    build_maps(anchors) -> gather_rows -> layer_recompute x N
    baselines  full refresh = the same calls with every affix token as an
               anchor; direct reuse = the same calls with none

Every step runs in the library's kernels; this module only allocates device
memory (torch), fills the small host-side offset arrays and issues the calls
on one stream, without synchronising.
"""

from __future__ import annotations

import contextlib
from typing import Callable, List, Optional

import numpy as np
import torch

from . import acache as A


class Model:
    """Device weights of a stack, one dict of tensors per layer
    (attn_norm, w_qkv, w_o, mlp_norm, w_gate_up, w_down)."""

    def __init__(self, dims: A.Dims, layers: List[dict]):
        self.dims = dims
        self.layers = layers
        self.lw = [A.layer_weights(w) for w in layers]

    @property
    def n_layers(self) -> int:
        return len(self.layers)

    @property
    def kv_width(self) -> int:
        return self.dims.n_kv_heads * self.dims.head_dim

    @property
    def dtype(self):
        return A.torch_dtype(self.dims)


class AffixBatch:
    """A batch of requests with one logical layout: S positions, the shared
    affix at [affix_begin, affix_begin + L), the masked span at
    [mask_begin, mask_begin + G).  Layer-0 inputs come from ``x_src`` rows,
    either indexed by b * S + position (hidden rows) or through ``remap``
    (token ids, x_src = embedding table).

    KV pools: one K and one V pool per layer, [n_slots, H_kv * d_h]
    (Section 4.1).  Flat plan (block_size None): slots [0, L) are the shared
    affix region and request b's recomputed rows use [L + b *
    private_stride, ...).  Paged plan: slots come in blocks of block_size
    from the library's block pool; the shared affix takes ceil(L / bs)
    blocks at creation (the first ones: slots [0, L) again), and each
    request a private block table of ceil(R / bs) blocks, grown when a call
    needs more rows and given back by release_private().  The pools hold
    enough blocks for the largest R the batch is built for (max_rows, else
    S: full recomputation)."""

    def __init__(self, model: Model, seq_len: int, affix_begin: int, affix_len: int, mask_begin: int,
                 mask_len: int, batch: int, x_src: torch.Tensor, remap: Optional[torch.Tensor] = None,
                 private_stride: Optional[int] = None, max_rows: Optional[int] = None, device="cuda",
                 block_size: Optional[int] = None):
        self.model = model
        self.S, self.ab, self.L = seq_len, affix_begin, affix_len
        self.mb, self.G, self.B = mask_begin, mask_len, batch
        self.stride = seq_len if private_stride is None else private_stride
        self.x_src = x_src
        self.remap = remap
        self.device = device
        self.bs = block_size
        self.table_version = 0
        r_max = seq_len if max_rows is None else max_rows
        if block_size:
            n_shared = -(-affix_len // block_size)
            self.pages = A.BlockPool(n_shared + batch * -(-r_max // block_size))
            self.shared_host = self.pages.alloc(n_shared)
            self.shared_blocks = self._i32(self.shared_host)
            self._table_host, self._table, self._table_nb = [], None, 0
            self.n_slots = self.pages.stats()["capacity"] * block_size
            j = np.arange(affix_len)
            self.affix_slots = self._i32(np.asarray(self.shared_host, dtype=np.int64)[j // block_size] * block_size
                                         + j % block_size)
        else:
            self.pages = None
            self.n_slots = affix_len + batch * self.stride
            self.affix_slots = torch.arange(affix_len, dtype=torch.int32, device=device)
        shape = (self.n_slots, model.kv_width)
        self.k_pools = [torch.zeros(shape, dtype=model.dtype, device=device) for _ in range(model.n_layers)]
        self.v_pools = [torch.zeros(shape, dtype=model.dtype, device=device) for _ in range(model.n_layers)]
        self.ws = A.workspace(model.dims, batch * r_max, batch, affix_len, device)
        self.layout = A.Layout(seq_len, affix_begin, affix_len, mask_begin, mask_len, 0, affix_len, self.stride)

    def _i32(self, a) -> torch.Tensor:
        return torch.from_numpy(np.ascontiguousarray(np.asarray(a), dtype=np.int32)).to(self.device)

    # ------------------------------------------------------------------ paging
    def private_table(self, R: int):
        """The private block table ([B * nb] device ids, nb) covering R rows
        per request; grows (new blocks, old ones returned) when R needs more."""
        nb = -(-R // self.bs)
        if nb > self._table_nb:
            self.release_private()
            self._table_host = self.pages.alloc(self.B * nb)
            self._table, self._table_nb = self._i32(self._table_host), nb
            self.table_version += 1
        return self._table, self._table_nb

    def release_private(self):
        """Give every request's private blocks back to the pool."""
        if self.pages is not None and self._table_host:
            self.pages.free(self._table_host)
            self._table_host, self._table, self._table_nb = [], None, 0
            self.table_version += 1

    def private_slots(self, R: int) -> np.ndarray:
        """[B, R] slot of request b's rank-i recomputed row (host copy)."""
        i = np.arange(R)
        if self.pages is None:
            return self.L + np.arange(self.B)[:, None] * self.stride + i[None, :]
        _, nb = self.private_table(R)
        tbl = np.asarray(self._table_host, dtype=np.int64).reshape(self.B, nb)
        return tbl[:, i // self.bs] * self.bs + i % self.bs

    def kv_bytes(self, blocks: int) -> int:
        """Bytes of K and V over every layer held by `blocks` blocks."""
        return blocks * self.bs * self.model.kv_width * 2 * self.model.n_layers * self.k_pools[0].element_size()

    # ------------------------------------------------------------------ pieces
    def anchor_count(self, ratio: float) -> int:
        """Eq. 6's K for anchor ratio `ratio` over this batch's affix."""
        return A.acache_anchor_count(ratio, self.L)

    def rows_per_request(self, k: int) -> int:
        return k + self.S - self.L

    def maps(self, anchors: Optional[torch.Tensor], k: int, stream=None, key_order: int = 0) -> dict:
        """key_order 1: each request's read slots list the affix keys first
        (the probe's order; see acache_layout.key_order)."""
        lay = self.layout
        if key_order:
            lay = A.Layout(*[getattr(lay, n) for n, _ in A.Layout._fields_])
            lay.key_order = key_order
        if self.pages is None:
            return A.acache_build_maps(lay, self.B, anchors, k, self.device, stream)
        tbl, nb = self.private_table(self.rows_per_request(k))
        return A.acache_build_maps_paged(lay, self.B, anchors, k, self.bs, self.shared_blocks, tbl, nb,
                                         self.device, stream)

    def gather_inputs(self, m: dict, stream=None) -> torch.Tensor:
        return A.acache_gather_rows(self.x_src, m["row_src"], self.remap, stream=stream)

    def request_groups(self, R: int):
        """Requests per layer call: the library addresses projection operands
        with 32-bit element offsets, so a batch whose rows times the widest
        projection input reach 2^31 elements runs in groups of requests."""
        d = self.model.dims
        widest = max(d.d_model, d.n_heads * d.head_dim, d.d_ff)
        per = max(1, ((1 << 31) - 1) // max(1, R * widest))
        return [(b0, min(self.B, b0 + per)) for b0 in range(0, self.B, per)]

    def run_layers(self, x: torch.Tensor, m: dict, k: int, score: Optional[dict] = None,
                   drop_non_anchor: bool = False, upto: Optional[int] = None, score_last_only: bool = False,
                   stream=None, layer_hook: Optional[Callable[[int, torch.Tensor], None]] = None):
        """drop_non_anchor: attention reads only the recomputed rows (DropNA,
        Section 5.3): their write slots serve as the read slots, R keys per
        request, and the non-anchor affix entries are never read.
        score_last_only: the last layer only adds its score (acache_layer_score)
        and x is left at the last layer's input.
        layer_hook(n, x): called on the host before layer n's launches are
        issued (x then holds layer n's input in stream order), and once more
        with n = the number of layers run after the last one; for inspection,
        e.g. copies of the rows on the same stream."""
        R = self.rows_per_request(k)
        groups = self.request_groups(R)
        read, nk = (m["write_slots"], R) if drop_non_anchor else (m["read_slots"], self.S)
        if score is not None and len(groups) > 1:
            raise ValueError("probe batch too large for one call")
        n_run = self.model.n_layers if upto is None else min(upto, self.model.n_layers)
        for n in range(n_run):
            if layer_hook is not None:
                layer_hook(n, x)
            layer = A.acache_layer_recompute
            if score is not None and score_last_only and n == self.model.n_layers - 1:
                layer = A.acache_layer_score
            for b0, b1 in groups:
                nb = b1 - b0
                cu_rows = [b * R for b in range(nb + 1)]
                cu_keys = [b * nk for b in range(nb + 1)]
                rows = slice(b0 * R, b1 * R)
                sc = score if score is None or n == 0 else dict(score, init=0)
                layer(self.model.dims, self.model.lw[n], cu_rows, cu_keys, x[rows], m["row_pos"][rows],
                      m["write_slots"][rows], read[b0 * nk:b1 * nk], self.k_pools[n], self.v_pools[n], self.ws,
                      score=sc, stream=stream)
        if layer_hook is not None:
            layer_hook(n_run, x)
        return x

    # ------------------------------------------------------------------ the method
    def materialize_affix(self, donor_x: torch.Tensor, donor_pos: torch.Tensor, write_slots: torch.Tensor,
                          read_slots: torch.Tensor, stream=None) -> torch.Tensor:
        """Materialise the shared affix cache once (Sections 3.3, 4.2): a full
        forward of a donor sequence whose affix rows write to the shared slots.
        donor_x [n, d] layer-0 inputs (consumed), donor_pos / write_slots [n],
        read_slots [n_keys] (the donor's logical view)."""
        n = donor_x.shape[0]
        for i in range(self.model.n_layers):
            A.acache_layer_recompute(self.model.dims, self.model.lw[i], [0, n], [0, read_slots.numel()], donor_x,
                                     donor_pos, write_slots, read_slots, self.k_pools[i], self.v_pools[i], self.ws,
                                     stream=stream)
        return donor_x

    def shift_affix(self, delta: int, stream=None):
        """Reuse the shared affix cache delta positions from where it was
        materialised: its K rows are re-rotated in place at every layer."""
        slots = self.affix_slots
        d = torch.full((self.L,), int(delta), dtype=torch.int32, device=self.device)
        for k in self.k_pools:
            A.acache_rerotate_k(self.model.dims, k, slots, k, slots, d, stream=stream)

    def probe(self, norm: int = A.ACACHE_NORM_AFFIX, stream=None, outputs: bool = True, layer_hook=None,
              attention_lse: bool = True):
        """One-shot probe (Section 3.2): forward the non-affix rows against the
        fixed shared affix cache and accumulate Eq. 5 over layers.  Returns
        (scores [B, L] fp32, x rows, maps).  outputs=False: the last layer
        computes only what its score reads (acache_layer_score), and the
        returned x is None.  layer_hook(n, x, scores): as run_layers', with
        the score buffer (its sum over the layers before n).  attention_lse:
        the keys are read affix first, so that a layer's attention takes the
        affix log-sum-exp for its score (False: keys in logical order, and
        the score makes its own pass over the affix keys)."""
        m = self.maps(None, 0, stream, key_order=1 if attention_lse else 0)
        x = self.gather_inputs(m, stream)
        # the first layer writes the scores (init) and the others add to them;
        # with no masked rows no layer scores, and they stay zero
        if self.G > 0:
            scores = torch.empty((self.B, self.L), dtype=torch.float32, device=self.device)
        else:
            scores = torch.zeros((self.B, self.L), dtype=torch.float32, device=self.device)
        # with no anchors and the affix first, every request reads its affix
        # keys, in order, through the shared slots from key index 0: the
        # attention may take their log-sum-exp for the score
        score = dict(q_rows=m["q_rows"], cu_q=[b * self.G for b in range(self.B + 1)],
                     affix_slots=self.affix_slots, scores=scores, norm=norm, init=int(self.G > 0))
        if attention_lse:
            score["affix_key_begin"] = 0
        hook = None if layer_hook is None else (lambda n, xx: layer_hook(n, xx, scores))
        self.run_layers(x, m, 0, score=score, score_last_only=not outputs, stream=stream, layer_hook=hook)
        return scores, (x if outputs else None), m

    def select_anchors(self, k: int, norm: int = A.ACACHE_NORM_AFFIX, stream=None, full_probe: bool = False):
        """Probe then Eq. 6.  Returns (anchors [B, k] int32 ascending, scores).
        The probe's last layer stops at its score unless full_probe."""
        scores, _, _ = self.probe(norm, stream, outputs=full_probe)
        if k == 0:
            return torch.empty((self.B, 0), dtype=torch.int32, device=self.device), scores
        return A.acache_topk(scores, k, stream=stream), scores

    def select_anchors_hkvd(self, k: int, stream=None):
        """The CacheBlend-style selector (KV deviation) in place of Eq. 4-5:
        a full-prompt forward of every request through the selection layer
        (the first whose affix K/V depend on context), then each affix
        token's squared K/V deviation from the shared cache, then Eq. 6's
        top-K.  Returns (anchors [B, k], scores [B, L])."""
        n = min(1, self.model.n_layers - 1)
        every = torch.arange(self.L, dtype=torch.int32, device=self.device).repeat(self.B, 1).contiguous()
        m = self.maps(every, self.L, stream)
        x = self.gather_inputs(m, stream)
        self.run_layers(x, m, self.L, upto=n + 1, stream=stream)
        fresh = m["write_slots"].view(self.B, self.S)[:, self.ab:self.ab + self.L]
        scores = A.acache_kv_deviation(self.model.dims, self.k_pools[n], self.v_pools[n], fresh, self.affix_slots,
                                       stream=stream)
        if k == 0:
            return torch.empty((self.B, 0), dtype=torch.int32, device=self.device), scores
        return A.acache_topk(scores, k, stream=stream), scores

    def refresh(self, anchors: Optional[torch.Tensor], k: int, drop_non_anchor: bool = False, stream=None,
                layer_hook=None):
        """Selective recomputation (Section 3.3): anchors plus every
        request-specific row through all layers; with drop_non_anchor the
        DropNA ablation (Section 5.3).  Returns (x rows [B*R, d], maps)."""
        m = self.maps(anchors, k, stream)
        x = self.gather_inputs(m, stream)
        self.run_layers(x, m, k, drop_non_anchor=drop_non_anchor, stream=stream, layer_hook=layer_hook)
        return x, m

    def full_refresh(self, stream=None):
        every = torch.arange(self.L, dtype=torch.int32, device=self.device).repeat(self.B, 1).contiguous()
        return self.refresh(every, self.L, stream)

    def direct_reuse(self, stream=None):
        return self.refresh(None, 0, stream)


class Head:
    """Final RMSNorm gain [d] and LM head [vocab, d] for the decode schedule."""

    def __init__(self, norm_g: torch.Tensor, w: torch.Tensor):
        self.norm_g = norm_g
        self.w = w


def block_row_index(batch: AffixBatch, k: int, block_begin: int, block_len: int) -> torch.Tensor:
    """Rows of the refresh output (k anchors per request) that hold logical
    positions [block_begin, block_begin + block_len) of every request.  A
    request's rows are its anchors then its non-affix positions, each in
    ascending order; the block lies in the masked span, after the affix."""
    S, ab, L, B = batch.S, batch.ab, batch.L, batch.B
    assert block_begin >= ab + L, "the generation block follows the affix"
    nonaffix = np.concatenate([np.arange(0, ab), np.arange(ab + L, S)])
    R = batch.rows_per_request(k)
    local = k + np.searchsorted(nonaffix, np.arange(block_begin, block_begin + block_len))
    rows = (np.arange(B)[:, None] * R + local[None, :]).reshape(-1)
    return torch.from_numpy(rows.astype(np.int32)).to(batch.device)


class DecodePlan:
    """Index arrays of the decode schedule, built on the host once: for each
    block, the refresh-output rows holding it and the token-id positions its
    commits go to."""

    def __init__(self, batch: AffixBatch, k: int, block_len: int, n_blocks: int, full: bool):
        import numpy as np
        B, S, dev = batch.B, batch.S, batch.device
        self.full, self.block_len, self.n_blocks = full, block_len, n_blocks
        self.k = batch.L if full else k
        self.anchors = (torch.arange(batch.L, dtype=torch.int32, device=dev).repeat(B, 1).contiguous()
                        if full else None)
        self.rows, self.pos, self.row_pos, self.local = [], [], [], []
        nonaffix = np.concatenate([np.arange(0, batch.ab), np.arange(batch.ab + batch.L, S)])
        i32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)
        for blk in range(n_blocks):
            p0 = batch.mb + blk * block_len
            self.rows.append(block_row_index(batch, self.k, p0, block_len))
            p = np.arange(p0, p0 + block_len)
            self.pos.append(i32((np.arange(B)[:, None] * S + p[None, :]).reshape(-1)))
            self.row_pos.append(i32(np.tile(p, B)))
            self.local.append(self.k + np.searchsorted(nonaffix, p))  # the rows' ranks in a request
        self._slots, self._version = None, None

    def write_slots(self, batch: AffixBatch, blk: int) -> torch.Tensor:
        """[B * block_len] private slots of block blk's rows: the slots their
        refresh rows wrote (Section 4.1), which the block keeps while it
        decodes.  Rebuilt when the batch's slot plan has changed."""
        if self._version != batch.table_version or self._slots is None:
            slots = batch.private_slots(batch.rows_per_request(self.k))
            self._slots = [torch.from_numpy(np.ascontiguousarray(slots[:, loc].reshape(-1), dtype=np.int32))
                           .to(batch.device) for loc in self.local]
            self._version = batch.table_version
        return self._slots[blk]


def decode_schedule(batch: AffixBatch, head: Head, plan: DecodePlan, k: int, logits: torch.Tensor,
                    committed: torch.Tensor, anchors: Optional[torch.Tensor] = None, stream=None):
    """The serving schedule over the masked span (Sections 3.1 and 4.3): one
    probe and top-K per request (selective mode), then per block a refresh
    (selective, or full recomputation), the final norm and LM head on the
    block's rows, and a greedy commit of every position of the block into the
    token ids the next refresh embeds.  committed [n_blocks, B * block_len]
    receives the chosen ids; logits [B * block_len, vocab] is scratch.
    anchors: a given anchor set [B, k] instead of the probe's (selective)."""
    if plan.full:
        anchors = plan.anchors
    elif anchors is None:
        anchors, _ = batch.select_anchors(k, stream=stream)
    for blk in range(plan.n_blocks):
        x, _ = batch.refresh(anchors, plan.k, stream=stream)
        h = A.acache_gather_rows(x, plan.rows[blk], stream=stream)
        y = A.acache_rmsnorm(batch.model.dims, h, head.norm_g, stream=stream)
        A.acache_linear(batch.model.dims, y, head.w, out=logits, ws=batch.ws, stream=stream)
        A.acache_argmax_commit(logits, out=committed[blk], commit_pos=plan.pos[blk], ids=batch.remap,
                               stream=stream)
    return committed


def capture(fn, warmup: int = 2):
    """Records the launches of fn() (the library's kernels, torch's fills and
    allocations) into a HIP graph: warmup calls on a side stream, then one
    call under capture.  Returns (graph, fn's outputs); graph.replay() reruns
    every launch with the same buffers and arguments, and rewrites the same
    output tensors.  fn must not synchronise with the host, and the library's
    kernel timer must not be armed while it is captured."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(warmup):
            fn()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        out = fn()
    return g, out


def _on(stream):
    """torch's own copies and fills go to the stream the library calls use."""
    return torch.cuda.stream(stream) if stream is not None else contextlib.nullcontext()


def decode_step(batch: AffixBatch, plan: DecodePlan, blk: int, m: dict, anchors: Optional[torch.Tensor] = None,
                split_shared: bool = True, stream=None):
    """One decoding step of block ``blk`` (Section 4.3, Appendix C.1): the
    block's rows, embedded from the current token ids, go through every
    layer with queries for those rows only; each layer writes their fresh
    K/V to the rows' private slots, then attention reads each request's
    whole logical context, the view the refresh (maps ``m``, anchor set
    ``anchors``) left.  With split_shared (bf16) the view is read as the
    shared affix minus the anchors, taken for all requests together, plus
    each request's private slots (acache_layer_decode); otherwise through
    the read-slot map.  Returns the block's last-layer rows [B * block_len, d]."""
    B, blen = batch.B, plan.block_len
    h = A.acache_gather_rows(batch.x_src, plan.pos[blk], batch.remap, stream=stream)
    wslots = plan.write_slots(batch, blk)
    k = plan.k
    if split_shared and batch.model.dims.dtype == A.ACACHE_BF16:
        R = batch.rows_per_request(k)
        anc = plan.anchors if plan.full else anchors
        if anc is None and k > 0:
            raise ValueError("the shared/private split needs the refresh's anchor set")
        for i in range(batch.model.n_layers):
            A.acache_layer_decode(batch.model.dims, batch.model.lw[i], B, blen, h, plan.row_pos[blk], wslots,
                                  batch.affix_slots, anc, k, m["write_slots"], R, batch.k_pools[i],
                                  batch.v_pools[i], batch.ws, stream=stream)
        return h
    cu_rows = [b * blen for b in range(B + 1)]
    cu_keys = [b * batch.S for b in range(B + 1)]
    for i in range(batch.model.n_layers):
        A.acache_layer_recompute(batch.model.dims, batch.model.lw[i], cu_rows, cu_keys, h, plan.row_pos[blk],
                                 wslots, m["read_slots"], batch.k_pools[i], batch.v_pools[i], batch.ws,
                                 stream=stream)
    return h


def decode_threshold_schedule(batch: AffixBatch, head: Head, plan: DecodePlan, k: int, tau: float,
                              anchors: Optional[torch.Tensor] = None, trace: Optional[list] = None,
                              max_steps: Optional[int] = None, stream=None):
    """Block-wise decoding with confidence-threshold commits (Sections 3.1,
    4.3, 5).  Per block: a refresh (selective, or full recomputation) whose
    block rows give the first predictions; then, until every position of the
    block is committed, decode steps that form queries for the block's rows
    only, write their fresh K/V to the rows' private slots and attend over the
    refresh's read-slot view, each followed by the final norm, the LM head
    and a commit of every uncommitted position with confidence >= tau (or
    the single most confident one).  Commits land in the token ids
    (``batch.remap``) that the next step and the next refresh embed; that is
    where the caller reads the generated tokens.

    The batch steps together: a request whose block is done commits nothing
    until the rest are.  The host reads the per-request commit counts after
    each step (one synchronisation) to know when the block is done.
    trace: if a list, receives per step a dict of host copies (block,
    logits, pick, conf, committed flags).  Returns the number of steps
    (commits) each block took; every step commits at least one position of
    each request whose block is not done, so a block takes at most
    block_len steps.  max_steps ends a block early (for measurement): its
    positions not yet committed keep the mask id."""
    if batch.remap is None:
        raise ValueError("decode steps embed token ids: the batch needs remap")
    B, blen, dev = batch.B, plan.block_len, batch.device
    dims = batch.model.dims
    if plan.full:
        anchors = plan.anchors
    elif anchors is None:
        anchors, _ = batch.select_anchors(k, stream=stream)
    n = B * blen
    logits = torch.empty((n, head.w.shape[0]), dtype=batch.model.dtype, device=dev)
    pick = torch.empty(n, dtype=torch.int32, device=dev)
    conf = torch.empty(n, dtype=torch.float32, device=dev)
    flags = torch.empty(n, dtype=torch.int32, device=dev)
    count = torch.empty(B, dtype=torch.int32, device=dev)
    count_host = torch.empty(B, dtype=torch.int32, pin_memory=True)
    steps = []
    for blk in range(plan.n_blocks):
        x, m = batch.refresh(anchors, plan.k, stream=stream)
        h = A.acache_gather_rows(x, plan.rows[blk], stream=stream)
        with _on(stream):
            flags.zero_()
        done, step = 0, 0
        while True:
            y = A.acache_rmsnorm(dims, h, head.norm_g, stream=stream)
            A.acache_linear(dims, y, head.w, out=logits, ws=batch.ws, stream=stream)
            A.acache_argmax_commit(logits, out=pick, conf=conf, stream=stream)
            A.acache_threshold_commit(blen, pick, conf, tau, flags, plan.pos[blk], batch.remap, count,
                                      stream=stream)
            with _on(stream):
                count_host.copy_(count, non_blocking=True)
            (stream if stream is not None else torch.cuda.current_stream()).synchronize()
            if trace is not None:
                trace.append(dict(block=blk, logits=logits.float().cpu().numpy(), pick=pick.cpu().numpy(),
                                  conf=conf.cpu().numpy(), committed=flags.cpu().numpy()))
            done += int(count_host.sum())
            step += 1
            if done >= n or (max_steps is not None and step >= max_steps):
                break
            h = decode_step(batch, plan, blk, m, anchors, stream=stream)
        steps.append(step)
    return steps
