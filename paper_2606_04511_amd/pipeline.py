"""Offloaded decode across layers with one-layer-ahead selection (paper Sec. 4.1 and 4.3, Alg. 2).

Per decode step and layer l (the model's projections and FFN are outside this path):
  * compute stream: select layer l+1's blocks from layer l's Forecast rows and layer l+1's
    compressed keys (Eq. 4); record `selected[l+1]`;
  * side stream: wait for `selected[l+1]` and for the attention that last read the staging
    slot about to be overwritten, then gather layer l+1's selected K/V blocks from its pinned
    host pool into that staging slot (`sparda_gather_blocks`); record `gathered[l+1]`;
  * compute stream: wait for `gathered[l]` (launched during layer l-1) and attend layer l from
    its staging slot.
Layer 0 keeps its KV cache in HBM and selects with its current-layer Forecast (Sec. 4.1).  Two
staging slots alternate between layers.  All device buffers are allocated up front; a step
allocates nothing.

Alg. 2 appends each decoded token's K/V to the cache.  Given the token's K/V per layer (new_kv),
a step appends it to layer 0's HBM cache; in an offloaded layer, whose blocks were gathered during
layer l-1 before the token existed, it writes the token into the staged copy of its own block
(`sparda_stage_append_kv`) before the attention, and after the attention stores it into the
layer's host pool on the side stream (`sparda_writeback_kv`, the asynchronous CPU write-back of
new KV entries of Sec. 5.3), where the stream order puts it before the next step's gathers.  A
compressed key that the token completes is computed from the cache (Alg. 2's incremental K~
update; for an offloaded layer from its host pool, after the write-back), and the next step's
selection of that layer waits for it.

With reuse=True each offloaded layer keeps its own staging buffer across decode steps (the NOSI
engine of the paper's efficiency setup, App. C): after layer l+1's selection,
`sparda_plan_staging` keeps the staged blocks that the new set still attends and that hold every
token up to the query, and the gather copies only the newly selected blocks (plus the open local
block, whose newest tokens arrived since the last copy).  The attention then reads the per-slot
block list the plan wrote.  This costs one staging buffer per offloaded layer instead of two in
total (2 B Hkv k 64 D bytes per layer: 1.07 GB at B64, 8 KV heads, k = 64).
"""
from __future__ import annotations

import math

import torch

from . import hostmem
from . import sparda as sp


def gather_workgroups(batch: int) -> int:
    """Persistent gather workgroups for a decode step at this batch size (the batch-adaptive CTA
    budget of Sec. 4.3 / App. D): the smallest count that reaches the host link's rate.  Measured
    on MI355X at 32K with 8 KV heads and k = 64, from B8 to B64: 4 workgroups move 37.3-37.7 GB/s,
    8 move 54.9-56.9 GB/s and 16-64 move 55.8-57.3 GB/s, while a concurrent decode attention slows
    more as the count grows (at B64: 186 us alone, 256 us beside 8 workgroups, 380 us beside 32).
    Unlike the H100 heuristic (16 CTAs below B32, 32 above), the link saturates at the same small
    count at every batch size here, so the budget stays at 8."""
    if batch < 1:
        raise ValueError("batch must be >= 1")
    return 8


class DecodePipeline:
    """L layers of one decode step.

    shape        -- sparda shape of one layer (batch, heads, k_total, t_cap, nc_cap ...)
    t_ctx        -- tokens in the context; the query sits at position t_ctx - 1
    q[l]         -- bf16 [B][Hq][1][D] device, query of layer l
    f[l]         -- bf16 [B][Hkv][1][D] device, Forecast rows of layer l (scores layer l+1)
    f0_cur       -- bf16 [B][Hkv][1][D] device, layer 0's current-layer Forecast
    kc[l]        -- bf16 [B][Hkv][nc_cap][D] device, compressed keys of layer l
    k0, v0       -- bf16 [B][Hkv][t_cap][D] device, layer 0's KV cache
    pools[l]     -- (host_k_ptr, host_v_ptr) of layer l (l >= 1): device-mapped pinned memory
                    laid out [B][Hkv][t_cap][D]; pools may be shared between layers (only when
                    steps write nothing back: a write-back goes to the layer's pool)
    n_workgroups -- persistent-grid size of the gather (its CU budget); None takes
                    gather_workgroups(batch)
    """

    def __init__(self, shape: sp.SpardaShape, t_ctx: int, q, f, f0_cur, kc, k0, v0, pools,
                 n_workgroups: int | None, device, sm_scale: float | None = None, reuse: bool = False):
        L = len(q)
        assert len(f) == L and len(kc) == L and len(pools) == L and L >= 1
        self.shape, self.t_ctx, self.L = shape, t_ctx, L
        self.q, self.f, self.f0_cur, self.kc, self.k0, self.v0, self.pools = q, f, f0_cur, kc, k0, v0, pools
        self.n_workgroups = gather_workgroups(shape.batch) if n_workgroups is None else n_workgroups
        self.scale = 1.0 / math.sqrt(shape.head_dim) if sm_scale is None else sm_scale
        B, H, K = shape.batch, shape.n_kv_heads, shape.k_total
        self.sel = [torch.empty(B, H, 1, K, dtype=torch.int16, device=device) for _ in range(L)]
        self.cnt = [torch.empty(B, H, 1, dtype=torch.int16, device=device) for _ in range(L)]
        self.o = [torch.empty(B, shape.n_q_heads, 1, shape.head_dim, dtype=torch.bfloat16, device=device)
                  for _ in range(L)]
        st = (B, H, K, shape.block_size, shape.head_dim)
        self.reuse = reuse
        n_stage = L if reuse else 2
        self.stage = [(torch.empty(st, dtype=torch.bfloat16, device=device),
                       torch.empty(st, dtype=torch.bfloat16, device=device)) if (not reuse or i >= 1) else None
                      for i in range(n_stage)]
        if reuse:
            i16 = dict(dtype=torch.int16, device=device)
            self.slot_blk = [torch.full((B, H, K), -1, **i16) for _ in range(L)]
            self.slot_len = [torch.zeros((B, H, K), **i16) for _ in range(L)]
            self.fetch = [torch.empty((B, H, K), **i16) for _ in range(L)]
            self.sel_staged = [torch.empty((B, H, K), **i16) for _ in range(L)]
            self.stage_cnt = [torch.empty((B, H), **i16) for _ in range(L)]
            self.n_fetch = [torch.zeros((B, H), dtype=torch.int32, device=device) for _ in range(L)]
        n_sel = sp.sparda_workspace_size(shape, sp.SPARDA_OP_FORECAST_SELECT, 1, t_ctx - 1)
        n_att = sp.sparda_workspace_size(shape, sp.SPARDA_OP_SPARSE_ATTN, 1, t_ctx - 1)
        self.ws_sel = torch.empty(max(n_sel, 16), dtype=torch.uint8, device=device)
        self.ws_att = torch.empty(max(n_att, 16), dtype=torch.uint8, device=device)
        self.side = torch.cuda.Stream(device=device)
        self.pool_dev = [None] + [(hostmem.device_pointer(hk), hostmem.device_pointer(hv)) for hk, hv in pools[1:]]
        self.ev_kc = [torch.cuda.Event() for _ in range(L)]
        self.kc_pending = [False] * L
        self.ev_sel = [torch.cuda.Event() for _ in range(L)]
        self.ev_gather = [torch.cuda.Event() for _ in range(L)]
        self.ev_attn = [torch.cuda.Event() for _ in range(L)]

    def _select(self, f_rows, layer):
        if self.kc_pending[layer]:  # a compressed key completed by the last token is being written
            torch.cuda.current_stream().wait_event(self.ev_kc[layer])
            self.kc_pending[layer] = False
        sp.sparda_forecast_select(self.shape, f_rows, 1, self.t_ctx - 1, self.kc[layer], self.sel[layer],
                                  self.cnt[layer], self.ws_sel)
        if self.reuse and layer >= 1:
            sp.sparda_plan_staging(self.shape, self.sel[layer].view(self.shape.batch, self.shape.n_kv_heads, -1),
                                   self.cnt[layer], self.t_ctx - 1, self.slot_blk[layer], self.slot_len[layer],
                                   self.fetch[layer], self.sel_staged[layer], self.stage_cnt[layer],
                                   self.n_fetch[layer])

    def _gather(self, layer, stream):
        hk, hv = self.pools[layer]
        if self.reuse:
            sk, sv = self.stage[layer]
            sp.sparda_gather_blocks(self.shape, hk, hv, self.fetch[layer], self.stage_cnt[layer], sk, sv,
                                    self.n_workgroups, stream)
            return
        sk, sv = self.stage[layer % 2]
        sp.sparda_gather_blocks(self.shape, hk, hv, self.sel[layer], self.cnt[layer], sk, sv, self.n_workgroups,
                                stream)

    def _attend(self, layer):
        sel, cnt = self.sel[layer], self.cnt[layer]
        if layer == 0:
            k, v, mode = self.k0, self.v0, 0
        elif self.reuse:
            (k, v), mode = self.stage[layer], 1
            sel, cnt = self.sel_staged[layer], self.stage_cnt[layer]
        else:
            k, v = self.stage[layer % 2]
            mode = 1
        sp.sparda_sparse_attn(self.shape, self.q[layer], 1, self.t_ctx - 1, k, v, mode, sel, cnt, self.scale,
                              self.o[layer], self.ws_att)

    def _new_windows(self, p):
        """Compressed keys [begin, end) that the token at position p completes."""
        lw, sw = self.shape.cmp_kernel, self.shape.cmp_stride
        last = (p + 1 - lw) // sw if p + 1 >= lw else -1
        prev = (p - lw) // sw if p >= lw else -1
        return prev + 1, last + 1

    def _append_layer0(self, k_new, v_new, p):
        """Alg. 2's append on the HBM-resident layer 0 (a device copy into its cache), then the
        compressed keys the token completes."""
        self.k0[:, :, p].copy_(k_new[:, :, 0])
        self.v0[:, :, p].copy_(v_new[:, :, 0])
        w0, w1 = self._new_windows(p)
        if w1 > w0:
            sp.sparda_compress_keys(self.shape, self.k0, p + 1, w0, w1, self.kc[0])

    def _staging_of(self, layer):
        if self.reuse:
            return self.stage[layer], self.sel_staged[layer], self.stage_cnt[layer]
        return self.stage[layer % 2], self.sel[layer], self.cnt[layer]

    def _writeback(self, layer, k_new, v_new, p, stream):
        """The token into the layer's host pool (Sec. 5.3's asynchronous write-back), then the
        compressed keys it completes, read from the pool; ev_kc[layer] marks the end."""
        hk, hv = self.pools[layer]
        sp.sparda_writeback_kv(self.shape, k_new, v_new, 1, p, hk, hv, self.n_workgroups, stream)
        w0, w1 = self._new_windows(p)
        if w1 > w0:
            sp.sparda_compress_keys(self.shape, self.pool_dev[layer][0], p + 1, w0, w1, self.kc[layer], stream)
            self.ev_kc[layer].record(stream)
            self.kc_pending[layer] = True

    def fetched_blocks(self) -> int:
        """Blocks the last step's gathers copied (reuse mode; synchronises)."""
        return int(sum(int(n.sum().item()) for n in self.n_fetch[1:]))

    def step(self, overlap: bool = True, t_ctx: int | None = None, new_kv=None):
        """Enqueue one decode step over all layers on the current stream (and the side stream).
        overlap=False runs each gather (and write-back) on the compute stream right before (after)
        its attention.  t_ctx moves the query to position t_ctx - 1 (the workspaces were sized for
        the first t_ctx and the positions of one decode run stay within the same workspace needs).
        new_kv[l] = (k_new, v_new), bf16 [B][Hkv][1][D] device: the decoded token's K/V of layer l
        at position t_ctx - 1, appended as the class docstring describes; None leaves the caches
        and host pools as they are (they must then already hold the token)."""
        if t_ctx is not None:
            self.t_ctx = t_ctx
        p = self.t_ctx - 1
        comp = torch.cuda.current_stream()
        if new_kv is not None:
            self._append_layer0(new_kv[0][0], new_kv[0][1], p)
        self._select(self.f0_cur, 0)
        for l in range(self.L):
            if l + 1 < self.L:
                self._select(self.f[l], l + 1)
                if overlap:
                    self.ev_sel[l + 1].record(comp)
                    self.side.wait_event(self.ev_sel[l + 1])
                    if l >= 1 and not self.reuse:  # the slot of layer l+1 was last read by layer l-1
                        self.side.wait_event(self.ev_attn[l - 1])
                    self._gather(l + 1, self.side)
                    self.ev_gather[l + 1].record(self.side)
            if l >= 1:
                if overlap:
                    comp.wait_event(self.ev_gather[l])
                else:
                    self._gather(l, comp)
                if new_kv is not None:
                    (sk, sv), ssel, scnt = self._staging_of(l)
                    sp.sparda_stage_append_kv(self.shape, new_kv[l][0], new_kv[l][1], p, ssel, scnt, sk, sv)
            self._attend(l)
            self.ev_attn[l].record(comp)
            if l >= 1 and new_kv is not None:
                if overlap:
                    self.side.wait_event(self.ev_attn[l])
                    self._writeback(l, new_kv[l][0], new_kv[l][1], p, self.side)
                else:
                    self._writeback(l, new_kv[l][0], new_kv[l][1], p, comp)
        return self.o
