"""GPU tests of the offloaded decode pipeline (one-layer-ahead selection + side-stream gather).

The oracle chain follows the paper: S_0 = select(F_0^cur, K~_0); S_{l+1} = select(F_l, K~_{l+1});
O_l = attend(Q_l, K_l, V_l, S_l), with layers >= 1 reading their KV from pinned host pools that
two layers share.  The race checks poison the staging buffers with NaN and hold the side stream
back with a bounded spin before each gather: correct event ordering must still give the oracle's
output, and a copy of the pipeline that drops the compute stream's wait must be caught.
"""
import math
import sys
import time

import numpy as np
import pytest
import torch

import oracle
import paper_2606_04511_amd.sparda as sp
from paper_2606_04511_amd import hostmem, inputs
from paper_2606_04511_amd.pipeline import DecodePipeline
from parity import abs_bits, compare_attention, compare_selection

pytestmark = pytest.mark.gpu

B, H, G, T, K, L, P = 2, 2, 4, 8192, 16, 4, 2
NB = T // 64


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def setup():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    sp.load()
    dev = torch.device("cuda:0")
    shape = sp.SpardaShape(batch=B, n_kv_heads=H, group_size=G, k_total=K, t_cap=T, nc_cap=NB)
    oshape = oracle.Shape(batch=B, n_kv_heads=H, group_size=G, k_total=K, t_cap=T, nc_cap=NB)
    w = inputs.Workload("pipe", batch=B, seq_len=T, n_q=1, n_kv_heads=H, group_size=G, k_total=K, seed=6000)
    q = [inputs.normal_bf16((B, H * G, 1, 128), 6000, 10 + l) for l in range(L)]
    f = [inputs.normal_bf16((B, H, 1, 128), 6000, 50 + l) for l in range(L)]
    f0 = inputs.normal_bf16((B, H, 1, 128), 6000, 99)
    kv = []  # kv[0] is layer 0 (HBM); kv[1 + p] is host pool p
    for i in range(1 + P):
        kv.append((inputs.keys_with_plants(w, f0[:, :, 0] if i == 0 else f[i - 1][:, :, 0], T, tensor_id=200 + i),
                   inputs.values(w, T, tensor_id=300 + i)))
    pools, bufs = [], []
    for p in range(P):
        hk = hostmem.PinnedBuffer(kv[1 + p][0].numel() * 2)
        hv = hostmem.PinnedBuffer(kv[1 + p][1].numel() * 2)
        hk.as_tensor(torch.bfloat16).copy_(kv[1 + p][0].reshape(-1))
        hv.as_tensor(torch.bfloat16).copy_(kv[1 + p][1].reshape(-1))
        bufs += [hk, hv]
        pools.append((hk.ptr, hv.ptr))
    layer_kv = [kv[0]] + [kv[1 + (l - 1) % P] for l in range(1, L)]
    layer_pool = [None] + [pools[(l - 1) % P] for l in range(1, L)]
    kc_ref = [oracle.compress_keys(oshape, inputs.to_u16(layer_kv[l][0]), T, 0, NB) for l in range(L)]
    kc = []
    for l in range(L):
        t = torch.zeros(B, H, NB, 128, dtype=torch.bfloat16, device=dev)
        sp.sparda_compress_keys(shape, layer_kv[l][0].to(dev), T, 0, NB, t)
        kc.append(t)
    torch.cuda.synchronize()
    for l in range(L):
        assert np.array_equal(inputs.to_u16(kc[l]), kc_ref[l])
    pipe_args = dict(shape=shape, t_ctx=T, q=[x.to(dev) for x in q], f=[x.to(dev) for x in f], f0_cur=f0.to(dev),
                     kc=kc, k0=kv[0][0].to(dev), v0=kv[0][1].to(dev), pools=layer_pool, n_workgroups=16,
                     device=dev)
    # the oracle chain
    ref_sel, ref_out, ref_w = [], [], []
    for l in range(L):
        frows = f0 if l == 0 else f[l - 1]
        s, c = oracle.forecast_select(oshape, inputs.to_u16(frows), 1, T - 1, kc_ref[l])
        ref_sel.append((s, c, frows))
        args = (oshape, inputs.to_u16(q[l]), 1, T - 1, inputs.to_u16(layer_kv[l][0]))
        v16 = inputs.to_u16(layer_kv[l][1])
        ref_out.append(oracle.sparse_attn(*args, v16, 0, s, c, 1.0 / math.sqrt(128)))
        ref_w.append(oracle.sparse_attn(*args, abs_bits(v16), 0, s, c, 1.0 / math.sqrt(128)))
    return dict(dev=dev, oshape=oshape, pipe_args=pipe_args, ref_sel=ref_sel, ref_out=ref_out, ref_w=ref_w,
                kc_ref=kc_ref, bufs=bufs)


def check(setup, pipe):
    torch.cuda.synchronize()
    for l in range(L):
        s, c, frows = setup["ref_sel"][l]
        gs, gc = pipe.sel[l].cpu().numpy(), pipe.cnt[l].cpu().numpy()
        compare_selection(setup["oshape"], inputs.to_u16(frows), setup["kc_ref"][l], 1, T - 1, gs, gc,
                          [(b, m, 0) for b in range(B) for m in range(H)])
        same = np.array_equal(gs, s)
        assert same, f"layer {l}: selection differs within the tie window; pick another seed"
        compare_attention(pipe.o[l].float().cpu().numpy(), setup["ref_out"][l], f"layer {l}", setup["ref_w"][l])


@pytest.mark.parametrize("overlap", [True, False])
def test_pipeline_matches_oracle_chain(setup, overlap):
    say(f"pipeline overlap={overlap}")
    pipe = DecodePipeline(**setup["pipe_args"])
    for _ in range(2):  # a second step reuses the staging slots and events
        pipe.step(overlap=overlap)
    check(setup, pipe)


class _DelayedGather(DecodePipeline):
    """Holds the side stream back (bounded spin) before every gather."""

    delay_cycles = 2_000_000

    def _gather(self, layer, stream):
        with torch.cuda.stream(stream):
            torch.cuda._sleep(self.delay_cycles)
        super()._gather(layer, stream)


class _NoWait(_DelayedGather):
    """A broken copy: the compute stream never waits for the gathers.  Its gathers are held back
    long enough (50M cycles, about 20 ms) that the compute stream's next layers have run before
    them, whatever else the GPU was doing before the test."""

    delay_cycles = 50_000_000

    def step(self, overlap=True):
        saved = torch.cuda.Stream.wait_event
        comp = torch.cuda.current_stream()

        def skip_compute_waits(stream, event):
            if stream == comp:
                return None
            return saved(stream, event)

        torch.cuda.Stream.wait_event = skip_compute_waits
        try:
            return super().step(overlap=True)
        finally:
            torch.cuda.Stream.wait_event = saved


def test_pipeline_event_ordering_with_delayed_side_stream(setup):
    say("pipeline race check")
    pipe = _DelayedGather(**setup["pipe_args"])
    for sk, sv in pipe.stage:
        sk.fill_(float("nan"))
        sv.fill_(float("nan"))
    torch.cuda.synchronize()
    pipe.step()
    check(setup, pipe)


def test_dropped_wait_is_detected(setup):
    """A copy of the pipeline whose compute stream never waits for the gathers reads staging that
    the delayed gathers have not filled (NaN-poisoned) and must miss the oracle.  torch hands out
    pool streams round-robin and HIP maps streams onto GPU_MAX_HW_QUEUES (4 here) hardware queues,
    so a side stream can share the compute stream's queue, where dispatches run in submission
    order and no race can occur; the check therefore tries successive fresh side streams, of
    which at least three in four sit on another queue."""
    say("pipeline dropped-wait check")
    caught = 0
    for attempt in range(8):
        pipe = _NoWait(**setup["pipe_args"])
        for sk, sv in pipe.stage:
            sk.fill_(float("nan"))
            sv.fill_(float("nan"))
        torch.cuda.synchronize()
        pipe.step()
        torch.cuda.synchronize()
        errs = []
        for l in range(1, L):
            o = pipe.o[l].float().cpu().numpy()
            errs.append(float(np.abs(np.nan_to_num(o, nan=1e9) - setup["ref_out"][l]).max()))
        say(f"  side stream {attempt}: max |o - oracle| per offloaded layer {[f'{e:.3g}' for e in errs]}")
        caught = sum(e > 2e-2 for e in errs)
        if caught:
            break
    assert caught > 0, "a pipeline without the gather wait went unnoticed on eight side streams"


def test_reuse_pipeline_matches_oracle_chain_and_refetches_nothing(setup):
    """Per-layer staging with step-to-step reuse (NaN-poisoned, side stream held back): the first
    step fetches every selected block, gives the oracle's outputs; a second step at the same
    position (the query's block is complete, p % 64 == 63) keeps every staged block, fetches
    nothing and gives the same outputs."""
    say("reuse pipeline")
    pipe = _DelayedGather(**setup["pipe_args"], reuse=True)
    for st in pipe.stage[1:]:
        st[0].fill_(float("nan"))
        st[1].fill_(float("nan"))
    torch.cuda.synchronize()
    pipe.step()
    check(setup, pipe)
    first = pipe.fetched_blocks()
    assert first == sum(int(c.sum()) for _, c, _ in setup["ref_sel"][1:])
    pipe.step()
    check(setup, pipe)
    assert pipe.fetched_blocks() == 0


# ----------------------------------------------------------------------------- decode steps with write-back

WB_B, WB_H, WB_G, WB_T, WB_K, WB_L, WB_STEPS = 2, 2, 4, 4096, 16, 4, 40
WB_P0 = 64 * 40 + 44  # the steps cross the end of block 40 at position 2623
NAN_BF16 = 0x7FC0


@pytest.mark.parametrize("overlap,reuse,delayed", [(True, False, True), (False, False, False), (True, True, True)])
def test_decode_steps_write_back_new_tokens(overlap, reuse, delayed):
    """A 40-step offloaded decode whose host pools and layer-0 cache start out holding only the
    tokens before the first position (later positions hold NaN): every later token reaches them
    only through the pipeline's append and write-back (Alg. 2; Sec. 5.3).  With one local block,
    the block a step completes is a candidate at the next step, so its compressed key must come
    from the written-back pool, and compressed keys not yet computed hold NaN.  Every step's sets
    and outputs match the oracle chain on the full caches; at the end the pools and the layer-0
    cache hold exactly the tokens up to the last position and the compressed keys the oracle's."""
    say(f"write-back steps overlap={overlap} reuse={reuse} delayed side stream={delayed}")
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    sp.load()
    dev = torch.device("cuda:0")
    B, H, G, T, K, L = WB_B, WB_H, WB_G, WB_T, WB_K, WB_L
    NB = T // 64
    shape = sp.SpardaShape(batch=B, n_kv_heads=H, group_size=G, k_total=K, t_cap=T, nc_cap=NB, n_local=1)
    oshape = oracle.Shape(batch=B, n_kv_heads=H, group_size=G, k_total=K, t_cap=T, nc_cap=NB, n_local=1)
    w = inputs.Workload("wb", batch=B, seq_len=T, n_q=1, n_kv_heads=H, group_size=G, k_total=K, n_local=1, seed=6100)
    q = [inputs.normal_bf16((B, H * G, 1, 128), 6100, 10 + l) for l in range(L)]
    f = [inputs.normal_bf16((B, H, 1, 128), 6100, 50 + l) for l in range(L)]
    f0 = inputs.normal_bf16((B, H, 1, 128), 6100, 99)
    full = [(inputs.keys_with_plants(w, (f0 if l == 0 else f[l - 1])[:, :, 0], T, tensor_id=200 + l),
             inputs.values(w, T, tensor_id=300 + l)) for l in range(L)]
    full16 = [(inputs.to_u16(k), inputs.to_u16(v)) for k, v in full]
    kc_ref = [oracle.compress_keys(oshape, full16[l][0], T, 0, NB) for l in range(L)]
    p0 = WB_P0
    done = p0 // 64  # blocks complete before the first step

    def truncated(x16):  # tokens before p0 only
        y = x16.copy()
        y[:, :, p0:] = NAN_BF16
        return y

    bufs, pools = [], [None]
    for l in range(1, L):
        pair = []
        for x16 in full16[l]:
            buf = hostmem.PinnedBuffer(x16.nbytes)
            buf.as_tensor(torch.int16).copy_(torch.from_numpy(truncated(x16).view(np.int16).reshape(-1)))
            bufs.append(buf)
            pair.append(buf.ptr)
        pools.append(tuple(pair))
    kc = []
    for l in range(L):
        t = kc_ref[l].copy()
        t[:, :, done:] = NAN_BF16
        kc.append(inputs.from_u16(t, dev))
    k0 = inputs.from_u16(truncated(full16[0][0]), dev)
    v0 = inputs.from_u16(truncated(full16[0][1]), dev)
    cls = _DelayedGather if delayed else DecodePipeline
    pipe = cls(shape=shape, t_ctx=p0 + 1, q=[x.to(dev) for x in q], f=[x.to(dev) for x in f], f0_cur=f0.to(dev),
               kc=kc, k0=k0, v0=v0, pools=pools, n_workgroups=8, device=dev, reuse=reuse)
    q16 = [inputs.to_u16(x) for x in q]
    frows16 = [inputs.to_u16(f0)] + [inputs.to_u16(f[l - 1]) for l in range(1, L)]
    worst = ratio = 0.0
    swaps = 0
    for step in range(WB_STEPS):
        p = p0 + step
        new_kv = [(full[l][0][:, :, p:p + 1].to(dev), full[l][1][:, :, p:p + 1].to(dev)) for l in range(L)]
        pipe.step(overlap=overlap, t_ctx=p + 1, new_kv=new_kv)
        torch.cuda.synchronize()
        for l in range(L):
            gs, gc = pipe.sel[l].cpu().numpy(), pipe.cnt[l].cpu().numpy()
            _, sw = compare_selection(oshape, frows16[l], kc_ref[l], 1, p, gs, gc,
                                      [(b, m, 0) for b in range(B) for m in range(H)])
            swaps += sw
            ref = oracle.sparse_attn(oshape, q16[l], 1, p, full16[l][0], full16[l][1], 0, gs, gc, 1.0 / math.sqrt(128))
            wab = oracle.sparse_attn(oshape, q16[l], 1, p, full16[l][0], abs_bits(full16[l][1]), 0, gs, gc,
                                     1.0 / math.sqrt(128))
            worst = max(worst, compare_attention(pipe.o[l].float().cpu().numpy(), ref, f"step {step} layer {l}", wab))
            ratio = max(ratio, compare_attention.last_tight_ratio)
    p_end = p0 + WB_STEPS  # tokens [0, p_end) exist now
    for l in range(1, L):
        for i, x16 in enumerate(full16[l]):
            got = bufs[2 * (l - 1) + i].as_tensor(torch.int16).numpy().view(np.uint16).reshape(x16.shape)
            assert np.array_equal(got[:, :, :p_end], x16[:, :, :p_end]), f"layer {l} pool {i}: tokens up to the end"
            assert np.all(got[:, :, p_end:] == NAN_BF16), f"layer {l} pool {i}: nothing past the last token"
    assert np.array_equal(inputs.to_u16(pipe.k0)[:, :, :p_end], full16[0][0][:, :, :p_end])
    assert np.array_equal(inputs.to_u16(pipe.v0)[:, :, :p_end], full16[0][1][:, :, :p_end])
    for l in range(L):
        got = inputs.to_u16(kc[l])
        assert np.array_equal(got[:, :, :p_end // 64], kc_ref[l][:, :, :p_end // 64]), f"layer {l}: K~"
        assert np.all(got[:, :, p_end // 64:] == NAN_BF16), f"layer {l}: K~ past the complete blocks"
    for b in bufs:
        b.free()
    say(f"  {WB_STEPS} steps x {L} layers: tie swaps {swaps}, attention max err {worst:.3g} "
        f"({ratio:.3f} of the tight bar); pools, layer-0 cache and K~ exact")
