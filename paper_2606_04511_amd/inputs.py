"""Seeded synthetic inputs shaped like the paper's 8B GQA setting.

This module draws random numbers and lays tensors out; it performs none of the method's
arithmetic (no pooling, scoring, selection or attention).  Both the GPU library's callers and the
CPU oracle's callers take their inputs from here, so both sides see identical bits.

Recipe (one generator per tensor, seeded from ``(seed, tensor id)``):
  * Q, K, V, F ~ N(0, 1) in float32, rounded to bf16 (round to nearest even).
  * Planted relevant blocks: for every (batch, KV group), ``round(0.05 * n_blocks)`` blocks are
    drawn without replacement from the candidate range of the last query position
    ``[n_init, blk(T-1) - n_local]``; every key in a planted block is shifted by
    ``2 * F_group / ||F_group||`` in float32 before the bf16 rounding, where ``F_group`` is the
    Forecast row of the last query position of that group.  Scores of planted blocks for that
    row are therefore about ``2 ||F|| ~ 22.6`` above the noise (std ~1.41), so the selection is
    not flat.
  * bf16 tensors are torch.bfloat16 on the requested device; ``to_u16`` gives the uint16 bit
    patterns that the oracle takes.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch

BLOCK = 64


@dataclass(frozen=True)
class Workload:
    """One synthetic workload (sizes only)."""
    name: str
    batch: int
    seq_len: int            # T: tokens in the context (decode) or the prefill length
    n_q: int                # query rows per (batch, group): 1 for decode, T for full prefill
    n_kv_heads: int = 8
    group_size: int = 4
    head_dim: int = 128
    k_total: int = 64
    n_init: int = 1
    n_local: int = 2
    seed: int = 1000
    layers: int = 1
    extras: dict = field(default_factory=dict, compare=False, hash=False)

    @property
    def n_q_heads(self) -> int:
        return self.n_kv_heads * self.group_size

    @property
    def n_blocks(self) -> int:
        return self.seq_len // BLOCK

    @property
    def q_pos0(self) -> int:
        return self.seq_len - self.n_q


# The five workloads of the benchmark table (decode at 4K/32K/128K, chunked prefill at 32K and
# the 32-layer offloaded decode pipeline at 128K).  Seeds are 1000 + index.
WORKLOADS = {
    "decode_b1_t4k": Workload("decode_b1_t4k", batch=1, seq_len=4096, n_q=1, k_total=16, seed=1000),
    "decode_b8_t32k": Workload("decode_b8_t32k", batch=8, seq_len=32768, n_q=1, k_total=64, seed=1001),
    "decode_b32_t128k": Workload("decode_b32_t128k", batch=32, seq_len=131072, n_q=1, k_total=64, seed=1002),
    "prefill_b1_t32k": Workload("prefill_b1_t32k", batch=1, seq_len=32768, n_q=32768, k_total=64, seed=1003),
    "pipeline_b64_t128k_l32": Workload("pipeline_b64_t128k_l32", batch=64, seq_len=131072, n_q=1, k_total=64,
                                       seed=1004, layers=32),
    # The paper's model configuration (MiniCPM4.1-8B, App. C: 32 query / 2 KV heads, a 96-block
    # budget holding the 32-block (2048-token) local window and one initial block), with keys on
    # the (32, 16) grid.
    "paper_decode_b32_t128k": Workload("paper_decode_b32_t128k", batch=32, seq_len=131072, n_q=1, n_kv_heads=2,
                                       group_size=16, k_total=96, n_local=32, seed=1005),
    "paper_prefill_b1_t32k": Workload("paper_prefill_b1_t32k", batch=1, seq_len=32768, n_q=32768, n_kv_heads=2,
                                      group_size=16, k_total=96, n_local=32, seed=1006),
}


def _gen(seed: int, tensor_id: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed((int(seed) * 1_000_003 + int(tensor_id)) & 0x7FFF_FFFF_FFFF_FFFF)
    return g


def normal_bf16(shape, seed: int, tensor_id: int, device="cpu") -> torch.Tensor:
    g = _gen(seed, tensor_id, device)
    x = torch.randn(*shape, generator=g, device=device, dtype=torch.float32)
    return x.to(torch.bfloat16)


def to_u16(t: torch.Tensor) -> np.ndarray:
    """bf16 tensor -> numpy uint16 bit patterns (host copy)."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def from_u16(a: np.ndarray, device="cpu") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device).view(torch.bfloat16)


def n_planted(n_blocks: int) -> int:
    return int(round(0.05 * n_blocks))


def planted_blocks(seed: int, batch: int, n_kv_heads: int, seq_len: int, n_init: int, n_local: int) -> np.ndarray:
    """int64 [B][Hkv][n_plant]: planted block ids, drawn from the last position's candidates."""
    last_blk = (seq_len - 1) // BLOCK
    lo, hi = n_init, last_blk - n_local  # inclusive candidate range
    n_cand = max(hi - lo + 1, 0)
    n_p = min(n_planted(seq_len // BLOCK), n_cand)
    rng = np.random.Generator(np.random.Philox(key=[seed, 77]))
    out = np.zeros((batch, n_kv_heads, n_p), np.int64)
    for b in range(batch):
        for m in range(n_kv_heads):
            out[b, m] = lo + rng.choice(n_cand, size=n_p, replace=False)
    return out


def keys_with_plants(w: Workload, f_last: torch.Tensor, t_cap: int, device="cpu", tensor_id: int = 2,
                     seed: int | None = None) -> torch.Tensor:
    """K cache bf16 [B][Hkv][t_cap][D]; tokens >= T are zero.  f_last: bf16 [B][Hkv][D], the
    Forecast row of the last query position of every group."""
    seed = w.seed if seed is None else seed
    B, H, D, T = w.batch, w.n_kv_heads, w.head_dim, w.seq_len
    plants = planted_blocks(seed, B, H, T, w.n_init, w.n_local)
    k = torch.zeros(B, H, t_cap, D, dtype=torch.bfloat16, device=device)
    for b in range(B):  # one batch element at a time bounds the float32 temporary
        g = _gen(seed, tensor_id * 100_000 + b, device)
        kb = torch.randn(H, T, D, generator=g, device=device, dtype=torch.float32)
        fl = f_last[b].to(torch.float32)
        shift = 2.0 * fl / fl.norm(dim=-1, keepdim=True)  # [H][D]
        for m in range(H):
            for j in plants[b, m]:
                kb[m, j * BLOCK:(j + 1) * BLOCK] += shift[m]
        k[b, :, :T] = kb.to(torch.bfloat16)
        del kb
    return k


def values(w: Workload, t_cap: int, device="cpu", tensor_id: int = 3, seed: int | None = None) -> torch.Tensor:
    seed = w.seed if seed is None else seed
    B, H, D, T = w.batch, w.n_kv_heads, w.head_dim, w.seq_len
    v = torch.zeros(B, H, t_cap, D, dtype=torch.bfloat16, device=device)
    for b in range(B):
        v[b, :, :T] = normal_bf16((H, T, D), seed, tensor_id * 100_000 + b, device)
    return v


def block_coded_values(batch: int, n_kv_heads: int, t_cap: int, device="cpu") -> torch.Tensor:
    """V cache bf16 [B][Hkv][t_cap][D] that identifies the block of every token: all 64 tokens of
    block j hold the same vector, 1.0 at dimension j mod 64 and at dimension 64 + (j div 64) mod 64,
    0.0 elsewhere (a two-coordinate code, unique for j < 4096).  An attention output over such
    values is, per dimension, the attention mass of the few attended blocks that share that
    coordinate, so leaving out, adding or exchanging one block changes some output element by
    that block's whole mass."""
    D = 128
    assert t_cap % BLOCK == 0
    j = torch.arange(t_cap // BLOCK, device=device)
    blk = torch.zeros(t_cap // BLOCK, D, dtype=torch.bfloat16, device=device)
    blk[j, j % 64] = 1.0
    blk[j, 64 + (j // 64) % 64] = 1.0
    v = blk.repeat_interleave(BLOCK, dim=0)  # [t_cap][D]
    return v.expand(batch, n_kv_heads, t_cap, D).contiguous()


def make_case(w: Workload, device="cpu", t_cap: int | None = None, seed: int | None = None) -> dict:
    """All inputs of one layer: q [B][Hq][n_q][D], f [B][Hkv][n_q][D], k, v [B][Hkv][t_cap][D]."""
    seed = w.seed if seed is None else seed
    t_cap = w.seq_len if t_cap is None else t_cap
    assert t_cap >= w.seq_len and t_cap % BLOCK == 0
    q = normal_bf16((w.batch, w.n_q_heads, w.n_q, w.head_dim), seed, 0, device)
    f = normal_bf16((w.batch, w.n_kv_heads, w.n_q, w.head_dim), seed, 1, device)
    k = keys_with_plants(w, f[:, :, -1, :], t_cap, device, seed=seed)
    v = values(w, t_cap, device, seed=seed)
    return {"q": q, "f": f, "k": k, "v": v, "t_cap": t_cap, "seed": seed,
            "plants": planted_blocks(seed, w.batch, w.n_kv_heads, w.seq_len, w.n_init, w.n_local)}
