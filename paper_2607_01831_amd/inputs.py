"""Seeded synthetic inputs for the Lynx hot path.

This module only draws random numbers and lays them out; it holds none of the
codec or attention arithmetic.  The same bytes feed the HIP path and the CPU
oracle.

Recipe (the paper's models and datasets are not used; synthetic tensors with
their shapes and outlier structure stand in for LLM activations):
  * K, V: fp32 draws from N(0, 1), rounded to BF16 (round to nearest even).
  * K outlier channels, following the paper's observation that a few K
    channels hold consistently large values across tokens (Sec. 3.2): the
    chosen (kv head, channel) columns are multiplied by a fixed factor before
    rounding to BF16.  V has none.
  * q, draft k_new/v_new: N(0, 1) rounded to BF16.
  * Paged pools: per-sequence lengths uniform on an integer range, blocks of
    16 tokens, block ids a random permutation of the pool.
  * One torch.Generator per (workload, tensor, layer, sequence); large
    tensors are drawn in fixed chunks of 4096 tokens so memory stays bounded.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import torch

HEAD_DIM = 128
CHUNK_TOKENS = 4096

# tensor ids used in the seed
T_K, T_V, T_Q, T_KNEW, T_VNEW, T_LENS, T_BLOCKS, T_OUTLIER = range(8)


@dataclass(frozen=True)
class Workload:
    name: str
    wid: int               # seed namespace
    layers: int
    batch: int
    Hq: int
    Hkv: int
    context: int           # tokens per sequence (upper bound when ragged)
    min_context: int = 0   # > 0: lengths uniform on [min_context, context]
    block_tokens: int = 0  # 0: contiguous layout
    drafts: int = 0        # k speculative queries for verification
    decode_steps: int = 1
    outliers_per_head: int = 0      # per kv head (tiny case)
    outlier_fraction: float = 0.0   # of all (kv head, channel) columns
    outlier_mult: float = 1.0
    extra: dict = field(default_factory=dict)

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv


WORKLOADS = {
    w.name: w for w in [
        Workload("tiny-gqa2-4k", 1, layers=1, batch=1, Hq=8, Hkv=4, context=4096,
                 drafts=1, outliers_per_head=4, outlier_mult=10.0),
        Workload("llama3-8b-32k", 2, layers=32, batch=1, Hq=32, Hkv=8, context=32768,
                 drafts=8, outlier_fraction=0.01, outlier_mult=8.0),
        Workload("llama3-8b-verify-128k", 3, layers=1, batch=1, Hq=32, Hkv=8,
                 context=131072, drafts=8, outlier_fraction=0.01, outlier_mult=8.0),
        Workload("paged-b16-16k-64k", 4, layers=1, batch=16, Hq=32, Hkv=8,
                 context=65536, min_context=16384, block_tokens=16,
                 outlier_fraction=0.01, outlier_mult=8.0),
        Workload("70b-overlap-b4-128k", 5, layers=1, batch=4, Hq=64, Hkv=8,
                 context=131072, drafts=4, decode_steps=16,
                 outlier_fraction=0.01, outlier_mult=8.0),
    ]
}


def seed_of(wid: int, tensor: int, layer: int = 0, seq: int = 0) -> int:
    return ((wid * 16 + tensor) * 64 + layer) * 64 + seq


def generator(seed: int, device="cpu") -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def outlier_columns(w: Workload, layer: int, Hkv: int | None = None) -> torch.Tensor:
    """Boolean [Hkv][128] mask of the K columns that carry outliers."""
    Hkv = Hkv or w.Hkv
    g = generator(seed_of(w.wid, T_OUTLIER, layer))
    mask = torch.zeros(Hkv, HEAD_DIM, dtype=torch.bool)
    if w.outliers_per_head:
        for h in range(Hkv):
            mask[h, torch.randperm(HEAD_DIM, generator=g)[: w.outliers_per_head]] = True
    elif w.outlier_fraction:
        n = round(w.outlier_fraction * Hkv * HEAD_DIM)
        mask.view(-1)[torch.randperm(Hkv * HEAD_DIM, generator=g)[:n]] = True
    return mask


def normal_bf16(shape, seed: int, device="cpu", col_mult: torch.Tensor | None = None,
                chunk_dim0: int = CHUNK_TOKENS) -> torch.Tensor:
    """N(0,1) fp32 draws rounded to BF16, drawn in chunks along dim 0.
    col_mult (broadcast over dim 0) multiplies selected columns first."""
    g = generator(seed, device)
    out = torch.empty(shape, dtype=torch.bfloat16, device=device)
    n0 = shape[0]
    for s in range(0, n0, chunk_dim0):
        e = min(n0, s + chunk_dim0)
        x = torch.randn((e - s, *shape[1:]), generator=g, device=device, dtype=torch.float32)
        if col_mult is not None:
            x *= col_mult.to(device)
        out[s:e] = x.to(torch.bfloat16)
    return out


def kv(w: Workload, which: str, layer: int = 0, seq: int = 0, T: int | None = None,
       device="cpu") -> torch.Tensor:
    """BF16 [T][Hkv][128] keys ('k') or values ('v') of one sequence/layer."""
    T = w.context if T is None else T
    if which == "k":
        mult = torch.ones(w.Hkv, HEAD_DIM)
        mult[outlier_columns(w, layer)] = w.outlier_mult
        return normal_bf16((T, w.Hkv, HEAD_DIM), seed_of(w.wid, T_K, layer, seq), device, mult)
    if which == "v":
        return normal_bf16((T, w.Hkv, HEAD_DIM), seed_of(w.wid, T_V, layer, seq), device)
    raise ValueError(which)


def queries(w: Workload, layer: int = 0, step: int = 0, nq: int = 1, device="cpu") -> torch.Tensor:
    """BF16 queries: [B][Hq][128] when nq == 1 (decode), else [B][nq][Hq][128]."""
    shape = (w.batch, nq, w.Hq, HEAD_DIM)
    q = normal_bf16(shape, seed_of(w.wid, T_Q, layer, step), device)
    return q[:, 0].contiguous() if nq == 1 else q


def drafts_kv(w: Workload, layer: int = 0, nq: int | None = None, device="cpu"):
    """BF16 draft-token K and V, each [B][nq][Hkv][128]."""
    nq = nq or w.drafts
    shape = (w.batch, nq, w.Hkv, HEAD_DIM)
    return (normal_bf16(shape, seed_of(w.wid, T_KNEW, layer), device),
            normal_bf16(shape, seed_of(w.wid, T_VNEW, layer), device))


def seq_lengths(w: Workload) -> torch.Tensor:
    """int32 [B] context lengths (ragged when min_context > 0)."""
    if w.min_context:
        g = generator(seed_of(w.wid, T_LENS))
        return torch.randint(w.min_context, w.context + 1, (w.batch,), generator=g,
                             dtype=torch.int64).to(torch.int32)
    return torch.full((w.batch,), w.context, dtype=torch.int32)


def paged_block_table(seq_lens: torch.Tensor, block_tokens: int, seed: int):
    """Random block table over a pool of exactly sum(ceil(T_b / bt)) blocks.
    Returns (block_table int32 [B][max_blocks], n_blocks); unused entries -1."""
    need = [(-(-int(t) // block_tokens)) for t in seq_lens.tolist()]
    n_blocks = sum(need)
    max_blocks = max(need) if need else 0
    perm = torch.randperm(n_blocks, generator=generator(seed)).to(torch.int32)
    table = torch.full((len(need), max(max_blocks, 1)), -1, dtype=torch.int32)
    pos = 0
    for b, n in enumerate(need):
        table[b, :n] = perm[pos:pos + n]
        pos += n
    return table, n_blocks


def contiguous_block_table(B: int) -> torch.Tensor:
    """Block table of the contiguous layout (one block per sequence)."""
    return torch.arange(B, dtype=torch.int32).view(B, 1)
