"""Shared set-up for the GPU parity tests: the same seeded inputs go through
the HIP path (via the C ABI binding) and through the CPU oracle.

Only moves bytes between torch, numpy and the two implementations; computes
no part of the method.
"""
from __future__ import annotations

import sys
from dataclasses import dataclass

import numpy as np
import torch

import oracle
from paper_2607_01831_amd import inputs, lynx

HEAD_DIM = 128


def note(msg: str) -> None:
    """Name the case on stdout before a GPU step (survives a lost box)."""
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def bits(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


@dataclass
class Cache:
    """One layer's encoded cache on both sides."""
    lens: list
    Hkv: int
    bt: int
    table: torch.Tensor          # int32 [B][max_blocks] (host)
    n_blocks: int
    L: lynx.Layout
    OL: oracle.Layout
    pool: lynx.KVPool            # device
    planes: dict | None = None   # oracle planes (numpy) or None when not computed
    meta: oracle.Meta | None = None
    k_list: list | None = None   # host BF16 inputs
    v_list: list | None = None

    @property
    def B(self):
        return len(self.lens)

    def table_dev(self):
        return self.table.cuda()

    def lens_dev(self):
        return torch.tensor(self.lens, dtype=torch.int32).cuda()


def build_cache(k_list, v_list, Hkv: int, bt: int | None = None, seed: int = 0,
                with_oracle: bool = True, merge: bool = True, max_tokens: int | None = None) -> Cache:
    """Encode sequences (host BF16 [T_b][Hkv][128]) with the HIP path into a
    pool (contiguous when bt is None, else paged with a random block table),
    and with the oracle when asked."""
    lens = [int(k.shape[0]) for k in k_list]
    B = len(lens)
    max_T = max(max(lens), 1)
    if bt is None:
        bt_eff = max_T
        table = torch.arange(B, dtype=torch.int32).view(B, 1)
        n_blocks = B
    else:
        bt_eff = bt
        table, n_blocks = inputs.paged_block_table(torch.tensor(lens), bt, seed)
        n_blocks = max(n_blocks, 1)
    max_blocks = table.shape[1]
    mt = max_tokens or max_T
    L = lynx.Layout(num_kv_heads=Hkv, block_tokens=bt_eff, max_blocks_per_seq=max_blocks,
                    num_blocks=n_blocks, max_tokens=mt)
    OL = oracle.Layout(Hkv=Hkv, bt=bt_eff, max_blocks=max_blocks, max_tokens=mt)
    pool = lynx.KVPool.allocate(L, B, codes=merge)
    tdev = table.cuda()
    for b in range(B):
        note(f"encode b={b} T={lens[b]} Hkv={Hkv} bt={bt_eff}")
        pool.encode(b, lens[b], tdev, k_list[b].cuda(), v_list[b].cuda())
    if merge:
        note("merge")
        pool.merge()
    torch.cuda.synchronize()
    c = Cache(lens, Hkv, bt_eff, table, n_blocks, L, OL, pool, k_list=k_list, v_list=v_list)
    if with_oracle:
        c.planes, c.meta = oracle.encode_batch(OL, lens, table.numpy(),
                                               [bits(k) for k in k_list],
                                               [bits(v) for v in v_list], n_blocks)
    return c


def device_meta_to_oracle(c: Cache) -> oracle.Meta:
    m = c.pool.meta
    return oracle.Meta(m.k_scale.cpu().numpy(), m.k_zero.cpu().numpy(),
                       m.v_scale.cpu().numpy(), m.v_zero.cpu().numpy())


def gpu_anchor_decode(c: Cache, q: torch.Tensor, with_lse=True):
    """q: BF16 [B][Hq][128] (host or device). Returns (out fp32 host, lse host)."""
    B, Hq = c.B, q.shape[1]
    qd = q.cuda().contiguous()
    out = torch.empty(B, Hq, HEAD_DIM, dtype=torch.bfloat16, device="cuda")
    lse = torch.empty(B, Hq, dtype=torch.float32, device="cuda") if with_lse else None
    max_len = max(c.lens) if c.lens else 0
    ws = lynx.workspace(c.L, B, Hq, 1, max_len)
    note(f"anchor_decode B={B} Hq={Hq} Hkv={c.Hkv} lens={c.lens[:4]}")
    lynx.lynx_attn_anchor_decode(c.L, B, Hq, max_len, c.lens_dev(), c.table_dev(), c.pool.k_anc,
                                 c.pool.v_anc, c.pool.meta, qd, out, lse, ws)
    torch.cuda.synchronize()
    return out.float().cpu().numpy(), (lse.cpu().numpy() if with_lse else None)


def gpu_verify(c: Cache, q: torch.Tensor, k_new=None, v_new=None):
    """q: BF16 [B][k][Hq][128]. Returns out fp32 host [B][k][Hq][128]."""
    B, nq, Hq = c.B, q.shape[1], q.shape[2]
    qd = q.cuda().contiguous()
    out = torch.empty(B, nq, Hq, HEAD_DIM, dtype=torch.bfloat16, device="cuda")
    max_len = max(c.lens) if c.lens else 0
    ws = lynx.workspace(c.L, B, Hq, nq, max_len)
    kn = None if k_new is None else k_new.cuda().contiguous()
    vn = None if v_new is None else v_new.cuda().contiguous()
    note(f"verify B={B} k={nq} Hq={Hq} Hkv={c.Hkv} tail={k_new is not None} lens={c.lens[:4]}")
    lynx.lynx_attn_verify(c.L, B, Hq, nq, max_len, c.lens_dev(), c.table_dev(), c.pool.k_codes,
                          c.pool.v_codes, c.pool.meta, qd, kn, vn, out, ws)
    torch.cuda.synchronize()
    return out.float().cpu().numpy()


def random_kv(T: int, Hkv: int, seed: int, outlier_cols: int = 2, mult: float = 8.0):
    g = torch.Generator().manual_seed(seed)
    k = torch.randn(T, Hkv, HEAD_DIM, generator=g)
    if outlier_cols:
        cols = torch.randperm(HEAD_DIM, generator=g)[:outlier_cols]
        k[:, :, cols] *= mult
    v = torch.randn(T, Hkv, HEAD_DIM, generator=g)
    return k.to(torch.bfloat16), v.to(torch.bfloat16)


def random_bf16(shape, seed: int):
    g = torch.Generator().manual_seed(seed)
    return torch.randn(*shape, generator=g).to(torch.bfloat16)
