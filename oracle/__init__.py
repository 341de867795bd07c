"""Lynx CPU oracle -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct CPU statement of the Lynx hot path (see
``lynx_oracle.c`` for the definitions and the paper passages they follow).
Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never imports, links or runs it, and this package imports
nothing from the product.

Arrays are numpy.  BF16 tensors travel as their raw uint16 bit patterns.
The serializer / deserializer of Sec. 4.2 and Sec. 5 (transmission buffers of
one KV object, and their scatter into the pages) is byte layout written here
in numpy over the C encode and merge.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from pathlib import Path

import numpy as np

from . import build as _build

HEAD_DIM = 128
K_GROUP = 128

_LIB = None


def _load():
    global _LIB
    if _LIB is not None:
        return _LIB
    override = os.environ.get("LYNX_ORACLE_LIB")  # mutation tests load a planted-bug build
    if override:
        path = Path(override)
    else:
        if not _build.LIBRARY.exists() or (
                _build.LIBRARY.stat().st_mtime < _build.SOURCE.stat().st_mtime):
            _build.build()
        path = _build.LIBRARY
    lib = ctypes.CDLL(str(path))
    P = ctypes.c_void_p
    I = ctypes.c_int
    lib.oracle_encode.argtypes = [I, I, I, I, I, I, P, P, P, P, P, P, P, P, P, P, P]
    lib.oracle_encode.restype = I
    lib.oracle_merge.argtypes = [P, P, P, ctypes.c_size_t]
    lib.oracle_merge.restype = None
    lib.oracle_dequant.argtypes = [I, I, I, I, I, I, I, P, P, P, P, P, P, P, P, P]
    lib.oracle_dequant.restype = I
    lib.oracle_anchor_decode.argtypes = [I, I, I, I, I, I, P, P, P, P, P, P, P, P,
                                         P, P, P, P, I]
    lib.oracle_anchor_decode.restype = I
    lib.oracle_verify.argtypes = [I, I, I, I, I, I, I, P, P, P, P, P, P, P, P, P,
                                  P, P, P, P, P, I]
    lib.oracle_verify.restype = I
    lib.oracle_anchor_decode_tail.argtypes = [I, I, I, I, I, I, P, P, P, P, P, P, P, P,
                                              P, I, P, P, P, P, P, I]
    lib.oracle_anchor_decode_tail.restype = I
    F = ctypes.c_float
    IP = ctypes.POINTER(ctypes.c_int)
    lib.oracle_encode_split.argtypes = [I, I, I, I, I, I, I, P, P, P, P, P, P, P, P, P, P, P]
    lib.oracle_encode_split.restype = I
    lib.oracle_merge_split.argtypes = [I, ctypes.c_size_t, P, P, P]
    lib.oracle_merge_split.restype = I
    lib.oracle_dequant_anchor_split.argtypes = [I, I, I, I, I, I, I, P, P, P, P, P, P, P, P, P]
    lib.oracle_dequant_anchor_split.restype = I
    lib.oracle_anchor_decode_split.argtypes = [I, I, I, I, I, I, I, P, P, P, P, P, P, P, P,
                                               P, P, P, P, I]
    lib.oracle_anchor_decode_split.restype = I
    lib.oracle_accept_sample.argtypes = [I, I, I, P, P, P, P, P, P]
    lib.oracle_accept_sample.restype = I
    lib.oracle_hsplit.argtypes = [I, I, I, IP, IP]
    lib.oracle_hsplit.restype = I
    lib.oracle_htables.argtypes = [F, I, P, P, P]
    lib.oracle_htables.restype = I
    lib.oracle_hencode.argtypes = [I, I, I, I, I, I, P, P, P, F, I, P, P, P, P, P, P, P, P, P, P, P, P]
    lib.oracle_hencode.restype = I
    lib.oracle_hdequant.argtypes = [I, I, I, I, I, I, I, I, P, P, P, F, P, P, P, P, P, P, P, P, P, P]
    lib.oracle_hdequant.restype = I
    _LIB = lib
    return lib


def _ptr(a):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data


def default_threads() -> int:
    return max(1, len(os.sched_getaffinity(0)))


@dataclass
class Layout:
    """Cache geometry: kv heads, tokens per block, block-table row stride and
    the per-sequence token stride of the logical metadata arrays."""
    Hkv: int
    bt: int
    max_blocks: int
    max_tokens: int

    @property
    def n_groups(self) -> int:
        return -(-self.max_tokens // K_GROUP)


@dataclass
class Meta:
    k_scale: np.ndarray  # fp32 [B][Hkv][n_groups][128]
    k_zero: np.ndarray
    v_scale: np.ndarray  # fp32 [B][Hkv][max_tokens]
    v_zero: np.ndarray

    @staticmethod
    def empty(L: Layout, B: int) -> "Meta":
        kshape = (B, L.Hkv, L.n_groups, HEAD_DIM)
        vshape = (B, L.Hkv, L.max_tokens)
        return Meta(np.zeros(kshape, np.float32), np.zeros(kshape, np.float32),
                    np.zeros(vshape, np.float32), np.zeros(vshape, np.float32))


def plane_bytes(L: Layout, n_blocks: int, row_bytes: int) -> int:
    return n_blocks * L.Hkv * L.bt * row_bytes


def encode(L: Layout, b: int, T: int, block_table: np.ndarray, k_bits: np.ndarray,
           v_bits: np.ndarray, planes: dict, meta: Meta) -> None:
    """Quantize/split/pack sequence b (k_bits, v_bits: uint16 [T][Hkv][128])
    into planes['k_anc'|'v_anc'|'k_res'|'v_res'] (uint8, flat) and meta row b."""
    lib = _load()
    bt_arr = np.ascontiguousarray(block_table, dtype=np.int32)
    k_bits = np.ascontiguousarray(k_bits, dtype=np.uint16)
    v_bits = np.ascontiguousarray(v_bits, dtype=np.uint16)
    assert k_bits.shape == (T, L.Hkv, HEAD_DIM) and v_bits.shape == k_bits.shape
    rc = lib.oracle_encode(L.Hkv, L.bt, L.max_blocks, L.max_tokens, b, T, _ptr(bt_arr),
                           _ptr(k_bits), _ptr(v_bits), _ptr(planes["k_anc"]),
                           _ptr(planes["v_anc"]), _ptr(planes["k_res"]),
                           _ptr(planes["v_res"]), _ptr(meta.k_scale), _ptr(meta.k_zero),
                           _ptr(meta.v_scale), _ptr(meta.v_zero))
    if rc != 0:
        raise ValueError(f"oracle_encode rejected its arguments ({rc})")


def merge(anc: np.ndarray, res: np.ndarray) -> np.ndarray:
    """Anchor + residual nibble planes (n bytes each) -> 2n code bytes."""
    anc = np.ascontiguousarray(anc, dtype=np.uint8).reshape(-1)
    res = np.ascontiguousarray(res, dtype=np.uint8).reshape(-1)
    assert anc.size == res.size
    codes = np.empty(2 * anc.size, np.uint8)
    _load().oracle_merge(_ptr(anc), _ptr(res), _ptr(codes), anc.size)
    return codes


def dequant(mode: str, L: Layout, b: int, T: int, block_table: np.ndarray,
            k_plane: np.ndarray, v_plane: np.ndarray, meta: Meta):
    """Reconstructed K, V of sequence b as fp64 [T][Hkv][128].
    mode 'anchor': nibble planes, zero + (16a + 7.5) scale;
    mode 'full':   code planes, zero + c scale."""
    m = {"anchor": 0, "full": 1}[mode]
    bt_arr = np.ascontiguousarray(block_table, dtype=np.int32)
    k_hat = np.empty((T, L.Hkv, HEAD_DIM), np.float64)
    v_hat = np.empty_like(k_hat)
    rc = _load().oracle_dequant(m, L.Hkv, L.bt, L.max_blocks, L.max_tokens, b, T,
                                _ptr(bt_arr), _ptr(k_plane), _ptr(v_plane),
                                _ptr(meta.k_scale), _ptr(meta.k_zero),
                                _ptr(meta.v_scale), _ptr(meta.v_zero), _ptr(k_hat),
                                _ptr(v_hat))
    if rc != 0:
        raise ValueError(f"oracle_dequant rejected its arguments ({rc})")
    return k_hat, v_hat


def anchor_decode(L: Layout, Hq: int, seq_lens: np.ndarray, block_table: np.ndarray,
                  k_anc: np.ndarray, v_anc: np.ndarray, meta: Meta, q_bits: np.ndarray,
                  unit_mask: np.ndarray | None = None, nthreads: int | None = None,
                  k_tail_bits: np.ndarray | None = None, v_tail_bits: np.ndarray | None = None):
    """One query per sequence (q_bits uint16 [B][Hq][128]) over the Anchor-only
    cache, followed, if given, by the BF16 tokens generated since the context
    arrived (k_tail_bits, v_tail_bits uint16 [B][n_tail][Hkv][128], all
    visible to the query).  Returns (out fp64 [B][Hq][128], lse fp64 [B][Hq]);
    units left out by unit_mask ([B][Hkv] flags) come back as NaN."""
    seq_lens = np.ascontiguousarray(seq_lens, dtype=np.int32)
    B = seq_lens.size
    q_bits = np.ascontiguousarray(q_bits, dtype=np.uint16)
    assert q_bits.shape == (B, Hq, HEAD_DIM)
    out = np.full((B, Hq, HEAD_DIM), np.nan)
    lse = np.full((B, Hq), np.nan)
    mask = None if unit_mask is None else np.ascontiguousarray(unit_mask, dtype=np.uint8)
    bt_arr = np.ascontiguousarray(block_table, dtype=np.int32)
    if k_tail_bits is None:
        rc = _load().oracle_anchor_decode(
            L.Hkv, L.bt, L.max_blocks, L.max_tokens, B, Hq, _ptr(seq_lens), _ptr(bt_arr),
            _ptr(k_anc), _ptr(v_anc), _ptr(meta.k_scale), _ptr(meta.k_zero),
            _ptr(meta.v_scale), _ptr(meta.v_zero), _ptr(q_bits), _ptr(out), _ptr(lse),
            _ptr(mask), nthreads or default_threads())
    else:
        k_tail_bits = np.ascontiguousarray(k_tail_bits, dtype=np.uint16)
        v_tail_bits = np.ascontiguousarray(v_tail_bits, dtype=np.uint16)
        n_tail = k_tail_bits.shape[1]
        assert k_tail_bits.shape == (B, n_tail, L.Hkv, HEAD_DIM)
        assert v_tail_bits.shape == k_tail_bits.shape
        rc = _load().oracle_anchor_decode_tail(
            L.Hkv, L.bt, L.max_blocks, L.max_tokens, B, Hq, _ptr(seq_lens), _ptr(bt_arr),
            _ptr(k_anc), _ptr(v_anc), _ptr(meta.k_scale), _ptr(meta.k_zero),
            _ptr(meta.v_scale), _ptr(meta.v_zero), _ptr(q_bits), n_tail, _ptr(k_tail_bits),
            _ptr(v_tail_bits), _ptr(out), _ptr(lse), _ptr(mask), nthreads or default_threads())
    if rc != 0:
        raise ValueError(f"oracle_anchor_decode failed ({rc})")
    return out, lse


def accept_greedy(target_logits: np.ndarray, draft_tokens: np.ndarray):
    """Greedy verification of k drafted tokens (Sec. 4.3: keep the longest
    prefix the target model agrees with, then correct the first divergence).

    target_logits: [B][k+1][V], the target model's scores for the token at
    each of the k draft positions and the one after them; draft_tokens:
    int [B][k].  The target's choice at a position is its highest score, the
    lowest vocabulary index among equal scores.  Returns (accepted int32 [B],
    next_token int32 [B]): the number of leading drafts equal to the target's
    choices, and the target's choice at the first position after them (the
    correction, or the bonus token when all k are kept)."""
    logits = np.asarray(target_logits)
    drafts = np.asarray(draft_tokens)
    B, k1, _ = logits.shape
    k = k1 - 1
    assert drafts.shape == (B, k)
    accepted = np.zeros(B, np.int32)
    next_token = np.zeros(B, np.int32)
    for b in range(B):
        n = 0
        while n < k:
            choice = int(np.argmax(logits[b, n]))  # first index of the maximum
            if choice != int(drafts[b, n]):
                break
            n += 1
        accepted[b] = n
        next_token[b] = int(np.argmax(logits[b, n]))
    return accepted, next_token



def accept_sample(p: np.ndarray, q: np.ndarray, draft_tokens: np.ndarray, u: np.ndarray):
    """Acceptance of k sampled drafts (Sec. 4.3 with the speculative-sampling
    rule; readings in lynx_oracle.c).  p: fp32 [B][k+1][V] target
    probabilities, q: fp32 [B][k][V] draft probabilities, draft_tokens: int
    [B][k], u: fp32 [B][k+1] uniforms.  Returns (accepted int32 [B],
    next_token int32 [B])."""
    p = np.ascontiguousarray(p, np.float32)
    q = np.ascontiguousarray(q, np.float32)
    drafts = np.ascontiguousarray(draft_tokens, np.int32)
    u = np.ascontiguousarray(u, np.float32)
    B, k1, V = p.shape
    k = k1 - 1
    assert q.shape == (B, k, V) and drafts.shape == (B, k) and u.shape == (B, k + 1)
    accepted = np.zeros(B, np.int32)
    next_token = np.zeros(B, np.int32)
    rc = _load().oracle_accept_sample(B, k, V, _ptr(p), _ptr(q), _ptr(drafts), _ptr(u),
                                      _ptr(accepted), _ptr(next_token))
    if rc != 0:
        raise ValueError("oracle_accept_sample rejected its arguments")
    return accepted, next_token

def verify(L: Layout, Hq: int, seq_lens: np.ndarray, block_table: np.ndarray,
           k_codes: np.ndarray, v_codes: np.ndarray, meta: Meta, q_bits: np.ndarray,
           k_new_bits: np.ndarray | None = None, v_new_bits: np.ndarray | None = None,
           unit_mask: np.ndarray | None = None, nthreads: int | None = None):
    """nq draft queries per sequence (q_bits uint16 [B][nq][Hq][128]) over the
    merged 8-bit cache plus, if given, the BF16 draft K/V ([B][nq][Hkv][128]),
    causal among drafts.  Returns (out fp64 [B][nq][Hq][128], lse [B][nq][Hq])."""
    seq_lens = np.ascontiguousarray(seq_lens, dtype=np.int32)
    B = seq_lens.size
    q_bits = np.ascontiguousarray(q_bits, dtype=np.uint16)
    nq = q_bits.shape[1]
    assert q_bits.shape == (B, nq, Hq, HEAD_DIM)
    if k_new_bits is not None:
        k_new_bits = np.ascontiguousarray(k_new_bits, dtype=np.uint16)
        v_new_bits = np.ascontiguousarray(v_new_bits, dtype=np.uint16)
        assert k_new_bits.shape == (B, nq, L.Hkv, HEAD_DIM)
        assert v_new_bits.shape == k_new_bits.shape
    out = np.full((B, nq, Hq, HEAD_DIM), np.nan)
    lse = np.full((B, nq, Hq), np.nan)
    mask = None if unit_mask is None else np.ascontiguousarray(unit_mask, dtype=np.uint8)
    bt_arr = np.ascontiguousarray(block_table, dtype=np.int32)
    rc = _load().oracle_verify(
        L.Hkv, L.bt, L.max_blocks, L.max_tokens, B, Hq, nq, _ptr(seq_lens), _ptr(bt_arr),
        _ptr(k_codes), _ptr(v_codes), _ptr(meta.k_scale), _ptr(meta.k_zero),
        _ptr(meta.v_scale), _ptr(meta.v_zero), _ptr(q_bits), _ptr(k_new_bits),
        _ptr(v_new_bits), _ptr(out), _ptr(lse), _ptr(mask),
        nthreads or default_threads())
    if rc != 0:
        raise ValueError(f"oracle_verify failed ({rc})")
    return out, lse


# --------------------------------------------------------------------------
# Convenience: a whole batch in the contiguous layout, or a paged pool.
# --------------------------------------------------------------------------

def encode_batch(L: Layout, seq_lens, block_table, k_list, v_list, n_blocks: int):
    """Encode every sequence b of a batch (k_list[b], v_list[b]: uint16
    [T_b][Hkv][128]) into fresh planes of n_blocks blocks.  Returns (planes, meta)."""
    B = len(seq_lens)
    nbytes = plane_bytes(L, n_blocks, 64)
    planes = {name: np.zeros(nbytes, np.uint8) for name in ("k_anc", "v_anc", "k_res", "v_res")}
    meta = Meta.empty(L, B)
    for b in range(B):
        encode(L, b, int(seq_lens[b]), block_table, k_list[b], v_list[b], planes, meta)
    return planes, meta


# --------------------------------------------------------------------------
# Serializer / deserializer (Sec. 4.2 Prioritized Transmission; Sec. 5
# Compression Kernel).  The serializer quantizes one KV object and writes the
# packed Anchor stream followed immediately by the shared scalars into one
# contiguous transmission buffer, and the Residual stream into another; the
# deserializer scatters a received Anchor buffer into the KV pages (Anchor
# phase) and later combines a received Residual buffer with the Anchors in
# the pages into the full 8-bit codes (Residual phase).
#
# Object: tokens [t0, t0 + n) of one sequence (one layer), all kv heads, with
# t0 a multiple of the 128-token K group so that its K groups are the
# sequence's.  Byte layout of the buffers (each section follows the previous
# one with no padding):
#   anchor:   K anchor rows [Hkv][n][64], V anchor rows [Hkv][n][64],
#             K scales, K zeros  fp32 [Hkv][ceil(n/128)][128],
#             V scales, V zeros  fp32 [Hkv][n]
#   residual: K residual rows [Hkv][n][64], V residual rows [Hkv][n][64]
# --------------------------------------------------------------------------

def serialized_sections(Hkv: int, n: int) -> dict:
    """Byte (offset, size) of every section of an object's buffers, and the
    two totals ('anchor_bytes', 'residual_bytes')."""
    g = -(-n // K_GROUP)
    rows = Hkv * n * 64
    kmeta = Hkv * g * HEAD_DIM * 4
    vmeta = Hkv * n * 4
    sizes = [("k_anc", rows), ("v_anc", rows), ("k_scale", kmeta), ("k_zero", kmeta),
             ("v_scale", vmeta), ("v_zero", vmeta)]
    out, off = {}, 0
    for name, size in sizes:
        out[name] = (off, size)
        off += size
    out["anchor_bytes"] = off
    out["k_res"] = (0, rows)
    out["v_res"] = (rows, rows)
    out["residual_bytes"] = 2 * rows
    return out


def serialize(Hkv: int, n: int, k_bits: np.ndarray, v_bits: np.ndarray):
    """Quantize an object (k_bits, v_bits: uint16 [n][Hkv][128], the tokens
    t0..t0+n-1 of a sequence) into its (anchor, residual) transmission
    buffers (uint8).  The object is encoded as a sequence of its own in a
    one-block cache, whose planes [Hkv][n][64] and metadata rows are exactly
    the sections of the buffers."""
    OL = Layout(Hkv=Hkv, bt=n, max_blocks=1, max_tokens=n)
    nbytes = plane_bytes(OL, 1, 64)
    planes = {name: np.zeros(nbytes, np.uint8) for name in ("k_anc", "v_anc", "k_res", "v_res")}
    meta = Meta.empty(OL, 1)
    encode(OL, 0, n, np.zeros((1, 1), np.int32), k_bits, v_bits, planes, meta)
    sec = serialized_sections(Hkv, n)
    anc = np.concatenate([planes["k_anc"], planes["v_anc"],
                          meta.k_scale.reshape(-1).view(np.uint8), meta.k_zero.reshape(-1).view(np.uint8),
                          meta.v_scale.reshape(-1).view(np.uint8), meta.v_zero.reshape(-1).view(np.uint8)])
    res = np.concatenate([planes["k_res"], planes["v_res"]])
    assert anc.size == sec["anchor_bytes"] and res.size == sec["residual_bytes"]
    return anc, res


def token_rows(L: Layout, block_table: np.ndarray, b: int, t0: int, n: int) -> np.ndarray:
    """Row index [Hkv][n] of (b, h, t0 + i) in the planes: the plane
    addressing ((block_table[b][t / bt] * Hkv + h) * bt + t % bt)."""
    t = t0 + np.arange(n)
    blk = np.asarray(block_table, dtype=np.int64)[b, t // L.bt]
    h = np.arange(L.Hkv)[:, None]
    return (blk[None, :] * L.Hkv + h) * L.bt + (t % L.bt)[None, :]


def deserialize_anchor(L: Layout, b: int, t0: int, n: int, block_table: np.ndarray,
                       anc_buf: np.ndarray, planes: dict, meta: Meta) -> None:
    """Anchor phase: scatter an object's anchor buffer into the anchor planes
    (planes['k_anc'|'v_anc'], flat uint8) and metadata row b of sequence b."""
    assert t0 % K_GROUP == 0 and t0 + n <= L.max_tokens
    sec = serialized_sections(L.Hkv, n)
    buf = np.asarray(anc_buf, dtype=np.uint8)
    assert buf.size == sec["anchor_bytes"]
    cols = np.arange(64)
    dst = (token_rows(L, block_table, b, t0, n) * 64)[:, :, None] + cols
    for name in ("k_anc", "v_anc"):
        off, size = sec[name]
        planes[name][dst] = buf[off:off + size].reshape(L.Hkv, n, 64)
    g = -(-n // K_GROUP)
    g0 = t0 // K_GROUP
    for name, arr in (("k_scale", meta.k_scale), ("k_zero", meta.k_zero)):
        off, size = sec[name]
        arr[b, :, g0:g0 + g, :] = buf[off:off + size].view(np.float32).reshape(L.Hkv, g, HEAD_DIM)
    for name, arr in (("v_scale", meta.v_scale), ("v_zero", meta.v_zero)):
        off, size = sec[name]
        arr[b, :, t0:t0 + n] = buf[off:off + size].view(np.float32).reshape(L.Hkv, n)


def deserialize_residual(L: Layout, b: int, t0: int, n: int, block_table: np.ndarray,
                         res_buf: np.ndarray, planes: dict, codes: dict) -> None:
    """Residual phase: combine an object's residual buffer with its anchor
    rows already in the pages (planes['k_anc'|'v_anc']) into the code planes
    (codes['k_codes'|'v_codes'], flat uint8, 128-byte rows) by the merge
    definition."""
    assert t0 % K_GROUP == 0 and t0 + n <= L.max_tokens
    sec = serialized_sections(L.Hkv, n)
    buf = np.asarray(res_buf, dtype=np.uint8)
    assert buf.size == sec["residual_bytes"]
    rows = token_rows(L, block_table, b, t0, n)
    src = (rows * 64)[:, :, None] + np.arange(64)
    dst = (rows * 128)[:, :, None] + np.arange(128)
    for anc_name, res_name, code_name in (("k_anc", "k_res", "k_codes"), ("v_anc", "v_res", "v_codes")):
        off, size = sec[res_name]
        anc = planes[anc_name][src].reshape(-1)
        res = buf[off:off + size]
        codes[code_name][dst] = merge(anc, res).reshape(L.Hkv, n, 128)


# --------------------------------------------------------------------------
# Hierarchical non-linear codec (Alg. 1, Sec. 4.1): pages of 256 tokens and
# chunks of 32 per channel, alpha-law transform to a magnitude code and a
# sign, split into a signed 4-bit anchor and a signed 4-bit correction.  The
# variants of the split and the readings of the garbled parts of Alg. 1
# are stated in lynx_oracle.c.
# --------------------------------------------------------------------------

H_PAGE = 256
H_CHUNK = 32


@dataclass
class HMeta:
    """fp32 metadata of the hierarchical codec for K and V of a batch."""
    k_gmin: np.ndarray    # [B][Hkv][ceil(max_tokens/256)][128]
    k_gscale: np.ndarray
    k_mu: np.ndarray      # [B][Hkv][ceil(max_tokens/32)][128]
    k_sigma: np.ndarray
    v_gmin: np.ndarray
    v_gscale: np.ndarray
    v_mu: np.ndarray
    v_sigma: np.ndarray

    @staticmethod
    def empty(L: Layout, B: int) -> "HMeta":
        pg = (B, L.Hkv, -(-L.max_tokens // H_PAGE), HEAD_DIM)
        ch = (B, L.Hkv, -(-L.max_tokens // H_CHUNK), HEAD_DIM)
        z = lambda shape: np.zeros(shape, np.float32)
        return HMeta(z(pg), z(pg), z(ch), z(ch), z(pg), z(pg), z(ch), z(ch))

    def ptrs(self):
        return [_ptr(a) for a in (self.k_gmin, self.k_gscale, self.k_mu, self.k_sigma,
                                  self.v_gmin, self.v_gscale, self.v_mu, self.v_sigma)]


H_VARIANTS = {"biased": 0, "centred": 1, "int4": 2}


def _variant(variant) -> int:
    return H_VARIANTS[variant] if isinstance(variant, str) else int(variant)


def hsplit(I: int, S: int, variant="biased"):
    """Stage 4 of Alg. 1 for one code: (anchor, residual) nibble values."""
    a, r = ctypes.c_int(), ctypes.c_int()
    rc = _load().oracle_hsplit(_variant(variant), int(I), int(S), ctypes.byref(a), ctypes.byref(r))
    if rc != 0:
        raise ValueError(f"oracle_hsplit rejected ({variant}, {I})")
    return a.value, r.value


def htables(alpha: float, variant="biased"):
    """(decision thresholds [M], reconstruction levels [M + 1], the centred
    split's anchor-only levels [8]) for alpha; M = 127, or 7 for 'int4'."""
    theta = np.zeros(127, np.float32)
    level = np.zeros(128, np.float32)
    alevel = np.zeros(8, np.float32)
    M = _load().oracle_htables(alpha, _variant(variant), _ptr(theta), _ptr(level), _ptr(alevel))
    if M < 0:
        raise ValueError(f"unknown variant {variant}")
    return theta[:M].copy(), level[:M + 1].copy(), alevel


def hencode(L: Layout, b: int, T: int, block_table: np.ndarray, k_bits: np.ndarray,
            v_bits: np.ndarray, alpha: float, planes: dict, hmeta: HMeta,
            variant="biased") -> None:
    """Hierarchical encode of sequence b (k_bits, v_bits: uint16 [T][Hkv][128])
    into planes['k_anc'|'v_anc'|'k_res'|'v_res'] ('int4': the anchor planes
    only) and hmeta row b."""
    bt_arr = np.ascontiguousarray(block_table, dtype=np.int32)
    k_bits = np.ascontiguousarray(k_bits, dtype=np.uint16)
    v_bits = np.ascontiguousarray(v_bits, dtype=np.uint16)
    assert k_bits.shape == (T, L.Hkv, HEAD_DIM) and v_bits.shape == k_bits.shape
    rc = _load().oracle_hencode(L.Hkv, L.bt, L.max_blocks, L.max_tokens, b, T, _ptr(bt_arr),
                                _ptr(k_bits), _ptr(v_bits), alpha, _variant(variant),
                                _ptr(planes["k_anc"]), _ptr(planes["v_anc"]),
                                _ptr(planes.get("k_res")), _ptr(planes.get("v_res")), *hmeta.ptrs())
    if rc != 0:
        raise ValueError(f"oracle_hencode rejected its arguments ({rc})")


def hdequant(mode: str, L: Layout, b: int, T: int, block_table: np.ndarray,
             k_plane: np.ndarray, v_plane: np.ndarray, alpha: float, hmeta: HMeta,
             variant="biased"):
    """Reconstructed K, V of sequence b as BF16 bits (uint16 [T][Hkv][128]):
    mode 'anchor' from the anchor nibble planes, 'full' from the merged code
    planes (not for 'int4')."""
    m = {"anchor": 0, "full": 1}[mode]
    bt_arr = np.ascontiguousarray(block_table, dtype=np.int32)
    k_out = np.zeros((T, L.Hkv, HEAD_DIM), np.uint16)
    v_out = np.zeros_like(k_out)
    rc = _load().oracle_hdequant(m, _variant(variant), L.Hkv, L.bt, L.max_blocks, L.max_tokens, b, T, _ptr(bt_arr),
                                 _ptr(k_plane), _ptr(v_plane), alpha, *hmeta.ptrs(), _ptr(k_out),
                                 _ptr(v_out))
    if rc != 0:
        raise ValueError(f"oracle_hdequant rejected its arguments ({rc})")
    return k_out, v_out


# --------------------------------------------------------------------------
# Split widths other than 4 + 4 (Sec. 8): an A-bit anchor c >> (8 - A) and an
# (8 - A)-bit residual, rows of 128 elements as little-endian bit strings
# (16 W bytes a row); the readings are stated in lynx_oracle.c.
# --------------------------------------------------------------------------

def encode_split(A: int, L: Layout, b: int, T: int, block_table: np.ndarray, k_bits: np.ndarray,
                 v_bits: np.ndarray, planes: dict, meta: Meta) -> None:
    """Encode sequence b into planes['k_anc'|'v_anc'] (rows of 16 A bytes),
    planes['k_res'|'v_res'] (rows of 16 (8 - A) bytes) and meta (as encode)."""
    bt_arr = np.ascontiguousarray(block_table, dtype=np.int32)
    k_bits = np.ascontiguousarray(k_bits, dtype=np.uint16)
    v_bits = np.ascontiguousarray(v_bits, dtype=np.uint16)
    rc = _load().oracle_encode_split(A, L.Hkv, L.bt, L.max_blocks, L.max_tokens, b, T, _ptr(bt_arr),
                                     _ptr(k_bits), _ptr(v_bits), _ptr(planes["k_anc"]),
                                     _ptr(planes["v_anc"]), _ptr(planes["k_res"]), _ptr(planes["v_res"]),
                                     _ptr(meta.k_scale), _ptr(meta.k_zero), _ptr(meta.v_scale),
                                     _ptr(meta.v_zero))
    if rc != 0:
        raise ValueError(f"oracle_encode_split rejected its arguments ({rc})")


def merge_split(A: int, anc: np.ndarray, res: np.ndarray) -> np.ndarray:
    """Rows of A-bit anchors and (8 - A)-bit residuals -> rows of 128 codes."""
    anc = np.ascontiguousarray(anc, dtype=np.uint8)
    res = np.ascontiguousarray(res, dtype=np.uint8)
    n_rows = anc.size // (16 * A)
    assert anc.size == n_rows * 16 * A and res.size == n_rows * 16 * (8 - A)
    codes = np.zeros(n_rows * HEAD_DIM, np.uint8)
    if _load().oracle_merge_split(A, n_rows, _ptr(anc), _ptr(res), _ptr(codes)) != 0:
        raise ValueError("oracle_merge_split rejected its arguments")
    return codes


def dequant_anchor_split(A: int, L: Layout, b: int, T: int, block_table: np.ndarray,
                         k_anc: np.ndarray, v_anc: np.ndarray, meta: Meta):
    """K, V of sequence b from the A-bit anchors alone, as BF16 bits
    (uint16 [T][Hkv][128])."""
    bt_arr = np.ascontiguousarray(block_table, dtype=np.int32)
    k_out = np.zeros((T, L.Hkv, HEAD_DIM), np.uint16)
    v_out = np.zeros_like(k_out)
    rc = _load().oracle_dequant_anchor_split(A, L.Hkv, L.bt, L.max_blocks, L.max_tokens, b, T,
                                             _ptr(bt_arr), _ptr(k_anc), _ptr(v_anc),
                                             _ptr(meta.k_scale), _ptr(meta.k_zero),
                                             _ptr(meta.v_scale), _ptr(meta.v_zero),
                                             _ptr(k_out), _ptr(v_out))
    if rc != 0:
        raise ValueError(f"oracle_dequant_anchor_split rejected its arguments ({rc})")
    return k_out, v_out


def anchor_decode_split(A: int, L: Layout, Hq: int, seq_lens: np.ndarray, block_table: np.ndarray,
                        k_anc: np.ndarray, v_anc: np.ndarray, meta: Meta, q_bits: np.ndarray,
                        unit_mask: np.ndarray | None = None, nthreads: int | None = None):
    """One query per sequence (q_bits uint16 [B][Hq][128]) over the A-bit
    anchors of a split width (rows of 16 A bytes), each standing for code
    2^R a + (2^R - 1) / 2 (R = 8 - A).  Returns (out fp64 [B][Hq][128],
    lse fp64 [B][Hq]); units left out by unit_mask come back as NaN."""
    seq_lens = np.ascontiguousarray(seq_lens, dtype=np.int32)
    B = seq_lens.size
    q_bits = np.ascontiguousarray(q_bits, dtype=np.uint16)
    assert q_bits.shape == (B, Hq, HEAD_DIM)
    out = np.full((B, Hq, HEAD_DIM), np.nan)
    lse = np.full((B, Hq), np.nan)
    mask = None if unit_mask is None else np.ascontiguousarray(unit_mask, dtype=np.uint8)
    bt_arr = np.ascontiguousarray(block_table, dtype=np.int32)
    rc = _load().oracle_anchor_decode_split(
        A, L.Hkv, L.bt, L.max_blocks, L.max_tokens, B, Hq, _ptr(seq_lens), _ptr(bt_arr),
        _ptr(k_anc), _ptr(v_anc), _ptr(meta.k_scale), _ptr(meta.k_zero), _ptr(meta.v_scale),
        _ptr(meta.v_zero), _ptr(q_bits), _ptr(out), _ptr(lse), _ptr(mask), nthreads or default_threads())
    if rc != 0:
        raise ValueError(f"oracle_anchor_decode_split rejected its arguments ({rc})")
    return out, lse
