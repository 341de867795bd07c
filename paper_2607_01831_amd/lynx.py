"""Python binding of liblynx.so (include/lynx.h): argument marshalling only.

Every function has the name and argument order of its C entry point.  Tensors
are torch CUDA tensors; their device pointers and the current HIP stream are
passed through ctypes.  Nothing here computes any part of the method: if the
library is missing the binding raises instead of falling back to anything.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass
from pathlib import Path

import torch

LIBRARY = Path(__file__).resolve().parent / "liblynx.so"

LYNX_OK, LYNX_EINVAL, LYNX_ENOTSUP, LYNX_EWORKSPACE, LYNX_EHIP = 0, -1, -2, -3, -4
HEAD_DIM = 128
K_GROUP = 128
MAX_DRAFTS = 64


class LynxError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} failed: {lynx_strerror(status)} ({status})")


class lynx_layout(ctypes.Structure):
    _fields_ = [("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("k_group_tokens", ctypes.c_int32), ("block_tokens", ctypes.c_int32),
                ("max_blocks_per_seq", ctypes.c_int32), ("num_blocks", ctypes.c_int32),
                ("max_tokens", ctypes.c_int32)]


class lynx_meta(ctypes.Structure):
    _fields_ = [("k_scale", ctypes.c_void_p), ("k_zero", ctypes.c_void_p),
                ("v_scale", ctypes.c_void_p), ("v_zero", ctypes.c_void_p)]


_lib = None


class lynx_hmeta(ctypes.Structure):
    _fields_ = [(name, ctypes.c_void_p) for name in
                ("k_gmin", "k_gscale", "k_mu", "k_sigma", "v_gmin", "v_gscale", "v_mu", "v_sigma")]


def load():
    """Load liblynx.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not LIBRARY.exists():
        raise RuntimeError(f"{LIBRARY} is not built: run `python -m paper_2607_01831_amd.build` "
                           "(or __graft_entry__.build()) first")
    lib = ctypes.CDLL(str(LIBRARY))
    P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    LP, MP = ctypes.POINTER(lynx_layout), ctypes.POINTER(lynx_meta)
    sigs = {
        "lynx_kv_encode": ([LP, I32, I32, P, P, P, P, P, P, P, MP, P], ctypes.c_int),
        "lynx_kv_merge": ([P, P, P, SZ, P], ctypes.c_int),
        "lynx_attn_workspace_bytes": ([LP, I32, I32, I32, I32], SZ),
        "lynx_attn_anchor_decode": ([LP, I32, I32, I32, P, P, P, P, MP, P, P, P, P, SZ, P],
                                    ctypes.c_int),
        "lynx_attn_anchor_decode_split": ([I32, LP, I32, I32, I32, P, P, P, P, MP, P, P, P, P, SZ, P],
                                          ctypes.c_int),
        "lynx_attn_anchor_decode_noalloc": ([LP, I32, I32, I32, P, P, P, P, MP, P, P, P, P],
                                            ctypes.c_int),
        "lynx_attn_verify": ([LP, I32, I32, I32, I32, P, P, P, P, MP, P, P, P, P, P, SZ, P],
                             ctypes.c_int),
        "lynx_attn_anchor_decode_tail": ([LP, I32, I32, I32, P, P, P, P, MP, P, I32, P, P, P, P, P,
                                          SZ, P], ctypes.c_int),
        "lynx_spec_accept_workspace_bytes": ([I32, I32, I32], SZ),
        "lynx_spec_accept_greedy": ([I32, I32, I32, P, P, P, P, P, SZ, P], ctypes.c_int),
        "lynx_spec_accept_sample": ([I32, I32, I32, P, P, P, P, P, P, P, SZ, P], ctypes.c_int),
        "lynx_serialized_bytes": ([I32, I32, ctypes.POINTER(SZ), ctypes.POINTER(SZ)], ctypes.c_int),
        "lynx_kv_serialize": ([I32, I32, P, P, P, P, P], ctypes.c_int),
        "lynx_kv_deserialize_anchor": ([LP, I32, I32, I32, P, P, P, P, MP, P], ctypes.c_int),
        "lynx_kv_deserialize_residual": ([LP, I32, I32, I32, P, P, P, P, P, P, P], ctypes.c_int),
        "lynx_hkv_encode": ([LP, I32, I32, P, P, P, ctypes.c_float, I32, P, P, P, P,
                             ctypes.POINTER(lynx_hmeta), P], ctypes.c_int),
        "lynx_hkv_dequant": ([LP, I32, I32, P, I32, P, P, ctypes.c_float, I32,
                              ctypes.POINTER(lynx_hmeta), P, P, P], ctypes.c_int),
        "lynx_kv_encode_split": ([LP, I32, I32, I32, P, P, P, P, P, P, P, MP, P], ctypes.c_int),
        "lynx_kv_merge_split": ([I32, SZ, P, P, P, P], ctypes.c_int),
        "lynx_kv_dequant_anchor_split": ([LP, I32, I32, I32, P, P, P, MP, P, P, P], ctypes.c_int),
        "lynx_strerror": ([ctypes.c_int], ctypes.c_char_p),
    }
    for name, (args, res) in sigs.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def lynx_strerror(status: int) -> str:
    return load().lynx_strerror(status).decode()


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError("liblynx takes device tensors")
    if not t.is_contiguous():
        raise ValueError("liblynx takes contiguous tensors")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return stream


def _check(fn: str, status: int):
    if status != LYNX_OK:
        raise LynxError(fn, status)


# Size checks of the tensors a call reads or writes.  The C ABI sees only
# pointers, so a short tensor would become an out-of-bounds device access:
# the binding rejects it first.
def _nbytes(t) -> int:
    return t.numel() * t.element_size()


def _need(fn: str, what: str, t, nbytes: int) -> None:
    if isinstance(t, torch.Tensor) and _nbytes(t) < nbytes:
        raise ValueError(f"{fn}: {what} holds {_nbytes(t)} bytes; the call uses {nbytes}")


def _need_meta(fn: str, L: "Layout", meta: "Meta", rows: int) -> None:
    """fp32 metadata rows 0 .. rows - 1 (sequences) of the layout."""
    k = rows * L.num_kv_heads * L.n_groups * HEAD_DIM * 4
    v = rows * L.num_kv_heads * L.max_tokens * 4
    for name, nbytes in (("k_scale", k), ("k_zero", k), ("v_scale", v), ("v_zero", v)):
        _need(fn, f"meta.{name}", getattr(meta, name), nbytes)


def _need_attn(fn: str, L: "Layout", B: int, seq_lens, block_table, planes, row_bytes: int,
               meta: "Meta") -> None:
    """The per-batch arguments every attention call reads."""
    if B <= 0:
        return
    _need(fn, "seq_lens", seq_lens, B * 4)
    _need(fn, "block_table", block_table, B * L.max_blocks_per_seq * 4)
    for i, t in enumerate(planes):
        _need(fn, f"plane {i}", t, L.plane_bytes(row_bytes))
    _need_meta(fn, L, meta, B)


@dataclass
class Layout:
    """Cache geometry (see lynx_layout in include/lynx.h)."""
    num_kv_heads: int
    block_tokens: int
    max_blocks_per_seq: int
    num_blocks: int
    max_tokens: int
    head_dim: int = HEAD_DIM
    k_group_tokens: int = K_GROUP

    def c(self) -> lynx_layout:
        return lynx_layout(self.num_kv_heads, self.head_dim, self.k_group_tokens,
                           self.block_tokens, self.max_blocks_per_seq, self.num_blocks,
                           self.max_tokens)

    @property
    def n_groups(self) -> int:
        return -(-self.max_tokens // K_GROUP)

    def plane_bytes(self, row_bytes: int = 64) -> int:
        return self.num_blocks * self.num_kv_heads * self.block_tokens * row_bytes


@dataclass
class Meta:
    """fp32 metadata tensors of a batch (device)."""
    k_scale: torch.Tensor  # [B][Hkv][n_groups][128]
    k_zero: torch.Tensor
    v_scale: torch.Tensor  # [B][Hkv][max_tokens]
    v_zero: torch.Tensor

    @staticmethod
    def empty(L: Layout, B: int, device="cuda") -> "Meta":
        ks = (B, L.num_kv_heads, L.n_groups, HEAD_DIM)
        vs = (B, L.num_kv_heads, L.max_tokens)
        f = dict(dtype=torch.float32, device=device)
        return Meta(torch.zeros(ks, **f), torch.zeros(ks, **f), torch.zeros(vs, **f),
                    torch.zeros(vs, **f))

    def c(self) -> lynx_meta:
        return lynx_meta(_ptr(self.k_scale), _ptr(self.k_zero), _ptr(self.v_scale),
                         _ptr(self.v_zero))


def lynx_kv_encode(L: Layout, b: int, T: int, block_table, k, v, k_anc, v_anc, k_res, v_res,
                   meta: Meta, stream=None) -> None:
    fn = "lynx_kv_encode"
    _need(fn, "k", k, T * L.num_kv_heads * HEAD_DIM * 2)
    _need(fn, "v", v, T * L.num_kv_heads * HEAD_DIM * 2)
    _need(fn, "block_table", block_table, (b + 1) * L.max_blocks_per_seq * 4)
    for name, t in (("k_anc", k_anc), ("v_anc", v_anc), ("k_res", k_res), ("v_res", v_res)):
        _need(fn, name, t, L.plane_bytes(64))
    _need_meta(fn, L, meta, b + 1)
    lay, met = L.c(), meta.c()
    _check("lynx_kv_encode", load().lynx_kv_encode(
        ctypes.byref(lay), b, T, _ptr(block_table), _ptr(k), _ptr(v), _ptr(k_anc), _ptr(v_anc),
        _ptr(k_res), _ptr(v_res), ctypes.byref(met), _stream(stream)))


def lynx_kv_merge(anc, res, codes, n_packed_bytes: int | None = None, stream=None) -> None:
    n = anc.numel() if n_packed_bytes is None else n_packed_bytes
    if n > anc.numel() or n > res.numel() or 2 * n > codes.numel():
        raise ValueError("lynx_kv_merge: the planes hold fewer bytes than asked for")
    _check("lynx_kv_merge", load().lynx_kv_merge(_ptr(anc), _ptr(res), _ptr(codes), n,
                                                 _stream(stream)))


def lynx_attn_workspace_bytes(L: Layout, B: int, Hq: int, num_queries: int,
                              max_seq_len: int) -> int:
    lay = L.c()
    return int(load().lynx_attn_workspace_bytes(ctypes.byref(lay), B, Hq, num_queries,
                                                 max_seq_len))


# Arrival counters at the head of every attention workspace (lynx.h).
ATTN_COUNTER_BYTES = 262144


def workspace(L: Layout, B: int, Hq: int, num_queries: int, max_seq_len: int,
              device="cuda") -> torch.Tensor:
    """A device buffer of lynx_attn_workspace_bytes() bytes (allocated by
    torch), zero-filled: the arrival counters at its head must start at zero."""
    n = lynx_attn_workspace_bytes(L, B, Hq, num_queries, max_seq_len)
    return torch.zeros(max(n, ATTN_COUNTER_BYTES), dtype=torch.uint8, device=device)


def lynx_attn_anchor_decode(L: Layout, B: int, Hq: int, max_seq_len: int, seq_lens,
                            block_table, k_anc, v_anc, meta: Meta, q, out, lse=None,
                            workspace_buf=None, stream=None) -> None:
    fn = "lynx_attn_anchor_decode"
    _need_attn(fn, L, B, seq_lens, block_table, (k_anc, v_anc), 64, meta)
    _need(fn, "q", q, B * Hq * HEAD_DIM * 2)
    _need(fn, "out", out, B * Hq * HEAD_DIM * 2)
    _need(fn, "lse", lse, B * Hq * 4)
    lay, met = L.c(), meta.c()
    ws = workspace_buf
    _check("lynx_attn_anchor_decode", load().lynx_attn_anchor_decode(
        ctypes.byref(lay), B, Hq, max_seq_len, _ptr(seq_lens), _ptr(block_table), _ptr(k_anc),
        _ptr(v_anc), ctypes.byref(met), _ptr(q), _ptr(out), _ptr(lse), _ptr(ws),
        0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)))


def lynx_attn_anchor_decode_split(anchor_bits: int, L: Layout, B: int, Hq: int, max_seq_len: int,
                                  seq_lens, block_table, k_anc, v_anc, meta: Meta, q, out, lse=None,
                                  workspace_buf=None, stream=None) -> None:
    """Decode over the A-bit anchor planes of a split width (rows of 16 A bytes)."""
    fn = "lynx_attn_anchor_decode_split"
    if anchor_bits not in (2, 4, 6):
        raise LynxError(fn, LYNX_EINVAL)
    _need_attn(fn, L, B, seq_lens, block_table, (k_anc, v_anc), 16 * anchor_bits, meta)
    _need(fn, "q", q, B * Hq * HEAD_DIM * 2)
    _need(fn, "out", out, B * Hq * HEAD_DIM * 2)
    _need(fn, "lse", lse, B * Hq * 4)
    lay, met = L.c(), meta.c()
    ws = workspace_buf
    _check(fn, load().lynx_attn_anchor_decode_split(
        anchor_bits, ctypes.byref(lay), B, Hq, max_seq_len, _ptr(seq_lens), _ptr(block_table),
        _ptr(k_anc), _ptr(v_anc), ctypes.byref(met), _ptr(q), _ptr(out), _ptr(lse), _ptr(ws),
        0 if ws is None else ws.numel() * ws.element_size(), _stream(stream)))


# Scratch held by the library for lynx_attn_anchor_decode_noalloc (lynx.h).
NOALLOC_SCRATCH_BYTES = 16 << 20


def lynx_attn_anchor_decode_noalloc(L: Layout, B: int, Hq: int, max_seq_len: int, seq_lens,
                                    block_table, k_anc, v_anc, meta: Meta, q, out, lse=None,
                                    stream=None) -> None:
    """lynx_attn_anchor_decode without a workspace: the library's own static
    scratch (calls that overlap on one GPU race)."""
    fn = "lynx_attn_anchor_decode_noalloc"
    _need_attn(fn, L, B, seq_lens, block_table, (k_anc, v_anc), 64, meta)
    _need(fn, "q", q, B * Hq * HEAD_DIM * 2)
    _need(fn, "out", out, B * Hq * HEAD_DIM * 2)
    _need(fn, "lse", lse, B * Hq * 4)
    lay, met = L.c(), meta.c()
    _check("lynx_attn_anchor_decode_noalloc", load().lynx_attn_anchor_decode_noalloc(
        ctypes.byref(lay), B, Hq, max_seq_len, _ptr(seq_lens), _ptr(block_table), _ptr(k_anc),
        _ptr(v_anc), ctypes.byref(met), _ptr(q), _ptr(out), _ptr(lse), _stream(stream)))


def lynx_attn_anchor_decode_tail(L: Layout, B: int, Hq: int, max_seq_len: int, seq_lens,
                                 block_table, k_anc, v_anc, meta: Meta, q, k_tail, v_tail, out,
                                 lse=None, workspace_buf=None, stream=None) -> None:
    """Anchor decode that also attends the BF16 tail k_tail / v_tail
    ([B][n_tail][Hkv][128], or None for n_tail = 0)."""
    fn = "lynx_attn_anchor_decode_tail"
    _need_attn(fn, L, B, seq_lens, block_table, (k_anc, v_anc), 64, meta)
    _need(fn, "q", q, B * Hq * HEAD_DIM * 2)
    _need(fn, "out", out, B * Hq * HEAD_DIM * 2)
    _need(fn, "lse", lse, B * Hq * 4)
    if k_tail is not None:
        nt = int(k_tail.shape[1])
        _need(fn, "k_tail", k_tail, B * nt * L.num_kv_heads * HEAD_DIM * 2)
        _need(fn, "v_tail", v_tail, B * nt * L.num_kv_heads * HEAD_DIM * 2)
    lay, met = L.c(), meta.c()
    ws = workspace_buf
    n_tail = 0 if k_tail is None else int(k_tail.shape[1])
    _check("lynx_attn_anchor_decode_tail", load().lynx_attn_anchor_decode_tail(
        ctypes.byref(lay), B, Hq, max_seq_len, _ptr(seq_lens), _ptr(block_table), _ptr(k_anc),
        _ptr(v_anc), ctypes.byref(met), _ptr(q), n_tail, _ptr(k_tail), _ptr(v_tail), _ptr(out),
        _ptr(lse), _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(),
        _stream(stream)))


def lynx_spec_accept_workspace_bytes(B: int, k: int, vocab: int) -> int:
    return int(load().lynx_spec_accept_workspace_bytes(B, k, vocab))


def lynx_spec_accept_greedy(target_logits, draft_tokens, accepted, next_token,
                            workspace_buf=None, stream=None) -> None:
    """target_logits fp32 [B][k+1][V], draft_tokens int32 [B][k]; writes
    accepted and next_token (int32 [B]).  workspace_buf: None allocates
    lynx_spec_accept_workspace_bytes() bytes with torch."""
    B, k1, V = (int(x) for x in target_logits.shape)
    ws = workspace_buf
    if ws is None:
        n = lynx_spec_accept_workspace_bytes(B, k1 - 1, V)
        ws = torch.empty(max(n, 16), dtype=torch.uint8, device=target_logits.device)
    _check("lynx_spec_accept_greedy", load().lynx_spec_accept_greedy(
        B, k1 - 1, V, _ptr(target_logits), _ptr(draft_tokens), _ptr(accepted), _ptr(next_token),
        _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def lynx_spec_accept_sample(target_probs, draft_probs, draft_tokens, uniforms, accepted,
                            next_token, workspace_buf=None, stream=None) -> None:
    """target_probs fp32 [B][k+1][V], draft_probs fp32 [B][k][V], draft_tokens
    int32 [B][k], uniforms fp32 [B][k+1]; writes accepted and next_token
    (int32 [B]).  workspace_buf: None allocates
    lynx_spec_accept_workspace_bytes() bytes with torch."""
    B, k1, V = (int(x) for x in target_probs.shape)
    ws = workspace_buf
    if ws is None:
        n = lynx_spec_accept_workspace_bytes(B, k1 - 1, V)
        ws = torch.empty(max(n, 16), dtype=torch.uint8, device=target_probs.device)
    _check("lynx_spec_accept_sample", load().lynx_spec_accept_sample(
        B, k1 - 1, V, _ptr(target_probs), _ptr(draft_probs), _ptr(draft_tokens), _ptr(uniforms),
        _ptr(accepted), _ptr(next_token), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def lynx_attn_verify(L: Layout, B: int, Hq: int, k: int, max_seq_len: int, seq_lens,
                     block_table, k_codes, v_codes, meta: Meta, q, k_new, v_new, out,
                     workspace_buf=None, stream=None) -> None:
    fn = "lynx_attn_verify"
    _need_attn(fn, L, B, seq_lens, block_table, (k_codes, v_codes), 128, meta)
    _need(fn, "q", q, B * k * Hq * HEAD_DIM * 2)
    _need(fn, "out", out, B * k * Hq * HEAD_DIM * 2)
    _need(fn, "k_new", k_new, B * k * L.num_kv_heads * HEAD_DIM * 2)
    _need(fn, "v_new", v_new, B * k * L.num_kv_heads * HEAD_DIM * 2)
    lay, met = L.c(), meta.c()
    ws = workspace_buf
    _check("lynx_attn_verify", load().lynx_attn_verify(
        ctypes.byref(lay), B, Hq, k, max_seq_len, _ptr(seq_lens), _ptr(block_table),
        _ptr(k_codes), _ptr(v_codes), ctypes.byref(met), _ptr(q), _ptr(k_new), _ptr(v_new),
        _ptr(out), _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(),
        _stream(stream)))


# ----------------------------------------------------------------------------
# Allocation helpers (torch device memory only)
# ----------------------------------------------------------------------------

@dataclass
class HMeta:
    """fp32 metadata of the hierarchical codec (device): page minimum and
    range [B][Hkv][ceil(max_tokens/256)][128], chunk mean and scale
    [B][Hkv][ceil(max_tokens/32)][128], for K and V."""
    k_gmin: torch.Tensor
    k_gscale: torch.Tensor
    k_mu: torch.Tensor
    k_sigma: torch.Tensor
    v_gmin: torch.Tensor
    v_gscale: torch.Tensor
    v_mu: torch.Tensor
    v_sigma: torch.Tensor

    @staticmethod
    def empty(L: Layout, B: int, device="cuda") -> "HMeta":
        pg = (B, L.num_kv_heads, -(-L.max_tokens // 256), HEAD_DIM)
        ch = (B, L.num_kv_heads, -(-L.max_tokens // 32), HEAD_DIM)
        z = lambda shape: torch.zeros(shape, dtype=torch.float32, device=device)
        return HMeta(z(pg), z(pg), z(ch), z(ch), z(pg), z(pg), z(ch), z(ch))

    def c(self) -> lynx_hmeta:
        return lynx_hmeta(*(_ptr(getattr(self, f)) for f, _ in lynx_hmeta._fields_))


def lynx_kv_encode_split(L: Layout, anchor_bits: int, b: int, T: int, block_table, k, v, k_anc, v_anc,
                         k_res, v_res, meta: Meta, stream=None) -> None:
    """k, v: BF16 [T][Hkv][128]; planes: uint8 device tensors of rows of
    16 anchor_bits (anchor) and 16 (8 - anchor_bits) (residual) bytes."""
    fn = "lynx_kv_encode_split"
    _need(fn, "k", k, T * L.num_kv_heads * HEAD_DIM * 2)
    _need(fn, "v", v, T * L.num_kv_heads * HEAD_DIM * 2)
    _need(fn, "block_table", block_table, (b + 1) * L.max_blocks_per_seq * 4)
    if 0 < anchor_bits < 8:
        for name, t, w in (("k_anc", k_anc, anchor_bits), ("v_anc", v_anc, anchor_bits),
                           ("k_res", k_res, 8 - anchor_bits), ("v_res", v_res, 8 - anchor_bits)):
            _need(fn, name, t, L.plane_bytes(16 * w))
    _need_meta(fn, L, meta, b + 1)
    lay, met = L.c(), meta.c()
    _check("lynx_kv_encode_split", load().lynx_kv_encode_split(
        ctypes.byref(lay), anchor_bits, b, T, _ptr(block_table), _ptr(k), _ptr(v), _ptr(k_anc),
        _ptr(v_anc), _ptr(k_res), _ptr(v_res), ctypes.byref(met), _stream(stream)))


def lynx_kv_merge_split(anchor_bits: int, anc, res, codes, stream=None) -> None:
    """Rows of A-bit anchors and (8 - A)-bit residuals -> rows of 128 codes."""
    n_rows = anc.numel() // (16 * anchor_bits)
    if (anc.numel() != n_rows * 16 * anchor_bits or res.numel() != n_rows * 16 * (8 - anchor_bits)
            or codes.numel() < n_rows * 128):
        raise ValueError("lynx_kv_merge_split: plane sizes do not match one another")
    _check("lynx_kv_merge_split", load().lynx_kv_merge_split(
        anchor_bits, n_rows, _ptr(anc), _ptr(res), _ptr(codes), _stream(stream)))


def lynx_kv_dequant_anchor_split(L: Layout, anchor_bits: int, b: int, T: int, block_table, k_anc, v_anc,
                                 meta: Meta, k_out, v_out, stream=None) -> None:
    """k_out, v_out: BF16 [T][Hkv][128] (device, written)."""
    fn = "lynx_kv_dequant_anchor_split"
    _need(fn, "block_table", block_table, (b + 1) * L.max_blocks_per_seq * 4)
    if 0 < anchor_bits < 8:
        _need(fn, "k_anc", k_anc, L.plane_bytes(16 * anchor_bits))
        _need(fn, "v_anc", v_anc, L.plane_bytes(16 * anchor_bits))
    _need_meta(fn, L, meta, b + 1)
    _need(fn, "k_out", k_out, T * L.num_kv_heads * HEAD_DIM * 2)
    _need(fn, "v_out", v_out, T * L.num_kv_heads * HEAD_DIM * 2)
    lay, met = L.c(), meta.c()
    _check("lynx_kv_dequant_anchor_split", load().lynx_kv_dequant_anchor_split(
        ctypes.byref(lay), anchor_bits, b, T, _ptr(block_table), _ptr(k_anc), _ptr(v_anc),
        ctypes.byref(met), _ptr(k_out), _ptr(v_out), _stream(stream)))


# codec variants of the hierarchical codec (lynx.h LYNX_HQ_*)
LYNX_HQ_BIASED, LYNX_HQ_CENTRED, LYNX_HQ_INT4 = 0, 1, 2


def lynx_hkv_encode(L: Layout, b: int, T: int, block_table, k, v, alpha: float, variant: int,
                    k_anc, v_anc, k_res, v_res, hmeta: HMeta, stream=None) -> None:
    """k_res, v_res may be None for LYNX_HQ_INT4."""
    fn = "lynx_hkv_encode"
    _need(fn, "k", k, T * L.num_kv_heads * HEAD_DIM * 2)
    _need(fn, "v", v, T * L.num_kv_heads * HEAD_DIM * 2)
    _need(fn, "block_table", block_table, (b + 1) * L.max_blocks_per_seq * 4)
    for name, t in (("k_anc", k_anc), ("v_anc", v_anc), ("k_res", k_res), ("v_res", v_res)):
        _need(fn, name, t, L.plane_bytes(64))
    pg = (b + 1) * L.num_kv_heads * -(-L.max_tokens // 256) * HEAD_DIM * 4
    ch = (b + 1) * L.num_kv_heads * -(-L.max_tokens // 32) * HEAD_DIM * 4
    for t in ("k", "v"):
        _need(fn, f"hmeta.{t}_gmin", getattr(hmeta, f"{t}_gmin"), pg)
        _need(fn, f"hmeta.{t}_gscale", getattr(hmeta, f"{t}_gscale"), pg)
        _need(fn, f"hmeta.{t}_mu", getattr(hmeta, f"{t}_mu"), ch)
        _need(fn, f"hmeta.{t}_sigma", getattr(hmeta, f"{t}_sigma"), ch)
    lay, met = L.c(), hmeta.c()
    _check("lynx_hkv_encode", load().lynx_hkv_encode(
        ctypes.byref(lay), b, T, _ptr(block_table), _ptr(k), _ptr(v), alpha, variant, _ptr(k_anc),
        _ptr(v_anc), _ptr(k_res), _ptr(v_res), ctypes.byref(met), _stream(stream)))


def lynx_hkv_dequant(L: Layout, b: int, T: int, block_table, full: bool, k_plane, v_plane,
                     alpha: float, variant: int, hmeta: HMeta, k_out, v_out, stream=None) -> None:
    """k_out, v_out: BF16 [T][Hkv][128] (device, written)."""
    fn = "lynx_hkv_dequant"
    _need(fn, "block_table", block_table, (b + 1) * L.max_blocks_per_seq * 4)
    _need(fn, "k_plane", k_plane, L.plane_bytes(128 if full else 64))
    _need(fn, "v_plane", v_plane, L.plane_bytes(128 if full else 64))
    _need(fn, "k_out", k_out, T * L.num_kv_heads * HEAD_DIM * 2)
    _need(fn, "v_out", v_out, T * L.num_kv_heads * HEAD_DIM * 2)
    pg = (b + 1) * L.num_kv_heads * -(-L.max_tokens // 256) * HEAD_DIM * 4
    ch = (b + 1) * L.num_kv_heads * -(-L.max_tokens // 32) * HEAD_DIM * 4
    for t in ("k", "v"):
        _need(fn, f"hmeta.{t}_gmin", getattr(hmeta, f"{t}_gmin"), pg)
        _need(fn, f"hmeta.{t}_gscale", getattr(hmeta, f"{t}_gscale"), pg)
        _need(fn, f"hmeta.{t}_mu", getattr(hmeta, f"{t}_mu"), ch)
        _need(fn, f"hmeta.{t}_sigma", getattr(hmeta, f"{t}_sigma"), ch)
    lay, met = L.c(), hmeta.c()
    _check("lynx_hkv_dequant", load().lynx_hkv_dequant(
        ctypes.byref(lay), b, T, _ptr(block_table), 1 if full else 0, _ptr(k_plane), _ptr(v_plane),
        alpha, variant, ctypes.byref(met), _ptr(k_out), _ptr(v_out), _stream(stream)))


def lynx_serialized_bytes(num_kv_heads: int, n_tokens: int) -> tuple[int, int]:
    """(anchor_bytes, residual_bytes) of an object of n_tokens tokens."""
    a, r = ctypes.c_size_t(), ctypes.c_size_t()
    _check("lynx_serialized_bytes", load().lynx_serialized_bytes(num_kv_heads, n_tokens,
                                                                 ctypes.byref(a), ctypes.byref(r)))
    return int(a.value), int(r.value)


def lynx_kv_serialize(num_kv_heads: int, n_tokens: int, k, v, anchor_buf, residual_buf,
                      stream=None) -> None:
    """k, v: BF16 [n_tokens][Hkv][128] (an object's tokens); the buffers are
    uint8 device tensors of lynx_serialized_bytes() bytes."""
    fn = "lynx_kv_serialize"
    _need(fn, "k", k, n_tokens * num_kv_heads * HEAD_DIM * 2)
    _need(fn, "v", v, n_tokens * num_kv_heads * HEAD_DIM * 2)
    if num_kv_heads > 0 and n_tokens > 0:
        na, nr = lynx_serialized_bytes(num_kv_heads, n_tokens)
        _need(fn, "anchor_buf", anchor_buf, na)
        _need(fn, "residual_buf", residual_buf, nr)
    _check("lynx_kv_serialize", load().lynx_kv_serialize(
        num_kv_heads, n_tokens, _ptr(k), _ptr(v), _ptr(anchor_buf), _ptr(residual_buf),
        _stream(stream)))


def lynx_kv_deserialize_anchor(L: Layout, b: int, t0: int, n_tokens: int, block_table, anchor_buf,
                               k_anc, v_anc, meta: Meta, stream=None) -> None:
    fn = "lynx_kv_deserialize_anchor"
    _need(fn, "block_table", block_table, (b + 1) * L.max_blocks_per_seq * 4)
    if n_tokens > 0:
        _need(fn, "anchor_buf", anchor_buf, lynx_serialized_bytes(L.num_kv_heads, n_tokens)[0])
    _need(fn, "k_anc", k_anc, L.plane_bytes(64))
    _need(fn, "v_anc", v_anc, L.plane_bytes(64))
    _need_meta(fn, L, meta, b + 1)
    lay, met = L.c(), meta.c()
    _check("lynx_kv_deserialize_anchor", load().lynx_kv_deserialize_anchor(
        ctypes.byref(lay), b, t0, n_tokens, _ptr(block_table), _ptr(anchor_buf), _ptr(k_anc),
        _ptr(v_anc), ctypes.byref(met), _stream(stream)))


def lynx_kv_deserialize_residual(L: Layout, b: int, t0: int, n_tokens: int, block_table,
                                 residual_buf, k_anc, v_anc, k_codes, v_codes,
                                 stream=None) -> None:
    fn = "lynx_kv_deserialize_residual"
    _need(fn, "block_table", block_table, (b + 1) * L.max_blocks_per_seq * 4)
    if n_tokens > 0:
        _need(fn, "residual_buf", residual_buf, lynx_serialized_bytes(L.num_kv_heads, n_tokens)[1])
    for name, t, rb in (("k_anc", k_anc, 64), ("v_anc", v_anc, 64), ("k_codes", k_codes, 128),
                        ("v_codes", v_codes, 128)):
        _need(fn, name, t, L.plane_bytes(rb))
    lay = L.c()
    _check("lynx_kv_deserialize_residual", load().lynx_kv_deserialize_residual(
        ctypes.byref(lay), b, t0, n_tokens, _ptr(block_table), _ptr(residual_buf), _ptr(k_anc),
        _ptr(v_anc), _ptr(k_codes), _ptr(v_codes), _stream(stream)))


@dataclass
class KVPool:
    """Nibble planes, metadata and (after merge) code planes of one layer."""
    layout: Layout
    B: int
    k_anc: torch.Tensor
    v_anc: torch.Tensor
    k_res: torch.Tensor
    v_res: torch.Tensor
    meta: Meta
    k_codes: torch.Tensor | None = None
    v_codes: torch.Tensor | None = None

    @staticmethod
    def allocate(L: Layout, B: int, device="cuda", codes: bool = True) -> "KVPool":
        n = L.plane_bytes(64)
        u8 = dict(dtype=torch.uint8, device=device)
        pool = KVPool(L, B, torch.zeros(n, **u8), torch.zeros(n, **u8), torch.zeros(n, **u8),
                      torch.zeros(n, **u8), Meta.empty(L, B, device))
        if codes:
            pool.k_codes = torch.zeros(2 * n, **u8)
            pool.v_codes = torch.zeros(2 * n, **u8)
        return pool

    @staticmethod
    def allocate_layers(L: Layout, B: int, layers: int, device="cuda", codes: bool = True):
        """Pools for `layers` layers whose planes are consecutive slices of one
        allocation per plane kind, so that a whole cache's residual planes can
        be transported and merged in one call each.  Returns (pools, whole),
        whole being a KVPool-like record of the full-length planes (its meta
        is that of layer 0 and is not used)."""
        n = L.plane_bytes(64)
        u8 = dict(dtype=torch.uint8, device=device)
        big = {name: torch.zeros(layers * n, **u8) for name in ("k_anc", "v_anc", "k_res", "v_res")}
        if codes:
            big["k_codes"] = torch.zeros(layers * 2 * n, **u8)
            big["v_codes"] = torch.zeros(layers * 2 * n, **u8)
        pools = []
        for l in range(layers):
            pool = KVPool(L, B, *(big[name][l * n:(l + 1) * n] for name in ("k_anc", "v_anc", "k_res", "v_res")),
                          Meta.empty(L, B, device))
            if codes:
                pool.k_codes = big["k_codes"][l * 2 * n:(l + 1) * 2 * n]
                pool.v_codes = big["v_codes"][l * 2 * n:(l + 1) * 2 * n]
            pools.append(pool)
        whole = KVPool(L, B, big["k_anc"], big["v_anc"], big["k_res"], big["v_res"], pools[0].meta,
                       big.get("k_codes"), big.get("v_codes"))
        return pools, whole

    def encode(self, b: int, T: int, block_table, k, v, stream=None) -> None:
        lynx_kv_encode(self.layout, b, T, block_table, k, v, self.k_anc, self.v_anc, self.k_res,
                       self.v_res, self.meta, stream)

    def merge(self, stream=None) -> None:
        lynx_kv_merge(self.k_anc, self.k_res, self.k_codes, stream=stream)
        lynx_kv_merge(self.v_anc, self.v_res, self.v_codes, stream=stream)


def contiguous_layout(Hkv: int, B: int, T: int) -> Layout:
    """One block of T tokens per sequence; block_table[b] = [b]."""
    return Layout(num_kv_heads=Hkv, block_tokens=T, max_blocks_per_seq=1, num_blocks=B,
                  max_tokens=T)
