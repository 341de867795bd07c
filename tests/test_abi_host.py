"""Host-side checks of liblynx.so that need no GPU: it loads, exports every
entry point include/lynx.h declares, and its synchronous argument validation
rejects bad calls before touching the device."""
import ctypes
import re
import subprocess
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parent.parent
HEADER = ROOT / "include" / "lynx.h"


def declared_functions():
    text = HEADER.read_text()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lynx_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    from paper_2607_01831_amd import lynx
    if not lynx.LIBRARY.exists():
        from paper_2607_01831_amd import build
        build.build()
    return lynx.load()


def test_header_declares_the_four_operations():
    fns = declared_functions()
    for name in ("lynx_kv_encode", "lynx_kv_merge", "lynx_attn_anchor_decode",
                 "lynx_attn_verify", "lynx_attn_workspace_bytes", "lynx_strerror"):
        assert name in fns


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", str(lib._name)], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\b(lynx_[a-z_]+)\b", out))
    assert set(declared_functions()) <= exported
    assert "oracle_" not in out  # the product library holds no oracle code


def test_strerror(lib):
    from paper_2607_01831_amd import lynx
    assert lynx.lynx_strerror(0) == "success"
    for s in (-1, -2, -3, -4):
        assert "unknown" not in lynx.lynx_strerror(s)


def _layout(**kw):
    from paper_2607_01831_amd import lynx
    base = dict(num_kv_heads=8, block_tokens=16, max_blocks_per_seq=4, num_blocks=64,
                max_tokens=64)
    base.update(kw)
    return lynx.Layout(**base)


def test_workspace_bytes_host_only(lib):
    from paper_2607_01831_amd import lynx
    L = _layout()
    n1 = lynx.lynx_attn_workspace_bytes(L, 2, 32, 1, 64)
    n8 = lynx.lynx_attn_workspace_bytes(L, 2, 32, 8, 64)
    assert 0 < n1 < n8
    assert lynx.lynx_attn_workspace_bytes(L, 2, 30, 1, 64) == 0       # Hq % Hkv != 0
    assert lynx.lynx_attn_workspace_bytes(L, 2, 32, 65, 64) == 0      # k > 64
    assert lynx.lynx_attn_workspace_bytes(_layout(head_dim=64), 2, 32, 1, 64) == 0


def test_validation_rejects_before_launch(lib):
    """Calls with bad arguments return an error code and launch nothing (the
    pointers below are never dereferenced: validation fails first)."""
    from paper_2607_01831_amd import lynx
    L = _layout()
    lay = L.c()
    meta = lynx.lynx_meta(16, 32, 48, 64)
    bad_meta = lynx.lynx_meta(16, 0, 48, 64)
    E = lynx
    # encode: NULL meta pointer, unsupported head_dim, T beyond capacity, misaligned input
    assert lib.lynx_kv_encode(ctypes.byref(lay), 0, 10, 16, 16, 16, 16, 16, 16, 16,
                              ctypes.byref(bad_meta), None) == E.LYNX_EINVAL
    lay64 = _layout(head_dim=64).c()
    assert lib.lynx_kv_encode(ctypes.byref(lay64), 0, 10, 16, 16, 16, 16, 16, 16, 16,
                              ctypes.byref(meta), None) == E.LYNX_ENOTSUP
    assert lib.lynx_kv_encode(ctypes.byref(lay), 0, 65, 16, 16, 16, 16, 16, 16, 16,
                              ctypes.byref(meta), None) == E.LYNX_EINVAL
    assert lib.lynx_kv_encode(ctypes.byref(lay), 0, 10, 16, 18, 16, 16, 16, 16, 16,
                              ctypes.byref(meta), None) == E.LYNX_EINVAL
    # merge: NULL, misaligned, overlapping output
    assert lib.lynx_kv_merge(None, 16, 4096, 64, None) == E.LYNX_EINVAL
    assert lib.lynx_kv_merge(16, 40, 4096, 64, None) == E.LYNX_EINVAL
    assert lib.lynx_kv_merge(4096, 16, 4096 + 32, 64, None) == E.LYNX_EINVAL  # codes overlap anc
    assert lib.lynx_kv_merge(16, 4096, 4096 - 64, 64, None) == E.LYNX_EINVAL  # codes overlap res
    assert lib.lynx_kv_merge(16, 32, 64, 0, None) == E.LYNX_OK  # nothing to do
    # attention: Hq not a multiple of Hkv, k out of range, tail half given, workspace
    args = (16, 16, 16, 16, ctypes.byref(meta), 16, 16)
    assert lib.lynx_attn_anchor_decode(ctypes.byref(lay), 1, 12, 64, *args, None, None, 0,
                                       None) == E.LYNX_EINVAL
    assert lib.lynx_attn_anchor_decode(ctypes.byref(lay), 1, 32, 65, *args, None, None, 0,
                                       None) == E.LYNX_EINVAL
    assert lib.lynx_attn_anchor_decode(ctypes.byref(lay), 1, 32, 64, *args, None, None, 0,
                                       None) == E.LYNX_EWORKSPACE
    assert lib.lynx_attn_anchor_decode(ctypes.byref(lay), 1, 32, 64, *args, None, 16, 64,
                                       None) == E.LYNX_EWORKSPACE
    vargs = (16, 16, 16, 16, ctypes.byref(meta), 16)
    assert lib.lynx_attn_verify(ctypes.byref(lay), 1, 32, 0, 64, *vargs, None, None, 16, 16,
                                1 << 20, None) == E.LYNX_EINVAL
    assert lib.lynx_attn_verify(ctypes.byref(lay), 1, 32, 65, 64, *vargs, None, None, 16, 16,
                                1 << 20, None) == E.LYNX_EINVAL
    assert lib.lynx_attn_verify(ctypes.byref(lay), 1, 32, 4, 64, *vargs, 16, None, 16, 16,
                                1 << 20, None) == E.LYNX_EINVAL
    # the no-allocation decode rejects a call that needs more than its static
    # scratch before touching the device: 64 sequences x 8 kv heads x 16
    # heads x 512 splits of partials
    big = _layout(max_tokens=1 << 18, block_tokens=1 << 18, max_blocks_per_seq=1).c()
    assert lib.lynx_attn_anchor_decode_noalloc(ctypes.byref(big), 64, 128, 1 << 18, *args, None,
                                               None) == E.LYNX_EWORKSPACE
    assert lib.lynx_attn_anchor_decode_noalloc(ctypes.byref(lay), 1, 12, 64, *args, None,
                                               None) == E.LYNX_EINVAL
    # B == 0 is a valid empty call
    assert lib.lynx_attn_anchor_decode(ctypes.byref(lay), 0, 32, 64, None, None, None, None,
                                       ctypes.byref(meta), None, None, None, None, 0,
                                       None) == E.LYNX_OK


def test_tail_and_acceptance_validation(lib):
    """The decode-with-tail and greedy-acceptance entry points reject bad
    arguments before launching anything (no pointer below is dereferenced)."""
    from paper_2607_01831_amd import lynx
    E = lynx
    L = _layout()
    lay = L.c()
    meta = lynx.lynx_meta(16, 32, 48, 64)
    base = (16, 16, 16, 16, ctypes.byref(meta), 16)
    # n_tail out of range; a tail count without its tensors; half a tail
    assert lib.lynx_attn_anchor_decode_tail(ctypes.byref(lay), 1, 32, 64, *base, 65, 16, 16, 16,
                                            None, 16, 1 << 20, None) == E.LYNX_EINVAL
    assert lib.lynx_attn_anchor_decode_tail(ctypes.byref(lay), 1, 32, 64, *base, 3, None, None, 16,
                                            None, 16, 1 << 20, None) == E.LYNX_EINVAL
    assert lib.lynx_attn_anchor_decode_tail(ctypes.byref(lay), 1, 32, 64, *base, 3, 16, None, 16,
                                            None, 16, 1 << 20, None) == E.LYNX_EINVAL
    assert lib.lynx_attn_anchor_decode_tail(ctypes.byref(lay), 1, 32, 64, *base, 3, 16, 16, 16,
                                            None, None, 0, None) == E.LYNX_EWORKSPACE
    # acceptance: workspace size, bad k / vocab, misaligned logits, short workspace
    n = lynx.lynx_spec_accept_workspace_bytes(4, 8, 128256)
    assert n == 4 * 9 * ((128256 + 4095) // 4096) * 16
    assert lynx.lynx_spec_accept_workspace_bytes(4, 0, 100) == 0
    assert lynx.lynx_spec_accept_workspace_bytes(4, 65, 100) == 0
    assert lynx.lynx_spec_accept_workspace_bytes(4, 8, 0) == 0
    assert lib.lynx_spec_accept_greedy(2, 0, 100, 16, 16, 16, 16, 16, 1 << 20, None) == E.LYNX_EINVAL
    assert lib.lynx_spec_accept_greedy(2, 4, 100, 20, 16, 16, 16, 16, 1 << 20, None) == E.LYNX_EINVAL
    assert lib.lynx_spec_accept_greedy(2, 4, 100, 16, 16, 16, 16, 16, 8, None) == E.LYNX_EWORKSPACE
    assert lib.lynx_spec_accept_greedy(0, 4, 100, None, None, None, None, None, 0, None) == E.LYNX_OK
    smp = lambda B=2, k=4, V=100, ptrs=(16, 16, 16, 16, 16, 16), wsb=1 << 20: \
        lib.lynx_spec_accept_sample(B, k, V, *ptrs, 16, wsb, None)
    assert smp(wsb=16) == E.LYNX_EWORKSPACE
    assert smp(k=0) == E.LYNX_EINVAL
    assert smp(k=65) == E.LYNX_EINVAL
    assert smp(V=0) == E.LYNX_EINVAL
    assert smp(V=(1 << 23) + 1) == E.LYNX_EINVAL
    assert smp(B=65536) == E.LYNX_EINVAL
    assert smp(ptrs=(16, 16, 16, None, 16, 16)) == E.LYNX_EINVAL
    assert smp(ptrs=(16, 16, 16, 16, 20, 16)) == E.LYNX_EINVAL
    assert smp(B=0, ptrs=(None,) * 6) == E.LYNX_OK


def test_serdes_sizes_and_validation(lib):
    """Object buffer sizes, and the serializer / deserializer reject bad
    arguments before launching anything (no pointer below is dereferenced)."""
    from paper_2607_01831_amd import lynx
    E = lynx
    # one kv head, 130 tokens: 2 x 130 x 64 row bytes + 2 x 2 x 128 x 4 K-scalar
    # bytes + 2 x 130 x 4 V-scalar bytes; residual 2 x 130 x 64
    assert lynx.lynx_serialized_bytes(1, 130) == (19728, 16640)
    assert lynx.lynx_serialized_bytes(8, 32768) == (144 * 32768 * 8, 128 * 32768 * 8)
    a, r = ctypes.c_size_t(), ctypes.c_size_t()
    assert lib.lynx_serialized_bytes(0, 10, ctypes.byref(a), ctypes.byref(r)) == E.LYNX_EINVAL
    assert lib.lynx_serialized_bytes(2, 0, ctypes.byref(a), ctypes.byref(r)) == E.LYNX_EINVAL
    # serialize: bad count, NULL / misaligned pointers, overlapping buffers
    assert lib.lynx_kv_serialize(0, 4, 16, 16, 16, 1 << 20, None) == E.LYNX_EINVAL
    assert lib.lynx_kv_serialize(2, 4, None, 16, 16, 1 << 20, None) == E.LYNX_EINVAL
    assert lib.lynx_kv_serialize(2, 4, 16, 16, 24, 1 << 20, None) == E.LYNX_EINVAL
    assert lib.lynx_kv_serialize(2, 4, 16, 16, 1 << 20, (1 << 20) + 64, None) == E.LYNX_EINVAL
    # deserialize: t0 not a multiple of 128, past the capacity, n < 1
    L = _layout(max_blocks_per_seq=16, num_blocks=64, max_tokens=256)
    lay = L.c()
    meta = lynx.lynx_meta(16, 32, 48, 64)
    args = (16, 16, 16, 16, ctypes.byref(meta), None)
    assert lib.lynx_kv_deserialize_anchor(ctypes.byref(lay), 0, 64, 10, *args) == E.LYNX_EINVAL
    assert lib.lynx_kv_deserialize_anchor(ctypes.byref(lay), 0, 128, 129, *args) == E.LYNX_EINVAL
    assert lib.lynx_kv_deserialize_anchor(ctypes.byref(lay), 0, 0, 0, *args) == E.LYNX_EINVAL
    assert lib.lynx_kv_deserialize_anchor(ctypes.byref(lay), -1, 0, 4, *args) == E.LYNX_EINVAL
    assert lib.lynx_kv_deserialize_residual(ctypes.byref(lay), 0, 64, 10, 16, 16, 16, 16, 16, 16,
                                            None) == E.LYNX_EINVAL
    assert lib.lynx_kv_deserialize_residual(ctypes.byref(lay), 0, 0, 4, 16, None, 16, 16, 16, 16,
                                            None) == E.LYNX_EINVAL


def test_split_width_validation(lib):
    """The split-width calls reject bad widths, sizes and overlaps before
    launching anything."""
    from paper_2607_01831_amd import lynx
    E = lynx
    L = _layout(max_blocks_per_seq=16, num_blocks=64, max_tokens=256)
    lay = L.c()
    m = lynx.lynx_meta(16, 32, 48, 64)
    enc = lambda A=2, T=10, planes=(16, 16, 16, 16): lib.lynx_kv_encode_split(
        ctypes.byref(lay), A, 0, T, 16, 16, 16, *planes, ctypes.byref(m), None)
    assert enc(A=3) == E.LYNX_EINVAL
    assert enc(A=8) == E.LYNX_EINVAL
    assert enc(T=257) == E.LYNX_EINVAL
    assert enc(planes=(16, 16, 24, 16)) == E.LYNX_EINVAL
    assert enc(T=0) == E.LYNX_OK
    assert lib.lynx_kv_merge_split(5, 10, 16, 4096, 8192, None) == E.LYNX_EINVAL
    assert lib.lynx_kv_merge_split(2, 0, None, None, None, None) == E.LYNX_OK
    assert lib.lynx_kv_merge_split(2, 10, 16, 4096, 24, None) == E.LYNX_EINVAL    # misaligned
    # codes over the anchor rows (10 rows: anchors 320 bytes, codes 1280)
    assert lib.lynx_kv_merge_split(2, 10, 1024, 8192, 512, None) == E.LYNX_EINVAL
    deq = lambda A=6, T=10: lib.lynx_kv_dequant_anchor_split(
        ctypes.byref(lay), A, 0, T, 16, 16, 16, ctypes.byref(m), 16, 16, None)
    assert deq(A=1) == E.LYNX_EINVAL
    assert deq(T=-1) == E.LYNX_EINVAL
    assert deq(T=0) == E.LYNX_OK
    # decode over split-width anchors: bad width, bad heads, workspace, empty batch
    args = (16, 16, 16, 16, ctypes.byref(m), 16, 16)
    dec = lambda A=2, B=1, Hq=32, ws=None, wsb=0: lib.lynx_attn_anchor_decode_split(
        A, ctypes.byref(lay), B, Hq, 64, *args, None, ws, wsb, None)
    assert dec(A=3) == E.LYNX_EINVAL
    assert dec(A=8) == E.LYNX_EINVAL
    assert dec(Hq=12) == E.LYNX_EINVAL
    assert dec() == E.LYNX_EWORKSPACE
    assert dec(ws=16, wsb=64) == E.LYNX_EWORKSPACE
    assert lib.lynx_attn_anchor_decode_split(6, ctypes.byref(lay), 0, 32, 64, None, None, None, None,
                                             ctypes.byref(m), None, None, None, None, 0,
                                             None) == E.LYNX_OK


def test_hierarchical_codec_validation(lib):
    """The hierarchical encode / dequant reject bad arguments before
    launching anything (no pointer below is dereferenced)."""
    from paper_2607_01831_amd import lynx
    E = lynx
    L = _layout(max_blocks_per_seq=16, num_blocks=64, max_tokens=256)
    lay = L.c()
    hm = lynx.lynx_hmeta(*[16 * (i + 1) for i in range(8)])
    enc = lambda alpha=255.0, T=10, hmp=ctypes.byref(hm), planes=(16, 16, 16, 16), variant=0: \
        lib.lynx_hkv_encode(ctypes.byref(lay), 0, T, 16, 16, 16, alpha, variant, *planes, hmp, None)
    assert enc(variant=3) == E.LYNX_EINVAL
    assert enc(variant=-1) == E.LYNX_EINVAL
    assert enc(variant=E.LYNX_HQ_CENTRED, planes=(16, 16, None, 16)) == E.LYNX_EINVAL
    assert enc(alpha=0.0) == E.LYNX_EINVAL
    assert enc(alpha=-1.0) == E.LYNX_EINVAL
    assert enc(alpha=float("nan")) == E.LYNX_EINVAL
    assert enc(T=257) == E.LYNX_EINVAL
    assert enc(hmp=None) == E.LYNX_EINVAL
    assert enc(planes=(16, 16, 24, 16)) == E.LYNX_EINVAL
    bad = lynx.lynx_hmeta(16, 32, 48, 64, 80, 96, 112, 0)
    assert enc(hmp=ctypes.byref(bad)) == E.LYNX_EINVAL
    assert enc(T=0) == E.LYNX_OK
    deq = lambda full=1, alpha=255.0, T=10, variant=0: lib.lynx_hkv_dequant(
        ctypes.byref(lay), 0, T, 16, full, 16, 16, alpha, variant, ctypes.byref(hm), 16, 16, None)
    assert deq(full=2) == E.LYNX_EINVAL
    assert deq(variant=7) == E.LYNX_EINVAL
    assert deq(full=1, variant=E.LYNX_HQ_INT4) == E.LYNX_EINVAL   # the 4-bit code has no residual
    assert deq(alpha=0.0) == E.LYNX_EINVAL
    assert deq(T=300) == E.LYNX_EINVAL
    assert deq(T=0) == E.LYNX_OK


def test_binding_rejects_short_tensors(lib):
    """The Python binding checks the tensors a call reads or writes against
    the sizes the layout implies and raises ValueError before the C ABI sees
    a pointer (host tensors suffice: the check comes first)."""
    import torch

    from paper_2607_01831_amd import lynx
    L = _layout(num_kv_heads=2, block_tokens=64, max_blocks_per_seq=1, num_blocks=2, max_tokens=64)
    B, Hq, T = 2, 4, 64
    u8 = lambda n: torch.zeros(n, dtype=torch.uint8)
    planes = [u8(L.plane_bytes(64)) for _ in range(4)]
    meta = lynx.Meta.empty(L, B, device="cpu")
    table = torch.arange(B, dtype=torch.int32).view(B, 1)
    lens = torch.full((B,), T, dtype=torch.int32)
    k = torch.zeros(T, 2, 128, dtype=torch.bfloat16)
    bad = [
        # encode: short K, a sequence past the metadata rows, short planes
        lambda: lynx.lynx_kv_encode(L, 0, T, table, k[:T - 1], k, *planes, meta),
        lambda: lynx.lynx_kv_encode(L, 2, T, table, k, k, *planes, meta),
        lambda: lynx.lynx_kv_encode(L, 0, T, table, k, k, planes[0][:100], *planes[1:], meta),
        # decode: seq_lens / block_table / q / out / lse shorter than the batch
        lambda: lynx.lynx_attn_anchor_decode(L, B, Hq, T, lens[:1], table, planes[0], planes[1],
                                             meta, torch.zeros(B, Hq, 128, dtype=torch.bfloat16),
                                             torch.zeros(B, Hq, 128, dtype=torch.bfloat16)),
        lambda: lynx.lynx_attn_anchor_decode(L, B, Hq, T, lens, table[:1], planes[0], planes[1],
                                             meta, torch.zeros(B, Hq, 128, dtype=torch.bfloat16),
                                             torch.zeros(B, Hq, 128, dtype=torch.bfloat16)),
        lambda: lynx.lynx_attn_anchor_decode_noalloc(L, B, Hq, T, lens, table, planes[0], planes[1],
                                                     meta, torch.zeros(1, Hq, 128, dtype=torch.bfloat16),
                                                     torch.zeros(B, Hq, 128, dtype=torch.bfloat16)),
        lambda: lynx.lynx_attn_anchor_decode(L, B, Hq, T, lens, table, planes[0], planes[1], meta,
                                             torch.zeros(B, Hq, 128, dtype=torch.bfloat16),
                                             torch.zeros(B, Hq, 128, dtype=torch.bfloat16),
                                             torch.zeros(B * Hq - 1)),
        # verify: code planes sized for nibbles, a short draft tail
        lambda: lynx.lynx_attn_verify(L, B, Hq, 2, T, lens, table, planes[0], planes[1], meta,
                                      torch.zeros(B, 2, Hq, 128, dtype=torch.bfloat16), None, None,
                                      torch.zeros(B, 2, Hq, 128, dtype=torch.bfloat16)),
        lambda: lynx.lynx_attn_verify(L, B, Hq, 2, T, lens, table, u8(L.plane_bytes(128)),
                                      u8(L.plane_bytes(128)), meta,
                                      torch.zeros(B, 2, Hq, 128, dtype=torch.bfloat16),
                                      torch.zeros(B, 1, 2, 128, dtype=torch.bfloat16),
                                      torch.zeros(B, 2, 2, 128, dtype=torch.bfloat16),
                                      torch.zeros(B, 2, Hq, 128, dtype=torch.bfloat16)),
        # split widths: a 2-bit anchor plane sized for nibbles is too short for 6 bits
        lambda: lynx.lynx_kv_encode_split(L, 6, 0, T, table, k, k, planes[0], planes[1],
                                          planes[2], planes[3], meta),
    ]
    for i, call in enumerate(bad):
        with pytest.raises(ValueError):
            call()
