"""Pins for the oracle's attention (anchor decode and verification), CPU only.

The oracle's attention is the textbook O = softmax(q K^T / sqrt(d)) V of
Sec. 2 over dequantized K/V.  It is pinned against torch's
scaled_dot_product_attention run in float64 on the CPU (a library routine
with its own implementation), against closed forms (one token; identical
keys give uniform weights), and against layout invariances (paged vs
contiguous, GQA head mapping, causal mask among drafts as in Sec. 4.3).
"""
import math

import numpy as np
import pytest
import torch

import oracle
from tests._util import bf16_bits, bits_to_f64

D = 128


def make_cache(rng, lens, Hkv, bt=None, outlier=True):
    """Encode random K/V for sequences of the given lengths with the oracle;
    bt None -> contiguous layout.  Returns (L, table, planes, meta, k, v)."""
    B = len(lens)
    ks, vs = [], []
    for T in lens:
        k = rng.standard_normal((T, Hkv, D)).astype(np.float32)
        if outlier:
            k[:, :, rng.integers(0, D, 2)] *= 8.0
        v = rng.standard_normal((T, Hkv, D)).astype(np.float32)
        ks.append(bf16_bits(k))
        vs.append(bf16_bits(v))
    max_T = max(max(lens), 1)
    if bt is None:
        L = oracle.Layout(Hkv=Hkv, bt=max_T, max_blocks=1, max_tokens=max_T)
        table = np.arange(B, dtype=np.int32).reshape(B, 1)
        n_blocks = B
    else:
        need = [-(-T // bt) for T in lens]
        n_blocks = max(sum(need), 1)
        perm = rng.permutation(n_blocks).astype(np.int32)
        table = np.full((B, max(max(need), 1)), -1, np.int32)
        pos = 0
        for b, n in enumerate(need):
            table[b, :n] = perm[pos:pos + n]
            pos += n
        L = oracle.Layout(Hkv=Hkv, bt=bt, max_blocks=table.shape[1], max_tokens=max_T)
    planes, meta = oracle.encode_batch(L, lens, table, ks, vs, n_blocks)
    return L, table, planes, meta, ks, vs


def sdpa_ref(q, k, v, mask=None):
    """torch SDPA, float64 on CPU.  q [H][n][D], k/v [H][T][D]."""
    return torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v),
        attn_mask=None if mask is None else torch.from_numpy(mask)).numpy()


@pytest.mark.parametrize("G,lens", [(1, [1]), (2, [300]), (4, [129, 17]), (8, [256, 1, 40])])
def test_anchor_decode_vs_sdpa(G, lens):
    rng = np.random.default_rng(G * 100 + len(lens))
    Hkv = 2
    Hq = G * Hkv
    L, table, planes, meta, _, _ = make_cache(rng, lens, Hkv)
    q = bf16_bits(rng.standard_normal((len(lens), Hq, D)).astype(np.float32))
    out, lse = oracle.anchor_decode(L, Hq, np.array(lens), table, planes["k_anc"],
                                    planes["v_anc"], meta, q, nthreads=2)
    for b, T in enumerate(lens):
        kh, vh = oracle.dequant("anchor", L, b, T, table, planes["k_anc"], planes["v_anc"], meta)
        # GQA: query head hq reads kv head hq // G
        kk = np.repeat(kh.transpose(1, 0, 2), G, axis=0)  # [Hq][T][D]
        vv = np.repeat(vh.transpose(1, 0, 2), G, axis=0)
        qq = bits_to_f64(q[b])[:, None, :]
        ref = sdpa_ref(qq, kk, vv)[:, 0, :]
        np.testing.assert_allclose(out[b], ref, rtol=1e-10, atol=1e-12)
        s = np.einsum("hd,htd->ht", qq[:, 0, :], kk) / math.sqrt(D)
        ref_lse = torch.logsumexp(torch.from_numpy(s), dim=1).numpy()
        np.testing.assert_allclose(lse[b], ref_lse, rtol=1e-12, atol=1e-12)


def test_single_token_closed_form():
    """T = 1: the softmax weight is 1, so the output is that token's value."""
    rng = np.random.default_rng(5)
    L, table, planes, meta, _, _ = make_cache(rng, [1], 1)
    q = bf16_bits(rng.standard_normal((1, 4, D)).astype(np.float32))
    out, _ = oracle.anchor_decode(L, 4, np.array([1]), table, planes["k_anc"], planes["v_anc"], meta, q)
    _, vh = oracle.dequant("anchor", L, 0, 1, table, planes["k_anc"], planes["v_anc"], meta)
    for h in range(4):
        np.testing.assert_array_equal(out[0, h], vh[0, 0])


def test_identical_keys_give_mean():
    """All keys equal -> uniform weights -> output is the mean of the values."""
    rng = np.random.default_rng(9)
    T = 200
    k = bf16_bits(np.tile(rng.standard_normal((1, 1, D)).astype(np.float32), (T, 1, 1)))
    v = bf16_bits(rng.standard_normal((T, 1, D)).astype(np.float32))
    L = oracle.Layout(Hkv=1, bt=T, max_blocks=1, max_tokens=T)
    table = np.zeros((1, 1), np.int32)
    planes, meta = oracle.encode_batch(L, [T], table, [k], [v], 1)
    q = bf16_bits(rng.standard_normal((1, 1, D)).astype(np.float32))
    out, lse = oracle.anchor_decode(L, 1, np.array([T]), table, planes["k_anc"], planes["v_anc"], meta, q)
    _, vh = oracle.dequant("anchor", L, 0, T, table, planes["k_anc"], planes["v_anc"], meta)
    np.testing.assert_allclose(out[0, 0], vh[:, 0, :].mean(axis=0), rtol=1e-12, atol=1e-13)


def test_paged_equals_contiguous_attention():
    rng = np.random.default_rng(21)
    lens = [70, 33, 129]
    Lp, tp, pp, mp, ks, vs = make_cache(rng, lens, 2, bt=16)
    Lc = oracle.Layout(Hkv=2, bt=max(lens), max_blocks=1, max_tokens=max(lens))
    tc = np.arange(3, dtype=np.int32).reshape(3, 1)
    pc, mc = oracle.encode_batch(Lc, lens, tc, ks, vs, 3)
    q = bf16_bits(rng.standard_normal((3, 8, D)).astype(np.float32))
    op, _ = oracle.anchor_decode(Lp, 8, np.array(lens), tp, pp["k_anc"], pp["v_anc"], mp, q)
    oc, _ = oracle.anchor_decode(Lc, 8, np.array(lens), tc, pc["k_anc"], pc["v_anc"], mc, q)
    np.testing.assert_array_equal(op, oc)


def test_unit_mask_selects_units():
    rng = np.random.default_rng(22)
    L, table, planes, meta, _, _ = make_cache(rng, [50, 60], 2)
    q = bf16_bits(rng.standard_normal((2, 4, D)).astype(np.float32))
    full, _ = oracle.anchor_decode(L, 4, np.array([50, 60]), table, planes["k_anc"], planes["v_anc"], meta, q)
    mask = np.array([[0, 1], [1, 0]], np.uint8)
    part, _ = oracle.anchor_decode(L, 4, np.array([50, 60]), table, planes["k_anc"], planes["v_anc"],
                                   meta, q, unit_mask=mask)
    np.testing.assert_array_equal(part[0, 2:], full[0, 2:])
    np.testing.assert_array_equal(part[1, :2], full[1, :2])
    assert np.isnan(part[0, :2]).all() and np.isnan(part[1, 2:]).all()


@pytest.mark.parametrize("nq,with_new", [(1, False), (3, True), (8, True), (64, True)])
def test_verify_vs_sdpa(nq, with_new):
    """Draft query i sees the context (8-bit dequant) and drafts 0..i (BF16)."""
    rng = np.random.default_rng(nq * 7 + with_new)
    lens = [90, 140]
    Hkv, G = 2, 4
    Hq = Hkv * G
    L, table, planes, meta, _, _ = make_cache(rng, lens, Hkv)
    kc = oracle.merge(planes["k_anc"], planes["k_res"])
    vc = oracle.merge(planes["v_anc"], planes["v_res"])
    q = bf16_bits(rng.standard_normal((2, nq, Hq, D)).astype(np.float32))
    kn = vn = None
    if with_new:
        kn = bf16_bits(rng.standard_normal((2, nq, Hkv, D)).astype(np.float32))
        vn = bf16_bits(rng.standard_normal((2, nq, Hkv, D)).astype(np.float32))
    out, lse = oracle.verify(L, Hq, np.array(lens), table, kc, vc, meta, q, kn, vn, nthreads=3)
    for b, T in enumerate(lens):
        kh, vh = oracle.dequant("full", L, b, T, table, kc, vc, meta)
        kk, vv = kh.transpose(1, 0, 2), vh.transpose(1, 0, 2)        # [Hkv][T][D]
        mask = np.zeros((nq, T), bool) | True
        if with_new:
            kk = np.concatenate([kk, bits_to_f64(kn[b]).transpose(1, 0, 2)], axis=1)
            vv = np.concatenate([vv, bits_to_f64(vn[b]).transpose(1, 0, 2)], axis=1)
            causal = np.tril(np.ones((nq, nq), bool))
            mask = np.concatenate([mask, causal], axis=1)
        kk, vv = np.repeat(kk, G, axis=0), np.repeat(vv, G, axis=0)
        qq = bits_to_f64(q[b]).transpose(1, 0, 2)                     # [Hq][nq][D]
        ref = sdpa_ref(qq, kk, vv, mask)                               # [Hq][nq][D]
        np.testing.assert_allclose(out[b], ref.transpose(1, 0, 2), rtol=1e-10, atol=1e-12)


def test_verify_without_drafts_is_decode_over_full_codes():
    """With no draft tokens each verification row is an ordinary decode over
    the 8-bit cache: rows with equal queries give equal outputs."""
    rng = np.random.default_rng(31)
    L, table, planes, meta, _, _ = make_cache(rng, [77], 1)
    kc = oracle.merge(planes["k_anc"], planes["k_res"])
    vc = oracle.merge(planes["v_anc"], planes["v_res"])
    q1 = rng.standard_normal((1, 1, 2, D)).astype(np.float32)
    q = bf16_bits(np.concatenate([q1, q1, -q1], axis=1))
    out, _ = oracle.verify(L, 2, np.array([77]), table, kc, vc, meta, q)
    np.testing.assert_array_equal(out[0, 0], out[0, 1])
    assert not np.allclose(out[0, 0], out[0, 2])


@pytest.mark.parametrize("n_tail,lens", [(1, [50, 0]), (5, [129, 33]), (64, [300, 1])])
def test_anchor_decode_tail_vs_sdpa(n_tail, lens):
    """Decode with the tokens generated since the context arrived: the query
    sees the anchor-only context and every BF16 tail token (an empty context
    leaves the tail alone)."""
    rng = np.random.default_rng(600 + n_tail)
    Hkv, G = 2, 4
    Hq = Hkv * G
    L, table, planes, meta, _, _ = make_cache(rng, lens, Hkv)
    B = len(lens)
    q = bf16_bits(rng.standard_normal((B, Hq, D)).astype(np.float32))
    kt = bf16_bits(rng.standard_normal((B, n_tail, Hkv, D)).astype(np.float32))
    vt = bf16_bits(rng.standard_normal((B, n_tail, Hkv, D)).astype(np.float32))
    out, lse = oracle.anchor_decode(L, Hq, np.array(lens), table, planes["k_anc"], planes["v_anc"],
                                    meta, q, nthreads=2, k_tail_bits=kt, v_tail_bits=vt)
    for b, T in enumerate(lens):
        kh, vh = oracle.dequant("anchor", L, b, T, table, planes["k_anc"], planes["v_anc"], meta)
        kk = np.concatenate([kh.transpose(1, 0, 2), bits_to_f64(kt[b]).transpose(1, 0, 2)], axis=1)
        vv = np.concatenate([vh.transpose(1, 0, 2), bits_to_f64(vt[b]).transpose(1, 0, 2)], axis=1)
        kk, vv = np.repeat(kk, G, axis=0), np.repeat(vv, G, axis=0)   # [Hq][T + n_tail][D]
        qq = bits_to_f64(q[b])[:, None, :]
        ref = sdpa_ref(qq, kk, vv)[:, 0, :]
        np.testing.assert_allclose(out[b], ref, rtol=1e-10, atol=1e-12)
        s = np.einsum("hd,htd->ht", qq[:, 0, :], kk) / math.sqrt(D)
        np.testing.assert_allclose(lse[b], torch.logsumexp(torch.from_numpy(s), dim=1).numpy(),
                                   rtol=1e-12, atol=1e-12)


def test_anchor_decode_empty_tail_is_plain_decode():
    rng = np.random.default_rng(611)
    L, table, planes, meta, _, _ = make_cache(rng, [70, 9], 2)
    q = bf16_bits(rng.standard_normal((2, 4, D)).astype(np.float32))
    empty = np.zeros((2, 0, 2, D), np.uint16)
    a, la = oracle.anchor_decode(L, 4, np.array([70, 9]), table, planes["k_anc"], planes["v_anc"], meta, q)
    b, lb = oracle.anchor_decode(L, 4, np.array([70, 9]), table, planes["k_anc"], planes["v_anc"], meta, q,
                                 k_tail_bits=empty, v_tail_bits=empty)
    np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(la, lb)
