"""Pins for the oracle's anchor decode over the A-bit anchors of a split width
(Sec. 4.2 Anchor phase with the other widths of Sec. 8), CPU only.  What the
pins rest on, other than the function itself:

  - A = 4 is the plain anchor decode: over the same plane bytes (the 4 + 4
    encode and the A = 4 split encode write the same bytes, pinned in
    test_oracle_split.py) the outputs and lse are identical;
  - the anchors obtained another way: each token's 8-bit codes from the plain
    4 + 4 encode and merge (pinned on their own), cut to their top A bits
    with integer shifts, give the anchor-only cache of the reading (code
    2^R a + (2^R - 1) / 2, R = 8 - A) in fp64; fp64 attention over that cache,
    written with numpy, agrees with the oracle to rounding;
  - the BF16 anchor pages of the split widths (oracle_dequant_anchor_split,
    pinned by hand-split codes and its error bound): fp64 attention over them
    agrees with the oracle within the worst-case bound that BF16 rounding of
    the keys and values allows (a loose bound: it ties the decode to the
    pages' convention against gross mistakes; the exact pin is the one above).
"""
import numpy as np
import pytest

import oracle
from tests._util import bf16_bits, bits_to_f64

HEAD_DIM = 128


def _cache(T, Hkv, bt, seed):
    rng = np.random.default_rng(seed)
    k = (rng.standard_normal((T, Hkv, HEAD_DIM)) * np.linspace(0.2, 6, HEAD_DIM)).astype(np.float32)
    v = rng.standard_normal((T, Hkv, HEAD_DIM)).astype(np.float32)
    L = oracle.Layout(Hkv=Hkv, bt=bt, max_blocks=-(-T // bt), max_tokens=T)
    table = rng.permutation(L.max_blocks).astype(np.int32).reshape(1, -1)
    return L, table, bf16_bits(k), bf16_bits(v)


def _encode(A, L, table, kb, vb, T):
    n_rows = L.max_blocks * L.Hkv * L.bt
    planes = {"k_anc": np.zeros(n_rows * 16 * A, np.uint8), "v_anc": np.zeros(n_rows * 16 * A, np.uint8),
              "k_res": np.zeros(n_rows * 16 * (8 - A), np.uint8), "v_res": np.zeros(n_rows * 16 * (8 - A), np.uint8)}
    meta = oracle.Meta.empty(L, 1)
    oracle.encode_split(A, L, 0, T, table, kb, vb, planes, meta)
    return planes, meta


def _encode_44(L, table, kb, vb, T):
    n = oracle.plane_bytes(L, L.max_blocks, 64)
    planes = {p: np.zeros(n, np.uint8) for p in ("k_anc", "v_anc", "k_res", "v_res")}
    meta = oracle.Meta.empty(L, 1)
    oracle.encode(L, 0, T, table, kb, vb, planes, meta)
    return planes, meta


def _queries(Hq, seed):
    rng = np.random.default_rng(seed)
    return bf16_bits(rng.standard_normal((1, Hq, HEAD_DIM)).astype(np.float32))


def _attention(q, K, V, G):
    """fp64 softmax(q K^T / sqrt(128)) V per query head (numpy); K, V [T][Hkv][128]."""
    Hq = q.shape[0]
    out = np.zeros((Hq, HEAD_DIM))
    lse = np.zeros(Hq)
    for hq in range(Hq):
        kvh = hq // G
        s = K[:, kvh, :] @ q[hq] / np.sqrt(HEAD_DIM)
        m = s.max()
        w = np.exp(s - m)
        out[hq] = (w @ V[:, kvh, :]) / w.sum()
        lse[hq] = m + np.log(w.sum())
    return out, lse


CASES = [(300, 2, 3, 16), (129, 1, 4, 128), (1, 2, 2, 1), (513, 2, 1, 32)]


@pytest.mark.parametrize("T,Hkv,G,bt", CASES)
def test_a4_is_the_plain_anchor_decode(T, Hkv, G, bt):
    L, table, kb, vb = _cache(T, Hkv, bt, seed=T + Hkv)
    planes, meta = _encode(4, L, table, kb, vb, T)
    p44, m44 = _encode_44(L, table, kb, vb, T)
    q = _queries(Hkv * G, seed=T)
    lens = np.array([T], np.int32)
    got, got_lse = oracle.anchor_decode_split(4, L, Hkv * G, lens, table, planes["k_anc"], planes["v_anc"],
                                              meta, q)
    want, want_lse = oracle.anchor_decode(L, Hkv * G, lens, table, p44["k_anc"], p44["v_anc"], m44, q)
    assert np.array_equal(got, want) and np.array_equal(got_lse, want_lse)


@pytest.mark.parametrize("A", [2, 6])
@pytest.mark.parametrize("T,Hkv,G,bt", CASES)
def test_against_anchors_cut_from_the_codes(A, T, Hkv, G, bt):
    L, table, kb, vb = _cache(T, Hkv, bt, seed=7 * A + T)
    planes, meta = _encode(A, L, table, kb, vb, T)
    p44, m44 = _encode_44(L, table, kb, vb, T)
    # the 8-bit codes of every (token, head), read through the block table
    kc = oracle.merge(p44["k_anc"], p44["k_res"]).reshape(-1, HEAD_DIM)
    vc = oracle.merge(p44["v_anc"], p44["v_res"]).reshape(-1, HEAD_DIM)
    R = 8 - A
    K = np.zeros((T, Hkv, HEAD_DIM))
    V = np.zeros((T, Hkv, HEAD_DIM))
    for t in range(T):
        for h in range(Hkv):
            row = (int(table[0, t // bt]) * Hkv + h) * bt + t % bt
            ak = (kc[row].astype(np.int64) >> R) << R
            av = (vc[row].astype(np.int64) >> R) << R
            half = ((1 << R) - 1) / 2.0
            K[t, h] = m44.k_zero[0, h, t // 128].astype(np.float64) + (ak + half) * m44.k_scale[0, h, t // 128]
            V[t, h] = float(m44.v_zero[0, h, t]) + (av + half) * float(m44.v_scale[0, h, t])
    q = _queries(Hkv * G, seed=A + T)
    got, got_lse = oracle.anchor_decode_split(A, L, Hkv * G, np.array([T], np.int32), table,
                                              planes["k_anc"], planes["v_anc"], meta, q)
    want, want_lse = _attention(bits_to_f64(q[0]), K, V, G)
    np.testing.assert_allclose(got[0], want, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(got_lse[0], want_lse, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("A", [2, 6])
def test_against_the_bf16_anchor_pages(A):
    """Within the bound BF16 rounding of the anchor pages allows: each key and
    value element is off by at most 2^-9 of itself, so a score by at most
    d = sum_d |q_d| |k_d| 2^-9 / sqrt(128), each softmax weight by a factor
    within exp(+-2 d), and the output by max|v| (2^-9 + exp(2 d) - 1)."""
    T, Hkv, G, bt = 400, 2, 3, 16
    L, table, kb, vb = _cache(T, Hkv, bt, seed=100 + A)
    planes, meta = _encode(A, L, table, kb, vb, T)
    kp, vp = oracle.dequant_anchor_split(A, L, 0, T, table, planes["k_anc"], planes["v_anc"], meta)
    K, V = bits_to_f64(kp), bits_to_f64(vp)
    q = _queries(Hkv * G, seed=200 + A)
    qf = bits_to_f64(q[0])
    got, _ = oracle.anchor_decode_split(A, L, Hkv * G, np.array([T], np.int32), table,
                                        planes["k_anc"], planes["v_anc"], meta, q)
    want, _ = _attention(qf, K, V, G)
    for hq in range(Hkv * G):
        kvh = hq // G
        d = (np.abs(K[:, kvh, :]) @ np.abs(qf[hq])).max() * 2.0 ** -9 / np.sqrt(HEAD_DIM)
        vmax = np.abs(V[:, kvh, :]).max() * (1 + 2.0 ** -9)
        bound = vmax * (2.0 ** -9 + np.expm1(2 * d))
        assert np.abs(got[0, hq] - want[hq]).max() <= bound, (hq, bound)
