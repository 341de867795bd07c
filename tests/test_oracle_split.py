"""Pins for the oracle's split widths other than 4 + 4 (an A-bit anchor and an
(8 - A)-bit residual of the uniform 8-bit code, A in {2, 4, 6}; the paper
leaves other widths to future work, Sec. 8), CPU only.  What the pins rest on,
other than the oracle itself:

  - the codes do not depend on the split: merging the A / (8 - A) planes gives
    the same codes as the 4 + 4 planes of the plain encode, for every A;
  - A = 4 is the 4 + 4 codec: same plane bytes as the plain encode, and its
    anchor dequantization agrees with the plain anchor dequantization
    (fp64 zero + (16 a + 7.5) scale) to within BF16 rounding;
  - the row layout against Python integers: a row read as one little-endian
    integer holds element e at bits e W .. e W + W - 1;
  - the split of every code by hand (c >> R, c & (2^R - 1));
  - the anchor-only error bound: within scale 2^R / 2 of the code's value
    (plus BF16 rounding).
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


def _encode_split(A, L, table, kb, vb, T):
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


@pytest.mark.parametrize("A", [2, 4, 6])
def test_codes_do_not_depend_on_the_split(A):
    T = 300
    L, table, kb, vb = _cache(T, 2, 16, seed=A)
    p44, m44 = _encode_44(L, table, kb, vb, T)
    pA, mA = _encode_split(A, L, table, kb, vb, T)
    for name in ("k_scale", "k_zero", "v_scale", "v_zero"):
        assert np.array_equal(getattr(m44, name), getattr(mA, name))
    for w in ("k", "v"):
        assert np.array_equal(oracle.merge_split(A, pA[w + "_anc"], pA[w + "_res"]),
                              oracle.merge(p44[w + "_anc"], p44[w + "_res"]))
    if A == 4:
        for name in p44:
            assert np.array_equal(p44[name], pA[name])


@pytest.mark.parametrize("A", [2, 4, 6])
def test_row_layout_against_python_integers(A):
    """One token, one head: read each plane row as a little-endian integer
    and take W-bit fields; they are the code's top A and bottom R bits."""
    T = 1
    L, table, kb, vb = _cache(T, 1, 1, seed=10 + A)
    planes, _ = _encode_split(A, L, table, kb, vb, T)
    p44, _ = _encode_44(L, table, kb, vb, T)
    codes = oracle.merge(p44["k_anc"], p44["k_res"])
    R = 8 - A
    for name, W, want in (("k_anc", A, codes >> R), ("k_res", R, codes & ((1 << R) - 1))):
        big = int.from_bytes(planes[name].tobytes(), "little")
        got = [(big >> (e * W)) & ((1 << W) - 1) for e in range(HEAD_DIM)]
        assert got == [int(x) for x in want]


@pytest.mark.parametrize("A", [2, 4, 6])
def test_split_of_every_code_by_hand(A):
    """Rows holding the codes 0..127 and 128..255: merge of the hand-made
    fields gives them back."""
    R = 8 - A
    for base in (0, 128):
        c = np.arange(base, base + HEAD_DIM)
        anc = int(sum(int(x >> R) << (e * A) for e, x in enumerate(c))).to_bytes(16 * A, "little")
        res = int(sum(int(x & ((1 << R) - 1)) << (e * R) for e, x in enumerate(c))).to_bytes(16 * R, "little")
        got = oracle.merge_split(A, np.frombuffer(anc, np.uint8), np.frombuffer(res, np.uint8))
        assert np.array_equal(got, c.astype(np.uint8))


@pytest.mark.parametrize("A", [2, 4, 6])
def test_anchor_dequantization(A):
    T = 260
    L, table, kb, vb = _cache(T, 2, 32, seed=20 + A)
    planes, meta = _encode_split(A, L, table, kb, vb, T)
    ka, va = oracle.dequant_anchor_split(A, L, 0, T, table, planes["k_anc"], planes["v_anc"], meta)
    R = 8 - A
    xs = {"k": bits_to_f64(kb), "v": bits_to_f64(vb)}
    ks = np.repeat(meta.k_scale[0].transpose(1, 0, 2), 128, axis=0)[:T].astype(np.float64)
    vs = np.repeat(meta.v_scale[0].T[:, :, None], HEAD_DIM, axis=2)[:T].astype(np.float64)
    for got, x, sc in ((ka, xs["k"], ks), (va, xs["v"], vs)):
        g = bits_to_f64(got)
        slack = 2 ** -8 * np.abs(g) + 1e-30
        # quantization (half a step) plus the anchor's half range
        assert np.all(np.abs(g - x) <= sc * (0.5 + 2 ** R / 2) + slack)
    if A == 4:
        p44, m44 = _encode_44(L, table, kb, vb, T)
        ref_k, ref_v = oracle.dequant("anchor", L, 0, T, table, p44["k_anc"], p44["v_anc"], m44)
        for got, ref in ((ka, ref_k), (va, ref_v)):
            g = bits_to_f64(got)
            assert np.all(np.abs(g - ref) <= 2 ** -8 * np.abs(ref) + 1e-30)


def test_bad_widths_are_rejected():
    L, table, kb, vb = _cache(8, 1, 8, seed=1)
    with pytest.raises(ValueError):
        oracle.merge_split(3, np.zeros(48, np.uint8), np.zeros(80, np.uint8))
    planes = {n: np.zeros(16 * 8 * 8, np.uint8) for n in ("k_anc", "v_anc", "k_res", "v_res")}
    with pytest.raises(ValueError):
        oracle.encode_split(5, L, 0, 8, table, kb, vb, planes, oracle.Meta.empty(L, 1))
