"""Pins for the oracle's codec (encode / merge / dequant), CPU only.

Each check is fixed by something other than the oracle itself: hand-derived
worked examples (tests/golden), the error bounds that linear quantization to
the nearest of 256 levels implies (Sec. 2.3) and that the anchor bucket centre
implies (Alg. 1 stage 4), brute-force nearest-level search on small inputs,
exhaustive enumeration of the split, and layout invariances.
"""
import json
from pathlib import Path

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
from tests._util import bf16_bits, bits_to_f64

GOLDEN = json.loads((Path(__file__).parent / "golden" / "codec_hand_examples.json").read_text())
F32_EPS = np.finfo(np.float32).eps


def contiguous(T, Hkv=1, max_tokens=None):
    max_tokens = max_tokens or max(T, 1)
    L = oracle.Layout(Hkv=Hkv, bt=max_tokens, max_blocks=1, max_tokens=max_tokens)
    return L, np.zeros((1, 1), np.int32)


def encode_one(k_bits, v_bits, L=None, table=None, n_blocks=1):
    T, Hkv, _ = k_bits.shape
    if L is None:
        L, table = contiguous(T, Hkv)
    planes, meta = oracle.encode_batch(L, [T], table, [k_bits], [v_bits], n_blocks)
    return L, table, planes, meta


def row_codes(planes, kind, L, t, h=0, table=None, b=0):
    """Codes of token row t via the oracle's merge of that row."""
    table = np.zeros((1, 1), np.int32) if table is None else table
    blk = table[b, t // L.bt]
    off = ((blk * L.Hkv + h) * L.bt + t % L.bt) * 64
    a = planes[f"{kind}_anc"][off:off + 64]
    r = planes[f"{kind}_res"][off:off + 64]
    return oracle.merge(a, r), a, r


# ---------------------------------------------------------------- goldens --

@pytest.mark.parametrize("case", GOLDEN["v_rows"], ids=lambda c: c["name"])
def test_golden_v_rows(case):
    row = np.full(128, case["rest"], np.float32)
    row[: len(case["row_prefix"])] = case["row_prefix"]
    v = bf16_bits(row.reshape(1, 1, 128))
    assert np.array_equal(bits_to_f64(v).reshape(-1), row.astype(np.float64)), "fixture not BF16-exact"
    k = bf16_bits(np.zeros((1, 1, 128), np.float32))
    L, table, planes, meta = encode_one(k, v)
    scale = np.float32(case["scale"]) if "scale" in case else \
        np.float32(case["scale_fraction"][0]) / np.float32(case["scale_fraction"][1])
    assert meta.v_scale[0, 0, 0] == scale
    assert meta.v_zero[0, 0, 0] == np.float32(case["zero"])
    codes, a, r = row_codes(planes, "v", L, 0)
    n = len(case["codes_prefix"])
    assert codes[:n].tolist() == case["codes_prefix"]
    assert (codes[n:] == case["codes_rest"]).all()
    nb = len(case["anchor_bytes_prefix"])
    assert a[:nb].tolist() == case["anchor_bytes_prefix"]
    assert r[:nb].tolist() == case["residual_bytes_prefix"]
    assert (a[nb:] == case["anchor_bytes_rest"]).all()
    assert (r[nb:] == case["residual_bytes_rest"]).all()
    if "anchor_values_prefix" in case:
        _, v_hat = oracle.dequant("anchor", L, 0, 1, table, planes["k_anc"], planes["v_anc"], meta)
        np.testing.assert_array_equal(v_hat[0, 0, :n], case["anchor_values_prefix"])


def test_golden_k_grouping():
    case = GOLDEN["k_case"]
    T = case["tokens"]
    x = np.zeros((T, 1, 128), np.float32)
    t = np.arange(T)
    x[:, 0, 0] = t
    x[:, 0, 1] = 2.5
    x[:, 0, 2] = np.where(t % 2 == 0, -1.0, 1.0)
    k = bf16_bits(x)
    assert np.array_equal(bits_to_f64(k), x.astype(np.float64))
    v = bf16_bits(np.zeros((T, 1, 128), np.float32))
    L, table, planes, meta = encode_one(k, v)
    for grp in case["groups"]:
        g, d = grp["g"], grp["channel"]
        scale = np.float32(grp["scale"]) if "scale" in grp else \
            np.float32(grp["scale_fraction"][0]) / np.float32(grp["scale_fraction"][1])
        assert meta.k_scale[0, 0, g, d] == scale, grp
        assert meta.k_zero[0, 0, g, d] == np.float32(grp["zero"]), grp
        for tok, code in grp["codes_at"].items():
            codes, _, _ = row_codes(planes, "k", L, int(tok))
            assert codes[d] == code, (grp, tok)
    _, a, r = row_codes(planes, "k", L, 129)
    assert a[:2].tolist() == case["token129_anchor_bytes_prefix"]
    assert r[:2].tolist() == case["token129_residual_bytes_prefix"]


# ------------------------------------------------------------- invariants --

def _bounds_check(x_f64, x_hat, scale, zero, half_width):
    """|x - x_hat| <= half_width * scale, plus fp32 rounding slack: the grid
    is built from fp32 scale/inv and fp32 (x - zero), a few ulps of the span."""
    span = np.maximum(np.abs(x_f64), np.abs(zero)) + 255.0 * scale
    slack = 8 * F32_EPS * span
    # A group whose inverse range 255/(max-min) overflows fp32 (range below
    # 255/FLT_MAX, about 7.5e-37) is stored as constant: error < that range.
    slack = np.where(scale == 0, 255.0 / float(np.finfo(np.float32).max), slack)
    err = np.abs(x_f64 - x_hat)
    assert (err <= half_width * scale + slack).all(), float((err - half_width * scale - slack).max())


def _random_kv(rng, T, Hkv, kind):
    if kind == "normal":
        x = rng.standard_normal((T, Hkv, 128)).astype(np.float32)
        x[:, :, rng.integers(0, 128, 3)] *= 10.0
    elif kind == "uniform_big":
        x = rng.uniform(-3e4, 3e4, (T, Hkv, 128)).astype(np.float32)
    elif kind == "tiny":
        x = (rng.standard_normal((T, Hkv, 128)) * 1e-38).astype(np.float32)  # denormal-range
    elif kind == "few_values":
        x = rng.choice(np.array([-2.0, -0.0, 0.0, 0.5, 3.0], np.float32), (T, Hkv, 128))
    else:
        raise ValueError(kind)
    return bf16_bits(x)


@pytest.mark.parametrize("kind", ["normal", "uniform_big", "tiny", "few_values"])
@pytest.mark.parametrize("T", [1, 15, 129, 300])
def test_error_bounds(kind, T):
    """8-bit error <= scale/2 (nearest of 256 levels); anchor-only error <= 8
    scales (bucket of 16 codes reconstructed at its centre)."""
    rng = np.random.default_rng(1000 * T + len(kind))
    Hkv = 2
    k, v = _random_kv(rng, T, Hkv, kind), _random_kv(rng, T, Hkv, kind)
    L, table, planes, meta = encode_one(k, v)
    codes = {n: oracle.merge(planes[f"{n}_anc"], planes[f"{n}_res"]) for n in ("k", "v")}
    k8, v8 = oracle.dequant("full", L, 0, T, table, codes["k"], codes["v"], meta)
    ka, va = oracle.dequant("anchor", L, 0, T, table, planes["k_anc"], planes["v_anc"], meta)
    kx, vx = bits_to_f64(k), bits_to_f64(v)
    g = np.arange(T) // 128
    ks = meta.k_scale[0][:, g, :].transpose(1, 0, 2).astype(np.float64)   # [T][Hkv][128]
    kz = meta.k_zero[0][:, g, :].transpose(1, 0, 2).astype(np.float64)
    vs = meta.v_scale[0][:, :T].T[:, :, None].astype(np.float64)          # [T][Hkv][1]
    vz = meta.v_zero[0][:, :T].T[:, :, None].astype(np.float64)
    _bounds_check(kx, k8, ks, kz, 0.5)
    _bounds_check(vx, v8, vs, vz, 0.5)
    _bounds_check(kx, ka, ks, kz, 8.0)
    _bounds_check(vx, va, vs, vz, 8.0)
    # zero is the group minimum and the top code reaches the maximum
    assert np.all(kz <= kx) and np.all(vz <= vx)


def test_nearest_level_brute_force():
    """On small random groups each code is, up to fp32 rounding of the grid,
    the nearest of the 256 levels zero + c*scale (searched exhaustively)."""
    rng = np.random.default_rng(7)
    T = 40
    k = _random_kv(rng, T, 1, "normal")
    v = _random_kv(rng, T, 1, "normal")
    L, table, planes, meta = encode_one(k, v)
    codes = oracle.merge(planes["v_anc"], planes["v_res"]).reshape(T, 128)
    levels = np.arange(256, dtype=np.float64)
    x = bits_to_f64(v)[:, 0, :]
    for t in range(T):
        s, z = float(meta.v_scale[0, 0, t]), float(meta.v_zero[0, 0, t])
        dist = np.abs(x[t][:, None] - (z + levels[None, :] * s))  # [128][256]
        best = dist.min(axis=1)
        chosen = dist[np.arange(128), codes[t]]
        assert (chosen <= best + 4 * F32_EPS * (abs(z) + 255 * s)).all()


def test_constant_and_two_valued_groups():
    T = 128
    x = np.zeros((T, 1, 128), np.float32)
    x[:, 0, 0] = 3.25                              # constant K column
    x[:, 0, 1] = np.where(np.arange(T) < 5, -7.0, 9.0)  # two-valued K column
    x[:, 0, 2] = -0.0                              # all negative zeros
    k = bf16_bits(x)
    vrow = np.full((T, 1, 128), -4.5, np.float32)  # constant V rows
    vrow[1, 0, :64] = 1.0                          # row 1 two-valued
    v = bf16_bits(vrow)
    L, table, planes, meta = encode_one(k, v)
    kc = oracle.merge(planes["k_anc"], planes["k_res"]).reshape(T, 128)
    vc = oracle.merge(planes["v_anc"], planes["v_res"]).reshape(T, 128)
    assert meta.k_scale[0, 0, 0, 0] == 0 and meta.k_zero[0, 0, 0, 0] == np.float32(3.25)
    assert (kc[:, 0] == 0).all()
    assert set(kc[:, 1].tolist()) == {0, 255}
    assert meta.k_zero[0, 0, 0, 1] == -7.0
    # -0 is stored as +0
    assert np.signbit(meta.k_zero[0, 0, 0, 2]) == False and meta.k_scale[0, 0, 0, 2] == 0
    assert meta.v_scale[0, 0, 0] == 0 and (vc[0] == 0).all()
    assert set(vc[1].tolist()) == {0, 255}
    k8, v8 = oracle.dequant("full", L, 0, T, table,
                            oracle.merge(planes["k_anc"], planes["k_res"]),
                            oracle.merge(planes["v_anc"], planes["v_res"]), meta)
    ka, va = oracle.dequant("anchor", L, 0, T, table, planes["k_anc"], planes["v_anc"], meta)
    # constant groups and the two endpoints of two-valued groups reconstruct exactly
    assert (k8[:, 0, 0] == 3.25).all() and (ka[:, 0, 0] == 3.25).all()
    assert (v8[0] == -4.5).all() and (va[0] == -4.5).all()
    assert np.allclose(k8[:, 0, 1], np.where(np.arange(T) < 5, -7.0, 9.0), rtol=0, atol=1e-5)


def test_split_merge_exhaustive():
    """Every code c in 0..255, placed at even and odd positions, comes back from
    anchor/residual planes, and the anchor is its high nibble: the split
    loses nothing (Sec. 4.2 residual phase rebuilds Q_full)."""
    # A V row per code pair: dims (2j, 2j+1) take codes (c, 255 - c) via exact
    # values 0..255 with the row's min 0 and max 255 pinned (scale 1).
    T = 256
    x = np.zeros((T, 1, 128), np.float32)
    for c in range(T):
        x[c, 0, :] = np.tile([c, 255 - c], 64)
        x[c, 0, 126:] = [0.0, 255.0]
    v = bf16_bits(x)
    k = bf16_bits(np.zeros_like(x))
    L, table, planes, meta = encode_one(k, v)
    assert (meta.v_scale[0, 0] == 1.0).all()
    codes = oracle.merge(planes["v_anc"], planes["v_res"]).reshape(T, 128)
    anc = planes["v_anc"].reshape(T, 64)
    for c in range(T):
        assert (codes[c, :126:2] == c).all() and (codes[c, 1:126:2] == 255 - c).all()
        assert anc[c, 0] == (c >> 4) | (((255 - c) >> 4) << 4)


def test_merge_is_bytewise_and_layout_agnostic():
    """Merge of a plane equals the concatenation of merges of its pieces."""
    rng = np.random.default_rng(3)
    a = rng.integers(0, 256, 4096, dtype=np.uint8)
    r = rng.integers(0, 256, 4096, dtype=np.uint8)
    whole = oracle.merge(a, r)
    parts = np.concatenate([oracle.merge(a[i:i + 100], r[i:i + 100]) for i in range(0, 4096, 100)])
    assert np.array_equal(whole, parts)
    # the high nibble of a code is always the anchor nibble
    ev = whole[0::2]
    assert np.array_equal(ev >> 4, a & 15) and np.array_equal(ev & 15, r & 15)


def test_paged_equals_contiguous():
    """Writing through a random block table only moves token rows."""
    rng = np.random.default_rng(11)
    Hkv, bt = 2, 16
    lens = [37, 64, 5]
    ks = [_random_kv(rng, T, Hkv, "normal") for T in lens]
    vs = [_random_kv(rng, T, Hkv, "normal") for T in lens]
    need = [-(-T // bt) for T in lens]
    n_blocks = sum(need)
    perm = rng.permutation(n_blocks).astype(np.int32)
    table = np.full((3, max(need)), -1, np.int32)
    pos = 0
    for b, n in enumerate(need):
        table[b, :n] = perm[pos:pos + n]
        pos += n
    Lp = oracle.Layout(Hkv=Hkv, bt=bt, max_blocks=max(need), max_tokens=max(lens))
    planes_p, meta_p = oracle.encode_batch(Lp, lens, table, ks, vs, n_blocks)
    for b, T in enumerate(lens):
        Lc, tc = contiguous(T, Hkv, max_tokens=max(lens))
        _, _, planes_c, meta_c = encode_one(ks[b], vs[b], Lc, tc)
        assert np.array_equal(meta_p.k_scale[b], meta_c.k_scale[0])
        assert np.array_equal(meta_p.v_zero[b, :, :T], meta_c.v_zero[0, :, :T])
        ka_p, va_p = oracle.dequant("anchor", Lp, b, T, table, planes_p["k_anc"], planes_p["v_anc"], meta_p)
        ka_c, va_c = oracle.dequant("anchor", Lc, 0, T, tc, planes_c["k_anc"], planes_c["v_anc"], meta_c)
        assert np.array_equal(ka_p, ka_c) and np.array_equal(va_p, va_c)


@settings(max_examples=40, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(T=st.integers(1, 260), seed=st.integers(0, 2**31 - 1),
       scale=st.sampled_from([1e-30, 1e-3, 1.0, 50.0, 1e30]))
def test_bounds_hypothesis(T, seed, scale):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal((T, 1, 128)) * scale).astype(np.float32)
    k = v = bf16_bits(x)
    L, table, planes, meta = encode_one(k, v)
    codes = oracle.merge(planes["k_anc"], planes["k_res"])
    k8, _ = oracle.dequant("full", L, 0, T, table, codes, codes, meta)
    g = np.arange(T) // 128
    ks = meta.k_scale[0][:, g, :].transpose(1, 0, 2).astype(np.float64)
    kz = meta.k_zero[0][:, g, :].transpose(1, 0, 2).astype(np.float64)
    _bounds_check(bits_to_f64(k), k8, ks, kz, 0.5)
