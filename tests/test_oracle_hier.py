"""Pins for the oracle's hierarchical non-linear codec (Alg. 1, Sec. 4.1), CPU
only.  What the pins rest on, other than the oracle itself:

  - the transform of stage 3 as the paper writes it, Y = 127 ln(1 + a|x|) /
    ln(1 + a), evaluated here with numpy: the decision thresholds sit where Y
    crosses k + 1/2, the reconstruction levels where Y = i;
  - the alpha -> 0 limit, where the transform becomes the uniform map
    I = round(127 |x|);
  - stage 4's stated properties over every code: the anchor is the
    magnitude rounded half down to a multiple of 16, the correction brings
    back the code exactly (up to the 4-bit reading at 121..127), the sign
    survives for a zero magnitude;
  - page and chunk statistics against numpy's min / max / sequential fp32
    sum on the same inputs;
  - a worked example computed by hand (alpha = 1);
  - error bounds of the reconstruction.

The split has three variants (stated in lynx_oracle.c): Alg. 1's biased
split with the 4-bit clamp, the centred split that keeps every code, and the
single 4-bit code.  The centred and 4-bit ones are pinned by the same kinds
of facts: the transform with M = 7 for the 4-bit code, the split's stated
properties over every code (the centred one is a bijection of the 256 signed
codes onto the byte), the agreement of the centred and biased variants
wherever the clamp does not act, a worked example, and error bounds with no
saturation term.

Parity note: alpha is not given by the paper, so nothing fixes the codec's
absolute accuracy; the pins fix that the oracle computes Alg. 1's stages.
"""
import numpy as np
import pytest

import oracle
from tests._util import bf16_bits, bits_to_f64

HEAD_DIM = 128


def y_of(x, alpha, M=127):
    return M * np.log1p(alpha * np.abs(np.asarray(x, np.float64))) / np.log1p(alpha)


@pytest.mark.parametrize("variant,M", [("biased", 127), ("centred", 127), ("int4", 7)])
@pytest.mark.parametrize("alpha", [1.0, 15.0, 255.0, 1e-6])
def test_thresholds_and_levels_follow_the_transform(alpha, variant, M):
    theta, level, alevel = oracle.htables(alpha, variant)
    assert len(theta) == M and len(level) == M + 1
    k = np.arange(M)
    # theta_k is the fp32 value nearest the crossing Y = k + 1/2: its fp32
    # neighbours lie on either side of the crossing (up to double rounding)
    below = np.nextafter(theta, np.float32(0))
    above = np.nextafter(theta, np.float32(2))
    tol = 1e-9 * (k + 1)
    assert np.all(y_of(below, alpha, M) <= k + 0.5 + tol)
    assert np.all(y_of(above, alpha, M) >= k + 0.5 - tol)
    assert np.all(np.diff(theta) > 0)
    # levels: Y(level_i) = i, level_0 = 0, level_M = 1
    assert level[0] == 0.0 and abs(level[M] - 1.0) <= 1e-7
    assert np.allclose(y_of(level, alpha, M), np.arange(M + 1), atol=2e-4 * max(1.0, alpha) ** 0.5)
    # the centred split's anchor-only levels: Y = 16 V + 7.5, the middle of
    # the bucket of codes 16 V .. 16 V + 15
    assert np.allclose(y_of(alevel, alpha), 16 * np.arange(8) + 7.5, atol=2e-4 * max(1.0, alpha) ** 0.5)


def test_split_over_every_code():
    for I in range(128):
        for S in (-1, 0, 1):
            qa, qr = oracle.hsplit(I, S)
            assert -8 <= qa <= 7 and -8 <= qr <= 7
            V = qa if qa >= 0 else -qa - 1
            # the sign survives even for a zero magnitude (sign-aware map)
            assert (qa < 0) == (S < 0)
            # the correction restores the code (codes above 120 saturate)
            assert 16 * V - qr == min(I, 120)
            if I <= 120:
                # anchor = I rounded to a multiple of 16, halves rounded down
                assert abs(16 * V - I) <= 8
                if I % 16 == 8:
                    assert 16 * V == I - 8
            else:
                assert V == 7


def test_centred_split_over_every_code():
    seen = set()
    for I in range(128):
        for S in (-1, 0, 1):
            qa, qr = oracle.hsplit(I, S, "centred")
            assert -8 <= qa <= 7 and -8 <= qr <= 7
            V = qa if qa >= 0 else -qa - 1
            assert (qa < 0) == (S < 0)
            # the anchor is the top three bits of the magnitude, the
            # correction centred on the bucket's middle brings back every code
            assert V == I >> 4
            assert 16 * V + 8 + qr == I
            seen.add(((qa & 15) << 4) | (qr & 15))
    # signed magnitudes 0..127 onto the 256 byte values: no two collide
    assert len(seen) == 256


def test_int4_split_over_every_code():
    for I in range(8):
        for S in (-1, 0, 1):
            qa, qr = oracle.hsplit(I, S, "int4")
            assert qr == 0 and (qa < 0) == (S < 0)
            assert (qa if qa >= 0 else -qa - 1) == I
    with pytest.raises(ValueError):
        oracle.hsplit(8, 1, "int4")


def _hcache(T, Hkv, x_k, x_v, alpha, bt=None, variant="biased"):
    bt = bt or T
    L = oracle.Layout(Hkv=Hkv, bt=bt, max_blocks=-(-T // bt), max_tokens=T)
    table = np.arange(L.max_blocks, dtype=np.int32).reshape(1, -1)
    n = oracle.plane_bytes(L, L.max_blocks, 64)
    planes = {name: np.zeros(n, np.uint8) for name in ("k_anc", "v_anc", "k_res", "v_res")}
    hm = oracle.HMeta.empty(L, 1)
    oracle.hencode(L, 0, T, table, bf16_bits(x_k), bf16_bits(x_v), alpha, planes, hm, variant)
    return L, table, planes, hm


def test_worked_example_by_hand():
    """alpha = 1, one 32-token page; channel 0 of K holds [0, 2, 1 x 30], the
    other channels are constant.  By hand: gmin 0, gscale 2, X = [0, 1, 0.5..];
    the chunk mean is (0 + 1 + 15) / 32 = 0.5, Xc = [-0.5, 0.5, 0..], sigma
    0.5, Xf = [-1, 1, 0..]; |Xf| = 1 gives Y = 127, I = 127, anchor magnitude
    (127 + 7) >> 4 = 8 clamped to 7 and correction 112 - 127 clamped to -8;
    token 0 (S < 0) anchors -8 (nibble 0x8), token 1 anchors 7 (0x7), both
    corrections -8 (0x8); zeros give 0.  Full reconstruction uses code 120:
    level (2^(120/127) - 1) = 0.92503, so x = (-+0.92503 * 0.5 + 0.5) * 2 =
    0.07497 and 1.92503; anchor only, code 112: level 0.84279, x = 0.15721
    and 1.84279."""
    T = 32
    xk = np.zeros((T, 1, HEAD_DIM), np.float32)
    xk[:, 0, 1:] = 3.0
    xk[:, 0, 0] = 1.0
    xk[0, 0, 0], xk[1, 0, 0] = 0.0, 2.0
    xv = np.full((T, 1, HEAD_DIM), -1.5, np.float32)
    L, table, planes, hm = _hcache(T, 1, xk, xv, alpha=1.0)
    assert hm.k_gmin[0, 0, 0, 0] == 0.0 and hm.k_gscale[0, 0, 0, 0] == 2.0
    assert hm.k_mu[0, 0, 0, 0] == 0.5 and hm.k_sigma[0, 0, 0, 0] == 0.5
    ka, kr = planes["k_anc"].reshape(T, 64), planes["k_res"].reshape(T, 64)
    assert ka[0, 0] == 0x08 and ka[1, 0] == 0x07 and not ka[2:, 0].any()
    assert kr[0, 0] == 0x08 and kr[1, 0] == 0x08 and not kr[2:, 0].any()
    # constant channels: range 0, everything 0, reconstructed exactly
    assert not ka[:, 1:].any() and not kr[:, 1:].any()
    assert not planes["v_anc"].any() and not planes["v_res"].any()
    codes_k = oracle.merge(planes["k_anc"], planes["k_res"])
    codes_v = oracle.merge(planes["v_anc"], planes["v_res"])
    fk, fv = oracle.hdequant("full", L, 0, T, table, codes_k, codes_v, 1.0, hm)
    ak, _ = oracle.hdequant("anchor", L, 0, T, table, planes["k_anc"], planes["v_anc"], 1.0, hm)
    f = bits_to_f64(fk)
    a = bits_to_f64(ak)
    assert abs(f[0, 0, 0] - 0.07497) < 1e-3 and abs(f[1, 0, 0] - 1.92503) < 8e-3
    assert abs(a[0, 0, 0] - 0.15721) < 1e-3 and abs(a[1, 0, 0] - 1.84279) < 8e-3
    assert np.all(f[2:, 0, 0] == 1.0) and np.all(f[:, 0, 1:] == 3.0)
    assert np.all(bits_to_f64(fv) == -1.5)


def test_statistics_against_numpy():
    rng = np.random.default_rng(5)
    T, Hkv, alpha = 600, 2, 255.0
    xk = rng.standard_normal((T, Hkv, HEAD_DIM)).astype(np.float32) * 3
    xv = rng.standard_normal((T, Hkv, HEAD_DIM)).astype(np.float32)
    L, table, planes, hm = _hcache(T, Hkv, xk, xv, alpha)
    for x, gmin, gsc, mu, sig in ((xk, hm.k_gmin, hm.k_gscale, hm.k_mu, hm.k_sigma),
                                  (xv, hm.v_gmin, hm.v_gscale, hm.v_mu, hm.v_sigma)):
        xb = bits_to_f64(bf16_bits(x)).astype(np.float32)
        for h in range(Hkv):
            for p in range(-(-T // 256)):
                pg = xb[256 * p:256 * (p + 1), h, :]
                lo, hi = pg.min(axis=0), pg.max(axis=0)
                assert np.array_equal(gmin[0, h, p], lo + np.float32(0))
                assert np.array_equal(gsc[0, h, p], hi - lo)
                X = (pg - lo) * (np.float32(1) / (hi - lo))
                for c in range(-(-pg.shape[0] // 32)):
                    ch = X[32 * c:32 * (c + 1)]
                    s = np.cumsum(ch, axis=0, dtype=np.float32)[-1]   # sequential fp32 sum
                    m = s / np.float32(ch.shape[0])
                    assert np.array_equal(mu[0, h, 8 * p + c], m)
                    assert np.array_equal(sig[0, h, 8 * p + c], np.abs(ch - m).max(axis=0))


def test_alpha_to_zero_is_uniform_rounding():
    """As alpha -> 0 the transform is 127 |x|: codes are round(127 |Xf|)."""
    rng = np.random.default_rng(9)
    T, alpha = 256, 1e-6
    xk = rng.standard_normal((T, 1, HEAD_DIM)).astype(np.float32)
    L, table, planes, hm = _hcache(T, 1, xk, xk, alpha)
    xb = bits_to_f64(bf16_bits(xk)).astype(np.float32)[:, 0, :]
    lo, hi = xb.min(axis=0), xb.max(axis=0)
    X = (xb - lo) * (np.float32(1) / (hi - lo))
    codes = oracle.merge(planes["k_anc"], planes["k_res"]).reshape(T, HEAD_DIM)
    qa = ((codes >> 4).astype(np.int32) ^ 8) - 8
    qr = ((codes & 15).astype(np.int32) ^ 8) - 8
    V = np.where(qa >= 0, qa, -qa - 1)
    got = 16 * V - qr
    for c in range(T // 32):
        ch = X[32 * c:32 * (c + 1)]
        m = np.cumsum(ch, axis=0, dtype=np.float32)[-1] / np.float32(32)
        xc = ch - m
        sig = np.abs(xc).max(axis=0)
        xf = np.minimum(np.abs(xc * (np.float32(1) / sig)), 1)
        want = np.minimum(np.floor(127.0 * xf.astype(np.float64) + 0.5), 120)
        frac = np.abs(127.0 * xf - np.floor(127.0 * xf) - 0.5)
        ok = frac > 1e-3   # away from the rounding ties (the transform is not exactly linear)
        assert np.array_equal(got[32 * c:32 * (c + 1)][ok], want[ok])


@pytest.mark.parametrize("alpha", [1.0, 255.0])
def test_reconstruction_error_bounds(alpha):
    """|x - x_hat| <= (half the widest level step, or the 121..127 saturation)
    * sigma * gscale for the full code; the anchor alone is off by at most
    the distance to the nearest multiple-of-16 level."""
    rng = np.random.default_rng(int(alpha))
    T, Hkv = 512, 2
    xk = (rng.standard_normal((T, Hkv, HEAD_DIM)) * np.linspace(0.1, 8, HEAD_DIM)).astype(np.float32)
    xv = rng.standard_normal((T, Hkv, HEAD_DIM)).astype(np.float32)
    L, table, planes, hm = _hcache(T, Hkv, xk, xv, alpha, bt=64)
    _, level, _ = oracle.htables(alpha)
    lv = level.astype(np.float64)
    step = np.max(np.diff(lv[:121]))
    sat = 1.0 - lv[120]
    anc_err = max(np.max(np.abs(lv[i] - lv[16 * ((min(i, 120) + 7) >> 4 if ((min(i, 120) + 7) >> 4) <= 7 else 7)]))
                  for i in range(128))
    codes = {p: oracle.merge(planes[p + "_anc"], planes[p + "_res"]) for p in ("k", "v")}
    fk, fv = oracle.hdequant("full", L, 0, T, table, codes["k"], codes["v"], alpha, hm)
    ak, av = oracle.hdequant("anchor", L, 0, T, table, planes["k_anc"], planes["v_anc"], alpha, hm)
    for x, full, anc, gsc, sig in ((xk, fk, ak, hm.k_gscale, hm.k_sigma), (xv, fv, av, hm.v_gscale, hm.v_sigma)):
        xb = bits_to_f64(bf16_bits(x))
        g = np.repeat(gsc[0].transpose(1, 0, 2), 256, axis=0)[:T]      # [T][Hkv][128]
        s = np.repeat(sig[0].transpose(1, 0, 2), 32, axis=0)[:T]
        scale = g.astype(np.float64) * s
        slack = 4 * np.spacing(np.abs(xb).astype(np.float32)).astype(np.float64) + 2 ** -8 * np.abs(xb)
        assert np.all(np.abs(bits_to_f64(full) - xb) <= max(step / 2, sat) * scale + slack + 1e-30)
        assert np.all(np.abs(bits_to_f64(anc) - xb) <= max(anc_err, sat) * scale + slack + 1e-30)


def _worked_example_input():
    T = 32
    xk = np.zeros((T, 1, HEAD_DIM), np.float32)
    xk[:, 0, 1:] = 3.0
    xk[:, 0, 0] = 1.0
    xk[0, 0, 0], xk[1, 0, 0] = 0.0, 2.0
    xv = np.full((T, 1, HEAD_DIM), -1.5, np.float32)
    return T, xk, xv


def test_worked_example_centred_by_hand():
    """The worked example above with the centred split.  Xf = [-1, 1, 0..]:
    I = 127 gives anchor magnitude 127 >> 4 = 7 and correction
    127 - 112 - 8 = 7, so token 0 anchors -8 (0x8), token 1 anchors 7 (0x7),
    both corrections 0x7; a zero gives anchor 0 and correction -8 (0x8).
    Full reconstruction is exact here: code 127 is level 1, x = (-+1 * 0.5 +
    0.5) * 2 = 0 and 2; code 0 is level 0, x = 1.  Anchor only, code 119.5:
    level 2^(119.5/127) - 1 = 0.91979, x = 0.08021 and 1.91979; code 7.5 for
    the zeros: level 0.04178, x = 1.04178, BF16 1.0390625."""
    T, xk, xv = _worked_example_input()
    L, table, planes, hm = _hcache(T, 1, xk, xv, alpha=1.0, variant="centred")
    ka, kr = planes["k_anc"].reshape(T, 64), planes["k_res"].reshape(T, 64)
    assert ka[0, 0] == 0x08 and ka[1, 0] == 0x07 and not ka[2:, 0].any()
    assert kr[0, 0] == 0x87 and kr[1, 0] == 0x87 and np.all(kr[2:, 0] == 0x88)
    codes_k = oracle.merge(planes["k_anc"], planes["k_res"])
    codes_v = oracle.merge(planes["v_anc"], planes["v_res"])
    fk, fv = oracle.hdequant("full", L, 0, T, table, codes_k, codes_v, 1.0, hm, "centred")
    ak, _ = oracle.hdequant("anchor", L, 0, T, table, planes["k_anc"], planes["v_anc"], 1.0, hm, "centred")
    f, a = bits_to_f64(fk), bits_to_f64(ak)
    assert f[0, 0, 0] == 0.0 and f[1, 0, 0] == 2.0 and np.all(f[2:, 0, 0] == 1.0)
    assert abs(a[0, 0, 0] - 0.08021) < 1e-3 and abs(a[1, 0, 0] - 1.91979) < 8e-3
    assert np.all(a[2:, 0, 0] == 1.0390625)
    assert np.all(f[:, 0, 1:] == 3.0) and np.all(bits_to_f64(fv) == -1.5)


def test_worked_example_int4_by_hand():
    """The same input as a 4-bit code (M = 7): |Xf| = 1 gives I = 7, so token
    0 is -8 (0x8), token 1 is 7 (0x7), zeros 0; level 7 is 1, so x = 0, 2
    and 1 exactly.  A second channel holds [0, 2, 1.5, 1 x 29]: gscale 2,
    X = [0, 1, 0.75, 0.5..], mean (0 + 1 + 0.75 + 14.5) / 32 = 0.5078125,
    sigma 0.5078125 (token 0).  Token 1: Xf = 0.4921875 / 0.5078125 =
    0.9692308, Y = 7 log2(1.9692308) = 6.844, I = 7, x = (0.5078125 +
    0.5078125) * 2 = 2.03125.  Token 2: Xf = 0.2421875 / 0.5078125 =
    0.4769231, Y = 7 log2(1.4769231) = 3.938, I = 4: level 2^(4/7) - 1 =
    0.4859943, x = (0.4859943 * 0.5078125 + 0.5078125) * 2 = 1.5092034,
    BF16 1.5078125."""
    T, xk, xv = _worked_example_input()
    xk[:, 0, 2] = 1.0
    xk[0, 0, 2], xk[1, 0, 2], xk[2, 0, 2] = 0.0, 2.0, 1.5
    L, table, planes, hm = _hcache(T, 1, xk, xv, alpha=1.0, variant="int4")
    assert not planes["k_res"].any() and not planes["v_res"].any()
    ka = planes["k_anc"].reshape(T, 64)
    assert ka[0, 0] == 0x08 and ka[1, 0] == 0x07
    assert ka[0, 1] & 15 == 0x8 and ka[1, 1] & 15 == 0x7 and ka[2, 1] & 15 == 4
    assert hm.k_mu[0, 0, 0, 2] == 0.5078125 and hm.k_sigma[0, 0, 0, 2] == 0.5078125
    ak, av = oracle.hdequant("anchor", L, 0, T, table, planes["k_anc"], planes["v_anc"], 1.0, hm, "int4")
    a = bits_to_f64(ak)
    assert a[0, 0, 0] == 0.0 and a[1, 0, 0] == 2.0 and np.all(a[2:, 0, 0] == 1.0)
    assert a[0, 0, 2] == 0.0 and a[1, 0, 2] == 2.03125 and a[2, 0, 2] == 1.5078125
    assert np.all(bits_to_f64(av) == -1.5)
    with pytest.raises(ValueError):
        oracle.hdequant("full", L, 0, T, table, planes["k_anc"], planes["v_anc"], 1.0, hm, "int4")


def test_int4_alpha_to_zero_is_uniform_rounding():
    """As alpha -> 0 the 4-bit transform is 7 |x|: codes are round(7 |Xf|)."""
    rng = np.random.default_rng(11)
    T, alpha = 256, 1e-6
    xk = rng.standard_normal((T, 1, HEAD_DIM)).astype(np.float32)
    L, table, planes, hm = _hcache(T, 1, xk, xk, alpha, variant="int4")
    xb = bits_to_f64(bf16_bits(xk)).astype(np.float32)[:, 0, :]
    lo, hi = xb.min(axis=0), xb.max(axis=0)
    X = (xb - lo) * (np.float32(1) / (hi - lo))
    nib = np.zeros((T, HEAD_DIM), np.int32)
    a = planes["k_anc"].reshape(T, 64).astype(np.int32)
    nib[:, 0::2], nib[:, 1::2] = a & 15, a >> 4
    qa = (nib ^ 8) - 8
    got = np.where(qa >= 0, qa, -qa - 1)
    for c in range(T // 32):
        ch = X[32 * c:32 * (c + 1)]
        m = np.cumsum(ch, axis=0, dtype=np.float32)[-1] / np.float32(32)
        xc = ch - m
        xf = np.minimum(np.abs(xc * (np.float32(1) / np.abs(xc).max(axis=0))), 1)
        want = np.floor(7.0 * xf.astype(np.float64) + 0.5)
        ok = np.abs(7.0 * xf - np.floor(7.0 * xf) - 0.5) > 1e-4
        assert np.array_equal(got[32 * c:32 * (c + 1)][ok], want[ok])
        # the sign is that of the centred value (zeros count as positive)
        assert np.all((qa[32 * c:32 * (c + 1)] < 0) == (xc < 0))


@pytest.mark.parametrize("alpha", [1.0, 255.0])
def test_centred_agrees_with_biased_below_the_clamp(alpha):
    """Both variants share stages 1-3: wherever the biased split's clamp does
    not act (code <= 120) the merged codes name the same code and the full
    reconstructions are bit-identical; the anchors differ only in the
    bucket rule."""
    rng = np.random.default_rng(3)
    T = 512
    xk = (rng.standard_normal((T, 1, HEAD_DIM)) * 2).astype(np.float32)
    xv = rng.standard_normal((T, 1, HEAD_DIM)).astype(np.float32)
    out = {}
    for v in ("biased", "centred"):
        L, table, planes, hm = _hcache(T, 1, xk, xv, alpha, bt=128, variant=v)
        codes = oracle.merge(planes["k_anc"], planes["k_res"]).reshape(T, HEAD_DIM)
        qa = ((codes >> 4).astype(np.int32) ^ 8) - 8
        qr = ((codes & 15).astype(np.int32) ^ 8) - 8
        V = np.where(qa >= 0, qa, -qa - 1)
        I = 16 * V - qr if v == "biased" else 16 * V + 8 + qr
        fk, _ = oracle.hdequant("full", L, 0, T, table, codes.reshape(-1),
                                oracle.merge(planes["v_anc"], planes["v_res"]), alpha, hm, v)
        out[v] = (I, np.sign(qa + 0.5), fk.reshape(T, HEAD_DIM), hm)
    Ib, sb, fb, hb = out["biased"]
    Ic, sc, fc, hc = out["centred"]
    assert np.array_equal(hb.k_mu, hc.k_mu) and np.array_equal(hb.k_sigma, hc.k_sigma)
    assert np.array_equal(sb, sc)
    low = Ic <= 120
    assert np.array_equal(Ib[low], Ic[low]) and np.all(Ib[~low] == 120)
    assert np.array_equal(fb[low], fc[low])
    # every chunk's extreme element has |Xf| = 1, code 127: only the
    # centred split keeps it
    assert (~low).sum() >= T // 32


def _interval_err(recon, theta, lo_code, hi_code):
    """Largest distance from recon to a point of the |Xf| interval that codes
    lo_code .. hi_code decide: [theta[lo - 1], theta[hi]] (0 and 1 at the
    ends)."""
    th = np.concatenate([[0.0], theta.astype(np.float64), [1.0]])
    return max(abs(recon - th[lo_code]), abs(th[hi_code + 1] - recon))


@pytest.mark.parametrize("variant", ["centred", "int4"])
@pytest.mark.parametrize("alpha", [1.0, 255.0])
def test_reconstruction_error_bounds_no_saturation(alpha, variant):
    """|x - x_hat| <= e * sigma * gscale, e the largest distance from a
    reconstruction level to the |Xf| interval its code decides (the
    thresholds): for the full code every code keeps its own level (the
    centred split keeps every code, so no saturation term); for the centred
    anchor alone a bucket of 16 codes shares the level at its centre."""
    rng = np.random.default_rng(int(alpha) + 7)
    T, Hkv = 512, 2
    xk = (rng.standard_normal((T, Hkv, HEAD_DIM)) * np.linspace(0.1, 8, HEAD_DIM)).astype(np.float32)
    xv = rng.standard_normal((T, Hkv, HEAD_DIM)).astype(np.float32)
    L, table, planes, hm = _hcache(T, Hkv, xk, xv, alpha, bt=64, variant=variant)
    theta, level, alevel = oracle.htables(alpha, variant)
    lv = level.astype(np.float64)
    M = len(theta)
    full_err = max(_interval_err(lv[i], theta, i, i) for i in range(M + 1))
    if variant == "centred":
        anc_err = max(_interval_err(float(alevel[V]), theta, 16 * V, 16 * V + 15) for V in range(8))
        codes = {p: oracle.merge(planes[p + "_anc"], planes[p + "_res"]) for p in ("k", "v")}
        fk, fv = oracle.hdequant("full", L, 0, T, table, codes["k"], codes["v"], alpha, hm, variant)
    else:
        anc_err = full_err
        fk = fv = None
    ak, av = oracle.hdequant("anchor", L, 0, T, table, planes["k_anc"], planes["v_anc"], alpha, hm, variant)
    for x, full, anc, gsc, sig in ((xk, fk, ak, hm.k_gscale, hm.k_sigma), (xv, fv, av, hm.v_gscale, hm.v_sigma)):
        xb = bits_to_f64(bf16_bits(x))
        g = np.repeat(gsc[0].transpose(1, 0, 2), 256, axis=0)[:T]
        s = np.repeat(sig[0].transpose(1, 0, 2), 32, axis=0)[:T]
        scale = g.astype(np.float64) * s
        slack = 4 * np.spacing(np.abs(xb).astype(np.float32)).astype(np.float64) + 2 ** -8 * np.abs(xb)
        if full is not None:
            assert np.all(np.abs(bits_to_f64(full) - xb) <= full_err * scale + slack + 1e-30)
        assert np.all(np.abs(bits_to_f64(anc) - xb) <= anc_err * scale + slack + 1e-30)
