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

Parity note: alpha is not given by the paper, so nothing fixes the codec's
absolute accuracy; the pins fix that the oracle computes Alg. 1's stages.
"""
import numpy as np
import pytest

import oracle
from tests._util import bf16_bits, bits_to_f64

HEAD_DIM = 128


def y_of(x, alpha):
    return 127.0 * np.log1p(alpha * np.abs(np.asarray(x, np.float64))) / np.log1p(alpha)


@pytest.mark.parametrize("alpha", [1.0, 15.0, 255.0, 1e-6])
def test_thresholds_and_levels_follow_the_transform(alpha):
    theta, level = oracle.htables(alpha)
    k = np.arange(127)
    # theta_k is the fp32 value nearest the crossing Y = k + 1/2: its fp32
    # neighbours lie on either side of the crossing (up to double rounding)
    below = np.nextafter(theta, np.float32(0))
    above = np.nextafter(theta, np.float32(2))
    tol = 1e-9 * (k + 1)
    assert np.all(y_of(below, alpha) <= k + 0.5 + tol)
    assert np.all(y_of(above, alpha) >= k + 0.5 - tol)
    assert np.all(np.diff(theta) > 0)
    # levels: Y(level_i) = i, level_0 = 0, level_127 = 1
    assert level[0] == 0.0 and abs(level[127] - 1.0) <= 1e-7
    assert np.allclose(y_of(level, alpha), np.arange(128), atol=2e-4 * max(1.0, alpha) ** 0.5)


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


def _hcache(T, Hkv, x_k, x_v, alpha, bt=None):
    bt = bt or T
    L = oracle.Layout(Hkv=Hkv, bt=bt, max_blocks=-(-T // bt), max_tokens=T)
    table = np.arange(L.max_blocks, dtype=np.int32).reshape(1, -1)
    n = oracle.plane_bytes(L, L.max_blocks, 64)
    planes = {name: np.zeros(n, np.uint8) for name in ("k_anc", "v_anc", "k_res", "v_res")}
    hm = oracle.HMeta.empty(L, 1)
    oracle.hencode(L, 0, T, table, bf16_bits(x_k), bf16_bits(x_v), alpha, planes, hm)
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
    _, level = oracle.htables(alpha)
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
