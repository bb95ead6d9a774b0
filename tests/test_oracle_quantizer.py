"""Pins for the oracle's quantizer (Eq. 1-4, Sec. 4.3-4.5) against independent facts.

Each test checks the oracle against something other than itself: a worked example
derived by hand from the equations, Eq. 1's set definitions, exhaustive search over
every quantization level, round-trip bounds implied by the bitwidths, and special
thresholds under which the method reduces to a textbook sign + min-max quantizer.
"""
import numpy as np
import pytest

from tests import bruteforce as bf

D = 128


def _rand_thr(rng):
    t = np.sort(rng.normal(0, 1.5, 4).astype(np.float32))
    # make the inner interval contain zero most of the time, as calibration does
    if rng.random() < 0.8:
        m = abs(float(rng.normal(0, 0.3)))
        t[1], t[2] = -m, m
        t = np.sort(t)
    return t


def _vec(rng, d=D, scale=1.0):
    x = rng.standard_t(3, d) * scale
    return np.clip(x, -60000, 60000).astype(np.float16)


# ---------------------------------------------------------------------------- #
def test_worked_example_by_hand(ref):
    """A 64-value vector worked through Eq. 1-4 and the fused encoding by hand.

    Thresholds (lo_o, lo_i, hi_i, hi_o) = (-4, -0.46875, 0.46875, 4).
      outer : x=6 (a=6-4=2), x=-5 (a=|-5+4|=1), x=10 (a=6) -> Min 1, Max 6, sigma=15/5=3
              codes c = 3, 0, 15 -> u = 16+3=19, 15-0=15, 16+15=31
      middle: x=4 (==hi_o, so middle, a=4-0.46875=3.53125), x=-4 (==lo_o, a=3.53125),
              x=1 (a=.53125), x=-2 (a=1.53125), 53 x 2.25 (a=1.78125)
              Min .53125, Max 3.53125, sigma = fl(7/3); c = 7, 7, 0, 2, 3
              -> u = 8+7=15, 7-7=0, 8+0=8, 7-2=5, 8+3=11
      inner : x=.46875 (==hi_i, inner), x=-.46875 (==lo_i), x=0 (upper side), x=-.078125
              Min 0, Max .46875, sigma = 32; c = 15, 15, 0, rint(2.5)=2 (half-even)
              -> u = 31, 0, 16, 13
    COO (6-bit index, bit 6 = outer, bit 7 = upper side), ascending index:
      j0 c0, j1 41, j4 84, j5 05, j8 88, j9 09, j10 ca
    meta fp16: inner (0, 0.03125), middle (0.53125, fl16(fl32(3/7))), outer (1, fl16(fl32(5/15)))
    """
    x = np.full(64, 2.25, np.float32)
    x[:11] = [6.0, -5.0, 4.0, -4.0, 0.46875, -0.46875, 1.0, -2.0, 0.0, -0.078125, 10.0]
    thr = np.array([-4.0, -0.46875, 0.46875, 4.0], np.float32)
    r = ref.quantize_vector(x.astype(np.float16), thr)
    want_code = [19, 15, 15, 0, 31, 0, 8, 5, 16, 13, 31] + [11] * 53
    want_group = [2, 2, 1, 1, 0, 0, 1, 1, 0, 0, 2] + [1] * 53
    assert r["code"].tolist() == want_code
    assert r["group"].tolist() == want_group
    assert r["coo"].tolist() == [0xC0, 0x41, 0x84, 0x05, 0x88, 0x09, 0xCA]
    assert r["counts"].tolist() == [7]
    assert r["meta"].tolist() == [0x0000, 0x2800, 0x3840, 0x36DB, 0x3C00, 0x3555]


def test_groups_follow_eq1_sets(ref):
    rng = np.random.default_rng(11)
    for _ in range(300):
        thr = _rand_thr(rng)
        x = _vec(rng)
        # plant values exactly on every threshold (Eq. 1 boundary cases)
        for k, t in enumerate(thr):
            x[k] = np.float16(t)
        r = ref.quantize_vector(x, thr)
        want = bf.eq1_membership(x.astype(np.float64), thr)
        assert np.array_equal(r["group"], want)
        # every outlier (inner or outer) has exactly one COO entry; middle values none
        n_out = int((want != 1).sum())
        assert len(r["coo"]) == n_out == int(r["counts"].sum())


def test_codes_are_nearest_levels(ref):
    """Eq. 2-3: per group, the code picks the nearest of 2^b levels spanning [Min, Max]
    of the shifted magnitudes (Eq. 4); b = 3 for middle and 4 for inner/outer."""
    rng = np.random.default_rng(12)
    for _ in range(300):
        thr = _rand_thr(rng)
        x = _vec(rng, scale=float(rng.choice([0.01, 1.0, 30.0])))
        r = ref.quantize_vector(x, thr)
        grp = bf.eq1_membership(x.astype(np.float64), thr)
        a, side = bf.shifted_magnitude(x.astype(np.float64), grp, thr)
        for g, b in ((0, 4), (1, 3), (2, 4)):
            sel = grp == g
            if not sel.any():
                continue
            u = r["code"][sel].astype(int)
            half = 1 << b
            s = side[sel]
            # the side is the code's top bit; the magnitude code runs away from the threshold
            assert np.array_equal((u >= half).astype(int), s)
            c = np.where(s == 1, u - half, half - 1 - u)
            assert c.min() >= 0 and c.max() <= half - 1
            bf.check_nearest_level(a[sel], c, half - 1)


def test_coo_byte_format_and_order(ref):
    """Sec. 4.5: 6 index bits (within a 64-value chunk), 1 group bit, 1 sign bit;
    entries keep ascending position order (the zero-remove shifter keeps order)."""
    rng = np.random.default_rng(13)
    for d in (64, 128, 256):
        for _ in range(50):
            thr = _rand_thr(rng)
            x = _vec(rng, d)
            r = ref.quantize_vector(x, thr)
            grp = bf.eq1_membership(x.astype(np.float64), thr)
            pos = np.nonzero(grp != 1)[0]
            coo = r["coo"].astype(int)
            assert np.array_equal(coo & 63, pos & 63)
            assert np.array_equal((coo >> 6) & 1, (grp[pos] == 2).astype(int))
            assert np.array_equal(coo >> 7, r["code"][pos] >> 4)
            assert np.array_equal(r["counts"], np.bincount(pos // 64, minlength=d // 64))


def test_round_trip_error_bound(ref):
    """|x - dequant(quant(x))| <= Delta_g / 2, plus the fp16 rounding of (Min, Delta)."""
    rng = np.random.default_rng(14)
    P, H = 16, 1
    lay = ref.layout(P, D)
    for trial in range(60):
        thr = _rand_thr(rng)
        xs = np.stack([_vec(rng, scale=float(rng.choice([0.1, 1, 10]))) for _ in range(P)])
        pool = np.zeros(lay["stride"] * 2, np.uint8)
        thr_all = np.stack([thr, thr])[None]
        ref.quantize_kv(pool, 1, P, H, D, thr_all, xs[:, None, :], xs[:, None, :],
                        np.zeros((1, 1), np.int32), [0], [0, P])
        for which in (0, 1):
            for t in range(P):
                xh, grp = ref.dequantize_slot(pool, P, H, D, thr_all, 0, 0, which, t, True)
                x = xs[t].astype(np.float64)
                g_want = bf.eq1_membership(x, thr)
                assert np.array_equal(grp, g_want)
                a, _ = bf.shifted_magnitude(x, g_want, thr)
                for g, lv in ((0, 15), (1, 7), (2, 15)):
                    sel = g_want == g
                    if not sel.any():
                        continue
                    rng_g = a[sel].max() - a[sel].min()
                    # grid step / 2, fp16 rounding of Min and Delta, fp32 rounding of the shift
                    bound = (rng_g / lv / 2 + 2.0 ** -11 * (a[sel].max() + rng_g)
                             + 4 * 2.0 ** -24 * (np.abs(x[sel]).max() + np.abs(thr).max()))
                    err = np.abs(xh[sel] - x[sel]).max()
                    assert err <= bound * (1 + 1e-9), (trial, which, t, g, err, bound)


def test_reduces_to_sign_3bit_minmax(ref):
    """Thresholds (-inf, 0, 0, +inf): no outer values, zeros are the only inner values and
    every nonzero value is middle with no shift -> a textbook sign + 3-bit min-max
    magnitude quantizer over the nonzero values."""
    rng = np.random.default_rng(15)
    thr = np.array([-np.inf, 0, 0, np.inf], np.float32)
    for _ in range(100):
        x = _vec(rng)
        x[rng.integers(0, D, 3)] = 0
        r = ref.quantize_vector(x, thr)
        xf = x.astype(np.float32)
        nz = xf != 0
        assert np.array_equal(r["group"] == 1, nz)
        m = np.abs(xf[nz])
        mn, mx = m.min(), m.max()
        sig = np.float32(7) / np.float32(mx - mn)
        c = np.clip(np.rint((m - mn) * sig), 0, 7).astype(int)
        sign = (xf[nz] > 0).astype(int)
        assert np.array_equal(r["code"][nz], np.where(sign == 1, 8 + c, 7 - c))


def test_reduces_to_sign_4bit_minmax_all_sparse(ref):
    """Thresholds (-inf, -inf, +inf, +inf): every value is inner (unshifted), stored as
    sign + 4-bit min-max magnitude with one COO entry each (worst-case sparse size)."""
    rng = np.random.default_rng(16)
    thr = np.array([-np.inf, -np.inf, np.inf, np.inf], np.float32)
    for _ in range(100):
        x = _vec(rng)
        r = ref.quantize_vector(x, thr)
        assert np.all(r["group"] == 0) and len(r["coo"]) == D
        m = np.abs(x.astype(np.float32))
        mn, mx = m.min(), m.max()
        sig = np.float32(15) / np.float32(mx - mn)
        c = np.clip(np.rint((m - mn) * sig), 0, 15).astype(int)
        sign = (x.astype(np.float32) >= 0).astype(int)
        assert np.array_equal(r["code"], np.where(sign == 1, 16 + c, 15 - c))
        assert r["counts"].tolist() == [64, 64]


def test_constant_vector_is_exact(ref):
    """Max == Min gives a zero range: every code is 0 and the value is reproduced."""
    thr = np.array([-2, -0.5, 0.5, 2], np.float32)
    for v in (3.0, -3.0, 1.0, -1.0, 0.25, -0.25, 0.0):
        x = np.full(D, v, np.float16)
        r = ref.quantize_vector(x, thr)
        c = r["code"].astype(int)
        assert len(set(c.tolist())) == 1
        assert r["meta"][1::2].tolist() == [0, 0, 0]  # every Delta is zero


def test_effective_bits_closed_form(ref):
    """Sec. 4.5: 4 dense bits per value plus one 8-bit COO entry per outlier.  At the
    paper's 4 %/6 % outer/inner ratios this is 4 + 8*0.10 = 4.8 bits, the 70 % reduction
    from 16 bits quoted in Sec. 1 (per-token scales not counted)."""
    rng = np.random.default_rng(17)
    lay = ref.layout(16, D)
    n_val = n_out = 0
    x = rng.standard_normal(200 * D).astype(np.float16)
    lo_o, hi_o = np.quantile(x, [0.02, 0.98])
    t = np.quantile(np.abs(x), 0.06)
    thr = np.array([lo_o, -t, t, hi_o], np.float32)
    for k in range(200):
        r = ref.quantize_vector(x[k * D:(k + 1) * D], thr)
        n_val += D
        n_out += len(r["coo"])
    bits = (4 * n_val + 8 * n_out) / n_val
    assert abs(n_out / n_val - 0.10) < 0.01
    assert abs(bits - 4.8) < 0.1
    assert abs((1 - 4.8 / 16) - 0.70) < 1e-12
    # layout: dense field is exactly 4 bits per value, sparse capacity one byte per value
    assert lay["sparse"] - lay["dense"] == 16 * D // 2
    assert lay["stride"] >= lay["sparse"] + 16 * D


def test_fp16_conversions_match_numpy(ref):
    """The oracle's binary16 conversions against numpy's (IEEE round-to-nearest-even)."""
    for b in range(0, 65536, 7):
        h = np.uint16(b).view(np.float16)
        if np.isnan(h):
            continue
        assert ref.half_to_float(b) == float(h)
    rng = np.random.default_rng(18)
    vals = np.concatenate([rng.standard_normal(2000) * 10.0 ** rng.integers(-9, 5, 2000),
                           [65504, 65519.99, 65520, 2 ** -25, 3 * 2 ** -26, 2 ** -24 * 1.5]])
    for v in vals.astype(np.float32):
        with np.errstate(over="ignore"):
            want = int(np.float16(v).view(np.uint16))
        assert ref.float_to_half(float(v)) == want, v
