"""Pins for the oracle's group-count variants (Sec. 6.2, number-of-groups study).

The variants generalize the three-group quantizer: two groups (no inner group, COO entry
= sign, pad bit, 6-bit index), four or five groups (two outer levels, one or two inner
levels; 9-bit COO entries padded to 16 bits) and four- or five-group encodings with 4-bit
outliers (sign in the nibble, 8-bit COO entries).  Checked here against the already
pinned three-group quantizer, the nested interval definitions, exhaustive search over
each group's levels, round-trip bounds, a textbook special case and the byte counts.
"""
import numpy as np
import pytest

from tests import bruteforce as bf

D = 128
VARIANTS = ["g3", "g2", "g4", "g5", "g4-o4", "g5-o4"]


def _vec(rng, d=D, scale=1.0):
    x = rng.standard_t(3, d) * scale
    return np.clip(x, -60000, 60000).astype(np.float16)


def _rand_thr8(rng):
    """Nested boundaries lo_ob <= lo_oa <= lo_ia <= lo_ib <= hi_ib <= hi_ia <= hi_oa <= hi_ob."""
    o = np.sort(np.abs(rng.normal(0, 2.0, 2))) + 0.5
    i = np.sort(np.abs(rng.normal(0, 0.3, 2)))
    if rng.random() < 0.2:      # coincident levels
        o[1] = o[0]
    if rng.random() < 0.2:
        i[0] = i[1]
    lo = -np.array([o[1], o[0], i[1], i[0]]) * rng.uniform(0.8, 1.2)
    hi = np.array([i[0], i[1], o[0], o[1]]) * rng.uniform(0.8, 1.2)
    t = np.concatenate([lo, hi]).astype(np.float32)
    return np.sort(t)


def _decode(ref, v, r, d=D):
    """Groups and full codes from an encoding, read by the test from the stated format."""
    info = ref.variant_info(v)
    mid, gb = info["n_in"], info["coo_bits"] - 6 - (1 if info["out_bits"] == 4 else 0)
    u = np.array([(r["nib"][j // 2] >> (4 * (j & 1))) & 15 for j in range(d)])
    grp = np.full(d, mid)
    coo = r["coo"].reshape(-1, info["coo_bytes"]).astype(int)
    e = coo[:, 0] | (coo[:, 1] << 8 if info["coo_bytes"] == 2 else 0)
    pos = []
    k = 0
    for c, n in enumerate(r["counts"]):
        for _ in range(int(n)):
            j = c * 64 + (e[k] & 63)
            rank = (e[k] >> 6) & ((1 << gb) - 1)
            grp[j] = rank if rank < mid else rank + 1
            if info["out_bits"] == 4:
                u[j] |= ((e[k] >> (6 + gb)) & 1) << 4
            pos.append(j)
            k += 1
    return info, grp, u, e, np.array(pos, int)


def test_g3_is_the_three_group_quantizer(ref):
    """Variant g3 with its eight boundaries built from four thresholds reproduces the
    (independently pinned) three-group quantizer byte for byte."""
    rng = np.random.default_rng(31)
    for trial in range(200):
        t = np.sort(rng.normal(0, 1.5, 4).astype(np.float32))
        if trial % 5 == 0:
            t = np.array([-np.inf, -np.inf, np.inf, np.inf], np.float32)
        x = _vec(rng, scale=float(rng.choice([0.1, 1, 10])))
        a = ref.quantize_vector(x, t)
        b = ref.variant_quantize_vector(ref.VARIANTS["g3"], x, ref.variant_thresholds(0, t))
        nib = ((a["code"][0::2] & 15) | ((a["code"][1::2] & 15) << 4)).astype(np.uint8)
        assert np.array_equal(b["nib"], nib)
        assert np.array_equal(b["coo"], a["coo"]) and np.array_equal(b["counts"], a["counts"])
        assert np.array_equal(b["meta"], a["meta"])


@pytest.mark.parametrize("name", VARIANTS)
def test_groups_follow_nested_sets(ref, name):
    v = ref.VARIANTS[name]
    rng = np.random.default_rng(32 + v)
    for _ in range(150):
        thr8 = _rand_thr8(rng)
        x = _vec(rng)
        for k, t in enumerate(thr8):      # values exactly on every boundary
            x[k] = np.float16(t)
        thr8 = thr8.astype(np.float16).astype(np.float32)   # boundaries representable in fp16
        r = ref.variant_quantize_vector(v, x, thr8)
        info, grp, _, _, pos = _decode(ref, v, r)
        want = bf.variant_membership(x.astype(np.float64), thr8, info["n_out"], info["n_in"])
        assert np.array_equal(grp, want)
        assert r["n_coo"] == int((want != info["n_in"]).sum()) == int(r["counts"].sum())


@pytest.mark.parametrize("name", VARIANTS)
def test_codes_are_nearest_levels(ref, name):
    """Eq. 2-3 per group: the code is the nearest of the group's levels over [Min, Max] of
    its shifted magnitudes; 3 magnitude bits for the middle, 4 (or 3) for outliers, the
    side on top."""
    v = ref.VARIANTS[name]
    rng = np.random.default_rng(40 + v)
    for _ in range(150):
        thr8 = _rand_thr8(rng)
        x = _vec(rng, scale=float(rng.choice([0.05, 1.0, 20.0])))
        r = ref.variant_quantize_vector(v, x, thr8)
        info, grp, u, _, _ = _decode(ref, v, r)
        a, side = bf.variant_shift(x.astype(np.float64), grp, thr8, info["n_out"], info["n_in"])
        for g in range(info["groups"]):
            sel = grp == g
            if not sel.any():
                continue
            b = 3 if g == info["n_in"] else info["out_bits"]
            half = 1 << b
            assert np.array_equal((u[sel] >= half).astype(int), side[sel])
            c = np.where(side[sel] == 1, u[sel] - half, half - 1 - u[sel])
            assert c.min() >= 0 and c.max() <= half - 1
            bf.check_nearest_level(a[sel], c, half - 1)


@pytest.mark.parametrize("name", VARIANTS)
def test_round_trip_error_bound(ref, name):
    """|x - dequant(quant(x))| <= Delta_g / 2 plus the fp16 rounding of (Min, Delta)."""
    v = ref.VARIANTS[name]
    rng = np.random.default_rng(50 + v)
    for _ in range(100):
        thr8 = _rand_thr8(rng)
        x = _vec(rng, scale=float(rng.choice([0.1, 1, 10])))
        r = ref.variant_quantize_vector(v, x, thr8)
        xh = ref.variant_dequantize_vector(v, r, thr8)
        info, grp, _, _, _ = _decode(ref, v, r)
        xd = x.astype(np.float64)
        a, _ = bf.variant_shift(xd, grp, thr8, info["n_out"], info["n_in"])
        for g in range(info["groups"]):
            sel = grp == g
            if not sel.any():
                continue
            lv = 7 if g == info["n_in"] else (1 << info["out_bits"]) - 1
            rg = a[sel].max() - a[sel].min()
            bound = (rg / lv / 2 + 2.0 ** -11 * (a[sel].max() + rg)
                     + 4 * 2.0 ** -24 * (np.abs(xd[sel]).max() + np.abs(thr8).max()))
            assert np.abs(xh[sel] - xd[sel]).max() <= bound * (1 + 1e-9)


@pytest.mark.parametrize("name", VARIANTS)
def test_coo_format_and_order(ref, name):
    """Entry = side bit above the group-rank bits above the 6-bit index (no side bit with
    4-bit outliers); two groups keep a zero pad bit; 9-bit entries take two bytes;
    entries in ascending position order with per-chunk counts."""
    v = ref.VARIANTS[name]
    rng = np.random.default_rng(60 + v)
    want_bits = {"g3": 8, "g2": 8, "g4": 9, "g5": 9, "g4-o4": 8, "g5-o4": 8}[name]
    for d in (64, 128, 256):
        for _ in range(30):
            thr8 = _rand_thr8(rng)
            x = _vec(rng, d)
            r = ref.variant_quantize_vector(v, x, thr8)
            info, grp, u, e, pos = _decode(ref, v, r, d)
            assert info["coo_bits"] == want_bits and info["coo_bytes"] == (2 if want_bits > 8 else 1)
            want_pos = np.nonzero(grp != info["n_in"])[0]
            assert np.array_equal(pos, want_pos)
            assert np.all(e < (1 << want_bits))
            if name == "g2":
                assert np.all((e >> 6) & 1 == 0)
            assert np.array_equal(r["counts"], np.bincount(want_pos // 64, minlength=d // 64))


def test_g2_reduces_to_sign_3bit_minmax(ref):
    """Two groups with infinite outer boundaries: every value is middle and unshifted,
    i.e. a textbook sign + 3-bit min-max quantizer over |x| (zeros on the upper side)."""
    rng = np.random.default_rng(70)
    thr8 = np.array([-np.inf, -np.inf, 0, 0, 0, 0, np.inf, np.inf], np.float32)
    for _ in range(100):
        x = _vec(rng)
        x[rng.integers(0, D, 2)] = 0
        r = ref.variant_quantize_vector(ref.VARIANTS["g2"], x, thr8)
        assert r["n_coo"] == 0
        xf = x.astype(np.float32)
        m = np.abs(xf)
        mn, mx = m.min(), m.max()
        c = np.clip(np.rint((m - mn) * (np.float32(7) / np.float32(mx - mn))), 0, 7).astype(int)
        u = np.where(xf >= 0, 8 + c, 7 - c)
        nib = (u[0::2] | (u[1::2] << 4)).astype(np.uint8)
        assert np.array_equal(r["nib"], nib)


@pytest.mark.parametrize("name", ["g4", "g5"])
def test_merged_levels_dequantize_as_g3(ref, name):
    """With each b level equal to its a level the extra groups are empty and the four- and
    five-group variants store the same codes and scales as three groups."""
    rng = np.random.default_rng(80)
    for _ in range(100):
        t = np.sort(rng.normal(0, 1.5, 4).astype(np.float32))
        x = _vec(rng)
        thr8 = np.array([t[0], t[0], t[1], t[1], t[2], t[2], t[3], t[3]], np.float32)
        a = ref.variant_dequantize_vector(0, ref.variant_quantize_vector(0, x, thr8), thr8)
        v = ref.VARIANTS[name]
        b = ref.variant_dequantize_vector(v, ref.variant_quantize_vector(v, x, thr8), thr8)
        assert np.array_equal(a, b)


@pytest.mark.parametrize("name", VARIANTS)
def test_bytes_per_vector_closed_form(ref, name):
    """Stored bytes = d/2 nibbles + one (or two) bytes per outlier + 4 bytes of (Min, Delta)
    per group + d/64 counts; with the total outlier share at 10 % the effective bits are
    4 + 0.1 * 8 (or 16) + the scale and count bytes."""
    v = ref.VARIANTS[name]
    info = ref.variant_info(v)
    rng = np.random.default_rng(90)
    x = rng.standard_normal((200, D)).astype(np.float16)
    xf = x.astype(np.float32).ravel()
    q = lambda p: np.float32(np.quantile(xf, p))
    t = lambda p: np.float32(np.quantile(np.abs(xf), p))
    if name == "g2":
        thr8 = np.array([q(.05), q(.05), 0, 0, 0, 0, q(.95), q(.95)], np.float32)
    else:
        ob = (q(.01), q(.99)) if info["n_out"] == 2 else (q(.02), q(.98))
        ib = t(.03) if info["n_in"] == 2 else t(.06)
        thr8 = np.array([ob[0], q(.02), -t(.06), -ib, ib, t(.06), q(.98), ob[1]], np.float32)
    n_coo = sum(ref.variant_quantize_vector(v, x[k], thr8)["n_coo"] for k in range(200))
    assert abs(n_coo / x.size - 0.10) < 0.01
    nbytes = 200 * (D // 2 + 4 * info["groups"] + D // 64) + n_coo * info["coo_bytes"]
    bits = 8 * nbytes / x.size
    want = 4 + 0.10 * 8 * info["coo_bytes"] + 8 * (4 * info["groups"] + D // 64) / D
    assert abs(bits - want) < 0.1
