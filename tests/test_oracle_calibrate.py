"""Pins for the oracle's offline threshold profiling (Sec. 4.3 "offline outlier threshold
profiling", Sec. 6.1 "Thresholds" / "Offline profiling").

Per run, the outer bounds are the k_o-th order statistics from each tail
(k_o = rne(n * r_o / 2)) and the inner bound t the k_i-th smallest magnitude
(k_i = rne(n * r_i)); thresholds are averaged over runs.  Checked by counting and by
numpy's selection routine, never by re-running the oracle's sort.
"""
import numpy as np
import pytest

from tests import bruteforce as bf


def _calib(rng, R, T, H, d, dist="t"):
    if dist == "t":
        x = rng.standard_t(3, (R, T, H, d)) * np.exp(0.5 * rng.standard_normal((1, 1, H, d)))
    elif dist == "pos":
        x = np.abs(rng.standard_normal((R, T, H, d))) + 5.0
    else:
        x = rng.standard_normal((R, T, H, d))
    return np.clip(x, -60000, 60000).astype(np.float16)


@pytest.mark.parametrize("ratios", [(0.04, 0.06), (0.10, 0.20), (0.0, 0.0), (0.02, 0.5)])
def test_single_run_order_statistics(ref, ratios):
    rng = np.random.default_rng(21)
    r_o, r_i = ratios
    R, T, H, d = 1, 64, 3, 64
    k = _calib(rng, R, T, H, d)
    v = _calib(rng, R, T, H, d)
    thr = ref.calibrate(k, v, r_o, r_i)
    n = T * d
    k_o = int(np.rint(n * np.float64(np.float32(r_o)) / 2))
    k_i = int(np.rint(n * np.float64(np.float32(r_i))))
    for h in range(H):
        for which, src in enumerate((k, v)):
            vals = src[0, :, h, :].astype(np.float64).ravel()
            lo_o, lo_i, hi_i, hi_o = thr[h, which].astype(np.float64)
            assert bf.order_stat_ok(vals, lo_o, k_o, "low")
            assert bf.order_stat_ok(vals, hi_o, k_o, "high")
            if k_i == 0:
                assert hi_i == 0 or hi_i == lo_o  # repaired into the outer interval
            else:
                t = hi_i
                mags = np.abs(vals)
                if lo_o <= -t and t <= hi_o:
                    assert bf.order_stat_ok(mags, t, k_i - 1, "low")
                    assert lo_i == -t
            assert lo_o <= lo_i <= hi_i <= hi_o


def test_average_over_runs_matches_selection(ref):
    """R runs: each threshold is the fp64 mean of the per-run order statistics, rounded
    once to fp32 (per-run statistics taken here with numpy's partition)."""
    rng = np.random.default_rng(22)
    R, T, H, d = 5, 40, 2, 128
    k = _calib(rng, R, T, H, d)
    v = _calib(rng, R, T, H, d, "n")
    thr = ref.calibrate(k, v, 0.04, 0.06)
    n = T * d
    k_o = int(np.rint(n * np.float64(np.float32(0.04)) / 2))
    k_i = int(np.rint(n * np.float64(np.float32(0.06))))
    for h in range(H):
        for which, src in enumerate((k, v)):
            lo, hi, tt = [], [], []
            for r in range(R):
                vals = src[r, :, h, :].astype(np.float64).ravel()
                lo.append(np.partition(vals, k_o)[k_o])
                hi.append(np.partition(vals, n - 1 - k_o)[n - 1 - k_o])
                m = np.abs(vals)
                tt.append(np.partition(m, k_i - 1)[k_i - 1])
            want = np.array([np.mean(lo), -np.mean(tt), np.mean(tt), np.mean(hi)], np.float32)
            assert np.allclose(thr[h, which], want, rtol=0, atol=0) or \
                np.all(np.abs(thr[h, which] - want) <= np.spacing(np.abs(want)))


def test_ordering_repair_all_positive(ref):
    """All-positive data: the symmetric inner bound -t falls below lo_o, so the inner
    interval is clamped into the outer one: lo_i = lo_o and hi_i = clamp(t, lo_i, hi_o)
    (Eq. 1's sets must stay disjoint and cover the line)."""
    rng = np.random.default_rng(23)
    k = _calib(rng, 1, 32, 1, 64, "pos")
    thr = ref.calibrate(k, k, 0.04, 0.06)
    lo_o, lo_i, hi_i, hi_o = thr[0, 0]
    vals = k[0, :, 0, :].astype(np.float64).ravel()
    k_i = int(np.rint(vals.size * np.float64(np.float32(0.06))))
    t = np.partition(np.abs(vals), k_i - 1)[k_i - 1]
    assert lo_o > 5.0 and lo_i == lo_o and hi_o > lo_o
    assert hi_i == np.float32(min(max(t, lo_i), hi_o))
    # and with a tiny inner share the interval collapses onto lo_o
    thr2 = ref.calibrate(k, k, 0.5, 0.0001)
    assert thr2[0, 0, 1] == thr2[0, 0, 0] == thr2[0, 0, 2]


def test_invalid_ratios_rejected(ref):
    k = np.zeros((1, 4, 1, 64), np.float16)
    for bad in ((1.0, 0.0), (-0.1, 0.0), (0.5, 0.6), (0.0, 1.5)):
        with pytest.raises(ValueError):
            ref.calibrate(k, k, *bad)


def test_negative_zero_canonical(ref):
    x = np.zeros((1, 8, 1, 64), np.float16)
    x[0, ::2] = np.float16(-0.0)
    thr = ref.calibrate(x, x, 0.04, 0.06)
    assert np.all(np.signbit(thr) == False)  # noqa: E712
