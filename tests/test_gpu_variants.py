"""GPU parity of the group-count variant encodings (Sec. 6.2, number-of-groups study):
nibbles, COO entries, chunk counts, (Min, Delta) and outlier counts bit-exact against the
oracle, and the GPU's fp32 dequantization against the oracle's fp64 one.  Inputs are the
synthetic workloads' K and V with thresholds calibrated by the oracle at each variant's
shares, plus heavy-tailed vectors under random nested boundaries."""
import numpy as np
import pytest
import torch

from paper_2503_18599_amd import synth
from tests.cases import np16

pytestmark = pytest.mark.gpu

DEV = "cuda"
VARIANTS = ["g3", "g2", "g4", "g5", "g4-o4", "g5-o4"]


@pytest.fixture(scope="module")
def B():
    from paper_2503_18599_amd import binding
    binding.lib()
    assert torch.cuda.is_available()
    return binding


def _shares(name):
    """(outer, inner) shares of the full levels and of the outermost/innermost levels."""
    if name == "g2":
        return (0.10, 0.0), None
    two_inner = name.startswith("g5")
    return (0.04, 0.06), (0.02, 0.03 if two_inner else 0.06)


_CALIB = {}


def _calibrated(ref, w, shares):
    key = (w.name, shares)
    if key not in _CALIB:
        kc, vc = np16(synth.calibration_set(w, "k")), np16(synth.calibration_set(w, "v"))
        _CALIB[key] = ref.calibrate(kc, vc, *shares)
    return _CALIB[key]


def _thr8(ref, w, name, which):
    full, lvl = _shares(name)
    a = _calibrated(ref, w, full)[:, which]
    b = _calibrated(ref, w, lvl)[:, which] if lvl else None
    return ref.variant_thresholds(ref.VARIANTS[name], a, b)


def _compare(B, ref, name, x, thr8):
    v = ref.VARIANTS[name]
    want = ref.variant_quantize(v, np16(x), thr8)
    got = B.variant_quantize(v, x.to(DEV), torch.from_numpy(np.ascontiguousarray(thr8)).to(DEV))
    for k in ("nib", "coo", "counts", "n_coo"):
        g = got[k].cpu().numpy()
        assert np.array_equal(g, want[k]), (name, k, int((g != want[k]).sum()))
    assert np.array_equal(got["meta"].cpu().numpy().view(np.uint16), want["meta"])
    # dequantization: GPU fp32 against the oracle's fp64
    xr = ref.variant_dequantize(v, want, thr8)
    xg = B.variant_dequantize(v, got, torch.from_numpy(np.ascontiguousarray(thr8)).to(DEV)).cpu().numpy()
    finite = np.abs(thr8[np.isfinite(thr8)]).max(initial=0.0)
    tol = 2.0 ** -21 * (np.abs(xr) + finite + 1e-30)
    assert np.all(np.abs(xg - xr) <= tol), (name, float(np.abs(xg - xr).max()))
    return want


@pytest.mark.parametrize("name", VARIANTS)
@pytest.mark.parametrize("cid,n_tok", [(1, 300), (2, 257), (4, 129)])
def test_variant_encoding_matches_oracle(B, ref, name, cid, n_tok):
    w = synth.WORKLOADS[cid]
    for which, kv in ((0, "k"), (1, "v")):
        x = synth.kv_values(w, kv, n_tok, w.seed("data"))
        thr8 = _thr8(ref, w, name, which)
        enc = _compare(B, ref, name, x, thr8)
        share = enc["n_coo"].sum() / x.numel()
        assert 0.05 < share < 0.16, (name, kv, share)   # about the calibrated 10 %


@pytest.mark.parametrize("name", VARIANTS)
@pytest.mark.parametrize("d", [64, 128])
def test_variant_random_boundaries(B, ref, name, d):
    rng = np.random.default_rng(7 + d)
    n, H = 50, 3
    x = torch.from_numpy(np.clip(rng.standard_t(3, (n, H, d)) * rng.choice([0.05, 1, 20], (n, H, 1)),
                                 -60000, 60000).astype(np.float16))
    thr8 = np.zeros((H, 8), np.float32)
    for h in range(H):
        o = np.sort(np.abs(rng.normal(0, 2.0, 2))) + 0.5
        i = np.sort(np.abs(rng.normal(0, 0.3, 2)))
        thr8[h] = np.sort(np.concatenate([-np.array([o[1], o[0], i[1], i[0]]), [i[0], i[1], o[0], o[1]]]))
    # values exactly on the boundaries and zeros
    xv = x.numpy()
    xv[0, :, :8] = thr8.astype(np.float16)
    xv[1, :, :5] = 0
    thr8 = thr8.astype(np.float16).astype(np.float32)
    _compare(B, ref, name, torch.from_numpy(xv), thr8)


@pytest.mark.parametrize("name", ["g2", "g5", "g5-o4"])
def test_variant_edge_boundaries(B, ref, name):
    """All-middle (infinite outer boundaries), all-outlier (everything beyond the outer
    boundaries), constant vectors, and an empty batch."""
    rng = np.random.default_rng(99)
    x = torch.from_numpy(np.clip(rng.standard_t(3, (20, 2, 128)), -60000, 60000).astype(np.float16))
    x[3] = 1.5
    x[4] = 0
    inf = np.float32(np.inf)
    all_mid = np.tile(np.array([-inf, -inf, -0.1, -0.05, 0.05, 0.1, inf, inf], np.float32), (2, 1))
    if name == "g2":
        all_mid[:, 2:6] = 0
    _compare(B, ref, name, x, all_mid)
    all_out = np.tile(np.array([0, 0, 0, 0, 0, 0, 0, 0], np.float32), (2, 1))
    _compare(B, ref, name, x, all_out)
    v = ref.VARIANTS[name]
    enc = B.variant_quantize(v, torch.empty(0, 2, 128, dtype=torch.float16, device=DEV),
                             torch.from_numpy(all_mid).to(DEV))
    assert enc["nib"].numel() == 0
