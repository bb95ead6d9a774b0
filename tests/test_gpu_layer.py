"""A decoder layer's decode step around the Oaken cache (QKV projection -> quantize ->
attention -> output projection -> MLP).  The Oaken part is checked against the oracle:
the layer's own projected K/V are quantized by the oracle into its copy of the cache and
the oracle's attention over it must match the layer's within the stated tolerance.  The
rest of the layer is checked against an fp32 CPU evaluation of the same weights (bf16
rounding of the GPU GEMMs bounds the difference), and the micro-batched step on two
streams must give the sequential step's result."""
import math

import numpy as np
import pytest
import torch

from paper_2503_18599_amd import synth
from paper_2503_18599_amd.layer import DecoderLayer
from tests.cases import Case, attention_tolerance, np16

pytestmark = pytest.mark.gpu

DEV = "cuda"
P = 16


@pytest.fixture(scope="module")
def B():
    from paper_2503_18599_amd import binding
    binding.lib()
    assert torch.cuda.is_available()
    return binding


@pytest.mark.parametrize("cid,paged", [(2, False), (4, False), (3, True)])
def test_layer_step_matches_oracle(B, ref, cid, paged):
    w = synth.scaled(synth.WORKLOADS[cid], n_seqs=5, ctx=300)
    case = Case(w)
    case.calibrate_oracle(ref)
    H, Hq, d = case.H, case.Hq, case.d
    lens = case.lens
    n = case.n_seqs
    # cache holding every token but each sequence's last, in the oracle and on the GPU
    pre = lens - 1
    rows = torch.cat([torch.arange(int(case.cu[s]), int(case.cu[s]) + int(pre[s])) for s in range(n)])
    cu_pre = torch.zeros(n + 1, dtype=torch.int32)
    cu_pre[1:] = torch.cumsum(pre, 0)
    lay = ref.layout(P, d)
    pool = np.zeros(case.num_blocks * H * 2 * lay["stride"], np.uint8)
    ref.quantize_kv(pool, case.num_blocks, P, H, d, case.thr, np16(case.k[rows]), np16(case.v[rows]),
                    case.bt.numpy(), np.zeros(n, np.int32), cu_pre.numpy())
    thr = torch.from_numpy(case.thr).to(DEV)
    cache = B.Cache(case.num_blocks, H, d, thr, sparse_pages=4 * case.num_blocks * H * 2 if paged else 0)
    bt = case.bt.to(DEV)
    B.quantize_kv(cache, case.k[rows].to(DEV), case.v[rows].to(DEV), bt, torch.zeros(n, dtype=torch.int32, device=DEV),
                  cu_pre.to(DEV), int(pre.max()))
    d_model, d_ff = Hq * d // 2, 2 * Hq * d
    layer = DecoderLayer(d_model, Hq, H, d, d_ff, cache, seed=7)
    layer.keep_attention = True
    g = torch.Generator().manual_seed(11)
    x = torch.randn(n, d_model, generator=g).to(torch.bfloat16).to(DEV)
    lens_d = lens.to(DEV)
    out = layer.step(x, bt, lens_d, int(lens.max()))
    attn = layer.last_attention.cpu().numpy()

    # Oaken part: the oracle quantizes the layer's own K/V and attends with its q
    q, k, v = layer.project(x)
    ref.quantize_kv(pool, case.num_blocks, P, H, d, case.thr, np16(k), np16(v), case.bt.numpy(),
                    pre.numpy().astype(np.int32), np.arange(n + 1, dtype=np.int32))
    want = ref.decode_attention(pool, case.num_blocks, P, H, d, case.thr, np16(q), case.bt.numpy(),
                                lens.numpy(), layer.scale)
    ok, max_abs, _ = attention_tolerance(attn, want)
    assert ok, max_abs

    # the rest of the layer in fp32 on the CPU from the same attention output
    f = lambda t: t.float().cpu()
    xf = f(x)
    h = xf + torch.from_numpy(attn).reshape(n, -1) @ f(layer.w_o)
    y = h * torch.rsqrt(h.pow(2).mean(-1, keepdim=True) + 1e-5)
    ref_out = h + (torch.nn.functional.silu(y @ f(layer.w_gate)) * (y @ f(layer.w_up))) @ f(layer.w_down)
    err = (f(out) - ref_out).abs().max().item()
    assert err <= 0.05 * ref_out.abs().max().item(), (err, ref_out.abs().max().item())

    # two micro-batches on two streams: the same step
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    out2 = layer.step_overlapped(x, bt, lens_d, int(lens.max()), streams)
    torch.cuda.synchronize()
    assert (f(out2) - f(out)).abs().max().item() <= 0.02 * f(out).abs().max().item()
