"""Decode-step benchmark of the Oaken hot path on one MI355X.

One step = quantize one new K/V token per sequence into the paged cache, then batched
decode attention over every sequence's full cache.  Default workload: a
Llama-2-13B-shaped layer (batch 256, 40 heads MHA, head_dim 128, context 2048 with the
new token, 16-token pages on a shuffled block table), synthetic seeded data.

Prints one JSON line with tokens/s, the attention kernel's achieved HBM bandwidth against
the 8 TB/s peak (algorithmic bytes / its average duration, timed with HIP events on the
launch stream), the CPU oracle timed on a bounded sample, and the sampled parity error.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_F32_PEAK_TFS = 157.3   # dense fp32 matrix-core peak of the MI355X
MFMA_F16_PEAK_TFS = 2500.0  # dense fp16 matrix-core peak of the MI355X


def log(msg: str):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed decode steps (default 20; 64 for the 32K-context workload)")
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=3, help="1..5 (3 = batch-256 Llama-2-13B layer)")
    ap.add_argument("--window", type=int, default=0,
                    help="sliding window in tokens (0: attend over the whole sequence)")
    ap.add_argument("--paged", action="store_true",
                    help="on-demand sparse pages: COO bytes in a separate pool of 256-byte pages")
    ap.add_argument("--layer", action="store_true",
                    help="time a full decoder layer's decode step (random bf16 weights) around the cache")
    ap.add_argument("--layer-batch", type=int, default=0,
                    help="sequences in the layer step (0: the whole workload batch)")
    ap.add_argument("--ratio-sweep", action="store_true",
                    help="group-ratio trade-off: effective bits vs attention error for several (outer, inner) ratios")
    ap.add_argument("--variants", action="store_true",
                    help="number-of-groups study: effective bits and error of each encoding variant")
    ap.add_argument("--prefill-chunk", type=int, default=0,
                    help="time chunked-prefill attention for the last N cached tokens of every sequence")
    ap.add_argument("--cold", type=int, default=-1,
                    help="1: write a 1 GiB scratch buffer between steps (outside the timed events) so that "
                         "no step finds the cache in the 256 MB Infinity Cache; 0: back to back; "
                         "default: cold for the workloads whose cache is under 1 GB (2 and 5)")
    ap.add_argument("--no-stream-probe", action="store_true")
    ap.add_argument("--cpu-sample-seqs", type=int, default=0,
                    help="sequences in the oracle's timed sample (default: 128, 4 for the 32K context)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="after timing, run one plain copy of this size (counter calibration)")
    return ap.parse_args()


def source_hash() -> str:
    h = hashlib.sha256()
    for f in ("attention.hip", "attention_mfma.hip", "oaken_internal.h"):
        with open(os.path.join(ROOT, "paper_2503_18599_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def stored_traffic(workload_name: str):
    """HBM bytes per attention launch from committed counter runs, if they were taken on
    the current kernel source (else None)."""
    p = os.path.join(ROOT, "profiles", "attention_traffic.json")
    if not os.path.exists(p):
        return None
    try:
        d = json.load(open(p))
    except (OSError, ValueError):
        return None
    if d.get("source_hash") != source_hash() or d.get("workload") != workload_name:
        return None
    return d.get("bytes_per_launch")


def layer_bench(args, w, cache, bt, lens, dev):
    """Decode step of a full decoder layer of the workload's shape: per-phase times of the
    sequential step (HIP events), and the step with the batch in two micro-batches on two
    streams."""
    import torch

    from paper_2503_18599_amd import binding as B
    from paper_2503_18599_amd.layer import PHASES, DecoderLayer

    n = args.layer_batch or w.n_seqs
    steps = args.steps or 20
    H, Hq, d = w.n_kv_heads, w.n_q_heads, w.head_dim
    d_model = Hq * d
    d_ff = {5120: 13824, 4096: 14336}.get(d_model, 4 * d_model)   # Llama-2-13B / Mistral-7B MLP widths
    layer = DecoderLayer(d_model, Hq, H, d, d_ff, cache, seed=1)
    x = (torch.randn(n, d_model, generator=torch.Generator().manual_seed(2)) * 0.5).to(torch.bfloat16).to(dev)
    bt_n, lens_n = bt[:n].contiguous(), lens[:n].to(dev)
    max_len = int(lens[:n].max())
    ws = torch.empty(max(1, B.attention_workspace_bytes(n, Hq, H, d, max_len)), dtype=torch.uint8, device=dev)
    for _ in range(args.warmup):
        layer.step(x, bt_n, lens_n, max_len, workspace=ws)
    torch.cuda.synchronize()
    ev = [{p: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for p in PHASES}
          for _ in range(steps)]
    t0 = time.perf_counter()
    for i in range(steps):
        layer.step(x, bt_n, lens_n, max_len, events=ev[i], workspace=ws)
    torch.cuda.synchronize()
    seq_s = (time.perf_counter() - t0) / steps
    phase_ms = {p: sum(e[p][0].elapsed_time(e[p][1]) for e in ev) / steps for p in PHASES}
    gpu_ms = sum(phase_ms.values())
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    halves = [n // 2, n - n // 2]
    wss = [torch.empty(max(1, B.attention_workspace_bytes(m, Hq, H, d, max_len)), dtype=torch.uint8, device=dev)
           for m in halves]
    for _ in range(args.warmup):
        layer.step_overlapped(x, bt_n, lens_n, max_len, streams, wss)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        layer.step_overlapped(x, bt_n, lens_n, max_len, streams, wss)
    torch.cuda.synchronize()
    ovl_s = (time.perf_counter() - t0) / steps
    log(f"layer step: sequential {seq_s * 1e3:.3f} ms (phases {phase_ms}), two streams {ovl_s * 1e3:.3f} ms")
    res = {
        "metric": "decoder-layer decode step tokens/sec (quantize + attention inside a full layer)",
        "value": round(n / min(seq_s, ovl_s), 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": steps, "warmup": args.warmup, "ms_per_step": round(min(seq_s, ovl_s) * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16+f32", "data": "synthetic",
        "config": {"workload": f"one {w.name} decoder layer (d_model {d_model}, {Hq}/{H} heads, MLP {d_ff}, "
                               f"random bf16 weights), batch {n}, context {w.ctx_min}..{w.ctx}"
                               + (", on-demand sparse pages" if args.paged else ""),
                   "global_batch": n, "seq_len": max_len, "parallelism": "single GPU"},
        "layer": {"sequential_ms": round(seq_s * 1e3, 4), "two_streams_ms": round(ovl_s * 1e3, 4),
                  "phase_ms": {p: round(v, 4) for p, v in phase_ms.items()},
                  "share": {p: round(v / gpu_ms, 4) for p, v in phase_ms.items()}},
    }
    print(json.dumps(res), flush=True)


def ratio_sweep(args):
    """Group-ratio trade-off (Sec. 6.2, accuracy vs compression ratio) on synthetic data:
    for each (outer, inner) share, calibrate thresholds, quantize a cache, and report the
    effective bits per element (from the stored bytes) and the decode-attention error
    against fp32 attention over the unquantized fp16 keys and values."""
    import numpy as np
    import torch

    from paper_2503_18599_amd import binding as B
    from paper_2503_18599_amd import synth

    dev = "cuda"
    w = synth.scaled(synth.WORKLOADS[args.workload], n_seqs=32, ctx=1024)
    H, Hq, d, n = w.n_kv_heads, w.n_q_heads, w.head_dim, w.n_seqs
    G = Hq // H
    lens = synth.seq_lengths(w)
    bt_cpu, nblk = synth.block_table(w, lens)
    bt = bt_cpu.to(dev)
    k = [synth.kv_values_seq(w, "k", s, int(lens[s]), dev) for s in range(n)]
    v = [synth.kv_values_seq(w, "v", s, int(lens[s]), dev) for s in range(n)]
    kk, vv = torch.cat(k), torch.cat(v)
    cu = torch.zeros(n + 1, dtype=torch.int32)
    cu[1:] = torch.cumsum(lens, 0)
    q = synth.queries(w, 0, dev)
    scale = float(np.float32(1.0 / math.sqrt(d)))
    # fp32 reference attention over the raw values
    ref = []
    for s in range(n):
        kt = k[s].float().repeat_interleave(G, 1).permute(1, 2, 0).contiguous()   # [Hq][d][L]
        vt = v[s].float().repeat_interleave(G, 1).permute(1, 0, 2).contiguous()   # [Hq][L][d]
        sc = torch.bmm(q[s].float()[:, None, :], kt)[:, 0, :] * scale
        ref.append(torch.bmm(torch.softmax(sc, -1)[:, None, :], vt)[:, 0, :])
    ref = torch.stack(ref)
    kc = synth.calibration_set(w, "k", dev)
    vc = synth.calibration_set(w, "v", dev)
    rows = []
    grid = [(0.0, 0.0), (0.02, 0.03), (0.04, 0.06), (0.0, 0.10), (0.10, 0.0), (0.06, 0.04), (0.06, 0.09), (0.08, 0.12)]
    for ro, ri in grid:
        thr = B.calibrate_thresholds(kc, vc, ro, ri)
        cache = B.Cache(nblk, H, d, thr)
        B.quantize_kv(cache, kk, vv, bt, torch.zeros(n, dtype=torch.int32, device=dev), cu.to(dev), int(lens.max()))
        out = B.decode_attention(cache, q, bt, lens.to(dev), int(lens.max()), scale)
        err = float(((out - ref).norm() / ref.norm()).item())
        rec = cache.pool.view(nblk, H, 2, cache.stride)
        n_out = int(rec[:, :, :, :16 * (d // 64)].to(torch.int64).sum())   # the records' COO counts
        n_el = int(lens.sum()) * H * 2 * d
        # bits per element: 4-bit code + one COO byte per outlier + 12 B meta and d/64 count bytes per vector
        bits = 4.0 + 8.0 * n_out / n_el + 8.0 * (12 + d // 64) / d
        rows.append({"outer": ro, "inner": ri, "outlier_fraction": round(n_out / n_el, 4),
                     "effective_bits": round(bits, 3), "attention_rel_err": round(err, 5)})
        log(f"outer {ro:.2f} inner {ri:.2f}: outliers {n_out / n_el:.4f}, {bits:.3f} bits, attention err {err:.5f}")
    print(json.dumps({"metric": "group-ratio trade-off (effective bits vs decode-attention relative L2 error)",
                      "config": {"workload": f"{w.name}: {n} sequences x {w.ctx} tokens, {Hq}/{H} heads, d {d}"},
                      "data": "synthetic", "reference": "fp32 attention over the unquantized fp16 K/V",
                      "sweep": rows}), flush=True)


def variant_sweep(args):
    """Number-of-groups study (Sec. 6.2) on synthetic data: for each encoding variant,
    calibrate its boundaries, encode and decode the keys and values, and report the
    effective bits per element (from the stored bytes), the relative error of K and V,
    the relative L2 error of fp32 attention over the decoded K/V against attention over
    the unquantized values, and the encoder's throughput."""
    import numpy as np
    import torch

    from paper_2503_18599_amd import binding as B
    from paper_2503_18599_amd import synth

    dev = "cuda"
    w = synth.scaled(synth.WORKLOADS[args.workload], n_seqs=32, ctx=1024)
    H, Hq, d, n = w.n_kv_heads, w.n_q_heads, w.head_dim, w.n_seqs
    G = Hq // H
    lens = synth.seq_lengths(w)
    k = [synth.kv_values_seq(w, "k", s, int(lens[s]), dev) for s in range(n)]
    v = [synth.kv_values_seq(w, "v", s, int(lens[s]), dev) for s in range(n)]
    kk, vv = torch.cat(k).contiguous(), torch.cat(v).contiguous()
    q = synth.queries(w, 0, dev)
    scale = float(np.float32(1.0 / math.sqrt(d)))
    cu = [0] + np.cumsum(lens.numpy()).tolist()

    def attention(kx, vx):
        out = []
        for s in range(n):
            ks, vs = kx[cu[s]:cu[s + 1]], vx[cu[s]:cu[s + 1]]
            kt = ks.float().repeat_interleave(G, 1).permute(1, 2, 0).contiguous()   # [Hq][d][L]
            vt = vs.float().repeat_interleave(G, 1).permute(1, 0, 2).contiguous()   # [Hq][L][d]
            sc = torch.bmm(q[s].float()[:, None, :], kt)[:, 0, :] * scale
            out.append(torch.bmm(torch.softmax(sc, -1)[:, None, :], vt)[:, 0, :])
        return torch.stack(out)

    ref = attention(kk, vv)
    kc = synth.calibration_set(w, "k", dev)
    vc = synth.calibration_set(w, "v", dev)
    shares = {"g3": ((0.04, 0.06), None), "g2": ((0.10, 0.0), None), "g4": ((0.04, 0.06), (0.02, 0.06)),
              "g5": ((0.04, 0.06), (0.02, 0.03)), "g4-o4": ((0.04, 0.06), (0.02, 0.06)),
              "g5-o4": ((0.04, 0.06), (0.02, 0.03))}
    rows = []
    for name, vid in B.VARIANTS.items():
        info = B.variant_info(vid)
        full, lvl = shares[name]
        ta = B.calibrate_thresholds(kc, vc, *full)
        tb = B.calibrate_thresholds(kc, vc, *lvl) if lvl else None
        dec, n_coo = [], 0
        for which, x in ((0, kk), (1, vv)):
            thr8 = B.variant_boundaries(vid, ta[:, which], None if tb is None else tb[:, which])
            enc = B.variant_quantize(vid, x, thr8)
            n_coo += int(enc["n_coo"].sum())
            dec.append(B.variant_dequantize(vid, enc, thr8))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        thr8 = B.variant_boundaries(vid, ta[:, 0], None if tb is None else tb[:, 0])
        for _ in range(3):
            B.variant_quantize(vid, kk, thr8)
        e0.record()
        for _ in range(10):
            B.variant_quantize(vid, kk, thr8)
        e1.record()
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) / 10 / 1e3
        n_vec = kk.shape[0] * H * 2
        n_el = n_vec * d
        nbytes = n_vec * (d // 2 + 4 * info["groups"] + d // 64) + n_coo * info["coo_bytes"]
        out = attention(dec[0], dec[1])
        err = float(((out - ref).norm() / ref.norm()).item())
        kerr = float(((dec[0] - kk.float()).norm() / kk.float().norm()).item())
        verr = float(((dec[1] - vv.float()).norm() / vv.float().norm()).item())
        rows.append({"variant": name, "groups": info["groups"], "coo_bits": info["coo_bits"],
                     "outlier_bits": info["out_bits"] + 1, "outlier_fraction": round(n_coo / n_el, 4),
                     "effective_bits": round(8.0 * nbytes / n_el, 3), "k_rel_err": round(kerr, 5),
                     "v_rel_err": round(verr, 5), "attention_rel_err": round(err, 5),
                     "encode_gbs": round(kk.numel() * 2 / t / 1e9, 1)})
        log(f"{name}: {rows[-1]}")
    print(json.dumps({"metric": "group-count variants (effective bits vs K/V and attention relative L2 error)",
                      "config": {"workload": f"{w.name}: {n} sequences x {w.ctx} tokens, {Hq}/{H} heads, d {d}"},
                      "data": "synthetic", "reference": "fp32 attention over the unquantized fp16 K/V",
                      "variants": rows}), flush=True)


def prefill_bench(args, w, cache, bt, lens, dev, bt_cpu):
    """Chunked-prefill attention: the last C cached tokens of every sequence attend causally
    over their prefixes.  A row block (up to 64 rows of query token x query head of one KV
    head) reads each page of its keys once, so the bytes of one pass over every chunk's
    visible prefix are the algorithmic bytes when a chunk fits one row block."""
    import numpy as np
    import torch

    from paper_2503_18599_amd import binding as B

    n, H, Hq, d = w.n_seqs, w.n_kv_heads, w.n_q_heads, w.head_dim
    cached = lens - 1                                    # tokens in the cache
    clen = torch.clamp(cached, max=args.prefill_chunk).to(torch.int32)
    start = (cached - clen).to(torch.int32)
    cu = torch.zeros(n + 1, dtype=torch.int32)
    cu[1:] = torch.cumsum(clen, 0)
    n_tok = int(cu[-1])
    q = (torch.randn(n_tok, Hq, d, generator=torch.Generator().manual_seed(3))).to(torch.float16).to(dev)
    max_len = int(lens.max())
    scale = float(np.float32(1.0 / math.sqrt(d)))
    out = torch.empty(n_tok, Hq, d, dtype=torch.float32, device=dev)
    win = max(0, args.window)
    ws = torch.empty(max(1, int(B.lib().oaken_prefill_attention_workspace_bytes(n_tok, Hq, H, d, max_len, win))),
                     dtype=torch.uint8, device=dev)
    args_d = (bt, start.to(dev), cu.to(dev), max_len, scale)
    for _ in range(args.warmup):
        B.prefill_attention(cache, q, *args_d, window=win, out=out, workspace=ws)
    torch.cuda.synchronize()
    steps = args.steps or 20
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        B.prefill_attention(cache, q, *args_d, window=win, out=out, workspace=ws)
    e1.record()
    torch.cuda.synchronize()
    t = e0.elapsed_time(e1) / steps / 1e3
    # one pass over each chunk's visible keys: positions [lo, last] of every KV head
    prefix = outlier_prefix(cache, bt_cpu, n, max_len)
    # query tokens per row block: blocks of 64 rows, or of 128 on the fp16 matrix cores when
    # the chunks hold more rows per KV head than 64 (head_dim 128; the library's rule)
    G = Hq // H
    # (the library's block rule: 128-row blocks past 64 rows per KV head at head_dim 128, else
    # blocks of 16, 32 or 64 rows sized to the mean chunk)
    rows = G * -(-n_tok // n)
    wide = d == 128 and rows > 64
    block_rows = 128 if wide else (16 if rows <= 16 else (32 if rows <= 32 else 64))
    tpb = max(1, block_rows // G)
    one_pass, passes = 0, 0
    for s in range(n):
        last = int(cached[s]) - 1
        lo = max(0, int(start[s]) + 1 - win) if win else 0
        if int(clen[s]) == 0:
            continue
        vec = (last + 1 - lo) * H * 2
        one_pass += vec * alg_bytes_per_vector(d) + int((prefix[s, :, :, last + 1] - prefix[s, :, :, lo]).sum())
        passes += (int(clen[s]) + tpb - 1) // tpb
    one_pass += n_tok * Hq * d * (2 + 4)
    gbs = one_pass / t / 1e9
    # matrix-core work: each (query token, query head) row takes 2d flops per visible key for
    # its scores and 2d for its output
    flops = 0
    for s in range(n):
        for i in range(int(clen[s])):
            p = int(start[s]) + i
            flops += 4 * d * Hq * (min(p + 1, win) if win else p + 1)
    tfs = flops / t / 1e12
    # the 64-row blocks contract on fp32 matrix cores; the 128-row blocks on fp16 ones, each
    # real operand as a high and a low fp16 part (2 products per score term, 3 per output
    # term: executed flops are 2.5x the algorithmic ones)
    peak = MFMA_F16_PEAK_TFS if wide else MFMA_F32_PEAK_TFS
    log(f"prefill attention: {n_tok} query tokens in {t * 1e6:.1f} us; one pass over the chunks' prefixes "
        f"{one_pass / 1e9:.3f} GB = {gbs:.0f} GB/s ({passes} row blocks for {n} chunks); "
        f"{flops / 1e9:.1f} GFLOP = {tfs:.1f} TFLOP/s on {'fp16' if wide else 'fp32'} matrix cores")
    hbm = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
           "frac": round(gbs / HBM_PEAK_GBS, 4), "bytes_one_pass": one_pass}
    mfma = {"bound": "mfma", "achieved": round(tfs, 2), "peak": peak, "unit": "TFLOP/s",
            "frac": round(tfs / peak, 4), "flops": flops}
    # the resource nearer to saturation is the roofline; the other is reported beside it
    roof, other = (mfma, hbm) if mfma["frac"] > hbm["frac"] else (hbm, mfma)
    res = {"metric": "chunked-prefill attention query tokens/sec", "value": round(n_tok / t, 1), "unit": "tokens/s",
           "n_gpus": 1, "steps": steps, "warmup": args.warmup, "ms_per_step": round(t * 1e3, 4),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": "f16x2-mfma+f32" if wide else "f32-mfma", "data": "synthetic",
           "config": {"workload": f"{w.name}: {n} sequences, chunks of the last {args.prefill_chunk} cached tokens "
                                  f"({n_tok} query tokens), {Hq}/{H} heads, d {d}, context {w.ctx_min}..{w.ctx}"
                                  + (f", sliding window {win}" if win else ""),
                      "global_batch": n, "seq_len": max_len, "parallelism": "single GPU"},
           "row_block_rows": block_rows,
           "roofline": dict(roof, traffic=None,
                            row_blocks_per_chunk=round(passes / max(1, sum(1 for s in range(n) if int(clen[s]) > 0)), 3)),
           "roofline_other": other}
    print(json.dumps(res), flush=True)


def alg_bytes_per_vector(d: int) -> int:
    """Bytes of one (token, KV head, K|V) vector without its COO entries: d/2 dense nibbles,
    d/64 count bytes, 12 bytes of fp16 metadata."""
    return d // 2 + d // 64 + 12


def outlier_prefix(cache, bt_cpu, n_seqs, max_pos):
    """int64 [n_seqs][H][2][max_pos + 1]: COO entries of positions < p, per sequence, KV head
    and K|V, from the records' counts."""
    import torch
    P, d, H = 16, cache.head_dim, cache.n_kv_heads
    nc = d // 64
    nblk = cache.num_blocks
    rec = cache.pool.view(nblk, H, 2, cache.stride)
    counts = rec[:, :, :, : P * nc].reshape(nblk, H, 2, P, nc).to(torch.int64).sum(-1).cpu()   # [blk,H,2,P]
    n_pages = (max_pos + P - 1) // P
    blocks = bt_cpu[:, :n_pages].to(torch.int64)                                               # [S, pages]
    per_pos = counts[blocks].permute(0, 2, 3, 1, 4).reshape(n_seqs, H, 2, n_pages * P)[..., :max_pos]
    out = torch.zeros(n_seqs, H, 2, max_pos + 1, dtype=torch.int64)
    out[..., 1:] = torch.cumsum(per_pos, -1)
    return out


def attention_bytes(cache, prefix, lens, window, Hq, n_seqs):
    """Algorithmic bytes of one attention launch over sequences of lengths `lens`: every key
    and value vector a query sees (dense, counts, metadata, its COO bytes), the queries,
    the outputs, the block-table entries and the lengths.  Split partials are overhead.
    Returns (KV-stream bytes, all algorithmic bytes, COO entries, vectors, pages)."""
    d, H = cache.head_dim, cache.n_kv_heads
    n_vec, n_out, pages = 0, 0, 0
    for s in range(n_seqs):
        L = int(lens[s])
        lo = max(0, L - window) if window else 0
        n_vec += (L - lo) * H * 2
        n_out += int((prefix[s, :, :, L] - prefix[s, :, :, lo]).sum())
        pages += (L + 15) // 16 - lo // 16
    kv = n_vec * alg_bytes_per_vector(d) + n_out
    return kv, kv + n_seqs * Hq * d * (2 + 4) + pages * 4 + n_seqs * 4, n_out, n_vec, pages


def stream_probe(cache, dev):
    """Measured streaming-read bandwidth on this device: a 4 GiB contiguous read, and the
    first 1456 bytes of every page record of the pool (counts, metadata, dense nibbles and
    about the mean COO stream at a 10 % outlier share: what decode attention reads per
    record)."""
    import torch

    from paper_2503_18599_amd import binding as B
    res = {}
    buf = torch.empty(4 << 30, dtype=torch.uint8, device=dev)
    buf.fill_(1)
    nrec_pool = cache.pool.numel() // cache.stride
    per_rec = min(1456, cache.stride // 16 * 16)
    for name, base, per, stride, n in (("plain_4gib", buf, 4096, 4096, (4 << 30) // 4096),
                                       ("record_prefix", cache.pool, per_rec, cache.stride, nrec_pool)):
        ck = torch.zeros(1, dtype=torch.int32, device=dev)
        for _ in range(3):
            B.probe_read(base, per, stride, n, ck)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        reps = 10
        e0.record()
        for _ in range(reps):
            B.probe_read(base, per, stride, n, ck)
        e1.record()
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) / reps / 1e3
        res[name] = {"gbs": round(per * n / t / 1e9, 1), "bytes": per * n, "us": round(t * 1e6, 2)}
        log(f"stream probe {name}: {per * n / 2**30:.2f} GiB in {t * 1e6:.1f} us = {per * n / t / 1e9:.0f} GB/s")
    del buf
    torch.cuda.empty_cache()
    return res


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.variants:
        return variant_sweep(args)
    if args.ratio_sweep:
        return ratio_sweep(args)
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU: the library has no "
                                   "multi-GPU path (sharding by sequence or KV head needs no "
                                   "exchange and is left to the caller)", "n_gpus": args.gpus}))
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2503_18599_amd import binding as B
    from paper_2503_18599_amd import synth

    dev = "cuda"
    torch.cuda.set_device(0)
    B.lib()
    w = synth.WORKLOADS[args.workload]
    H, Hq, d = w.n_kv_heads, w.n_q_heads, w.head_dim
    n = w.n_seqs
    K = args.steps if args.steps is not None else (w.decode_steps if w.prefill else 20)
    W = args.warmup
    cold = bool(args.cold) if args.cold >= 0 else args.workload in (2, 5)
    log(f"workload {w.name}: B={n} Hq={Hq} Hkv={H} d={d} ctx={w.ctx_min}..{w.ctx}; {K} steps, cold={cold}")

    # ---- setup: thresholds, cache prefill ----------------------------------------
    kc = synth.calibration_set(w, "k", dev)
    vc = synth.calibration_set(w, "v", dev)
    thr = B.calibrate_thresholds(kc, vc, 0.04, 0.06)
    del kc, vc
    if w.prefill:
        # the whole context is quantized by one prefill-time call (timed); the decode steps
        # then append at positions ctx, ctx + 1, ...
        L0 = torch.full((n,), w.ctx, dtype=torch.int32)
        bt_cpu, nblk = synth.block_table(w, L0, extra_tokens=max(K, W) + 1)
        pre = [w.ctx] * n
        lens = L0 + 1                        # (the layer and chunked-prefill modes append one token)
    else:
        lens = synth.seq_lengths(w)          # incl. the token each decode step appends
        bt_cpu, nblk = synth.block_table(w, lens)
        pre = [int(L) - 1 for L in lens]
    bt = bt_cpu.to(dev)
    cache = B.Cache(nblk, H, d, thr, sparse_pages=2 * nblk * H * 2 if args.paged else 0)
    log(f"pool {cache.pool.numel() / 2**30:.2f} GiB, {nblk} pages")
    prefill_res = None
    if w.prefill:
        k_all = torch.cat([synth.kv_values_seq(w, "k", s, pre[s], dev) for s in range(n)])
        v_all = torch.cat([synth.kv_values_seq(w, "v", s, pre[s], dev) for s in range(n)])
        cu = torch.zeros(n + 1, dtype=torch.int32)
        cu[1:] = torch.cumsum(torch.tensor(pre, dtype=torch.int32), 0)
        cu_d, z = cu.to(dev), torch.zeros(n, dtype=torch.int32, device=dev)
        B.quantize_kv(cache, k_all, v_all, bt, z, cu_d, max(pre))     # warm-up (same bytes again below)
        torch.cuda.synchronize()
        reps = 3
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for e0, e1 in ev:
            e0.record()
            B.quantize_kv(cache, k_all, v_all, bt, z, cu_d, max(pre))
            e1.record()
        torch.cuda.synchronize()
        t_pf = sum(a.elapsed_time(b) for a, b in ev) / reps / 1e3
        n_vec = sum(pre) * H * 2
        pfx = outlier_prefix(cache, bt_cpu, n, w.ctx)
        n_out = int(pfx[:, :, :, w.ctx].sum())
        in_b = n_vec * d * 2
        out_b = n_vec * alg_bytes_per_vector(d) + n_out
        gbs = (in_b + out_b) / t_pf / 1e9
        prefill_res = {"tokens": sum(pre), "us": round(t_pf * 1e6, 1), "tokens_per_s": round(sum(pre) / t_pf, 1),
                       "bytes_in": in_b, "bytes_out": out_b,
                       "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                    "frac": round(gbs / HBM_PEAK_GBS, 4)}}
        log(f"prefill quantization: {sum(pre)} tokens x {H} heads in {t_pf * 1e6:.1f} us ({gbs:.0f} GB/s)")
        del k_all, v_all
        torch.cuda.empty_cache()
    else:
        t0 = time.time()
        chunk = 16
        for s0 in range(0, n, chunk):
            ss = list(range(s0, min(n, s0 + chunk)))
            k = torch.cat([synth.kv_values_seq(w, "k", s, pre[s], dev) for s in ss])
            v = torch.cat([synth.kv_values_seq(w, "v", s, pre[s], dev) for s in ss])
            cu = torch.zeros(len(ss) + 1, dtype=torch.int32)
            cu[1:] = torch.cumsum(torch.tensor([pre[s] for s in ss], dtype=torch.int32), 0)
            B.quantize_kv(cache, k, v, bt[s0:s0 + len(ss)].contiguous(),
                          torch.zeros(len(ss), dtype=torch.int32, device=dev), cu.to(dev), max(pre[s] for s in ss))
            del k, v
        torch.cuda.synchronize()
        log(f"cache built: {sum(pre)} tokens (inputs drawn on the GPU) in {time.time() - t0:.1f}s")
    capacity = None
    if args.paged:
        free, overflow = cache.sparse_status()
        if overflow:
            raise SystemExit("sparse page pool overflowed")
        used_pages = cache.sparse_pages - free
        capacity = {"dense_pool_bytes": cache.pool.numel(), "sparse_pages_used": used_pages,
                    "pool_bytes": cache.pool.numel() + used_pages * B.SPARSE_PAGE_BYTES,
                    "fixed_record_pool_bytes": nblk * H * 2 * B.record_bytes(d)}
        log(f"sparse pages used: {used_pages}; pool {capacity['pool_bytes'] / 2**30:.2f} GiB "
            f"vs {capacity['fixed_record_pool_bytes'] / 2**30:.2f} GiB with fixed records")

    if args.layer:
        return layer_bench(args, w, cache, bt, lens, dev)
    if args.prefill_chunk:
        return prefill_bench(args, w, cache, bt, lens, dev, bt_cpu)

    # ---- decode steps ----------------------------------------------------------------
    # step i appends one token per sequence at start_i and attends over lens_i tokens: a
    # growing context for the prefill workload, the same last position otherwise
    n_new = max(K, W)
    if w.prefill:
        starts = [torch.full((n,), w.ctx + i, dtype=torch.int32, device=dev) for i in range(n_new)]
        lens_l = [torch.full((n,), w.ctx + i + 1, dtype=torch.int32) for i in range(n_new)]
        k_new = [synth.new_token_values(w, "k", i, dev) for i in range(n_new)]
        v_new = [synth.new_token_values(w, "v", i, dev) for i in range(n_new)]
    else:
        starts = [(lens - 1).to(torch.int32).to(dev)] * n_new
        lens_l = [lens] * n_new
        k_new = [synth.new_token_values(w, "k", 0, dev)] * n_new
        v_new = [synth.new_token_values(w, "v", 0, dev)] * n_new
    lens_d = [L.to(dev) for L in lens_l]
    cu1 = torch.arange(n + 1, dtype=torch.int32, device=dev)
    q = synth.queries(w, 0, dev)
    max_len = max(int(L.max()) for L in lens_l)
    scale = float(np.float32(1.0 / math.sqrt(d)))
    out = torch.empty(n, Hq, d, dtype=torch.float32, device=dev)
    win = max(0, args.window)
    ws_bytes = B.attention_workspace_bytes(n, Hq, H, d, max_len, win)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=dev)
    scratch = torch.empty(1 << 30, dtype=torch.uint8, device=dev) if cold else None

    def step(i, ev=None):
        if ev is not None:
            ev[0].record()
        B.quantize_kv(cache, k_new[i], v_new[i], bt, starts[i], cu1, 1)
        if ev is not None:
            ev[1].record()
        B.decode_attention(cache, q, bt, lens_d[i], max_len, scale, out=out, workspace=ws, window=win)
        if ev is not None:
            ev[2].record()

    for i in range(W):
        if cold:
            scratch.fill_(i & 0xff)
        step(i)
    torch.cuda.synchronize()
    evs = [tuple(torch.cuda.Event(enable_timing=True) for _ in range(3)) for _ in range(K)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(K):
        if cold:
            scratch.fill_((i + 7) & 0xff)   # outside the step's events
        step(i, evs[i])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    quant_s = [a.elapsed_time(b) / 1e3 for a, b, _ in evs]
    attn_s = [b.elapsed_time(c) / 1e3 for _, b, c in evs]
    step_s = sum(quant_s) + sum(attn_s)
    attn_avg_s = sum(attn_s) / K
    log(f"{K} steps in {elapsed * 1e3:.2f} ms wall; events: quantize avg {sum(quant_s) / K * 1e6:.1f} us, "
        f"attention avg {attn_avg_s * 1e6:.1f} us")
    if cold:
        del scratch
        torch.cuda.empty_cache()

    if args.copy_probe_mib:
        src = torch.ones(args.copy_probe_mib * 2**20 // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst

    # ---- algorithmic bytes of the attention launches ---------------------------------
    prefix = outlier_prefix(cache, bt_cpu, n, max_len)
    kv_tot, alg_tot, out_tot, vec_tot = 0, 0, 0, 0
    memo = {}
    for i in range(K):
        key = id(lens_l[i])
        if key not in memo:
            memo[key] = attention_bytes(cache, prefix, lens_l[i], win, Hq, n)
        kv_i, alg_i, out_i, vec_i, pages_i = memo[key]
        kv_tot += kv_i
        alg_tot += alg_i + (pages_i * H * 2 * 8 if args.paged else 0)   # (paged: each record's first two page ids)
        out_tot += out_i
        vec_tot += vec_i
    achieved = alg_tot / sum(attn_s) / 1e9
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": stored_traffic(w.name) if not (win or args.paged or w.prefill) else None,
                "bytes_per_launch": int(alg_tot / K), "kv_stream_bytes_per_launch": int(kv_tot / K),
                "kernel_us": round(attn_avg_s * 1e6, 2),
                "overhead_bytes_per_launch": {"split_partials_written_and_read": 2 * ws_bytes},
                "outlier_fraction": round(out_tot / (vec_tot * d), 4)}
    quant_res = {"us_per_step": round(sum(quant_s) / K * 1e6, 2),
                 "attention_us_per_step": round(attn_avg_s * 1e6, 2)}

    stream = None
    if not args.no_stream_probe:
        stream = stream_probe(cache, dev)
        stream["attention_frac_of_plain"] = round(achieved / stream["plain_4gib"]["gbs"], 4)
        stream["attention_frac_of_record_prefix"] = round(achieved / stream["record_prefix"]["gbs"], 4)

    # ---- CPU oracle on a bounded sample + sampled parity -------------------------------
    cpu = None
    parity = None
    if not args.no_cpu_baseline:
        import oracle
        S = min(n, args.cpu_sample_seqs or (4 if w.prefill else 128))
        sample = list(range(0, n, max(1, n // S)))[:S]
        thr_np = thr.cpu().numpy()
        lay = oracle.layout(16, d)
        last = K - 1
        L_fin = [int(lens_l[last][s]) for s in sample]
        nb_s = [(L + 15) // 16 for L in L_fin]
        bt_s = np.zeros((S, max(nb_s)), np.int32)
        off = 0
        for i, nb in enumerate(nb_s):
            bt_s[i, :nb] = np.arange(off, off + nb)
            off += nb
        pool_s = np.zeros(off * H * 2 * lay["stride"], np.uint8)
        pre_s = np.array([pre[s] for s in sample], np.int32)
        kk = torch.cat([synth.kv_values_seq(w, "k", s, int(p), dev) for s, p in zip(sample, pre_s)]).cpu().numpy()
        vv = torch.cat([synth.kv_values_seq(w, "v", s, int(p), dev) for s, p in zip(sample, pre_s)]).cpu().numpy()
        cu = np.concatenate([[0], np.cumsum(pre_s)]).astype(np.int32)
        threads = oracle.max_threads()
        t0 = time.perf_counter()
        oracle.quantize_kv(pool_s, off, 16, H, d, thr_np, kk, vv, bt_s, np.zeros(S, np.int32), cu)
        t_pre = time.perf_counter() - t0
        del kk, vv
        ar = np.arange(S + 1, dtype=np.int32)
        # decode steps before the last one (the prefill workload's growing context)
        for i in range(last if w.prefill else 0):
            oracle.quantize_kv(pool_s, off, 16, H, d, thr_np, k_new[i].cpu().numpy()[sample],
                               v_new[i].cpu().numpy()[sample], bt_s, starts[i].cpu().numpy()[sample], ar)
        kn = k_new[last].cpu().numpy()[sample]
        vn = v_new[last].cpu().numpy()[sample]
        st_s = starts[last].cpu().numpy()[sample]
        qs = q.cpu().numpy()[sample]
        lens_s = np.array(L_fin, np.int32)
        log(f"oracle sample: {S} sequences built in {t_pre:.1f} s ({threads} threads); timing one decode step")

        def one_step(idx):
            oracle.quantize_kv(pool_s, off, 16, H, d, thr_np, kn[idx], vn[idx], bt_s[idx], st_s[idx],
                               np.arange(len(idx) + 1, dtype=np.int32))
            return oracle.decode_attention(pool_s, off, 16, H, d, thr_np, qs[idx], bt_s[idx], lens_s[idx], scale,
                                           window=win)

        times = []
        for _ in range(3):   # median of three steps (re-quantizing the same slot is idempotent)
            t0 = time.perf_counter()
            want = one_step(np.arange(S))
            times.append(time.perf_counter() - t0)
        cpu_s = sorted(times)[1]
        # one thread, on an eighth of the sample
        S1 = max(1, S // 8)
        oracle.set_threads(1)
        t0 = time.perf_counter()
        one_step(np.arange(S1))
        cpu1_s = time.perf_counter() - t0
        oracle.set_threads(threads)
        cpu = {"value": round(S / cpu_s, 2), "unit": "tokens/s", "cores": threads, "kind": "oracle",
               "sample": f"{S} of {n} sequences (context {L_fin[0]}, all {Hq} heads), one decode step "
                         f"(quantize + attention), median of 3: {cpu_s:.2f} s",
               "one_thread": {"value": round(S1 / cpu1_s, 3), "unit": "tokens/s", "cores": 1,
                              "sample": f"{S1} sequences, one decode step: {cpu1_s:.2f} s"}}
        if w.prefill:
            cpu["prefill_quantize_tokens_per_s"] = round(int(pre_s.sum()) / t_pre, 1)
        got = out.cpu().numpy()[sample]
        err = np.abs(got.astype(np.float64) - want)
        okm = err <= 2e-3 + 1e-2 * np.abs(want)
        parity = {"seqs": S, "max_abs": float(err.max()), "pass": bool(okm.all())}
        log(f"oracle {cpu_s:.2f}s ({threads} threads), {cpu1_s:.2f}s for {S1} at 1 thread; "
            f"parity max_abs={err.max():.2e} pass={bool(okm.all())}")

    value = n * K / (step_s if cold else elapsed)
    res = {
        "metric": "decode-attention tokens/sec + achieved HBM GB/s (% of peak) at batch 256",
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round((step_s if cold else elapsed) / K * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i8mfma-4limb+f32",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: batch {n}, {Hq} query / {H} KV heads, head_dim {d}, "
                               + (f"context {w.ctx} quantized by one prefill call, then {K} decode steps "
                                  f"(context {w.ctx + 1}..{w.ctx + K})" if w.prefill else
                                  f"context {w.ctx_min}..{w.ctx} incl. the new token")
                               + ", 16-token pages, shuffled block table"
                               + (f", sliding window {win}" if win else "")
                               + (", on-demand 256-byte sparse pages" if args.paged else "")
                               + "; step = quantize 1 token/seq + attention",
                   "global_batch": n, "seq_len": max_len, "parallelism": "single GPU"},
        "timing": ("HIP events per step; a 1 GiB scratch write between steps (outside the events) evicts "
                   "the 256 MB Infinity Cache" if cold else "wall clock over the steps, back to back")
                  + f"; wall {elapsed / K * 1e3:.4f} ms/step",
        "roofline": roofline,
        "step_breakdown": quant_res,
        "stream_read": stream,
        **({"prefill_quantize": prefill_res} if prefill_res else {}),
        "cpu_baseline": cpu,
        **({"capacity": capacity} if capacity else {}),
        "parity_sample": parity,
        "attention_source": source_hash(),
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
