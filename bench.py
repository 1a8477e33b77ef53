#!/usr/bin/env python3
"""Benchmark of the block-sparse causal GQA prefill operator on one MI355X.

One step = one fp2_prefill call (block means, fused scoring and selection,
sparse attention with the mean correction) over one synthetic layer whose
inputs are already resident in HBM. Default workload: 128K tokens, 32 query /
8 KV heads, head_dim 128, block 128, paged KV (page 64), fp8 e4m3 with
per-head scales, threshold calibrated to ~5% kept blocks, correction on.

Prints ONE JSON line with the dense-equivalent throughput, the latency, the
kept-block ratio, a roofline entry for the attention kernel (the dominant
kernel; its duration from HIP events the library records right around its
launch), the oracle timed on the host cores on a bounded sample, and a
`configs` array with every benchmark configuration (2K, 32K bf16, the 128K
fp8 layer at 10 / 5 / 2 % kept with the correction on and off, the ragged
batch of 8, the 128K 64/8-head layer in bf16 and fp8 with its error against
dense attention). --variants adds the paper-literal 128-row selection tile.
The roofline's HBM traffic comes from the committed rocprofv3 counter summary
of the attention kernel, and the estimation stage's traffic (pool + estimate
kernels) from its own summary, each only while the kernel sources are the
ones the counters were taken on (else null).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "128K prefill attn latency + dense-equiv TFLOP/s (bf16/fp8); kept-block ratio"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attend_kernel_llama128k_fp8_pmc.txt")
KERNEL_SOURCES = ["paper_2608_19758_amd/csrc/attend.hip", "paper_2608_19758_amd/csrc/kernels.h",
                  "paper_2608_19758_amd/csrc/common.h"]
PEAK_TFLOPS = {"bf16": 2500.0, "fp8": 5000.0}
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama128k_fp8")
    ap.add_argument("--target", default="0.05", help="kept-ratio target the alpha was calibrated for")
    ap.add_argument("--variants", action="store_true",
                    help="also measure the paper-literal 128-row selection tile on the headline "
                         "workload and the mask-to-CSR conversion")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-config array (every benchmark configuration)")
    ap.add_argument("--chunked", action="store_true",
                    help="also measure chunked prefill of the default workload through the "
                         "serving backend (prefix KV), its short tail chunks with and without KV "
                         "splits, and a continuous-batching forward of four requests")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-units", type=int, default=768,
                    help="(sequence, KV head, query block) units the oracle runs for the CPU baseline")
    ap.add_argument("--profile-only", action="store_true",
                    help="only run the timed loop of the default workload (for rocprofv3)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 256 MiB device copy three times (scales the "
                         "FETCH_SIZE / WRITE_SIZE counters)")
    return ap.parse_args()


def kernel_sources_sha256():
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


ESTIMATION_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "estimation_llama128k_fp8_pmc.txt")
ESTIMATION_SOURCES = ["paper_2608_19758_amd/csrc/pool.hip", "paper_2608_19758_amd/csrc/estimate.hip",
                      "paper_2608_19758_amd/csrc/kernels.h", "paper_2608_19758_amd/csrc/common.h"]


def estimation_sources_sha256():
    import hashlib
    h = hashlib.sha256()
    for rel in ESTIMATION_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def committed_estimation_traffic():
    """HBM bytes per estimation call (pool + estimate kernels) from the
    committed counter summary, scaled like the attention's; None if missing or
    taken on other kernel sources."""
    try:
        with open(ESTIMATION_TRAFFIC_FILE) as f:
            kv = dict(line.split(":", 1) for line in f if ":" in line and not line.startswith("#"))
    except OSError:
        return None
    kv = {k.strip(): v.strip() for k, v in kv.items()}
    if kv.get("source_sha256") != estimation_sources_sha256():
        return None
    try:
        return float(kv["stage_traffic_bytes"])
    except (KeyError, ValueError):
        return None


def committed_traffic():
    """HBM bytes per attention launch from the committed counter summary:
    FETCH_SIZE and WRITE_SIZE (KiB per dispatch) times the factors a plain
    copy of known size gives; None if the summary is missing or was taken on
    other kernel sources."""
    try:
        with open(TRAFFIC_FILE) as f:
            kv = dict(line.split(":", 1) for line in f if ":" in line and not line.startswith("#"))
    except OSError:
        return None
    kv = {k.strip(): v.strip() for k, v in kv.items()}
    if kv.get("source_sha256") != kernel_sources_sha256():
        return None
    try:
        return (float(kv["fetch_kib_per_dispatch"]) * 1024 * float(kv["fetch_scale"])
                + float(kv["write_kib_per_dispatch"]) * 1024 * float(kv["write_scale"]))
    except (KeyError, ValueError):
        return None


def copy_calibration():
    import torch
    n = 256 << 20
    x = torch.randint(0, 255, (n,), dtype=torch.uint8, device="cuda")
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    for _ in range(3):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n, "copies": 3}), flush=True)


def measured_peaks():
    """Reference rates measured on this GPU in the same run: a 1 GiB device
    copy (bytes read + written per second); the library's MFMA and exp loops
    (fp2_calibrate: the matrix instructions the kernels issue, and v_exp_f32,
    on every SIMD with no memory traffic); and the library GEMMs (hipBLASLt
    through torch) at 8192^3 in bf16 and fp8 e4m3 -- next to the vendor peaks
    the roofline uses."""
    import torch
    import paper_2608_19758_amd as fp2

    def timed(fn, reps=5):
        fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps * 1e-3

    res = {}
    n = 1 << 30
    x = torch.empty(n, dtype=torch.uint8, device="cuda")
    y = torch.empty_like(x)
    res["copy_gbs"] = round(2 * n / timed(lambda: y.copy_(x)) / 1e9, 1)
    del x, y
    sink = torch.zeros(1, dtype=torch.float32, device="cuda")
    for key, kind, iters, unit in (("mfma_bf16_tflops", "mfma_bf16", 50000, 1e12),
                                   ("mfma_fp8_tflops", "mfma_fp8", 25000, 1e12),
                                   ("exp_per_s", "exp", 25000, 1.0)):
        ops = fp2.calibrate(kind, iters, sink)
        res[key] = float("%.4g" % (ops / timed(lambda: fp2.calibrate(kind, iters, sink)) / unit))
    m = 8192
    a = torch.randn(m, m, device="cuda", dtype=torch.bfloat16)
    bt = torch.randn(m, m, device="cuda", dtype=torch.bfloat16)
    res["gemm_bf16_tflops"] = round(2 * m ** 3 / timed(lambda: a @ bt) / 1e12, 1)
    try:
        a8 = a.to(torch.float8_e4m3fn)
        b8 = bt.to(torch.float8_e4m3fn).t().contiguous().t()
        one = torch.ones((), device="cuda", dtype=torch.float32)
        res["gemm_fp8_tflops"] = round(2 * m ** 3 / timed(
            lambda: torch._scaled_mm(a8, b8, scale_a=one, scale_b=one,
                                     out_dtype=torch.bfloat16)) / 1e12, 1)
    except Exception as e:   # the fp8 GEMM path may be missing from this torch build
        res["gemm_fp8_tflops"] = None
        print("[bench] fp8 GEMM reference unavailable: %s" % e, file=sys.stderr, flush=True)
    del a, bt
    torch.cuda.empty_cache()
    return res


def setup(name, target, correction=None, tile_rows=0, base=None):
    """Inputs resident on the GPU, buffers and the prefill call of one
    workload at one calibrated threshold. base: a setup of the same workload
    whose generated inputs are reused (other threshold or correction)."""
    import torch
    import paper_2608_19758_amd as fp2
    import synth

    if base is not None and base["spec"].name == name:
        wl, d = base["wl"], base["d"]
        spec = wl.spec
    else:
        spec = synth.named(name)
        wl = synth.generate(spec)
        d = wl.device_inputs("cuda")
        if spec.dtype == "bf16":
            for k in ("q", "k_cache", "v_cache"):
                d[k] = d[k].view(torch.bfloat16)
    corr = spec.mean_correction if correction is None else int(correction)
    alpha = synth.alpha_for(name, target)
    p = fp2.make_params(batch=spec.batch, num_q_heads=spec.num_q_heads,
                        num_kv_heads=spec.num_kv_heads, max_seq_len=spec.max_seq_len,
                        page_size=spec.page_size, max_pages_per_seq=wl.max_pages, alpha=alpha,
                        sink_blocks=spec.sink_blocks, window_blocks=spec.window_blocks,
                        recent_blocks=spec.recent_blocks, mean_correction=corr,
                        dtype=spec.dtype, query_tile_rows=tile_rows)
    out, mask, _ = fp2.alloc_outputs(p, spec.total_tokens)
    ws = fp2.alloc_workspace(p)
    bt = d["block_table"] if spec.page_size else None
    kw = dict(cu_seqlens_host=wl.cu_seqlens, q_scale=d["q_scale"], k_scale=d["k_scale"],
              v_scale=d["v_scale"])

    def run_prefill(out=out, p=p):
        fp2.prefill(p, d["q"], d["k_cache"], d["v_cache"], d["cu_seqlens"], bt, out=out,
                    block_mask=mask, workspace=ws, **kw)

    def run_csr():
        return fp2.mask_to_csr(p, mask, d["cu_seqlens"], workspace=ws)

    return dict(spec=spec, wl=wl, alpha=alpha, p=p, d=d, out=out, mask=mask, ws=ws,
                target=target, correction=corr, run_prefill=run_prefill, run_csr=run_csr)


def time_loop(fn, steps, warmup):
    """Average ms per call with HIP events on the current stream (the stream
    the library launches on), bracketed by device synchronisation."""
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(steps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    return e0.elapsed_time(e1) / steps, (t1 - t0) * 1e3 / steps


def timed_prefill(cfg, steps, warmup):
    """K prefill steps timed with HIP events on the library's stream, and in
    each step the library records one more event pair right around the
    attention kernel and one around the estimation kernels (fp2_time_kernels):
    (ms per step, wall ms per step, estimation-kernel ms, attention-kernel
    ms), averages over the K steps."""
    import torch
    import paper_2608_19758_amd as fp2
    for _ in range(warmup):
        cfg["run_prefill"]()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    for row in ev:
        for e in row:
            e.record()   # creates the event the library records into
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record()
    try:
        for i in range(steps):
            fp2.time_kernels(estimate=(ev[i][0], ev[i][1]), attend=(ev[i][2], ev[i][3]))
            cfg["run_prefill"]()
    finally:
        fp2.time_kernels()
    e1.record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    est = sum(r[0].elapsed_time(r[1]) for r in ev) / steps
    att = sum(r[2].elapsed_time(r[3]) for r in ev) / steps
    return e0.elapsed_time(e1) / steps, (t1 - t0) * 1e3 / steps, est, att


def measure(cfg, steps, warmup):
    from paper_2608_19758_amd import accounting as acc
    sp = cfg["spec"]
    t_pre, wall, t_est, t_attn = timed_prefill(cfg, steps, warmup)
    mask = cfg["mask"].cpu().numpy()
    if cfg["p"].query_tile_rows:
        # kept pairs over visible (tile, key block) pairs of the 128-row tiles
        pt = cfg["p"].query_tile_rows // (sp.num_q_heads // sp.num_kv_heads)
        vis = sum(sum(t * pt // 128 + 1 for t in range((L + pt - 1) // pt)) for L in sp.seqlens)
        kept_ratio = float((mask & 1).sum()) / max(1, vis * sp.num_kv_heads)
    else:
        kept_ratio = acc.block_counts(mask, sp.seqlens, sp.block_size, False)[0] / max(
            1, sum(((L + 127) // 128) * ((L + 127) // 128 + 1) // 2 for L in sp.seqlens)
            * sp.num_kv_heads)
    dense = acc.dense_equiv_flops(sp.seqlens, sp.num_q_heads)
    fk, fc = acc.attention_flops(mask, sp.seqlens, sp.num_q_heads, sp.num_kv_heads,
                                 correction=bool(cfg["correction"]),
                                 tile_rows=cfg["p"].query_tile_rows)
    t_attn = max(1e-6, t_attn)
    main_peak = PEAK_TFLOPS[sp.dtype]
    # time-weighted peak of the MFMA types the kernel issues: the kept tiles
    # and the correction chunks both run on the workload dtype's MFMA (fp8
    # inputs score the pooled means' e4m3 codes), so it is the dtype's peak
    corr_peak = main_peak
    mix = (fk + fc) / (fk / main_peak + fc / corr_peak) if (fk + fc) else main_peak
    achieved = (fk + fc) / (t_attn * 1e-3) / 1e12
    est_bytes = acc.estimation_bytes(sp.seqlens, sp.num_q_heads, sp.num_kv_heads,
                                     elem=1 if sp.dtype == "fp8" else 2)
    sflop = acc.scoring_flops(sp.seqlens, sp.num_q_heads)   # bf16 MFMA (scoring key in bf16)
    return dict(
        ms_per_step=t_pre, wall_ms_per_step=wall, estimate_ms=t_est, attention_ms=t_attn,
        dense_tflops=dense / (t_pre * 1e-3) / 1e12, kept_ratio=kept_ratio,
        attention=dict(executed_tflop=(fk + fc) / 1e12, kept_tflop=fk / 1e12, corr_tflop=fc / 1e12,
                       achieved_tflops=achieved, peak_tflops=main_peak,
                       frac=achieved / main_peak, mix_peak_tflops=mix, frac_mix=achieved / mix),
        estimation=dict(alg_bytes=est_bytes, gbs=est_bytes / (t_est * 1e-3) / 1e9,
                        hbm_frac=est_bytes / (t_est * 1e-3) / 1e9 / PEAK_HBM_GBS,
                        scoring_tflop=sflop / 1e12,
                        mfma_frac=sflop / (t_est * 1e-3) / 1e12 / PEAK_TFLOPS["bf16"],
                        exps_per_s=sflop / (2 * sp.head_dim) / (t_est * 1e-3)),
    )


def config_entry(cfg, r, cid):
    """One entry of the per-config array."""
    sp = cfg["spec"]
    return {"config": cid, "workload": sp.name, "dtype": sp.dtype, "batch": sp.batch,
            "seqlens": sp.seqlens if sp.batch <= 8 else None,
            "num_q_heads": sp.num_q_heads, "num_kv_heads": sp.num_kv_heads,
            "kept_target": float(cfg["target"]), "alpha": cfg["alpha"],
            "mean_correction": cfg["correction"],
            "ms": round(r["ms_per_step"], 4),
            "dense_tflops": round(r["dense_tflops"], 2),
            "kept_ratio": round(r["kept_ratio"], 5),
            "attention_kernel_ms": round(r["attention_ms"], 4),
            "attention_executed_tflops": round(r["attention"]["achieved_tflops"], 1),
            "attention_mfma_frac": round(r["attention"]["frac"], 4),
            "attention_mfma_frac_mix": round(r["attention"]["frac_mix"], 4),
            "estimate_ms": round(r["estimate_ms"], 4),
            "estimation_hbm_frac": round(r["estimation"]["hbm_frac"], 4),
            "estimation_scoring_mfma_frac": round(r["estimation"]["mfma_frac"], 4)}


def error_vs_dense(cfg):
    """The sparse output against dense attention computed by the same kernels
    with every causal block kept (alpha = 0): max-abs and relative Frobenius
    error over every output element."""
    import torch
    import paper_2608_19758_amd as fp2
    sp = cfg["spec"]
    p0 = fp2.make_params(batch=sp.batch, num_q_heads=sp.num_q_heads,
                         num_kv_heads=sp.num_kv_heads, max_seq_len=sp.max_seq_len,
                         page_size=sp.page_size, max_pages_per_seq=cfg["wl"].max_pages, alpha=0.0,
                         sink_blocks=sp.sink_blocks, window_blocks=sp.window_blocks,
                         recent_blocks=sp.recent_blocks, mean_correction=cfg["correction"],
                         dtype=sp.dtype)
    dense = torch.empty_like(cfg["out"])
    cfg["run_prefill"]()
    cfg["run_prefill"](out=dense, p=p0)
    torch.cuda.synchronize()
    worst, num, den = 0.0, 0.0, 0.0
    for t0 in range(0, dense.shape[0], 16384):
        a = cfg["out"][t0:t0 + 16384].float()
        b = dense[t0:t0 + 16384].float()
        worst = max(worst, float((a - b).abs().max()))
        num += float(((a - b) ** 2).sum())
        den += float((b ** 2).sum())
    del dense
    return {"max_abs": float("%.4g" % worst), "rel_fro": float("%.4g" % ((num / max(den, 1e-300)) ** 0.5)),
            "reference": "dense causal attention by the same kernels at alpha = 0"}


def run_configs(head_cfg, head_m, steps, warmup):
    """Every benchmark configuration: tiny 2K, 32K bf16, the 128K fp8 layer at
    10 / 5 / 2 % kept with the correction on and off, the ragged batch of 8,
    and the 128K 64/8-head layer in bf16 and fp8 with its error against dense
    attention. The headline measurement is reused for its own entry."""
    import torch
    entries = []
    plan = [(0, "tiny2k", "0.30", None), (1, "llama32k", "0.18", None)]
    plan += [(2, "llama128k_fp8", t, c) for t in ("0.10", "0.05", "0.02") for c in (1, 0)]
    plan += [(3, "ragged8", "0.18", None), (4, "wide128k_bf16", "0.009", None),
             (4, "wide128k_fp8", "0.009", None)]
    base = head_cfg
    for cid, name, tgt, corr in plan:
        hs = head_cfg["spec"]
        if (name, tgt) == (hs.name, head_cfg["target"]) and \
                (corr is None or corr == head_cfg["correction"]):
            entries.append(config_entry(head_cfg, head_m, cid))
            entries[-1]["headline"] = True
            continue
        c = setup(name, tgt, corr, base=base if base is not None and base["spec"].name == name
                  else None)
        big = c["spec"].max_seq_len >= 65536 or c["spec"].batch > 1
        r = measure(c, max(5, steps // 2) if big else steps, max(2, warmup // 2))
        e = config_entry(c, r, cid)
        if cid == 4:
            e["error_vs_dense"] = error_vs_dense(c)
        entries.append(e)
        print("[bench] config %s" % json.dumps(e), file=sys.stderr, flush=True)
        if c["spec"].name != head_cfg["spec"].name:
            del c
            torch.cuda.empty_cache()
    return entries


def chunked(cfg, steps, warmup):
    """Chunked prefill of the headline sequence through the serving backend
    (paper_2608_19758_amd.serving): the same 128K tokens as sequential
    forwards over chunks of C tokens, chunk c attending to the c*C tokens
    before it as a cached prefix (the serving mode of the paper's
    chunked-prefill experiments), timed as the sum of the per-layer
    forward_extend calls with the per-forward metadata prepared beforehand;
    short tail chunks (the last T tokens after a 128K - T prefix) with the
    cost-balanced KV splits against kv_splits = 1; and one continuous-batching
    forward mixing four requests at different prefix lengths. Chunk sequences
    and tails are also timed with the block-means cache (complete prefix
    blocks copied instead of pooled again)."""
    import torch
    import paper_2608_19758_amd.serving as serving
    sp, wl, d = cfg["spec"], cfg["wl"], cfg["d"]
    L = sp.seqlens[0]
    dev = d["q"].device

    def backend(max_batch, max_ext, splits=0):
        c = serving.BackendConfig(num_q_heads=sp.num_q_heads, num_kv_heads=sp.num_kv_heads,
                                  page_size=sp.page_size, max_batch=max_batch,
                                  max_extend_len=max_ext, max_kv_len=L, dtype=sp.dtype,
                                  alpha=cfg["alpha"], sink_blocks=sp.sink_blocks,
                                  window_blocks=sp.window_blocks,
                                  recent_blocks=sp.recent_blocks,
                                  mean_correction=bool(sp.mean_correction), kv_splits=splits)
        return serving.PrefillBackend(c)

    def table(be, rows):
        bt = torch.zeros((rows, be.cfg.max_pages_per_seq), dtype=torch.int32, device=dev)
        bt[:, :d["block_table"].shape[1]] = d["block_table"][0]
        return bt

    kw = dict(q_scale=d["q_scale"], k_scale=d["k_scale"], v_scale=d["v_scale"])
    res = {"chunks": [], "tails": [], "batched": None}
    for C in (16384, 8192):
        be = backend(1, C)
        bt = table(be, 1)
        mc = be.alloc_means_cache(wl.num_pages)
        out = torch.empty((C, sp.num_q_heads, sp.head_dim), dtype=torch.bfloat16, device=dev)
        r = {"chunk": C}
        # without and with the block-means cache (chunk c takes the complete
        # blocks of its prefix, which the chunks before it pooled)
        for key, cache in (("total_ms", None), ("total_ms_means_cache", mc)):
            calls = []
            for c0 in range(0, L, C):
                meta = be.init_forward_metadata([C], [c0], bt,
                                                cached_prefix_lens=None if cache is None else [c0])
                calls.append((meta, d["q"][c0:c0 + C]))

            def all_chunks():
                for meta, q in calls:
                    be.forward_extend(q, d["k_cache"], d["v_cache"], meta, out=out,
                                      means_cache=cache, **kw)
            t, _ = time_loop(all_chunks, max(3, steps // 4), max(1, warmup // 2))
            r[key] = round(t, 4)
            r["calls"] = len(calls)
        res["chunks"].append(r)
        print("[bench] chunked %d x %d: %.3f ms, with the means cache %.3f ms"
              % (r["calls"], C, r["total_ms"], r["total_ms_means_cache"]), file=sys.stderr,
              flush=True)
        del be, calls, mc
    for T in (128, 1024, 4096):
        r = {"tail_tokens": T, "prefix": L - T}
        for splits, key in ((0, "ms_planned_splits"), (1, "ms_no_splits"),
                            (0, "ms_planned_splits_means_cache")):
            be = backend(1, T, splits)
            q = d["q"][L - T:]
            out = torch.empty((T, sp.num_q_heads, sp.head_dim), dtype=torch.bfloat16, device=dev)
            mc = None
            if key.endswith("means_cache"):
                # one call fills the cache with the means of every block
                mc = be.alloc_means_cache(wl.num_pages)
                fill = be.init_forward_metadata([T], [L - T], table(be, 1))
                be.forward_extend(q, d["k_cache"], d["v_cache"], fill, out=out, means_cache=mc,
                                  **kw)
            meta = be.init_forward_metadata([T], [L - T], table(be, 1),
                                            cached_prefix_lens=None if mc is None else [L - T])
            fwd = lambda: be.forward_extend(q, d["k_cache"], d["v_cache"], meta, out=out,   # noqa: E731
                                            means_cache=mc, **kw)
            r[key] = round(time_loop(fwd, steps, warmup)[0], 4)
            if mc is not None:
                # the same forward captured once in a HIP graph and replayed
                side = torch.cuda.Stream()
                side.wait_stream(torch.cuda.current_stream())
                with torch.cuda.stream(side):
                    fwd()
                torch.cuda.current_stream().wait_stream(side)
                torch.cuda.synchronize()
                graph = torch.cuda.CUDAGraph()
                with torch.cuda.graph(graph):
                    fwd()
                r[key + "_graph"] = round(time_loop(graph.replay, steps, warmup)[0], 4)
                del graph
            del be, mc
        res["tails"].append(r)
        print("[bench] tail %d: planned splits %.3f ms, none %.3f ms, planned + means cache %.3f ms"
              " (%.3f ms replayed from a HIP graph)"
              % (T, r["ms_planned_splits"], r["ms_no_splits"], r["ms_planned_splits_means_cache"],
                 r["ms_planned_splits_means_cache_graph"]), file=sys.stderr, flush=True)
    # four requests of the same sequence data at different stages of their
    # prefill, in one forward (continuous batching)
    ext, pre = [8192, 8192, 4096, 1024], [0, 32768, 90112, 130048]
    be = backend(4, 8192)
    meta = be.init_forward_metadata(ext, pre, table(be, 4))
    q = torch.cat([d["q"][p:p + e] for e, p in zip(ext, pre)])
    out = torch.empty((q.shape[0], sp.num_q_heads, sp.head_dim), dtype=torch.bfloat16, device=dev)
    t, _ = time_loop(lambda: be.forward_extend(q, d["k_cache"], d["v_cache"], meta, out=out, **kw),
                     steps, warmup)
    mc = be.alloc_means_cache(wl.num_pages)
    be.forward_extend(q, d["k_cache"], d["v_cache"], meta, out=out, means_cache=mc, **kw)   # fill
    meta_c = be.init_forward_metadata(ext, pre, table(be, 4), cached_prefix_lens=pre)
    tc, _ = time_loop(lambda: be.forward_extend(q, d["k_cache"], d["v_cache"], meta_c, out=out,
                                                means_cache=mc, **kw), steps, warmup)
    dense = sum(sp.num_q_heads * 4 * sp.head_dim * (e * p + e * (e + 1) / 2) for e, p in zip(ext, pre))
    res["batched"] = {"extend": ext, "prefix": pre, "ms": round(t, 4),
                      "ms_means_cache": round(tc, 4),
                      "dense_equiv_tflops": round(dense / (t * 1e-3) / 1e12, 1)}
    print("[bench] batched forward %s after %s: %.3f ms, with the means cache %.3f ms"
          % (ext, pre, t, tc), file=sys.stderr, flush=True)
    del be
    torch.cuda.empty_cache()
    return res


def cpu_baseline(cfg, nunits):
    """The oracle on a bounded sample of the same workload: every KV head,
    query blocks at an even stride (heaviest included); estimation plus
    attention of those units under the oracle's own mask."""
    import numpy as np
    import oracle
    sp, wl = cfg["spec"], cfg["wl"]
    B, g = sp.block_size, sp.num_q_heads // sp.num_kv_heads
    n = (sp.seqlens[0] + B - 1) // B
    per_head = max(1, nunits // sp.num_kv_heads)
    Is = sorted(set(np.linspace(n - 1, 0, per_head).round().astype(int).tolist()))
    units = [(0, h, I) for h in range(sp.num_kv_heads) for I in Is]
    inp = oracle.Inputs(wl)
    op = inp.params(cfg["alpha"])
    t0 = time.perf_counter()
    mask = oracle.estimate(inp, op, units=units)
    oracle.attend(inp, op, mask, units=units)
    dt = time.perf_counter() - t0
    L = sp.seqlens[0]
    flops = 0.0
    for _, _, I in units:
        p0, p1 = I * B, min(L, (I + 1) * B)
        pos = np.arange(p0, p1)
        flops += float(g * 4 * sp.head_dim * (pos + 1).sum())
    cpu_model = None
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((ln.split(":", 1)[1].strip() for ln in f
                              if ln.startswith("model name")), None)
    except OSError:
        pass
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s (dense-equivalent)",
            "cores": op.nthreads, "kind": "oracle", "cpu_model": cpu_model,
            "sample": "%d units (all %d KV heads x %d query blocks at an even stride, incl. the last) "
                      "of %s: estimation + attention, %.1f s" % (len(units), sp.num_kv_heads,
                                                                 len(Is), sp.name, dt),
            "seconds": dt}


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on exactly one GPU: this operator build has no multi-GPU path "
              "(the path would shard by KV head); got --gpus %d, WORLD_SIZE %d"
              % (args.gpus, world), file=sys.stderr)
        sys.exit(2)
    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"

    if args.copy_calibration:
        copy_calibration()
        return
    cfg = setup(args.workload, args.target)
    if args.profile_only:
        t, _ = time_loop(cfg["run_prefill"], args.steps, args.warmup)
        print(json.dumps({"profile_only": True, "ms_per_step": t}), flush=True)
        return
    m = measure(cfg, args.steps, args.warmup)
    sp = cfg["spec"]
    print("[bench] %s: %.3f ms, %.1f dense-equiv TFLOP/s, kept %.4f" % (
        sp.name, m["ms_per_step"], m["dense_tflops"], m["kept_ratio"]), file=sys.stderr, flush=True)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, args.cpu_units)
        print("[bench] cpu baseline: %s" % cpu["sample"], file=sys.stderr, flush=True)

    chunk_res = chunked(cfg, args.steps, args.warmup) if args.chunked else None
    peaks = measured_peaks()
    print("[bench] measured on this GPU: %s" % json.dumps(peaks), file=sys.stderr, flush=True)

    configs = []
    if not args.no_configs:
        configs = run_configs(cfg, m, args.steps, args.warmup)
    variants = []
    if args.variants:
        # the paper-literal selection tile (128 packed rows) on the headline
        # workload, and the mask-to-CSR conversion of the headline mask
        csr_ms = time_loop(cfg["run_csr"], max(5, args.steps // 2), 2)[0]
        print("[bench] mask to CSR: %.3f ms" % csr_ms, file=sys.stderr, flush=True)
        c = setup(args.workload, args.target, None, 128, base=cfg)
        r = measure(c, max(5, args.steps // 2), max(2, args.warmup // 2))
        e = config_entry(c, r, 2)
        e["query_tile_rows"] = 128
        variants.append(e)
        print("[bench] variant %s" % json.dumps(e), file=sys.stderr, flush=True)
        del c
        torch.cuda.empty_cache()

    att = m["attention"]
    headline = (args.workload, args.target) == ("llama128k_fp8", "0.05")
    traffic = committed_traffic() if headline else None
    etraffic = committed_estimation_traffic() if headline else None
    line = {
        "metric": METRIC,
        "value": round(m["dense_tflops"], 3),
        "unit": "TFLOP/s (dense-equivalent)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(m["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": sp.dtype,
        "data": "synthetic",
        "config": {"workload": sp.name, "seq_len": sp.max_seq_len, "batch": sp.batch,
                   "num_q_heads": sp.num_q_heads, "num_kv_heads": sp.num_kv_heads,
                   "head_dim": sp.head_dim, "block_size": sp.block_size,
                   "page_size": sp.page_size, "alpha": cfg_alpha(args),
                   "kept_target": float(args.target), "sink_blocks": sp.sink_blocks,
                   "window_blocks": sp.window_blocks, "mean_correction": sp.mean_correction},
        "kept_ratio": round(m["kept_ratio"], 5),
        "latency_ms": {"prefill": round(m["ms_per_step"], 4),
                       "estimate_kernels": round(m["estimate_ms"], 4),
                       "attention_kernel": round(m["attention_ms"], 4)},
        # the attention kernel: executed FLOPs (kept blocks and the
        # correction's pooled keys, both on the dtype's MFMA) over its own
        # duration (HIP events recorded by the library right around its
        # launch in every timed step), against the dtype's MFMA peak; frac_mix
        # against the time-weighted peak of the MFMA types issued (equal to
        # frac since the correction runs on the same type)
        "roofline": {"bound": "mfma", "kernel": "attend_kernel",
                     "achieved": round(att["achieved_tflops"], 2),
                     "peak": round(att["peak_tflops"], 1), "unit": "TFLOP/s",
                     "frac": round(att["frac"], 4),
                     "frac_mix": round(att["frac_mix"], 4),
                     "peak_mix": round(att["mix_peak_tflops"], 1),
                     "kernel_ms": round(m["attention_ms"], 4),
                     "executed_tflop": round(att["executed_tflop"], 4),
                     "traffic": None if traffic is None else round(traffic / 1e9, 3),
                     "traffic_unit": "GB per launch"},
        # the index stage (pooling + scoring + selection): its HBM fraction, and
        # the fractions of the resources that bind it at 128K (bf16 MFMA for
        # the scores, one exponential per (query row, pooled key))
        "estimation": {"ms": round(m["estimate_ms"], 4),
                       "hbm_gbs": round(m["estimation"]["gbs"], 1),
                       "hbm_frac": round(m["estimation"]["hbm_frac"], 4),
                       "scoring_mfma_frac": round(m["estimation"]["mfma_frac"], 4),
                       "exps_per_s": float("%.4g" % m["estimation"]["exps_per_s"]),
                       # counter-measured bytes of the pool + estimate kernels per call
                       # (committed rocprofv3 summary) and the rate they imply
                       "traffic": None if etraffic is None else round(etraffic / 1e9, 4),
                       "traffic_unit": "GB per call",
                       "measured_gbs": None if etraffic is None
                       else round(etraffic / 1e9 / (m["estimate_ms"] / 1e3), 1)},
        # reference rates measured in this run (device copy, library GEMMs)
        "measured_peaks": peaks,
        "cpu_baseline": None if cpu is None else {k: (round(v, 6) if isinstance(v, float) else v)
                                                  for k, v in cpu.items() if k != "seconds"},
    }
    if configs:
        line["configs"] = configs
    if variants:
        line["variants"] = variants
        line["mask_to_csr_ms"] = round(csr_ms, 4)
    if chunk_res:
        line["chunked_prefill"] = chunk_res
    print(json.dumps(line), flush=True)


def cfg_alpha(args):
    import synth
    return synth.alpha_for(args.workload, args.target)


if __name__ == "__main__":
    main()
