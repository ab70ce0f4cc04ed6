"""Benchmark: checkpointed LoRA training steps (MeBP, Algorithm 1) on one MI355X.

One step = embedding, forward over every layer storing the layer-boundary checkpoints,
final RMSNorm + tied int4 LM head + cross-entropy and its gradient, then every layer in
reverse: recompute from its checkpoint, backpropagate into the LoRA A/B gradients and the
layer-input gradient. Inputs are synthetic, seeded, resident in device memory before the
timed region. Prints one JSON line.

The default workload is the largest single-GPU shape: Gemma3-4B-shaped (34 layers, hidden
2560, 8 x 256 heads / 4 KV, GeGLU 10240, vocab 262144, batch 8 x 2048 tokens, LoRA r16 on
all seven projections). The Qwen2.5-0.5B-shaped step is measured too and reported as an
extra field.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# MI355X published dense peaks
PEAK_TFLOPS_16BIT = 2516.6  # fp16 / bf16 dense MFMA, TFLOP/s
PEAK_HBM_GBS = 8000.0


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def algorithmic_flops(cfg):
    """Work the method must do per step (see the design notes): base GEMMs
    fwd + recompute + input-gradient = 6 N P L; LM head logits + gradient = 4 N d V;
    attention 16 dh per visible (query, key) pair per query head; LoRA 8 N r (in + out)."""
    from mebp_inputs import PROJ
    N, L = cfg.n_tokens, cfg.n_layers
    P = sum(o * i for o, i in (cfg.proj_shape(p) for p in PROJ))
    base = 6.0 * N * P * L
    head = 4.0 * N * cfg.hidden * cfg.vocab
    attn = 0.0
    for l in range(L):
        W = cfg.layer_window(l)
        pairs = sum(min(t + 1, W) if W else t + 1 for t in range(cfg.seq))
        attn += 16.0 * cfg.head_dim * pairs * cfg.n_heads * cfg.batch
    lora = sum(8.0 * N * cfg.lora_rank * sum(cfg.proj_shape(p)) for p in cfg.lora_modules) * L
    return base + head + attn + lora


def kernel_source_digest():
    """Digest of the HIP sources, so HBM counters taken from an older build are not reused."""
    import hashlib
    h = hashlib.sha256()
    src = os.path.join(ROOT, "paper_2510_03425_amd", "csrc")
    for name in sorted(os.listdir(src)):
        with open(os.path.join(src, name), "rb") as f:
            h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE
    summary of this workload, or None when there is none or the sources changed since."""
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_{workload}.txt")
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            if line.startswith("digest ") or line.startswith("traffic "):
                key, _, rest = line.partition(" ")
                fields.setdefault(key, []).append(rest.split())
    if [kernel_source_digest()] not in fields.get("digest", []):
        return None
    for row in fields.get("traffic", []):
        if row[0] == kernel:
            return float(row[1])
    return None


# Timing-report names -> the HIP kernels they launch (demangled-name patterns), for reading
# rocprofv3 output of the same run.
KERNEL_PATTERNS = {
    "gemm_nt_f16out": r"k_gemm_nt(_big|_lds)?<(\d+, \d+, )?0(, (true|false))?(, \d+)?(, (true|false))?>",
    "gemm_nt_f32out": r"k_gemm_nt(_big|_lds)?<(\d+, \d+, )?1(, (true|false))?(, \d+)?(, (true|false))?>",
    "gemm_nt_logits": r"k_gemm_nt(_big|_lds)?<(\d+, \d+, )?2(, (true|false))?(, \d+)?(, (true|false))?>",
    "gemm_tn_f32out": r"k_gemm_tn(_big|_lds)?<(\d+, )?0(, (true|false))?>",
    "gemm_tn_act_bwd": r"k_gemm_tn(_big|_lds)?<(\d+, )?1(, (true|false))?>",
    "gemm_tn_probs_dh": r"k_gemm_tn(_big|_lds)?<(\d+, )?2(, (true|false))?>",
    "gemm_tn_bf16out": r"k_gemm_tn(_big|_lds)?<(\d+, )?3(, (true|false))?>",
    "lora_rows": r"k_lora_rows<",
    "lora_outer": r"k_lora_outer<",
    "attn_fwd": r"k_attn_fwd",
    "attn_bwd_dkdv": r"k_attn_bwd_(dkdv|kv32p?)<",
    "attn_bwd_dq": r"k_attn_bwd_dq<",
}


def _kname(raw):
    n = raw.replace("(anonymous namespace)::", "").replace("void ", "").replace("mebp::", "")
    return n.split("(")[0]


def rocprof_summary(trace_dir, top=32):
    """Per-kernel count / average / total of a rocprofv3 --kernel-trace CSV (text table)."""
    import csv
    import glob
    import re
    path = glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True)[0]
    agg = {}
    for r in csv.DictReader(open(path)):
        n = _kname(r["Kernel_Name"])
        d = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        a = agg.setdefault(n, [0, 0.0])
        a[0] += 1
        a[1] += d
    tot = sum(a[1] for a in agg.values())
    out = [f"{'kernel':52s} {'calls':>7s} {'avg_us':>9s} {'total_ms':>10s} {'pct':>6s}"]
    for n, (c, t) in sorted(agg.items(), key=lambda kv: -kv[1][1])[:top]:
        out.append(f"{n[:52]:52s} {c:7d} {t / c:9.2f} {t / 1e3:10.3f} {100 * t / tot:6.2f}")
    out.append(f"{'(all kernels)':52s} {sum(a[0] for a in agg.values()):7d} {'':9s} {tot / 1e3:10.3f}")
    grouped = ["", "grouped by timing-report name (avg over every launch of the matching kernels):"]
    for logical, pat in KERNEL_PATTERNS.items():
        hits = [(c, t) for n, (c, t) in agg.items() if re.search(pat, n) and "reduce" not in n]
        if hits:
            c, t = sum(h[0] for h in hits), sum(h[1] for h in hits)
            grouped.append(f"  {logical:22s} {c:7d} launches  avg {t / c:9.2f} us")
    return "\n".join(out + grouped)


def pmc_per_dispatch(pmc_dir, counter):
    """{kernel name: [value per dispatch]} of one counter from a rocprofv3 --pmc CSV."""
    import csv
    import glob
    path = glob.glob(os.path.join(pmc_dir, "**", "*counter_collection.csv"), recursive=True)[0]
    per = {}
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter:
            continue
        key = (r["Dispatch_Id"], _kname(r["Kernel_Name"]))
        per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
    out = {}
    for (_, n), v in per.items():
        out.setdefault(n, []).append(v)
    return out


def pmc_command_lines(workload):
    """Header lines naming the rocprofv3 counter passes the summaries are made from."""
    a = "--steps 2 --warmup 1 --profile-steps 1" if workload == "qwen2.5-0.5b" else "--steps 1 --warmup 0 --profile-steps 0"
    run = f"python3 -u bench.py --workload {workload} {a} --graph 0 --no-cpu-baseline --extra-workload ''"
    return [f"# command: cd /tmp && export TMPDIR=/tmp && cd /root/repo && rocprofv3 --pmc <counters> --output-format csv "
            f"-d gpurun_out/cnt_{workload}/<pass> -o run -- {run}",
            "# passes: fetch = FETCH_SIZE; write = WRITE_SIZE; sq = SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE "
            "SQ_INSTS_VALU SQ_INSTS_MFMA (counter table only)",
            "# calibration: the FETCH_SIZE and WRITE_SIZE passes around python3 -u bench.py --calibrate-copy 1024 "
            "(-d gpurun_out/pmc_cal_fetch, gpurun_out/pmc_cal_write)",
            f"# summary: python bench.py --workload {workload} --calibrate-copy 1024 --traffic-summary | --counter-summary "
            "<the pass folders>"]


def traffic_summary(args, fetch_dir, write_dir, cal_fetch_dir, cal_write_dir):
    """Scale FETCH_SIZE / WRITE_SIZE (KiB per dispatch) by what the same counters read for a
    plain device copy of known size, and write per-kernel HBM bytes per launch."""
    import re
    cal_n = args.calibrate_copy << 20 if args.calibrate_copy else 1 << 30
    cf = pmc_per_dispatch(cal_fetch_dir, "FETCH_SIZE")
    cw = pmc_per_dispatch(cal_write_dir, "WRITE_SIZE")
    ck = [n for n in cf if "copy" in n.lower() or "elementwise" in n.lower()]
    big = lambda d: max((v for n in d for v in d[n] if n in ck or not ck), default=0.0)
    f_cal, w_cal = big(cf) * 1024.0, big(cw) * 1024.0  # KiB -> bytes, largest dispatch = the copy
    kf, kw = cal_n / f_cal, cal_n / w_cal
    fe = pmc_per_dispatch(fetch_dir, "FETCH_SIZE")
    wr = pmc_per_dispatch(write_dir, "WRITE_SIZE")
    lines = [f"# HBM traffic per launch (rocprofv3 FETCH_SIZE, WRITE_SIZE), workload {args.workload}",
             *pmc_command_lines(args.workload),
             f"# copy calibration: {cal_n} B read counted as {f_cal:.0f} B (x{kf:.4f}), "
             f"{cal_n} B written counted as {w_cal:.0f} B (x{kw:.4f})",
             "# traffic <timing-report name> <bytes per launch> <fetch> <write> <dispatches>",
             f"digest {kernel_source_digest()}"]
    for logical, pat in KERNEL_PATTERNS.items():
        f = [v for n, vs in fe.items() if re.search(pat, n) and "reduce" not in n for v in vs]
        w = [v for n, vs in wr.items() if re.search(pat, n) and "reduce" not in n for v in vs]
        if not f or not w:
            continue
        fb, wb = sum(f) / len(f) * 1024.0 * kf, sum(w) / len(w) * 1024.0 * kw
        lines.append(f"traffic {logical} {fb + wb:.0f} {fb:.0f} {wb:.0f} {len(f)}")
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_{args.workload}.txt")
    with open(path, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def counter_summary(args, fetch_dir, write_dir, sq_dir, cal_fetch_dir, cal_write_dir):
    """Per-kernel table from rocprofv3 --pmc runs of the same command: serialized duration (the
    counter runs' own timestamps), HBM bytes per launch (FETCH_SIZE + WRITE_SIZE scaled by a
    plain-copy calibration) and GB/s against the 8 TB/s peak, and MFMA busy cycles as a share
    of all SIMD cycles (SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x GRBM_GUI_ACTIVE / 8 XCDs))."""
    import csv
    import glob
    cal_n = args.calibrate_copy << 20 if args.calibrate_copy else 1 << 30
    cf, cw = pmc_per_dispatch(cal_fetch_dir, "FETCH_SIZE"), pmc_per_dispatch(cal_write_dir, "WRITE_SIZE")
    kf = cal_n / (max(max(v) for v in cf.values()) * 1024.0)
    kw = cal_n / (max(max(v) for v in cw.values()) * 1024.0)

    def per_dispatch(d, counters):
        path = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)[0]
        out = {}
        for r in csv.DictReader(open(path)):
            key = (r["Dispatch_Id"], _kname(r["Kernel_Name"]))
            rec = out.setdefault(key, {"dur": (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3})
            if r["Counter_Name"] in counters:
                rec[r["Counter_Name"]] = rec.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        return out
    fe = per_dispatch(fetch_dir, ["FETCH_SIZE"])
    wr = per_dispatch(write_dir, ["WRITE_SIZE"])
    sq = per_dispatch(sq_dir, ["SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE", "SQ_INSTS_VALU", "SQ_INSTS_MFMA"])
    agg = {}
    for (d, n), rec in fe.items():
        a = agg.setdefault(n, {"n": 0, "dur": 0.0, "f": 0.0, "w": 0.0, "mb": 0.0, "gr": 0.0, "valu": 0.0, "mfma": 0.0,
                               "nsq": 0})
        a["n"] += 1
        a["dur"] += rec["dur"]
        a["f"] += rec.get("FETCH_SIZE", 0.0) * 1024.0 * kf
    for (d, n), rec in wr.items():
        if n in agg:
            agg[n]["w"] += rec.get("WRITE_SIZE", 0.0) * 1024.0 * kw
    for (d, n), rec in sq.items():
        if n in agg:
            a = agg[n]
            a["mb"] += rec.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
            a["gr"] += rec.get("GRBM_GUI_ACTIVE", 0.0)
            a["valu"] += rec.get("SQ_INSTS_VALU", 0.0)
            a["mfma"] += rec.get("SQ_INSTS_MFMA", 0.0)
            a["nsq"] += 1
    lines = [f"# per-kernel counters, workload {args.workload} (rocprofv3 --pmc, kernels serialized by the counter runs)",
             *pmc_command_lines(args.workload),
             f"# copy calibration: reads x{kf:.4f}, writes x{kw:.4f} (a plain {cal_n} B device copy)",
             f"# HBM GB/s = (fetch + write bytes) / serialized duration, against {PEAK_HBM_GBS:.0f} GB/s; MFMA busy = "
             "SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x GRBM_GUI_ACTIVE / 8 XCDs)",
             f"{'kernel':48s} {'calls':>6s} {'avg_us':>9s} {'MB/launch':>10s} {'GB/s':>8s} {'%HBM':>6s} {'%MFMA':>6s} "
             f"{'VALU/MFMA':>9s} {'total_ms':>9s}"]
    tot = sum(a["dur"] for a in agg.values())
    for n, a in sorted(agg.items(), key=lambda kv: -kv[1]["dur"]):
        if a["dur"] < 0.002 * tot:
            continue
        dur = a["dur"] / a["n"]
        mbytes = (a["f"] + a["w"]) / a["n"] / 1e6
        gbs = mbytes * 1e6 / (dur * 1e-6) / 1e9
        mf = 100.0 * a["mb"] * 8.0 / (1024.0 * a["gr"]) if a["gr"] else 0.0
        vm = a["valu"] / a["mfma"] if a["mfma"] else float("nan")
        lines.append(f"{n[:48]:48s} {a['n']:6d} {dur:9.2f} {mbytes:10.2f} {gbs:8.1f} {100 * gbs / PEAK_HBM_GBS:6.1f} "
                     f"{mf:6.1f} {vm:9.2f} {a['dur'] / 1e3:9.2f}")
    lines.append(f"digest {kernel_source_digest()}")
    path = os.path.join(ROOT, "profiles", f"kernel_counters_{args.workload}.txt")
    with open(path, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def optimizer_bench(cfg, reps=20):
    """Time mebp_lora_adamw_step over every LoRA tensor of `cfg` (fresh device tensors of the
    adapter shapes; the update is elementwise, so the values do not matter). Returns the
    average duration of one update (all launches) and its HBM rate at 28 bytes per
    parameter (read p, g, m, v; write p, m, v)."""
    import torch
    from mebp_inputs import PROJ
    from paper_2510_03425_amd import _lib as L
    from paper_2510_03425_amd.device import make_config, stream_handle
    n = cfg.n_layers
    params, m, v = ((L.MebpLayerLoraState * n)() for _ in range(3))
    grads = (L.MebpLayerLoraGrad * n)()
    keep, count = [], 0
    for l in range(n):
        for i, p in enumerate(PROJ):
            if p not in cfg.lora_modules:
                continue
            o, k = cfg.proj_shape(p)
            for shape, fa, fg in (((cfg.lora_rank, k), "A", "dA"), ((o, cfg.lora_rank), "B", "dB")):
                ts = [torch.randn(shape, device="cuda") * 0.01 for _ in range(3)] + [torch.zeros(shape, device="cuda")]
                keep += ts
                getattr(params[l], fa)[i] = ts[0].data_ptr()
                getattr(grads[l], fg)[i] = ts[1].data_ptr()
                getattr(m[l], fa)[i] = ts[2].data_ptr()
                getattr(v[l], fa)[i] = ts[3].data_ptr()
                count += shape[0] * shape[1]
    ccfg = make_config(cfg)
    hp = L.MebpAdamwHparams(lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01, grad_scale=1.0, step=1)
    for t in range(3):
        hp.step = t + 1
        L.mebp_lora_adamw_step(ccfg, params, grads, m, v, hp, stream_handle())
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for t in range(reps):
        hp.step = t + 4
        L.mebp_lora_adamw_step(ccfg, params, grads, m, v, hp, stream_handle())
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) / reps * 1e3
    gbs = 28.0 * count / (us * 1e-6) / 1e9
    return {"shape": f"{cfg.name}-shaped adapters", "params": count, "us_per_update": round(us, 2),
            "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4)}


def experiments(cfg, seqs=(128, 256, 512, 1024, 2048, 4096)):
    """Counterparts of the paper's sequence-length table and decompression-share table.

    seq_sweep: the whole checkpointed step of `cfg`'s model at batch 1 and each sequence
    length (the same weights; ids are the first T of one seeded draw), HIP-graph replay.

    decompression_in_gemm: the cost of the decompression fused into the GEMMs (see
    decompression_overhead).

    decompression_as_separate_pass: the paper's runtime decompresses each block's weights
    before its graph runs. What such a separate pass would cost on this GPU is timed with
    the stand-alone decompression kernel (int4 -> bf16 into a scratch matrix, every
    projection of every layer), and set against the measured forward pass (every layer's
    mebp_layer_forward_ckpt) and backward pass (every layer's mebp_layer_recompute_backward)
    of the fused design at the workload's own batch and length.

    checkpoint_offload: step time and peak device memory with the checkpoints in pinned
    host memory (4-slot device ring) against device checkpoints."""
    import torch
    from mebp_inputs import PROJ, make_inputs
    from paper_2510_03425_amd import _lib as L
    from paper_2510_03425_amd.device import DeviceModel, stream_handle

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    out = {"workload": f"{cfg.name}-shaped", "seq_sweep": []}
    big = cfg.with_(batch=1, seq=max(seqs))
    t0 = time.time()
    inp = make_inputs(big, seed=0)
    log(f"inputs drawn in {time.time() - t0:.1f}s")
    for T in seqs:
        c = cfg.with_(batch=1, seq=T)
        inp.cfg, ids_all = c, inp.ids
        inp.ids = ids_all[:, :T].copy()
        dm = DeviceModel(inp, device="cuda:0")
        inp.ids = ids_all
        dm.train_step(None)
        torch.cuda.synchronize()
        s_cap = torch.cuda.Stream()
        s_cap.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s_cap):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=s_cap):
                dm.train_step(None)
        torch.cuda.current_stream().wait_stream(s_cap)
        ms = timed(g.replay, 10 if T <= 1024 else 4)
        out["seq_sweep"].append({"batch": 1, "seq_len": T, "ms_per_step": round(ms, 3), "tokens_per_s": round(T / ms * 1e3, 1)})
        log(f"seq {T}: {ms:.3f} ms/step, {T / ms * 1e3:.0f} tokens/s")
        del g, dm
        torch.cuda.synchronize()
    inp.cfg = big

    # Table 2 analog: the fused decompression's cost inside the GEMMs
    out["decompression_in_gemm"] = decompression_overhead(cfg)

    # decompression as a separate pass, at the workload's own shape
    inp2 = make_inputs(cfg, seed=0)
    dm = DeviceModel(inp2, device="cuda:0")
    Lyr = cfg.n_layers
    biggest = max(o * i for o, i in (cfg.proj_shape(p) for p in PROJ))
    scratch = torch.empty(biggest, dtype=torch.int16, device="cuda:0")

    def decompress_all():
        for l in range(Lyr):
            for i, p in enumerate(PROJ):
                o, k = cfg.proj_shape(p)
                L.mebp_dequant_q4(dm.base[l].w[i], o, k, cfg.group, 0, scratch.data_ptr(), stream_handle())

    ck = dm.alloc_ckpt()
    dm.embed(ck[0])

    def forward_all():
        for l in range(Lyr):
            dm.layer_forward(l, ck[l], ck[l + 1])

    dy = torch.randn_like(ck[0])
    dxb = torch.empty_like(dy)

    def backward_all():
        for l in reversed(range(Lyr)):
            dm.layer_backward(l, ck[l], dy, dxb)

    t_dec = timed(decompress_all, 5)
    t_fwd = timed(forward_all, 3)
    t_bwd = timed(backward_all, 3)
    wbytes = sum(o * i for o, i in (cfg.proj_shape(p) for p in PROJ)) * Lyr
    out["decompression_as_separate_pass"] = {
        "batch": cfg.batch, "seq_len": cfg.seq, "weights": wbytes,
        "separate_pass_ms": round(t_dec, 3), "separate_pass_GBps": round(wbytes * (0.5625 + 2) / (t_dec * 1e-3) / 1e9, 1),
        "forward_ms": round(t_fwd, 3), "backward_ms": round(t_bwd, 3),
        "share_of_forward_if_separate": round(t_dec / (t_fwd + t_dec), 4),
        "share_of_backward_if_separate": round(t_dec / (t_bwd + t_dec), 4)}
    log(f"decompression pass {t_dec:.3f} ms; forward {t_fwd:.3f} ms; backward {t_bwd:.3f} ms")
    del scratch, ck, dy, dxb

    # checkpoints in pinned host memory through a 4-slot device ring, against the step with
    # every checkpoint in device memory (both replayed as HIP graphs); the device memory each
    # configuration holds is measured on a model of its own (torch's allocator peak: every
    # device buffer comes from it)
    N, d, slots = cfg.n_tokens, cfg.hidden, 4

    def graph_of(fn):
        fn()
        torch.cuda.synchronize()
        s_cap = torch.cuda.Stream()
        s_cap.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s_cap):
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr, stream=s_cap):
                fn()
        torch.cuda.current_stream().wait_stream(s_cap)
        return gr

    def fresh_peak():
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        torch.cuda.reset_peak_memory_stats()

    del dm
    fresh_peak()
    dm = DeviceModel(inp2, device="cuda:0")
    g_dev = graph_of(lambda: dm.train_step(None))
    t_dev = timed(g_dev.replay, 5)
    peak_dev = torch.cuda.max_memory_allocated()
    ws_bytes = dm.ws_bytes
    weights = sum(t.numel() * t.element_size() for t in dm.keep)
    del g_dev, dm
    fresh_peak()
    dm = DeviceModel(inp2, device="cuda:0")
    host = torch.empty((Lyr + 1, N, d), dtype=torch.float32).pin_memory()
    ring = torch.empty((slots, N, d), dtype=torch.float32, device="cuda:0")
    g_off = graph_of(lambda: dm.train_step_offload(host, ring, None))
    t_off = timed(g_off.replay, 5)
    peak_off = torch.cuda.max_memory_allocated()
    out["checkpoint_offload"] = {
        "ring_slots": slots, "ms_per_step_device_ckpt": round(t_dev, 3), "ms_per_step_offload": round(t_off, 3),
        "peak_device_bytes_device_ckpt": int(peak_dev), "peak_device_bytes_offload": int(peak_off),
        "device_ckpt_bytes": (Lyr + 1) * N * d * 4, "device_ring_bytes": slots * N * d * 4,
        "host_ckpt_bytes": (Lyr + 1) * N * d * 4, "weights_lora_norm_bytes": weights, "workspace_bytes": ws_bytes}
    log(f"offload: {t_off:.3f} ms/step vs {t_dev:.3f} ms/step with device checkpoints; peak device memory "
        f"{peak_off / 2**30:.2f} GiB vs {peak_dev / 2**30:.2f} GiB")
    del g_off, dm, ring, host
    print(json.dumps(out), flush=True)


def decompression_overhead(cfg, reps=5):
    """Counterpart of the paper's decompression-share table for this design, on the
    workload's projection shapes (M = B*T tokens). Forward products: the decompression is
    fused into the GEMM; the production kernel runs once on the int4 weights and once on
    the same weights already decompressed to fp16 (the same kernel with the decompression
    taken out; mebp_test_gemm kinds NT_LDS / NT_LDS_W16). Input-gradient products: the
    training path decompresses the weights into a transient bf16 copy right before the
    large-tile kernel reads them, so int4 = that pass (mebp_dequant_q4 to bf16) plus the
    kernel on the copy (TN_BIG_W16) and 16-bit = the kernel alone; the int4-fused variant
    of the same kernel (TN_BIG) is reported beside them. Per step every projection runs
    twice forward (forward pass and recompute) and once backward, in each of the L layers.
    overhead = t_int4 / t_16bit - 1 (negative: the int4 path is faster, its weight operand
    being a quarter of the bytes)."""
    import numpy as np
    import torch
    from mebp_inputs import PROJ, quantize_q4
    from paper_2510_03425_amd import _lib as L
    from paper_2510_03425_amd.device import stream_handle

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    M, st = cfg.n_tokens, stream_handle()
    rows, tot = {}, {"fwd_int4": 0.0, "fwd_16": 0.0, "bwd_int4": 0.0, "bwd_16": 0.0, "bwd_int4_fused": 0.0}
    for p in PROJ:
        n_out, n_in = cfg.proj_shape(p)
        rng = np.random.default_rng(0)
        q4, sb = quantize_q4((rng.standard_normal((n_out, n_in), dtype=np.float32) * 0.02))
        tq, ts = torch.from_numpy(q4).cuda(), torch.from_numpy(sb.view(np.int16)).cuda()
        wq = L.MebpQ4(q4=tq.data_ptr(), scale=ts.data_ptr())
        wf = torch.empty((n_out, n_in), dtype=torch.float32, device="cuda")
        L.mebp_dequant_q4(wq, n_out, n_in, cfg.group, wf.data_ptr(), 0, st)
        w_h, w_b = wf.half().contiguous(), wf.bfloat16().contiguous()
        x = (torch.randn(M, n_in, device="cuda") * 0.5).half()
        g = (torch.randn(M, n_out, device="cuda") * 0.01).bfloat16()
        out_f = torch.empty(M, n_out, device="cuda")
        out_b = torch.empty(M, n_in, device="cuda")
        w16 = L.MebpQ4(q4=w_h.data_ptr(), scale=0)
        b16 = L.MebpQ4(q4=w_b.data_ptr(), scale=0)
        w_t = torch.empty((n_out, n_in), dtype=torch.int16, device="cuda")  # the transient bf16 copy
        t16 = L.MebpQ4(q4=w_t.data_ptr(), scale=0)
        r = {"fwd_int4": timed(lambda: L.mebp_test_gemm(L.TEST_GEMM_NT_LDS, wq, n_out, n_in, x.data_ptr(), M,
                                                         out_f.data_ptr(), st)),
             "fwd_16": timed(lambda: L.mebp_test_gemm(L.TEST_GEMM_NT_LDS_W16, w16, n_out, n_in, x.data_ptr(), M,
                                                       out_f.data_ptr(), st)),
             "bwd_int4": timed(lambda: (L.mebp_dequant_q4(wq, n_out, n_in, cfg.group, 0, w_t.data_ptr(), st),
                                        L.mebp_test_gemm(L.TEST_GEMM_TN_BIG_W16, t16, n_out, n_in, g.data_ptr(), M,
                                                         out_b.data_ptr(), st))),
             "bwd_16": timed(lambda: L.mebp_test_gemm(L.TEST_GEMM_TN_BIG_W16, b16, n_out, n_in, g.data_ptr(), M,
                                                       out_b.data_ptr(), st)),
             "bwd_int4_fused": timed(lambda: L.mebp_test_gemm(L.TEST_GEMM_TN_BIG, wq, n_out, n_in, g.data_ptr(), M,
                                                               out_b.data_ptr(), st))}
        rows[p] = {k: round(v, 4) for k, v in r.items()}
        for k in tot:
            tot[k] += r[k] * cfg.n_layers * (2 if k.startswith("fwd") else 1)
        del tq, ts, wf, w_h, w_b, w_t, x, g, out_f, out_b
        torch.cuda.empty_cache()
    res = {"tokens": M, "per_projection_ms": rows,
           "forward_ms_per_step": {"int4": round(tot["fwd_int4"], 2), "16bit": round(tot["fwd_16"], 2)},
           "backward_ms_per_step": {"int4": round(tot["bwd_int4"], 2), "16bit": round(tot["bwd_16"], 2),
                                    "int4_fused_kernel": round(tot["bwd_int4_fused"], 2)},
           "overhead_forward": round(tot["fwd_int4"] / tot["fwd_16"] - 1, 4),
           "overhead_backward": round(tot["bwd_int4"] / tot["bwd_16"] - 1, 4)}
    log(f"decompression inside the GEMMs ({cfg.name}): forward {res['overhead_forward']:+.1%}, backward "
        f"{res['overhead_backward']:+.1%} (int4 against pre-decompressed 16-bit weights)")
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="gemma3-4b")
    ap.add_argument("--extra-workload", default="qwen2.5-0.5b",
                    help="a second workload timed after the first and reported as an extra field ('' for none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-steps", type=int, default=3, help="extra steps with per-kernel event timing")
    ap.add_argument("--graph", type=int, default=1, help="replay the step as one captured HIP graph (1) or launch eagerly (0)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB five times (HBM counter calibration)")
    ap.add_argument("--rocprof-summary", metavar="DIR", help="print a summary of a rocprofv3 kernel trace (no GPU)")
    ap.add_argument("--traffic-summary", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "CAL_FETCH_DIR", "CAL_WRITE_DIR"),
                    help="HBM bytes per launch from rocprofv3 FETCH_SIZE / WRITE_SIZE runs of this bench and of "
                         "--calibrate-copy (no GPU); writes profiles/hbm_traffic_<workload>.txt")
    ap.add_argument("--counter-summary", nargs=5,
                    metavar=("FETCH_DIR", "WRITE_DIR", "SQ_DIR", "CAL_FETCH_DIR", "CAL_WRITE_DIR"),
                    help="per-kernel HBM GB/s and MFMA busy share from rocprofv3 --pmc runs (no GPU); writes "
                         "profiles/kernel_counters_<workload>.txt")
    ap.add_argument("--arch", action="store_true",
                    help="the model family's architecture details on top of the shape: QKV bias (Qwen2.5), per-head "
                         "QK-norm, sandwich norms and embedding scale (Gemma3)")
    ap.add_argument("--experiments", action="store_true",
                    help="instead of the benchmark: step time against sequence length (B = 1, T = 128 .. 4096) and "
                         "the cost of decompressing every layer's weights as a separate pass, at --workload")
    args = ap.parse_args()
    if args.counter_summary:
        counter_summary(args, *args.counter_summary)
        return
    if args.rocprof_summary:
        print(rocprof_summary(args.rocprof_summary))
        return
    if args.traffic_summary:
        traffic_summary(args, *args.traffic_summary)
        return
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU (asked for --gpus {args.gpus}); the multi-GPU path is not "
              "part of this build", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n, "reads": n, "writes": n, "launches": 5}), flush=True)
        return

    from mebp_inputs import CONFIGS, make_inputs
    from paper_2510_03425_amd import _lib as L
    from paper_2510_03425_amd.device import DeviceModel

    cfg = CONFIGS[args.workload]
    if args.arch:
        fam = dict(qkv_bias=True) if cfg.name.startswith("qwen") else \
            dict(qk_norm=True, sandwich_norm=True, embed_scale=True)
        cfg = cfg.with_(name=cfg.name + "+arch", **fam)
    if args.experiments:
        experiments(cfg)
        return
    res = measure(cfg, args, profile=True)
    extra = None
    if args.extra_workload and args.extra_workload != cfg.name:
        ecfg = CONFIGS[args.extra_workload]
        e = measure(ecfg, argparse.Namespace(**{**vars(args), "steps": 20, "warmup": 3}), profile=False)
        extra = {"workload": f"{ecfg.name}-shaped full LoRA step", "global_batch": ecfg.batch, "seq_len": ecfg.seq,
                 "ms_per_step": e["ms"], "tokens_per_s": round(e["value"], 1), "step_mfma_frac": e["step_frac"],
                 "launch": e["launch"]}
    # the optimizer step that follows a training step (AdamW over every LoRA tensor), at this
    # workload's adapters and at the largest adapter set (Gemma3-4B shape, all 7 projections)
    optim = {"bound": "hbm", "workload": optimizer_bench(cfg), "largest": optimizer_bench(CONFIGS["gemma3-4b"])}
    log(f"adamw: {optim['workload']['us_per_update']} us per update of {optim['workload']['params']} params; "
        f"{optim['largest']['params']} params: {optim['largest']['us_per_update']} us, {optim['largest']['achieved']} GB/s")

    cpu = None if args.no_cpu_baseline else cpu_baseline(cfg, res["inp"], res["loss"])
    out = {
        "metric": "LoRA train tokens/s per checkpointed step",
        "value": round(res["value"], 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(res["ms"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16/bf16 MFMA, fp32 accumulate",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}-shaped full LoRA step", "layers": cfg.n_layers, "hidden": cfg.hidden,
                   "heads": f"{cfg.n_heads}x{cfg.head_dim}/{cfg.n_kv_heads}kv", "ffn": cfg.ffn, "vocab": cfg.vocab,
                   "global_batch": cfg.batch, "seq_len": cfg.seq, "lora": f"r{cfg.lora_rank} a{cfg.lora_alpha:g} "
                   + ",".join(cfg.lora_modules), "weights": "int4 group-32, fp16 scales", "parallelism": "none"},
        "step_mfma_frac": res["step_frac"],
        "launch": res["launch"],
        "loss": res["loss"],
        "roofline": res["roofline"],
        "cpu_baseline": cpu,
        "memory": res["memory"],
        "extra_workload": extra,
        "optimizer_adamw": optim,
    }
    print(json.dumps(out), flush=True)


def measure(cfg, args, profile=True):
    """Time `args.steps` whole steps of `cfg` (HIP-graph replay unless --graph 0) after
    `args.warmup` eager ones; with `profile`, also the per-kernel event pass, the in-stream
    duration of the leading kernels and the roofline of the dominant one, and the device
    memory the step holds."""
    import torch
    from mebp_inputs import make_inputs
    from paper_2510_03425_amd import _lib as L
    from paper_2510_03425_amd.device import DeviceModel

    t0 = time.time()
    inp = make_inputs(cfg, seed=0)
    log(f"inputs {cfg.name} drawn in {time.time() - t0:.1f}s")
    torch.cuda.synchronize()
    torch.cuda.reset_peak_memory_stats()
    dm = DeviceModel(inp, device="cuda:0")
    dx0 = None
    stream = torch.cuda.current_stream()

    for _ in range(args.warmup):
        dm.train_step(dx0)
    torch.cuda.synchronize()
    log("warmup done")

    def capture():
        # one whole step (every kernel of the library, no allocation, no host sync) captured
        # on a side stream; the eager steps before it already validated the inputs
        s_cap = torch.cuda.Stream()
        s_cap.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s_cap):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=s_cap):
                dm.train_step(dx0)
        torch.cuda.current_stream().wait_stream(s_cap)
        g.replay()
        torch.cuda.synchronize()
        return g

    run_step = lambda: dm.train_step(dx0)
    graph = None
    if args.graph:
        graph = capture()
        run_step = graph.replay
        log("captured the step as a HIP graph")

    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        run_step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms = ev0.elapsed_time(ev1) / args.steps
    tokens = cfg.n_tokens
    value = tokens / (ms / 1e3)
    log(f"{cfg.name}: {ms:.3f} ms/step, {value:.0f} tokens/s (wall {wall / args.steps * 1e3:.3f} ms/step)")
    loss = dm.loss.item()
    step_flops = algorithmic_flops(cfg)
    res = {"ms": ms, "value": value, "loss": loss, "inp": inp, "launch": "hip_graph" if graph is not None else "eager",
           "step_frac": round(step_flops / (ms / 1e3) / 1e12 / PEAK_TFLOPS_16BIT, 4), "roofline": None,
           "memory": None}
    if not profile:
        del graph, dm
        torch.cuda.synchronize()
        return res

    # device memory held by the step: every device buffer comes from torch's allocator (the
    # library allocates nothing), so its peak is the step's footprint
    ckpt_bytes = (cfg.n_layers + 1) * cfg.n_tokens * cfg.hidden * 4
    free, total = torch.cuda.mem_get_info()
    res["memory"] = {"peak_device_bytes": int(torch.cuda.max_memory_allocated()),
                     "workspace_bytes": int(dm.ws_bytes), "checkpoint_bytes": ckpt_bytes,
                     "weights_lora_grads_bytes": int(sum(t.numel() * t.element_size() for t in dm.keep)
                                                     + sum(t.numel() * 4 for d in dm.dA + dm.dB for t in d.values())),
                     "device_used_bytes": int(total - free), "device_total_bytes": int(total)}
    log(f"memory: peak allocated {res['memory']['peak_device_bytes'] / 2**30:.2f} GiB (workspace "
        f"{dm.ws_bytes / 2**30:.2f} GiB, checkpoints {ckpt_bytes / 2**30:.2f} GiB)")

    # profile pass: a few extra eager steps with HIP events around every launch, recorded on
    # the stream the library launches on (the step's stream)
    roof = None
    if args.profile_steps > 0:
        L.mebp_kernel_timing(True, 1 << 16)
        for _ in range(args.profile_steps):
            dm.train_step(dx0)
        torch.cuda.synchronize()
        rep = L.mebp_kernel_timing_report()
        L.mebp_kernel_timing(False)
        total_k = sum(r["ms"] for r in rep)
        rep.sort(key=lambda r: -r["ms"])
        for r in rep[:20]:
            log(f"  {r['kernel']:24s} {r['ms'] / args.profile_steps:8.3f} ms/step  {r['launches'] // args.profile_steps:4d}"
                f" launches  {r['flops'] / r['ms'] / 1e9 if r['ms'] else 0:8.1f} TFLOP/s"
                f"  {r['bytes'] / r['ms'] / 1e6 if r['ms'] else 0:8.1f} GB/s")
        gemm = [r for r in rep if r["kernel"].startswith("gemm_")]
        if gemm:
            gf, gms = sum(r["flops"] for r in gemm), sum(r["ms"] for r in gemm)
            log(f"  all dequant GEMMs: {gf / gms / 1e9:.1f} TFLOP/s = {gf / gms / 1e9 / PEAK_TFLOPS_16BIT:.3f} of peak,"
                f" {gms / total_k:.3f} of kernel time")
        # In-stream duration of the leading kernels: the same eager steps again with every
        # launch of one kernel issued BURST times back to back inside its event pair (on the
        # kernel's own stream). The extra time over the single-launch pass, divided by the
        # extra launches, is the kernel's back-to-back duration: the event and dispatch latency
        # that a pair around one launch also counts cancels out. The repeated kernels
        # recompute the same outputs; this is checked.
        BURST = 5
        ref_loss = dm.loss.clone()
        ref_grad = dm.grad_probe().clone()
        best = None
        for r in rep[:4]:
            name, per_step = r["kernel"], r["launches"] // args.profile_steps
            if L.lib().mebp_kernel_repeat(name.encode(), BURST) != 0:
                # kernels that update a buffer in place cannot be repeated; their single-launch
                # event time (an upper bound) stands
                dur_ms, how = r["ms"] / r["launches"], "single-launch events"
            else:
                try:
                    L.mebp_kernel_timing(True, 1 << 16)
                    for _ in range(args.profile_steps):
                        dm.train_step(dx0)
                    torch.cuda.synchronize()
                    rb = [x for x in L.mebp_kernel_timing_report() if x["kernel"] == name][0]
                finally:
                    L.mebp_kernel_timing(False)
                    L.mebp_kernel_repeat(None, 1)
                assert torch.equal(dm.loss, ref_loss) and torch.equal(dm.grad_probe(), ref_grad), \
                    f"repeating {name} changed the result"
                dur_ms = (rb["ms"] - r["ms"]) / (rb["launches"] - r["launches"])
                how = f"bursts of {BURST} minus single launches"
            log(f"  in-stream {name}: {dur_ms * 1e3:.2f} us per launch ({how}) x {per_step} launches/step"
                f" (single-launch events {r['ms'] / r['launches'] * 1e3:.2f} us)")
            if best is None or dur_ms * per_step > best[1] * best[2]:
                best = (r, dur_ms, per_step)
        dom, per_launch_ms, per_step = best
        traffic = measured_traffic(dom["kernel"], cfg.name)
        # the dense contractions (dequant GEMMs, attention) are priced against the MFMA peak;
        # the LoRA, norm and elementwise kernels are bound by HBM and priced by their bytes
        mfma_bound = dom["kernel"].startswith(("gemm_", "attn_fwd", "attn_bwd")) and dom["flops"] > 0
        if mfma_bound:
            ach = dom["flops"] / dom["launches"] / (per_launch_ms / 1e3) / 1e12
            roof = {"bound": "mfma", "achieved": round(ach, 2), "peak": PEAK_TFLOPS_16BIT, "unit": "TFLOP/s",
                    "frac": round(ach / PEAK_TFLOPS_16BIT, 4), "traffic": traffic}
        else:
            ach = dom["bytes"] / dom["launches"] / (per_launch_ms / 1e3) / 1e9
            roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                    "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": traffic}
        roof.update({"kernel": dom["kernel"], "launches_per_step": per_step,
                     "avg_launch_us": round(per_launch_ms * 1e3, 2),
                     "kernel_share_of_step": round(per_launch_ms * per_step / ms, 3)})
        if gemm:
            roof["all_gemms_frac"] = round(gf / gms / 1e9 / PEAK_TFLOPS_16BIT, 4)
    res["roofline"] = roof
    del graph, dm
    torch.cuda.synchronize()
    return res


def host_info():
    """CPU model, BLAS and thread count of the host the oracle runs on."""
    import numpy as np
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = "unknown"
    try:
        deps = np.show_config(mode="dicts")["Build Dependencies"]["blas"]
        blas = f"{deps.get('name')} {deps.get('version', '')}".strip()
    except Exception:
        pass
    threads = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_info
        info = threadpool_info()
        threads = max((i.get("num_threads", 1) for i in info), default=threads)
        blas = ", ".join(sorted({f"{i.get('internal_api')} {i.get('version')}" for i in info if i.get("user_api") == "blas"})) or blas
    except Exception:
        pass
    return {"cores": threads, "cpu": model, "blas": blas, "host_cpus": len(os.sched_getaffinity(0))}


def cpu_baseline(cfg, inp, gpu_loss):
    """The fp64 oracle timed on this host's cores, as a baseline (not a target).

    Whole steps for shapes the oracle finishes in seconds. For the large shapes one step
    would take hours, so a bounded sample is timed and extrapolated linearly: one layer
    (forward of the first loop, then recompute + backward of the second) on one whole
    sequence of the batch (every row, every column; the oracle's attention costs the same
    for local and global layers), scaled by layers x sequences, plus the LM head on a sample
    of rows (loss and gradient rows are independent of each other), scaled by rows."""
    import numpy as np
    import oracle as O
    hi = host_info()
    N, L = cfg.n_tokens, cfg.n_layers
    if algorithmic_flops(cfg) <= 1e12:  # whole steps take seconds
        n_steps, t0 = 0, time.perf_counter()
        while True:
            ref = O.train_step(cfg, inp, keep_ckpts=False)
            n_steps += 1
            dt = time.perf_counter() - t0
            if dt > 10.0 or n_steps >= 3:
                break
        log(f"oracle {n_steps} step(s) {dt:.1f}s on {hi['cores']} threads; loss gpu {gpu_loss:.6f} oracle {ref.loss:.6f}")
        return {"value": round(n_steps * N / dt, 3), "unit": "tokens/s", "kind": "oracle", **hi,
                "sample": f"{n_steps} full fp64 step(s) of the same workload ({N} tokens each) in {dt:.1f} s",
                "loss_oracle": ref.loss}
    one = cfg.with_(batch=1)
    T, d = cfg.seq, cfg.hidden
    E = O.decompress_embedding(cfg, inp)
    x = O.embed(E, inp.ids[:1], O.embed_scale(cfg))
    dy = np.random.default_rng(5).standard_normal(x.shape)
    t0 = time.perf_counter()
    P = O.decompress_layer(one, inp, 0)
    O.layer_forward(one, 0, P, x)
    O.layer_backward(one, 0, P, x, dy)
    t_layer = time.perf_counter() - t0
    rows = np.arange(min(128, T - 1))
    tgt = inp.ids[0, 1:][rows]
    t0 = time.perf_counter()
    O.lm_head_ce_rows(cfg, E, inp.norm_final, x[rows], tgt, cfg.batch * (T - 1))
    t_rows = time.perf_counter() - t0
    total = t_layer * L * cfg.batch + t_rows * N / len(rows)
    log(f"oracle sample: one layer on one sequence {t_layer:.1f}s, LM head on {len(rows)} rows {t_rows:.1f}s "
        f"-> {total:.0f}s per step extrapolated ({hi['cores']} threads)")
    return {"value": round(N / total, 4), "unit": "tokens/s", "kind": "oracle", **hi, "extrapolated": True,
            "sample": f"extrapolated: one layer (decompression, forward, recompute + backward) on one whole sequence "
                      f"of {T} tokens in {t_layer:.1f} s, x {L} layers x {cfg.batch} sequences; LM head on {len(rows)} "
                      f"rows in {t_rows:.1f} s, x {N} rows / {len(rows)}; {total:.0f} s per step"}


if __name__ == "__main__":
    main()
