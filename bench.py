"""Benchmark of the Hidden Decoding hot path on one MI355X.

One step = one pass of the whole hot path over one batch of synthetic input, the
36-layer stack at the Qwen3-8B-like shape (B=1, L=4096 tokens, n=4 streams, N=16384
expanded rows, Hq=32, Hkv=8, D=128, bf16):
  * the stream expansion of 4096 token ids through n=4 tables of 151936 x 4096,
  * the forward of 36 attention layers (mixing layers at 8, 17, 26, 35, intra-stream
    layers elsewhere),
  * the final-stream gather of the 4096 x 4096 hidden states that the loss reads,
    eq. (hd_loss), and its adjoint,
  * the backward of the 36 layers in reverse order,
  * the expansion's backward (sparse gradient of the n tables),
each layer on its own seeded q/k/v/dO, all resident in HBM before timing starts.

Prints one JSON line.  value = useful TFLOP/s of the whole step (useful flop counts
only visible query/key pairs: 4*D per pair forward, 10*D backward).  The roofline
entry is for the kernel with the largest share of the step (from one untimed step with
HIP events around every launch), timed with HIP events that the library records on the
launch stream around that kernel's launches in the timed steps.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "SFA fwd+bwd useful TFLOP/s and % of bf16 MFMA peak, n=4 L=4096 (1 GPU)"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="stack36",
                    choices=["stack36"] + [f"{w}-{m}" for w in ("qwen8b", "frontier")
                                           for m in ("intra", "mix", "local", "final",
                                                     "final-local")]
                    + [f"sweep-n{n}-{m}" for n in (1, 2, 4, 8) for m in ("intra", "mix", "local")]
                    + ["decode-stack36", "decode-intra", "decode-mix", "decode-local"])
    ap.add_argument("--window", type=int, default=None,
                    help="window of local layers in expanded positions "
                         "(default: the workloads' 4096)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-tokens", type=int, default=768)
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES (3 times) and exit; "
                         "used to scale HBM traffic counters")
    return ap.parse_args()


def copy_calibration(nbytes):
    import torch

    src = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": nbytes, "launches": 3}))


def per_kernel_flops(shape, mode, window, final=False):
    """Algorithmic flop per kernel family for one layer (useful pairs only)."""
    from paper_2607_08186_amd import workloads as W

    if final:
        pairs = W.visible_pairs_final(shape, window if mode == W.LOCAL else 0)
    else:
        pairs = W.visible_pairs(shape, mode, window)
    D = shape.D
    # forward: S = QK^T and O = PV; dK/dV pass: S, dP, dV, dK; dQ pass: dQ only
    # (it recomputes S and dP, which the useful count does not credit twice)
    return {"fwd": 4 * D * pairs, "dkdv": 8 * D * pairs, "dq": 2 * D * pairs}


def kernel_family(name):
    if name.startswith("embed_bwd"):
        return "expand_bwd"
    for fam in ("fwd", "dkdv", "dq", "preprocess", "expand"):
        if fam in name:
            return fam
    return name


def time_steps(hd, torch, step, steps):
    """Run one untimed step with every library launch bracketed by HIP events (the
    per-kernel breakdown), then `steps` timed steps in which only the launches of the
    dominant kernel of that breakdown carry events (recorded on their launch stream),
    so the timed region holds no other event.  -> (elapsed s of the timed steps,
    breakdown [(name, launches, total ms)] of the one step, (name, launches, total ms)
    of the dominant kernel over the timed steps)."""
    torch.cuda.synchronize()
    hd.hd_timing_filter(None)
    hd.hd_timing_enable(True)
    hd.hd_timing_collect()  # drop anything recorded before
    step()
    torch.cuda.synchronize()
    hd.hd_timing_enable(False)
    breakdown = hd.hd_timing_collect()
    dom_name = max(breakdown, key=lambda r: r[2])[0]
    hd.hd_timing_filter(dom_name)
    hd.hd_timing_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        step()
        print(f"[bench] step {i + 1}/{steps} enqueued", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    hd.hd_timing_enable(False)
    hd.hd_timing_filter(None)
    dom = [r for r in hd.hd_timing_collect() if r[0] == dom_name]
    if len(dom) != 1:
        raise RuntimeError(f"no timing events for {dom_name} over the timed steps")
    return elapsed, breakdown, dom[0]


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(every run here uses a single MI355X); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.workload.startswith("decode"):
        run_decode(args)
        return

    import torch

    import paper_2607_08186_amd as hd
    from paper_2607_08186_amd import synth
    from paper_2607_08186_amd import workloads as W

    if not os.path.exists(hd.binding.LIB_PATH):
        from paper_2607_08186_amd import build as hip_build

        hip_build.build()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()

    # ---------------------------------------------------------------- workload
    window = args.window if args.window is not None else W.LOCAL_WINDOW
    if window < 1:
        raise SystemExit("--window must be >= 1")
    if args.workload == "stack36":
        shape = W.QWEN8B.shape
        modes = W.stack_modes()
        with_embed = True
        wl_desc = (f"stack36: expand_embed (n=4 tables of {W.STACK_VOCAB}x{W.STACK_DMODEL}) + "
                   f"fwd of 36 layers (mix at {list(W.STACK_MIX_LAYERS)}, intra elsewhere) + "
                   "final-stream gather of the hidden states and its adjoint + "
                   "bwd in reverse, each layer B=1 L=4096 n=4 Hq=32 Hkv=8 D=128, + "
                   "expand_embed backward")
        std = W.QWEN8B.qkv_std
        spike = None
        final = False
    else:
        final = "final" in args.workload
        parts = args.workload.replace("final-local", "local").replace("final", "mix").split("-")
        m = {"intra": W.INTRA, "mix": W.MIX, "local": W.LOCAL}[parts[-1]]
        if parts[0] == "qwen8b":
            wl = W.QWEN8B
        elif parts[0] == "frontier":
            wl = W.FRONTIER
        else:
            wl = {w.shape.n: w for w in W.SWEEP}[int(parts[1][1:])]
        shape, modes, with_embed = wl.shape, [m], False
        wl_desc = f"{wl.name} {W.MODE_NAMES[m]} fwd+bwd"
        if final:
            wl_desc = (f"{wl.name} final-stream {W.MODE_NAMES[m]} layer fwd+bwd (queries at "
                       "the final stream of each token, keys over all n streams)")
        if m == W.LOCAL:
            wl_desc += f" (window {window} expanded positions)"
        std, spike = wl.qkv_std, wl.k_spike
    s = shape
    nl = len(modes)
    scale = s.scale

    # ------------------------------------------------- resident synthetic inputs
    t_gen = time.time()
    layers = []
    for li in range(nl):
        seed = synth.seed_for("bench", args.workload, li)
        qrows = s.L if final else s.N  # final-stream layers: one query row per token
        q = synth.device_normal((s.B, qrows, s.Hq, s.D), std, seed + 1, dev, torch.bfloat16)
        k = synth.device_normal((s.B, s.N, s.Hkv, s.D), std, seed + 2, dev, torch.bfloat16)
        v = synth.device_normal((s.B, s.N, s.Hkv, s.D), std, seed + 3, dev, torch.bfloat16)
        do = synth.device_normal((s.B, qrows, s.Hq, s.D), W.QWEN8B.dout_std, seed + 4, dev,
                                 torch.bfloat16)
        if spike is not None:  # scale a seeded 1% of K rows by 8 (exact in bf16)
            flat = k.view(-1, s.D)
            g = torch.Generator(device=dev)
            g.manual_seed(seed + 5)
            pick = torch.randperm(flat.shape[0], generator=g, device=dev)[
                :int(spike[0] * flat.shape[0])]
            flat[pick] *= spike[1]
        o = torch.empty_like(q)
        lse = torch.empty((s.B, s.Hq, qrows), dtype=torch.float32, device=dev)
        layers.append(dict(q=q, k=k, v=v, do=do, o=o, lse=lse, mode=modes[li]))
    dq = torch.empty_like(layers[0]["q"])
    dk = torch.empty_like(layers[0]["k"])
    dv = torch.empty_like(layers[0]["v"])
    if final:
        ws_bytes = hd.hd_sfa_bwd_final_workspace_bytes(s.B, s.L, s.n, s.Hq, s.Hkv, s.D,
                                                       window if W.LOCAL in modes else 0,
                                                       hd.HD_DTYPE_BF16)
    else:
        ws_bytes = max(hd.hd_sfa_bwd_workspace_bytes(s.B, s.L, s.n, s.Hq, s.Hkv, s.D, m,
                                                     hd.HD_DTYPE_BF16) for m in set(modes))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    if with_embed:
        ids = torch.randint(0, W.STACK_VOCAB, (1, s.L), dtype=torch.int32, device=dev,
                            generator=torch.Generator(device=dev).manual_seed(11))
        tables = synth.device_normal((s.n, W.STACK_VOCAB, W.STACK_DMODEL), W.STACK_EMBED_STD,
                                     12, dev, torch.bfloat16)
        emb = torch.empty((1, s.N, W.STACK_DMODEL), dtype=torch.bfloat16, device=dev)
        # the expansion's backward: upstream gradient of the expanded rows -> sparse
        # table gradient (distinct ids, rows)
        demb = synth.device_normal((1, s.N, W.STACK_DMODEL), 1.0, 13, dev, torch.bfloat16)
        uniq = torch.empty(s.L, dtype=torch.int32, device=dev)
        drows = torch.empty((s.n, s.L, W.STACK_DMODEL), dtype=torch.float32, device=dev)
        nuniq = torch.empty(1, dtype=torch.int32, device=dev)
        ews_bytes = hd.hd_expand_embed_bwd_workspace_bytes(1, s.L)
        ews = torch.empty(ews_bytes, dtype=torch.uint8, device=dev)
        # the loss input: final-stream rows of the top hidden states (the expansion's
        # output stands in for them: same [1][N][Dm] layout), and the adjoint of an
        # upstream gradient of those rows
        hfin = torch.empty((1, s.L, W.STACK_DMODEL), dtype=torch.bfloat16, device=dev)
        dfin = synth.device_normal((1, s.L, W.STACK_DMODEL), 1.0, 14, dev, torch.bfloat16)
        dh = torch.empty((1, s.N, W.STACK_DMODEL), dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()
    t_gen = time.time() - t_gen

    def step():
        if with_embed:
            hd.hd_expand_embed(ids, tables, emb, 1, s.L, s.n, W.STACK_VOCAB, W.STACK_DMODEL,
                               stream=stream)
        for ly in layers:
            if final:
                hd.hd_sfa_fwd_final(ly["q"], ly["k"], ly["v"], ly["o"], ly["lse"], s.B, s.L, s.n,
                                    s.Hq, s.Hkv, s.D, window if ly["mode"] == W.LOCAL else 0,
                                    scale, stream=stream)
            elif ly["mode"] == W.LOCAL:
                hd.hd_sfa_fwd_local(ly["q"], ly["k"], ly["v"], ly["o"], ly["lse"], s.B, s.L,
                                    s.n, s.Hq, s.Hkv, s.D, window, scale, stream=stream)
            else:
                hd.hd_sfa_fwd(ly["q"], ly["k"], ly["v"], ly["o"], ly["lse"], s.B, s.L, s.n,
                              s.Hq, s.Hkv, s.D, ly["mode"], scale, stream=stream)
        if with_embed:
            hd.hd_final_stream_gather(emb, hfin, 1, s.L, s.n, W.STACK_DMODEL, stream=stream)
            hd.hd_final_stream_gather_bwd(dfin, dh, 1, s.L, s.n, W.STACK_DMODEL, stream=stream)
        for ly in reversed(layers):
            if final:
                hd.hd_sfa_bwd_final(ly["q"], ly["k"], ly["v"], ly["o"], ly["lse"], ly["do"], dq,
                                    dk, dv, s.B, s.L, s.n, s.Hq, s.Hkv, s.D,
                                    window if ly["mode"] == W.LOCAL else 0, scale, ws, ws_bytes,
                                    stream=stream)
            elif ly["mode"] == W.LOCAL:
                hd.hd_sfa_bwd_local(ly["q"], ly["k"], ly["v"], ly["o"], ly["lse"], ly["do"], dq,
                                    dk, dv, s.B, s.L, s.n, s.Hq, s.Hkv, s.D, window, scale, ws,
                                    ws_bytes, stream=stream)
            else:
                hd.hd_sfa_bwd(ly["q"], ly["k"], ly["v"], ly["o"], ly["lse"], ly["do"], dq, dk,
                              dv, s.B, s.L, s.n, s.Hq, s.Hkv, s.D, ly["mode"], scale, ws,
                              ws_bytes, stream=stream)
        if with_embed:
            hd.hd_expand_embed_bwd(ids, demb, 1, s.L, s.n, W.STACK_VOCAB, W.STACK_DMODEL, uniq,
                                   drows, nuniq, ews, ews_bytes, stream=stream)

    for _ in range(args.warmup):
        step()
    elapsed, ktimes, dom = time_steps(hd, torch, step, args.steps)
    per_mode = copy_ceiling = None
    if args.workload == "stack36":
        per_mode = time_layer_modes(hd, torch, layers, s, scale, dq, dk, dv, ws, ws_bytes,
                                    stream, W)
        copy_ceiling = time_expand_vs_copy(hd, torch, ids, tables, emb, s, W, stream)

    if final:
        flop_step = sum(14 * s.D * W.visible_pairs_final(s, window if m == W.LOCAL else 0)
                        for m in modes)
    else:
        flop_step = sum(W.useful_flop(s, m, window=window) for m in modes)
    ms_per_step = elapsed * 1e3 / args.steps
    value = flop_step * args.steps / elapsed / 1e12

    # ------------------------------------------------------ per-kernel roofline
    fam_flops = {}
    for m in modes:
        for fam, f in per_kernel_flops(s, m, window, final).items():
            fam_flops[fam] = fam_flops.get(fam, 0) + f
    # breakdown: the one fully bracketed step; share = that kernel's time in it over the
    # timed steps' ms per step
    per_kernel = []
    fam_ms = {}
    for name, launches, total_ms in ktimes:
        fam = kernel_family(name)
        fam_ms[fam] = fam_ms.get(fam, 0.0) + total_ms
        per_kernel.append({"kernel": name, "launches_per_step": launches,
                           "avg_ms": round(total_ms / launches, 5),
                           "share": round(total_ms / ms_per_step, 4)})
    dom_fam = kernel_family(dom[0])
    dom_launches = dom[1]
    avg_ms = dom[2] / dom_launches
    if dom_fam in fam_flops:
        per_launch = fam_flops[dom_fam] * args.steps / dom_launches
        achieved = per_launch / (avg_ms * 1e-3) / 1e12
        roofline = {"kernel": dom[0], "bound": "mfma", "achieved": round(achieved, 2),
                    "peak": W.MI355X_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(achieved / W.MI355X_BF16_PEAK_TFLOPS, 4),
                    "traffic": measured_traffic(dom[0], args.workload),
                    "flop_per_launch": per_launch, "avg_launch_ms": round(avg_ms, 5)}
    else:
        roofline = {"kernel": dom[0], "bound": "hbm", "achieved": None, "peak": 8000.0,
                    "unit": "GB/s", "frac": None, "traffic": None}
    breakdown = {}
    for fam, ms in fam_ms.items():
        ent = {"ms_per_step": round(ms, 4)}
        if fam in fam_flops:
            ent["tflops"] = round(fam_flops[fam] / (ms * 1e-3) / 1e12, 2)
        if fam == "expand":
            nbytes = W.embed_bytes(1, s.L, s.n, W.STACK_DMODEL)
            ent["gbs"] = round(nbytes / (ms * 1e-3) / 1e9, 1)
            ent["bytes_per_launch"] = nbytes
            if copy_ceiling is not None:
                ent["back_to_back_ms"] = copy_ceiling["expand_ms"]
                ent["back_to_back_gbs"] = copy_ceiling["expand_gbs"]
                ent["copy_gbs"] = copy_ceiling["gbs"]
                ent["of_copy"] = round(copy_ceiling["expand_gbs"] / copy_ceiling["gbs"], 3)
                ent["cold_gbs"] = copy_ceiling["cold_expand_gbs"]
                ent["cold_copy_gbs"] = copy_ceiling["cold_gbs"]
                ent["cold_of_copy"] = round(copy_ceiling["cold_expand_gbs"] / copy_ceiling["cold_gbs"], 3)
        if fam in ("final_gather", "final_gather_bwd"):
            nbytes = W.final_gather_bytes(1, s.L, s.n, W.STACK_DMODEL, fam == "final_gather_bwd")
            ent["gbs"] = round(nbytes / (ms * 1e-3) / 1e9, 1)
            ent["bytes_per_launch"] = nbytes
        if fam == "expand_bwd":
            nbytes = W.embed_bwd_bytes(1, s.L, s.n, W.STACK_DMODEL, int(nuniq.cpu()[0]))
            ent["gbs"] = round(nbytes / (ms * 1e-3) / 1e9, 1)
            ent["bytes_per_launch"] = nbytes
        breakdown[fam] = ent

    out = {
        "metric": METRIC, "value": round(value, 3), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded device normal draws; no dataset or weights)",
        "config": {"workload": wl_desc, "B": s.B, "L": s.L, "n": s.n, "Hq": s.Hq,
                   "Hkv": s.Hkv, "D": s.D, "layers": nl,
                   **({"window": window} if W.LOCAL in modes else {}),
                   "useful_tflop_per_step": round(flop_step / 1e12, 4)},
        "frac_of_peak": round(value / W.MI355X_BF16_PEAK_TFLOPS, 4),
        "roofline": roofline, "breakdown": breakdown, "per_kernel": per_kernel,
        "input_gen_s": round(t_gen, 2),
    }
    if per_mode is not None:
        out["per_mode"] = per_mode
    if copy_ceiling is not None:
        out["copy_ceiling"] = copy_ceiling
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.cpu_sample_tokens, flop_step, ms_per_step)
    print(json.dumps(out), flush=True)


def time_layer_modes(hd, torch, layers, s, scale, dq, dk, dv, ws, ws_bytes, stream, W, reps=10):
    """fwd+bwd of one intra-stream and one mixing layer of the step (its first layer of
    each kind, same inputs), each alone: `reps` back-to-back passes between two events
    on the launch stream, after one untimed pass.  Each layer is timed with the one-pass
    backward (the workspace the step uses) and again with the backward in query bands
    at the smallest workspace it accepts."""
    res = {}
    for mode in (W.INTRA, W.MIX):
        ly = next(x for x in layers if x["mode"] == mode)

        def one(nbytes):
            hd.hd_sfa_fwd(ly["q"], ly["k"], ly["v"], ly["o"], ly["lse"], s.B, s.L, s.n, s.Hq,
                          s.Hkv, s.D, mode, scale, stream=stream)
            hd.hd_sfa_bwd(ly["q"], ly["k"], ly["v"], ly["o"], ly["lse"], ly["do"], dq, dk, dv,
                          s.B, s.L, s.n, s.Hq, s.Hkv, s.D, mode, scale, ws, nbytes,
                          stream=stream)

        def timed(nbytes):
            one(nbytes)
            t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            t0.record(stream)
            for _ in range(reps):
                one(nbytes)
            t1.record(stream)
            torch.cuda.synchronize()
            return t0.elapsed_time(t1) / reps

        ms = timed(ws_bytes)
        tf = W.useful_flop(s, mode) / (ms * 1e-3) / 1e12
        ent = {"ms": round(ms, 4), "tflops": round(tf, 2),
               "frac_of_peak": round(tf / W.MI355X_BF16_PEAK_TFLOPS, 4),
               "useful_tflop": round(W.useful_flop(s, mode) / 1e12, 4), "reps": reps}
        low = hd.hd_sfa_bwd_min_workspace_bytes(s.B, s.L, s.n, s.Hq, s.Hkv, s.D, mode,
                                                hd.HD_DTYPE_BF16)
        ms_b = timed(low)
        tf_b = W.useful_flop(s, mode) / (ms_b * 1e-3) / 1e12
        ent["query_bands_min_workspace"] = {
            "ms": round(ms_b, 4), "tflops": round(tf_b, 2), "workspace_bytes": low,
            "one_pass_workspace_bytes": hd.hd_sfa_bwd_workspace_bytes(
                s.B, s.L, s.n, s.Hq, s.Hkv, s.D, mode, hd.HD_DTYPE_BF16)}
        res[W.MODE_NAMES[mode]] = ent
    return res


def time_expand_vs_copy(hd, torch, ids, tables, emb, s, W, stream, reps=20):
    """The expansion and a plain device-to-device copy of as many bytes as the expansion
    moves (read + write counted), each launched `reps` times back to back between two
    events on the launch stream: the same protocol for both, so that their ratio
    compares the kernels (a single launch bracketed by events also carries the events'
    own overhead, a few microseconds, which is large against a 40-microsecond kernel)."""
    src = emb.view(-1)
    dst = torch.empty_like(src)
    nbytes = 2 * src.numel() * src.element_size()

    def b2b(fn):
        fn()
        torch.cuda.synchronize()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for _ in range(reps):
            fn()
        t1.record(stream)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / reps

    flush = torch.empty(1 << 30, dtype=torch.uint8, device=src.device)

    def cold(fn):
        """Median of single launches, each after writing 1 GiB elsewhere (which evicts
        the 256 MB Infinity Cache and the L2s), as the step's expansion finds them."""
        ts = []
        for i in range(reps // 2):
            flush.fill_(i & 255)
            t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            t0.record(stream)
            fn()
            t1.record(stream)
            torch.cuda.synchronize()
            ts.append(t0.elapsed_time(t1))
        return sorted(ts)[len(ts) // 2]

    copy = lambda: dst.copy_(src)  # noqa: E731
    expand = lambda: hd.hd_expand_embed(ids, tables, emb, 1, s.L, s.n, W.STACK_VOCAB,  # noqa: E731
                                        W.STACK_DMODEL, stream=stream)
    ms_copy, ms_exp = b2b(copy), b2b(expand)
    cold_copy, cold_exp = cold(copy), cold(expand)
    del flush
    gbs = lambda ms: round(nbytes / (ms * 1e-3) / 1e9, 1)  # noqa: E731
    return {"bytes": nbytes, "ms": round(ms_copy, 5), "gbs": gbs(ms_copy),
            "expand_ms": round(ms_exp, 5), "expand_gbs": gbs(ms_exp),
            "cold_ms": round(cold_copy, 5), "cold_gbs": gbs(cold_copy),
            "cold_expand_ms": round(cold_exp, 5), "cold_expand_gbs": gbs(cold_exp),
            "reps": reps,
            "what": "torch copy_ of the expansion's output size (read + write bytes) and the "
                    "expansion itself, each timed back to back over the reps (warm: the "
                    "previous repetition leaves data in the Infinity Cache) and as single "
                    "launches after a cache flush (cold, medians; these carry the events' "
                    "own few microseconds)"}


DECODE_BATCH = 16  # sequences decoded together


def run_decode(args):
    """One parallel-stream decode step: for each layer, the n streams of every sequence's
    new token against that layer's KV cache (all sequences at a full 4096-token context,
    Qwen3-8B-like heads).  value = GB/s of cache rows read (each cached key/value row of a
    layer is read once per step, whatever the layer type)."""
    import torch

    import paper_2607_08186_amd as hd
    from paper_2607_08186_amd import synth
    from paper_2607_08186_amd import workloads as W

    if not os.path.exists(hd.binding.LIB_PATH):
        from paper_2607_08186_amd import build as hip_build

        hip_build.build()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    s = W.QWEN8B.shape
    B, Lcap, n = DECODE_BATCH, s.L, s.n
    window = args.window if args.window is not None else W.LOCAL_WINDOW
    kind = args.workload.split("-")[1]
    modes = (W.stack_modes() if kind == "stack36" else
             [{"intra": W.INTRA, "mix": W.MIX, "local": W.LOCAL}[kind]])
    ctx_len = Lcap - 1
    ctx = torch.full((B,), ctx_len, dtype=torch.int32, device=dev)
    t_gen = time.time()
    layers = []
    for li, m in enumerate(modes):
        seed = synth.seed_for("decode-bench", li)
        layers.append(dict(
            mode=m,
            q=synth.device_normal((B, n, s.Hq, s.D), W.QWEN8B.qkv_std, seed + 1, dev, torch.bfloat16),
            k=synth.device_normal((B, n * Lcap, s.Hkv, s.D), W.QWEN8B.qkv_std, seed + 2, dev,
                                  torch.bfloat16),
            v=synth.device_normal((B, n * Lcap, s.Hkv, s.D), W.QWEN8B.qkv_std, seed + 3, dev,
                                  torch.bfloat16),
            o=torch.empty((B, n, s.Hq, s.D), dtype=torch.bfloat16, device=dev),
            lse=torch.empty((B, s.Hq, n), dtype=torch.float32, device=dev)))
    ws_bytes = max(hd.hd_sfa_decode_workspace_bytes(B, Lcap, n, s.Hq, s.Hkv, s.D, m, window,
                                                    ctx_len) for m in set(modes))
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()
    t_gen = time.time() - t_gen

    def step():
        for ly in layers:
            hd.hd_sfa_decode(ly["q"], ly["k"], ly["v"], ctx, ctx_len, ly["o"], ly["lse"], B, Lcap,
                             n, s.Hq, s.Hkv, s.D, ly["mode"], window, s.scale, ws, ws_bytes,
                             stream=stream)

    for _ in range(args.warmup):
        step()
    elapsed, ktimes, dom = time_steps(hd, torch, step, args.steps)

    def cache_bytes(m):
        rows = (ctx_len + 1) * n
        if m == W.LOCAL:
            rows = min(rows, window + n - 1)  # the last window positions of the n queries
        return B * rows * s.Hkv * s.D * 2 * 2
    bytes_step = sum(cache_bytes(m) for m in modes)
    ms_step = elapsed * 1e3 / args.steps
    value = bytes_step * args.steps / elapsed / 1e9
    per_kernel = [{"kernel": name, "launches_per_step": nl, "avg_ms": round(ms / nl, 5),
                   "share": round(ms / ms_step, 4)} for name, nl, ms in ktimes]
    avg_ms = dom[2] / dom[1]
    per_launch = bytes_step * args.steps / dom[1] if "partial" in dom[0] or "decode_bf16" in dom[0] else None
    roofline = {"kernel": dom[0], "bound": "hbm", "unit": "GB/s", "peak": W.MI355X_HBM_PEAK_GBS,
                "achieved": round(per_launch / (avg_ms * 1e-3) / 1e9, 1) if per_launch else None,
                "frac": round(per_launch / (avg_ms * 1e-3) / 1e9 / W.MI355X_HBM_PEAK_GBS, 4)
                if per_launch else None,
                "traffic": measured_traffic(dom[0], args.workload), "bytes_per_launch": per_launch,
                "avg_launch_ms": round(avg_ms, 5)}
    out = {
        "metric": "SFA parallel-stream decode KV-cache read GB/s", "value": round(value, 1),
        "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded device normal draws)",
        "config": {"workload": f"{args.workload}: {DECODE_BATCH} sequences x {ctx_len + 1} "
                               f"tokens in cache, n={n} Hq={s.Hq} Hkv={s.Hkv} D={s.D}, "
                               f"{len(modes)} layer(s)",
                   "layers": len(modes), **({"window": window} if W.LOCAL in modes else {})},
        "roofline": roofline, "per_kernel": per_kernel, "input_gen_s": round(t_gen, 2),
    }
    print(json.dumps(out), flush=True)


# sources each kernel family is built from (a change voids stored counter readings)
KERNEL_SOURCES = {
    "sfa_decode_bf16": ["sfa_decode_bf16.hip", "decode_internal.h", "sfa_lds.h", "hd_device.h",
                        "hd_internal.h"],
    "sfa_dkdv_bf16": ["sfa_bwd_bf16.hip", "sfa_lds.h", "hd_device.h", "hd_internal.h"],
    "sfa_dq_bf16": ["sfa_bwd_bf16.hip", "sfa_lds.h", "hd_device.h", "hd_internal.h"],
    "sfa_fwd_bf16": ["sfa_fwd_bf16.hip", "sfa_lds.h", "hd_device.h", "hd_internal.h"],
}


def kernel_source_hash(kernel):
    import hashlib
    fam = next((f for f in KERNEL_SOURCES if kernel.startswith(f)), None)
    if fam is None:
        return None
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[fam]:
        with open(os.path.join(ROOT, "paper_2607_08186_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 counter summary
    (FETCH_SIZE and WRITE_SIZE, each scaled by the factor a plain copy of known size
    reads), or None when there is none for this kernel and workload or the kernel's
    sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and not line.startswith("#"):
                key, val = line.split(":", 1)
                kv[key.strip()] = val.strip()
    if kv.get("source_sha") != kernel_source_hash(kernel):
        return None
    return int(float(kv["hbm_bytes_per_launch"]))


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(Ls, flop_step, ms_step):
    """The fp64 oracle on a bounded sample of the same workload: one intra-stream and
    one mixing layer of the stack, fwd + bwd, all 32 query heads, first Ls tokens, on
    every thread this process may use (forward and backward both parallel over the 32
    query heads).  The oracle's cost is proportional to the useful flop it does (it
    evaluates visible pairs only), so the whole step's oracle time is extrapolated
    from the sampled rate and labelled as such."""
    import numpy as np  # noqa: F401

    import oracle
    from paper_2607_08186_amd import synth
    from paper_2607_08186_amd import workloads as W

    base = W.QWEN8B.shape
    sh = W.Shape(1, Ls, base.n, base.Hq, base.Hkv, base.D)
    nthreads = oracle.default_threads()
    ins = synth.sfa_inputs(sh.B, sh.L, sh.n, sh.Hq, sh.Hkv, sh.D, seed=synth.seed_for("cpu"),
                           dtype="bf16", qkv_std=W.QWEN8B.qkv_std)
    flop = 0
    t0 = time.perf_counter()
    for mode in (W.INTRA, W.MIX):
        kw = dict(L=sh.L, n=sh.n, mode=mode, scale=sh.scale, nthreads=nthreads)
        oracle.sfa_fwd(ins["q"], ins["k"], ins["v"], **kw)
        oracle.sfa_bwd(ins["q"], ins["k"], ins["v"], ins["dout"], **kw)
        flop += W.useful_flop(sh, mode)
        print(f"[bench] cpu oracle mode {mode} done", file=sys.stderr, flush=True)
    dt = time.perf_counter() - t0
    rate = flop / dt
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:
        affinity = None
    step_s = flop_step / rate
    return {"value": round(rate / 1e12, 6), "unit": "TFLOP/s", "cores": nthreads,
            "kind": "oracle", "seconds": round(dt, 2),
            "threads": nthreads, "nproc": os.cpu_count(), "affinity_cpus": affinity,
            "omp_num_threads": os.environ.get("OMP_NUM_THREADS"), "cpu_model": _cpu_model(),
            "sample": (f"one intra + one mix layer, fwd+bwd, B=1 L={Ls} n={sh.n} "
                       f"Hq={sh.Hq} Hkv={sh.Hkv} D={sh.D} (prefix of the step's layer shape), "
                       f"fp64, {nthreads} threads, fwd and bwd parallel over the {sh.Hq} "
                       "query heads"),
            "extrapolated_step_s": round(step_s, 1),
            "extrapolated_step_vs_gpu": round(step_s * 1e3 / ms_step, 1),
            "extrapolation": ("EXTRAPOLATED, not measured: the whole step's useful flop "
                              "divided by the sampled oracle rate (the oracle's cost is "
                              "proportional to the visible pairs it evaluates)")}


if __name__ == "__main__":
    main()
