"""Throughput of the speculative-cascade verify step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--sets S] [--no-cpu-baseline]
                    [--copy-calib-mb N] [--rule NAME --alpha A]
    python bench.py --traffic-from FETCH.csv WRITE.csv --copy-calib-mb N

A step is one spc_verify call (the statistics tiles, which also merge and
decide each row, then the draw pass) on the Gemma-vocabulary workload: B=32 sequences, gamma=7 drafted positions,
V=256000, bfloat16 logits, Diff rule alpha=0.05, temperature 1 (seeded
synthetic Zipf(1.2) logits).  --rule / --alpha time the same shape under
another rule (opt, or a token-specific rule token-v1/v2/v3, which add the
second statistics pass).  Inputs are resident in HBM before timing; S
distinct input sets (default 3 x 262 MB) are rotated so the 256 MB
Infinity Cache cannot serve a repeat.

Prints one JSON line: verified positions/s (B*gamma per step) for the whole
path, plus the statistics kernel's roofline (algorithmic logit bytes / its
mean duration, from HIP events recorded around it on the launch stream on
every EVERY-th step of the timed region, by default every 32nd -- the four
event records of a sampled step cost about 10 us of GPU time, which at every
4th step added 2.4 us to the mean step and at every 32nd adds about 0.3 us)
and the fp64
oracle's throughput on the host cores (reported baseline).  Step-time
percentiles come from the spacing of those events (EVERY-step windows).

HBM traffic of the statistics kernel (k_tiles) comes from two rocprofv3 counter runs of
this script (FETCH_SIZE, then WRITE_SIZE) with --copy-calib-mb, which first
runs an elementwise float32 negation of N MiB (reads N MiB, writes N MiB):
each counter is scaled by the ratio of the copy's known bytes to what the same
counter reads for it.  --traffic-from reduces the two counter tables to one
record, stored in profiles/ with the sha256 of the kernel source; the
benchmark line reports it only while that source is unchanged.
"""
import argparse
import csv
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0  # MI355X HBM3E, published
KERNEL_SRC = os.path.join(ROOT, "paper_2405_19261_amd", "csrc", "spc_kernels.hip")
TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "k_tiles_gemma-vocab_b32_g7_traffic.txt")
ROOF_KERNEL = "k_tiles"  # the kernel the roofline object describes
STEP_KERNELS = ("k_tiles", "k_res", "k_jobs", "k_small")
MALL_BYTES = 256 << 20  # MI355X Infinity Cache
COPY_KERNEL_TAG = "neg_kernel"  # the calibration copy is torch.neg


class HipEvents:
    """hipEvent_t handles created straight from the HIP runtime."""

    def __init__(self):
        import torch  # noqa: F401  (loads libamdhip64)
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]

    def create(self):
        e = ctypes.c_void_p()
        assert self.hip.hipEventCreate(ctypes.byref(e)) == 0
        return e.value

    def elapsed_ms(self, a, b):
        assert self.hip.hipEventSynchronize(ctypes.c_void_p(b)) == 0
        t = ctypes.c_float()
        assert self.hip.hipEventElapsedTime(ctypes.byref(t), ctypes.c_void_p(a),
                                            ctypes.c_void_p(b)) == 0
        return t.value

    def destroy(self, e):
        self.hip.hipEventDestroy(ctypes.c_void_p(e))


def kernel_sha256():
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def per_dispatch_kib(path, counter, tag, required=True):
    """Mean counter value (KiB) per dispatch of kernels whose name holds tag
    (the kernel name up to its template arguments)."""
    def match(name):  # a library kernel by its own name, else any name holding tag
        return f"::{tag}<" in name if tag.startswith("k_") else tag in name
    vals = [float(r["Counter_Value"]) for r in csv.DictReader(open(path))
            if r["Counter_Name"] == counter and match(r["Kernel_Name"])]
    if not vals:
        if required:
            raise SystemExit(f"no {counter} rows for kernels matching {tag!r} in {path}")
        return None, 0
    return sum(vals) / len(vals), len(vals)


def traffic_record(fetch_csv, write_csv, copy_mb):
    """HBM bytes per statistics-kernel launch from the two counter tables."""
    copy_bytes = copy_mb * 2 ** 20
    f_copy, n_fc = per_dispatch_kib(fetch_csv, "FETCH_SIZE", COPY_KERNEL_TAG)
    w_copy, n_wc = per_dispatch_kib(write_csv, "WRITE_SIZE", COPY_KERNEL_TAG)
    f_k, n_fk = per_dispatch_kib(fetch_csv, "FETCH_SIZE", ROOF_KERNEL)
    w_k, n_wk = per_dispatch_kib(write_csv, "WRITE_SIZE", ROOF_KERNEL)
    fetch_scale = copy_bytes / (f_copy * 1024.0)
    write_scale = copy_bytes / (w_copy * 1024.0)
    fetch_b = f_k * 1024.0 * fetch_scale
    write_b = w_k * 1024.0 * write_scale
    # the step's other kernels, scaled alike
    others = {}
    for name in STEP_KERNELS:
        if name == ROOF_KERNEL:
            continue
        f, nf = per_dispatch_kib(fetch_csv, "FETCH_SIZE", name, required=False)
        w, nw = per_dispatch_kib(write_csv, "WRITE_SIZE", name, required=False)
        if f is not None and w is not None:
            others[name] = dict(fetch_bytes=f * 1024.0 * fetch_scale,
                                write_bytes=w * 1024.0 * write_scale, dispatches=[nf, nw])
    return dict(kernel=ROOF_KERNEL, kernel_src_sha256=kernel_sha256(), copy_mib=copy_mb,
                copy_fetch_kib=f_copy, copy_write_kib=w_copy, fetch_scale=fetch_scale,
                write_scale=write_scale, k_fetch_kib=f_k, k_write_kib=w_k,
                dispatches=dict(copy_fetch=n_fc, copy_write=n_wc, k_fetch=n_fk, k_write=n_wk),
                fetch_bytes=fetch_b, write_bytes=write_b, traffic_bytes=fetch_b + write_b,
                other_kernels=others)


def stored_traffic():
    """Traffic bytes per launch from the stored record, or None if there is
    none or the kernel source changed since it was taken."""
    try:
        for line in open(TRAFFIC_RECORD):
            if line.startswith("record: "):
                rec = json.loads(line[len("record: "):])
                if rec.get("kernel_src_sha256") == kernel_sha256():
                    return rec["traffic_bytes"]
    except OSError:
        pass
    return None


def copy_calibration(mb):
    """Elementwise float32 negation of mb MiB: reads mb MiB, writes mb MiB."""
    import torch
    n = mb * 2 ** 20 // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    del src, dst


def cpu_baseline(wl, inp, gpu_out, min_seconds=10.0):
    """fp64 oracle on the host cores over whole steps of the same workload
    until min_seconds have passed; also checks the GPU outputs of that step."""
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import oracle
    import parity
    h = parity.host_inputs(inp)
    n = 0
    t0 = time.perf_counter()
    while True:
        o = parity.run_oracle(h)
        n += 1
        el = time.perf_counter() - t0
        if el >= min_seconds:
            break
    rep = parity.compare(gpu_out, o, h, wl.dtype)
    cores = oracle.num_threads()
    # the same step on one thread (the oracle's results do not depend on the
    # thread count), for a per-core figure
    oracle.set_num_threads(1)
    try:
        t1 = time.perf_counter()
        parity.run_oracle(h)
        el1 = time.perf_counter() - t1
    finally:
        oracle.set_num_threads(cores)
    return dict(value=n * wl.B * wl.gamma / el, unit="positions/s",
                cores=cores, kind="oracle",
                sample=f"{n} whole step(s) of the timed workload (B={wl.B}, gamma={wl.gamma}, "
                       f"V={wl.V} bf16), fp64, OpenMP over sequences, {el:.1f} s; "
                       f"one_thread: 1 step, {el1:.1f} s",
                logit_gbps=n * wl.logit_bytes() / el / 1e9,
                one_thread_value=wl.B * wl.gamma / el1, cpu_model=cpu_model()), dict(rep)


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def bench_draft(args, wl, dev):
    """The drafter's sampling step on B rows of V logits (one position per
    sequence), at the workload's temperature."""
    import torch
    from paper_2405_19261_amd import spc
    from paper_2405_19261_amd import workloads as W
    sets = [W.generate(wl, 2000 + i, dev)["q"][:, 0].contiguous() for i in range(max(args.sets, 8))]
    u = torch.rand(wl.B, generator=torch.Generator(device=dev).manual_seed(1), device=dev)
    out = torch.empty(wl.B, dtype=torch.int32, device=dev)
    for i in range(args.warmup):
        spc.spc_draft_sample(sets[i % len(sets)], wl.temperature, uniforms=u, out=out)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(args.steps):
        spc.spc_draft_sample(sets[i % len(sets)], wl.temperature, uniforms=u, out=out)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / args.steps
    nbytes = wl.B * wl.V * (2 if wl.dtype == "bf16" else 4)
    print(json.dumps(dict(
        metric="drafter sampling steps/s", value=1e6 / us, unit="steps/s", n_gpus=1,
        steps=args.steps, warmup=args.warmup, us_per_step=us, higher_is_better=True,
        dtype="f32", data="synthetic",
        config=dict(workload=f"draft sampling: B={wl.B} rows of V={wl.V} {wl.dtype}, "
                             f"T={wl.temperature}", input_sets=len(sets)),
        roofline=dict(bound="hbm", achieved=nbytes / us / 1e3, peak=PEAK_HBM_GBPS, unit="GB/s",
                      frac=nbytes / us / 1e3 / PEAK_HBM_GBPS, bytes_per_step=nbytes))), flush=True)
    return 0


def decode_params(wl):
    """Rule, alpha and temperature of the decoding loop: the workload's
    scalars, or for the stress mix per-sequence arrays drawn (seeded) from its
    rule and temperature sets."""
    import torch
    from paper_2405_19261_amd import workloads as W
    if wl.rule >= 0:
        return wl.rule, wl.alpha, wl.temperature
    g = torch.Generator().manual_seed(1000 * wl.cfg)
    pick = torch.randint(0, len(W.CFG5_RULES), (wl.B,), generator=g)
    rule = torch.tensor([r for r, _ in W.CFG5_RULES], dtype=torch.int32)[pick]
    alpha = torch.tensor([a for _, a in W.CFG5_RULES], dtype=torch.float32)[pick]
    temp = torch.tensor(W.CFG5_TEMPS, dtype=torch.float32)[
        torch.randint(0, len(W.CFG5_TEMPS), (wl.B,), generator=g)]
    return rule, alpha, temp


def bench_decode(args, wl, dev, backend=None):
    """Rounds of the decoding loop (draft gamma tokens, score, verify, roll
    back) on synthetic models of the workload's vocabulary; emitted tokens/s
    over the whole loop, host bookkeeping included.  ``backend`` defaults to
    the library's."""
    import torch
    from paper_2405_19261_amd import decode
    dev = torch.device(dev)

    def sync():
        if dev.type == "cuda":
            torch.cuda.synchronize()

    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    q_lm, p_lm = decode.synthetic_pair(wl.V, seed=1, dtype=dt, device=dev)
    first = torch.randint(0, wl.V, (wl.B,), generator=torch.Generator().manual_seed(0))
    rule, alpha, temp = decode_params(wl)
    kw = dict(gamma=wl.gamma, rule=rule, alpha=alpha, temperature=temp, graph=args.graph,
              backend=backend)
    decode.spec_decode(q_lm, p_lm, first, rounds=2, seed=5, **kw)  # warm-up
    sync()
    t0 = time.perf_counter()
    res = decode.spec_decode(q_lm, p_lm, first, rounds=args.decode, seed=6, **kw)
    sync()
    el = time.perf_counter() - t0
    n = sum(len(t) for t in res.tokens)
    params = (f"rule {wl.rule} alpha={wl.alpha:g} T={wl.temperature}" if wl.rule >= 0 else
              "per-sequence rule {Chow 0.4, Diff 0.05, OPT 0.1} and T {0.5, 0.7, 1.0}")
    line = dict(
        metric="emitted tokens/s (decoding loop, synthetic models)", value=n / el,
        unit="tokens/s", n_gpus=1, rounds=args.decode, higher_is_better=True, dtype="f32",
        data="synthetic", ms_per_round=el * 1e3 / args.decode,
        tokens_per_round=res.tokens_per_round(),
        config=dict(workload=f"decoding loop: B={wl.B} gamma={wl.gamma} V={wl.V} {wl.dtype}, "
                             f"{params}; synthetic Markov drafter/verifier (table lookups)"
                             + ("; one HIP graph replay per round (capture included)"
                                if args.graph else "")))
    print(json.dumps(line), flush=True)
    return line


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--sets", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calib-mb", type=int, default=0)
    ap.add_argument("--event-every", type=int, default=32)
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"))
    ap.add_argument("--rule", default=None,
                    choices=["chow", "diff", "opt", "always", "never",
                             "token-v1", "token-v2", "token-v3", "lossy", "bild", "chowlog",
                             "difflog", "optlog"])
    ap.add_argument("--cfg", type=int, default=3, choices=[1, 2, 3, 4, 5],
                    help="workload (default 3, the Gemma-vocabulary step); 4 and 5 run "
                         "through spc_verify_ex with per-sequence arrays")
    ap.add_argument("--alpha", type=float, default=None)
    ap.add_argument("--draft", action="store_true",
                    help="time the drafter's sampling step (spc_draft_sample) on the "
                         "workload's drafter rows [B, V] instead of the verify step")
    ap.add_argument("--decode", type=int, default=0, metavar="ROUNDS",
                    help="time ROUNDS rounds of the decoding loop (decode.py) on synthetic "
                         "models of the workload's shape")
    ap.add_argument("--graph", action="store_true",
                    help="with --decode: capture one round into a HIP graph and replay it")
    args = ap.parse_args()
    if args.traffic_from:
        if args.copy_calib_mb <= 0:
            ap.error("--traffic-from needs the --copy-calib-mb the counter runs used")
        print(json.dumps(traffic_record(*args.traffic_from, args.copy_calib_mb)))
        return 0
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the verify path has no multi-GPU mode "
              f"(--gpus {args.gpus} requested)", file=sys.stderr)
        return 2

    import torch
    from paper_2405_19261_amd import spc
    from paper_2405_19261_amd import workloads as W

    wl = W.WORKLOADS[args.cfg]
    if args.rule is not None or args.alpha is not None:
        rule = wl.rule if args.rule is None else {v: k for k, v in W.RULE_NAMES.items()}[args.rule]
        wl = wl.with_(rule=rule, alpha=wl.alpha if args.alpha is None else args.alpha)
    rule_desc = (f"{W.RULE_NAMES[wl.rule]} alpha={wl.alpha:g}" if wl.rule in W.RULE_NAMES
                 else "per-sequence rules")
    per_seq = args.cfg == 5  # the mixed batch: per-sequence arrays
    # the rules the per-sequence arrays hold (the library skips passes for the others)
    rule_mask = (sum(1 << r for r, _ in W.CFG5_RULES) if args.cfg == 5 else 1 << wl.rule) \
        if per_seq else 0
    if args.cfg != 3:
        args.no_cpu_baseline = True
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calib_mb > 0:
        copy_calibration(args.copy_calib_mb)
    if args.draft:
        return bench_draft(args, wl, dev)
    if args.decode:
        bench_decode(args, wl, dev)
        return 0
    sets = [W.generate(wl, 1000 + i, dev) for i in range(args.sets)]
    B, gamma, V = wl.B, wl.gamma, wl.V
    outs = [(torch.empty(B, dtype=torch.int32, device=dev),
             torch.empty(B, dtype=torch.int32, device=dev),
             torch.empty((B, gamma + 1), dtype=torch.uint8, device=dev)) for _ in sets]
    stream = torch.cuda.current_stream()
    ev = HipEvents()
    n = args.steps
    every = max(1, args.event_every)
    sampled = list(range(0, n, every))
    hot = {i: tuple(ev.create() for _ in range(4)) for i in sampled}
    outer = (ev.create(), ev.create())

    def call(i, ev_tiles=None):
        s = sets[i % len(sets)]
        if per_seq:
            temp = torch.zeros_like(s["temperature"]) if wl.greedy else s["temperature"]
            spc.spc_verify_ex(s["q"], s["p"], s["draft"], s["uniforms"], 0, 0.0, 1.0,
                              rule_per_seq=s["rule"], alpha_per_seq=s["alpha"],
                              temp_per_seq=temp, rules_present=rule_mask, ev_tiles=ev_tiles,
                              out=outs[i % len(sets)], stream=stream)
        else:
            # temperature 0 is the batch-wide greedy step (spc_greedy_verify)
            spc.spc_verify_ex(s["q"], s["p"], s["draft"], None if wl.greedy else s["uniforms"],
                              wl.rule, wl.alpha, 0.0 if wl.greedy else wl.temperature,
                              ev_tiles=ev_tiles, out=outs[i % len(sets)], stream=stream)

    sraw = ctypes.c_void_p(stream.cuda_stream)

    def step(i, events=None):
        # a sampled step records four events on the call's stream: around the
        # whole call, and (inside the library) around its statistics kernel
        if events is None:
            call(i)
            return
        ev.hip.hipEventRecord(ctypes.c_void_p(events[0]), sraw)
        call(i, (events[1], events[2]))
        ev.hip.hipEventRecord(ctypes.c_void_p(events[3]), sraw)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # timed region: exactly `steps` steps; every `every`-th one brackets the
    # call and its statistics kernel with events
    torch.cuda.synchronize()
    ev.hip.hipEventRecord(ctypes.c_void_p(outer[0]), ctypes.c_void_p(stream.cuda_stream))
    t0 = time.perf_counter()
    for i in range(n):
        step(i, hot.get(i))
    ev.hip.hipEventRecord(ctypes.c_void_p(outer[1]), ctypes.c_void_p(stream.cuda_stream))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    total_ms = ev.elapsed_ms(*outer)
    hot_ms = sorted(ev.elapsed_ms(hot[i][1], hot[i][2]) for i in sampled)
    call_ms = sorted(ev.elapsed_ms(hot[i][0], hot[i][3]) for i in sampled)
    windows = sorted(ev.elapsed_ms(hot[a][0], hot[b][0]) / (b - a)
                     for a, b in zip(sampled, sampled[1:]))
    ms_per_step = total_ms / n
    hot_mean = sum(hot_ms) / len(hot_ms)

    def pct(xs, q):
        return xs[min(len(xs) - 1, int(q * (len(xs) - 1) + 0.5))] if xs else None
    pos_per_s = B * gamma / (ms_per_step / 1e3)
    stats_bytes = wl.logit_bytes()  # the statistics kernel reads q and p once
    achieved = stats_bytes / (hot_mean / 1e3) / 1e9
    traffic = stored_traffic()

    line = dict(
        metric="verified positions/s and achieved HBM GB/s (B=32, γ=7, V=256000 bf16)",
        value=pos_per_s, unit="positions/s", n_gpus=1, steps=n, warmup=args.warmup,
        ms_per_step=ms_per_step, higher_is_better=True, scaling="weak", vs_baseline=None,
        dtype="f32", data="synthetic",
        config=dict(workload=(("gemma-vocab verify step: B=32 gamma=7 V=256000 bf16 logits, "
                              f"{rule_desc}, T=1, Zipf(1.2)+N(0,1) verifier, "
                              "0.8*verifier+N(0,1) drafter (10% rows +N(0,3))")
                             if args.cfg == 3 else f"{wl.name} ({rule_desc})"),
                    global_batch=B, positions_per_step=B * gamma,
                    algorithmic_bytes_per_step=wl.algorithmic_bytes(),
                    path_gbps=wl.algorithmic_bytes() / (ms_per_step / 1e3) / 1e9,
                    input_sets=len(sets), wall_s=wall,
                    cache=("cold: the rotated input sets exceed twice the 256 MB Infinity Cache"
                           if len(sets) * wl.logit_bytes() > 2 * MALL_BYTES else
                           "hot: every input set fits in the 256 MB Infinity Cache"),
                    step_us_p10_p50_p90=[None if pct(windows, q) is None else pct(windows, q) * 1e3
                                         for q in (0.1, 0.5, 0.9)],
                    step_us_windows=f"{len(windows)} windows of {every} steps"),
        roofline=dict(bound="hbm", kernel="k_tiles", achieved=achieved, peak=PEAK_HBM_GBPS,
                      unit="GB/s", frac=achieved / PEAK_HBM_GBPS, traffic=traffic,
                      mean_us=hot_mean * 1e3, min_us=hot_ms[0] * 1e3,
                      p10_p50_p90_us=[pct(hot_ms, q) * 1e3 for q in (0.1, 0.5, 0.9)],
                      launches_timed=len(hot_ms), bytes_per_launch=stats_bytes),
        # the whole step against the same roof: algorithmic bytes of the step
        # (both logit tensors once, drafts, uniforms, outputs) / step time
        step_roofline=dict(bound="hbm", achieved=wl.algorithmic_bytes() / (ms_per_step / 1e3) / 1e9,
                           peak=PEAK_HBM_GBPS, unit="GB/s",
                           frac=wl.algorithmic_bytes() / (ms_per_step / 1e3) / 1e9 / PEAK_HBM_GBPS,
                           call_us_p10_p50_p90=[pct(call_ms, q) * 1e3 for q in (0.1, 0.5, 0.9)]),
    )
    if not args.no_cpu_baseline:
        torch.cuda.synchronize()
        out0 = outs[0]
        s0 = sets[0]
        spc.spc_verify(s0["q"], s0["p"], s0["draft"], s0["uniforms"], wl.rule, wl.alpha,
                       wl.temperature, out=out0, stream=stream)
        torch.cuda.synchronize()
        g = dict(accept_len=out0[0].cpu().numpy(), next_token=out0[1].cpu().numpy(),
                 defer=out0[2].cpu().numpy())
        base, rep = cpu_baseline(wl, s0, g)
        line["cpu_baseline"] = base
        line["parity_vs_oracle"] = rep
    for evs in hot.values():
        for e in evs:
            ev.destroy(e)
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
