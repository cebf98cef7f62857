"""Throughput of the speculative-cascade verify step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--sets S] [--no-cpu-baseline]

A step is one spc_verify call (statistics pass + residual sampling pass) on
the Gemma-vocabulary workload: B=32 sequences, gamma=7 drafted positions,
V=256000, bfloat16 logits, Diff rule alpha=0.05, temperature 1 (seeded
synthetic Zipf(1.2) logits).  Inputs are resident in HBM before timing; S
distinct input sets (default 3 x 262 MB) are rotated so the 256 MB
Infinity Cache cannot serve a repeat.

Prints one JSON line: verified positions/s (B*gamma per step) for the whole
path, plus the statistics kernel's roofline (algorithmic logit bytes / its
mean duration, from HIP events recorded around it on the launch stream) and
the fp64 oracle's throughput on the host cores (reported baseline).
"""
import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0  # MI355X HBM3E, published


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
    return dict(value=n * wl.B * wl.gamma / el, unit="positions/s",
                cores=oracle.num_threads(), kind="oracle",
                sample=f"{n} whole step(s) of the timed workload (B={wl.B}, gamma={wl.gamma}, "
                       f"V={wl.V} bf16), fp64, OpenMP over sequences, {el:.1f} s",
                logit_gbps=n * wl.logit_bytes() / el / 1e9), dict(rep)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--sets", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the verify path has no multi-GPU mode "
              f"(--gpus {args.gpus} requested)", file=sys.stderr)
        return 2

    import torch
    from paper_2405_19261_amd import spc
    from paper_2405_19261_amd import workloads as W

    wl = W.WORKLOADS[3]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    sets = [W.generate(wl, 1000 + i, dev) for i in range(args.sets)]
    B, gamma, V = wl.B, wl.gamma, wl.V
    outs = [(torch.empty(B, dtype=torch.int32, device=dev),
             torch.empty(B, dtype=torch.int32, device=dev),
             torch.empty((B, gamma + 1), dtype=torch.uint8, device=dev)) for _ in sets]
    stream = torch.cuda.current_stream()
    ev = HipEvents()
    n = args.steps
    hot = [(ev.create(), ev.create()) for _ in range(n)]
    outer = (ev.create(), ev.create())

    def step(i, events=None):
        s = sets[i % len(sets)]
        if events is None:
            spc.spc_verify(s["q"], s["p"], s["draft"], s["uniforms"], wl.rule, wl.alpha,
                           wl.temperature, out=outs[i % len(sets)], stream=stream)
        else:
            spc.spc_verify_ex(s["q"], s["p"], s["draft"], s["uniforms"], wl.rule, wl.alpha,
                              wl.temperature, ev_hot_begin=events[0], ev_hot_end=events[1],
                              out=outs[i % len(sets)], stream=stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # timed region: exactly `steps` steps, each bracketing the statistics
    # kernel with its own pair of events
    torch.cuda.synchronize()
    ev.hip.hipEventRecord(ctypes.c_void_p(outer[0]), ctypes.c_void_p(stream.cuda_stream))
    t0 = time.perf_counter()
    for i in range(n):
        step(i, hot[i])
    ev.hip.hipEventRecord(ctypes.c_void_p(outer[1]), ctypes.c_void_p(stream.cuda_stream))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    total_ms = ev.elapsed_ms(*outer)
    hot_ms = [ev.elapsed_ms(a, b) for a, b in hot]
    ms_per_step = total_ms / n
    hot_mean = sum(hot_ms) / n
    pos_per_s = B * gamma / (ms_per_step / 1e3)
    stats_bytes = wl.logit_bytes()  # the statistics kernel reads q and p once
    achieved = stats_bytes / (hot_mean / 1e3) / 1e9

    line = dict(
        metric="verified positions/s and achieved HBM GB/s (B=32, γ=7, V=256000 bf16)",
        value=pos_per_s, unit="positions/s", n_gpus=1, steps=n, warmup=args.warmup,
        ms_per_step=ms_per_step, higher_is_better=True, scaling="weak", vs_baseline=None,
        dtype="f32", data="synthetic",
        config=dict(workload="gemma-vocab verify step: B=32 gamma=7 V=256000 bf16 logits, "
                             "Diff alpha=0.05, T=1, Zipf(1.2)+N(0,1) verifier, "
                             "0.8*verifier+N(0,1) drafter (10% rows +N(0,3))",
                    global_batch=B, positions_per_step=B * gamma,
                    algorithmic_bytes_per_step=wl.algorithmic_bytes(),
                    path_gbps=wl.algorithmic_bytes() / (ms_per_step / 1e3) / 1e9,
                    input_sets=len(sets), wall_s=wall),
        roofline=dict(bound="hbm", kernel="k_stats", achieved=achieved, peak=PEAK_HBM_GBPS,
                      unit="GB/s", frac=achieved / PEAK_HBM_GBPS, traffic=None,
                      mean_us=hot_mean * 1e3, min_us=min(hot_ms) * 1e3,
                      bytes_per_launch=stats_bytes),
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
    for a, b in hot:
        ev.destroy(a)
        ev.destroy(b)
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
