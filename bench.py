"""Benchmark of NaCl's one-shot encoding-phase KV-cache eviction on one MI355X.

One step = the eviction of every layer of the workload (score -> select ->
compact per layer, layers back to back on one stream), inputs resident in HBM.
Prints one JSON line:

  value     prefill tokens per second evicted per layer = B * L * layers / t_step
  roofline  the dominant kernel against its roofline, from its average
            duration measured with HIP events on the launch stream
  stages    every kernel's average duration and achieved rate
  cpu_baseline  the CPU oracle on a bounded sample of the same workload

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
"""

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # dense bf16 MFMA
F32_PEAK_TFLOPS = 157.3        # dense fp32 MFMA

# FETCH_SIZE / WRITE_SIZE scale factors and the per-launch traffic of the
# dominant kernel, from the rocprofv3 counter runs summarised under profiles/.
# None until measured for the current kernel.
MEASURED_TRAFFIC = None


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="prefill_32k")
    ap.add_argument("--layers", type=int, default=0, help="override the layer count (profiling only)")
    ap.add_argument("--stage-reps", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-heads", type=int, default=32)
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(eviction shards by head or batch with no communication; see DESIGN.md)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2408_03675_amd import nacl
    from synth import WORKLOADS, alg_bytes, alg_flops, make_layer

    w = WORKLOADS[args.workload]
    layers = args.layers or w.layers
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    nacl.load_library()

    log(f"[bench] workload {w.name}: layers={layers} B={w.B} H={w.H} L={w.L} D={w.D} P={w.P} "
        f"C={w.C} Cr={w.Cr} dtype={w.dtype}")
    t0 = time.time()
    data = [make_layer(w, l, device=dev) for l in range(layers)]
    torch.cuda.synchronize()
    log(f"[bench] generated {layers} layers in {time.time() - t0:.1f}s")
    q0, k0, v0 = data[0]
    pos_dev = torch.tensor(w.proxy_pos, dtype=torch.int32, device=dev)
    prob = nacl.Problem.from_tensors(q0, k0, v0, w.proxy_pos, sm_scale=w.scale, proxy_pos_dev=pos_dev)
    ws = nacl.workspace(prob, dev)
    BH = w.B * w.H
    outs = []
    for _ in range(layers):
        outs.append((torch.empty((w.B, w.H, w.L), dtype=torch.float32, device=dev),
                     torch.empty((w.B, w.H, w.C), dtype=torch.int32, device=dev),
                     torch.empty((w.B, w.H, w.C, w.D), dtype=q0.dtype, device=dev),
                     torch.empty((w.B, w.H, w.C, w.D), dtype=q0.dtype, device=dev)))

    def step():
        for l in range(layers):
            q, k, v = data[l]
            F, keep, ko, vo = outs[l]
            nacl.evict(prob, q, k, v, w.C, w.Cr, nacl.SAMPLE_SOFTMAX, w.rng_seed, l, ws=ws,
                       scores=F, keep_idx=keep, k_out=ko, v_out=vo)

    stream = torch.cuda.current_stream(dev)
    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        log(f"[bench] warmup {i + 1}/{args.warmup} done")
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    total_ms = e0.elapsed_time(e1)
    ms_per_step = total_ms / args.steps
    tok_per_s = w.B * w.L * layers / (ms_per_step / 1e3)
    log(f"[bench] {args.steps} steps: {ms_per_step:.3f} ms/step, {ms_per_step / layers * 1e3:.1f} us/layer")

    # Per-kernel durations through the public entry points, timed with events
    # on the launch stream: score with the caller's log-sum-exp runs only the
    # column-reduction kernel; without it, pass 1 + combine run too.
    lse_ws = torch.empty((w.B, w.H, w.P), dtype=torch.float32, device=dev)

    def timed(fn):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        ev[0].record(stream)
        for _ in range(args.stage_reps):
            for l in range(layers):
                fn(l)
        ev[1].record(stream)
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / (args.stage_reps * layers) * 1e3  # us per launch

    def f_score(l):
        q, k, v = data[l]
        nacl.score(prob, q, k, ws, out=outs[l][0])

    def f_pass2(l):
        q, k, v = data[l]
        nacl.score(prob, q, k, ws, lse=lse_ws, out=outs[l][0])

    def f_select(l):
        nacl.select(prob, outs[l][0], w.C, w.Cr, nacl.SAMPLE_SOFTMAX, w.rng_seed, l, ws=ws, out=outs[l][1])

    def f_compact(l):
        q, k, v = data[l]
        nacl.compact(prob, k, v, outs[l][1], k_out=outs[l][2], v_out=outs[l][3])

    # A finite log-sum-exp for the pass-2-only timing: 0 gives the same work.
    lse_ws.zero_()
    t_score = timed(f_score)
    t_pass2 = timed(f_pass2)
    t_select = timed(f_select)
    t_compact = timed(f_compact)
    step()  # restore the real outputs of every layer
    torch.cuda.synchronize()
    ab = alg_bytes(w)
    fl = alg_flops(w)
    peak_tf = F32_PEAK_TFLOPS if w.dtype == "f32" else BF16_PEAK_TFLOPS
    t_pass1 = t_score - t_pass2
    stages = {
        "score_pass1_combine_us": round(t_pass1, 2),
        "score_pass2_us": round(t_pass2, 2),
        "score_us": round(t_score, 2),
        "select_us": round(t_select, 2),
        "compact_us": round(t_compact, 2),
        "layer_us": round(ms_per_step / layers * 1e3, 2),
        "score_alg_GBps": round(ab["score"] / (t_score * 1e3), 1),
        "score_mfma_util_alg": round(fl / (t_score * 1e-6) / (peak_tf * 1e12), 4),
        "score_mfma_util_exec": round(2 * fl / (t_score * 1e-6) / (peak_tf * 1e12), 4),
        "pass2_mfma_util": round(fl / (t_pass2 * 1e-6) / (peak_tf * 1e12), 4),
        "select_alg_GBps": round(ab["select"] / (t_select * 1e3), 1),
        "compact_alg_GBps": round(ab["compact"] / (t_compact * 1e3), 1),
        "select_compact_hbm_frac": round((ab["select"] + ab["compact"]) /
                                         ((t_select + t_compact) * 1e3) / HBM_PEAK_GBS, 4),
    }
    log(f"[bench] stages {json.dumps(stages)}")

    # Dominant single kernel: the longest of pass 2 and compaction (pass 1 +
    # combine is two launches).
    if t_compact >= t_pass2:
        dom = {"kernel": "compact_kernel", "bound": "hbm", "us": t_compact,
               "achieved": ab["compact"] / (t_compact * 1e3), "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    else:
        dom = {"kernel": "score_pass2_kernel", "bound": "hbm", "us": t_pass2,
               "achieved": ab["score"] / (t_pass2 * 1e3), "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    traffic = None
    if MEASURED_TRAFFIC and MEASURED_TRAFFIC.get("kernel") == dom["kernel"] \
            and MEASURED_TRAFFIC.get("workload") == w.name:
        traffic = MEASURED_TRAFFIC["bytes_per_launch"]
    roofline = {"bound": dom["bound"], "achieved": round(dom["achieved"], 1), "peak": dom["peak"],
                "unit": dom["unit"], "frac": round(dom["achieved"] / dom["peak"], 4),
                "traffic": traffic, "kernel": dom["kernel"], "avg_us": round(dom["us"], 2)}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, data[0], args.cpu_heads)
        log(f"[bench] cpu baseline {json.dumps(cpu)}")

    line = {
        "metric": "prefill tokens/sec evicted per layer (32k ctx)",
        "value": round(tok_per_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded Gaussian Q/K/V with injected attention sinks and heavy hitters)",
        "config": {"workload": w.name, "layers": layers, "batch": w.B, "heads": w.H, "seq_len": w.L,
                   "head_dim": w.D, "proxies": w.P, "budget_C": w.C, "random_Cr": w.Cr,
                   "protected": w.n_protect, "sampling": "softmax", "parallelism": "single GPU"},
        "roofline": roofline,
        "stages": stages,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def cpu_baseline(w, layer0, n_heads):
    """The oracle, as it stands, on heads of batch row 0 of layer 0 (host
    copies of the GPU inputs).  tokens/s = L * n_heads / H / t: the rate at
    which it would evict one sequence's layer."""
    import numpy as np
    import torch
    from threadpoolctl import threadpool_info
    from oracle import evict as o_evict

    q, k, v = layer0
    n_heads = min(n_heads, w.H)
    qh = q[0:1, :n_heads].float().cpu().numpy()
    kh = k[0:1, :n_heads].float().cpu().numpy()
    vh = v[0:1, :n_heads].float().cpu().numpy()
    t0 = time.perf_counter()
    o_evict(qh, kh, vh, w.proxy_pos, w.n_protect, w.C, w.Cr, 0, w.rng_seed, 0, w.scale)
    dt = time.perf_counter() - t0
    blas = [i.get("num_threads") for i in threadpool_info() if i.get("user_api") == "blas"]
    threads = max(blas) if blas else 1
    return {"value": round(w.L * n_heads / w.H / dt, 1), "unit": "tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"layer 0, batch row 0, heads 0..{n_heads - 1} of {w.name} "
                      f"({n_heads}/{w.B * w.H} of one layer's heads), float64 NumPy, {dt:.1f}s",
            "host_cpus": len(os.sched_getaffinity(0))}


if __name__ == "__main__":
    main()
