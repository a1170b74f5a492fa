"""Benchmark of NaCl's one-shot encoding-phase KV-cache eviction on one MI355X.

One step = the eviction of every layer of the workload (score -> select ->
compact per layer; consecutive layers alternate between --streams HIP
streams, each with its own workspace, so one layer's selection and
compaction overlap the next layer's scoring), inputs resident in HBM.
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

# HBM traffic of the dominant kernel per launch, from two rocprofv3 --pmc runs
# (FETCH_SIZE, then WRITE_SIZE) scaled by the same counters on a plain copy of
# known size; summarised under profiles/.  It is reported only while the
# kernel source hashes to the value it was measured on.
MEASURED_TRAFFIC = {"workload": "prefill_32k", "kernel": "score_split_kernel", "bytes_per_launch": 2202688896,
                    "source_sha": "c0c0db1d43746326"}


def _source_sha(rel):
    import hashlib
    with open(os.path.join(ROOT, rel), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


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
    ap.add_argument("--streams", type=int, default=2, help="HIP streams the layers alternate between")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="run the CPU oracle on whole layers until this much time has passed")
    ap.add_argument("--probe", choices=["score", "select", "compact", "copy"],
                    help="run one kernel three times on layer 0 and exit (for rocprofv3 counter runs)")
    ap.add_argument("--pass-breakdown", action="store_true",
                    help="also time the score kernel's second pass alone (caller-supplied LSE)")
    ap.add_argument("--generation", action="store_true",
                    help="instead of the benchmark, time generation-phase re-eviction at decode shapes "
                         "(append m rows, evict the C + m cache back to C in place)")
    ap.add_argument("--prefill", action="store_true",
                    help="instead of the benchmark, time one layer of Appendix A.7's pipeline: the prefill "
                         "attention with its log-sum-exp, then the eviction fed with it (score in one pass), "
                         "beside the eviction that computes the log-sum-exp itself")
    ap.add_argument("--configs", action="store_true",
                    help="instead of the benchmark, print one JSON line per parity workload (GPU times, "
                         "score roofline fraction, oracle rate on a bounded sample of heads)")
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(eviction shards by head or batch, with no communication between GPUs)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2408_03675_amd import nacl
    from paper_2408_03675_amd.layer_loop import LayerLoop
    from synth import WORKLOADS, alg_bytes, alg_flops, make_layer

    if args.configs:
        run_configs()
        return
    if args.generation:
        run_generation(args.workload)
        return
    if args.prefill:
        run_prefill(args.workload)
        return
    w = WORKLOADS[args.workload]
    layers = args.layers or w.layers
    if args.probe:
        layers = 1
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
    prob = nacl.Problem.from_tensors(q0, k0, v0, w.proxy_pos, n_protect=w.n_protect, sm_scale=w.scale,
                                     proxy_pos_dev=pos_dev)
    loop = LayerLoop(prob, data, w.C, w.Cr, nacl.SAMPLE_SOFTMAX, w.rng_seed, streams=args.streams, device=dev)
    n_streams = len(loop.streams)
    ws = loop.workspaces[0]
    outs = loop.outs

    if args.probe:
        run_probe(args.probe, w, prob, ws, data[0], outs[0])
        return

    stream = torch.cuda.current_stream(dev)
    step = loop.run

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

    # Per-stage durations through the public entry points, timed with events
    # on the launch stream.  nacl_score = an init kernel (zeroes the work
    # queue counters) + the score kernel (score_split_kernel for bf16,
    # D = 128 and at least 128 proxies, else score_kernel); nacl_select =
    # gumbel_keys_kernel + select_kernel_regs (select_kernel_global past 32k
    # tokens); nacl_compact = compact_kernel.  Inside nacl_evict the score
    # kernel also draws the Gumbel keys and the key kernel is skipped.
    def timed(fn):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        ev[0].record(stream)
        for _ in range(args.stage_reps):
            for l in range(layers):
                fn(l)
        ev[1].record(stream)
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / (args.stage_reps * layers) * 1e3  # us per call

    def f_score(l):
        q, k, v = data[l]
        nacl.score(prob, q, k, ws, out=outs[l][0])

    def f_select(l):
        nacl.select(prob, outs[l][0], w.C, w.Cr, nacl.SAMPLE_SOFTMAX, w.rng_seed, l, ws=ws, out=outs[l][1])

    def f_compact(l):
        q, k, v = data[l]
        nacl.compact(prob, k, v, outs[l][1], k_out=outs[l][2], v_out=outs[l][3])

    t_score = timed(f_score)
    t_select = timed(f_select)
    t_compact = timed(f_compact)
    t_pass2 = None
    if args.pass_breakdown:
        lse0 = torch.zeros((w.B, w.H, w.P), dtype=torch.float32, device=dev)  # same work as any finite LSE

        def f_pass2(l):
            q, k, v = data[l]
            nacl.score(prob, q, k, ws, lse=lse0, out=outs[l][0])
        t_pass2 = timed(f_pass2)
    step()  # restore the real outputs of every layer
    torch.cuda.synchronize()
    # Sticky health words: every call since the workspaces were zeroed,
    # warm-up and timed steps included, completed its waits normally.
    status = loop.health()
    if status:
        raise RuntimeError(f"a kernel reported health bits {status:#x}; the timed results are invalid")
    ab = alg_bytes(w)
    fl = alg_flops(w)
    split = w.dtype == "bf16" and w.D == 128 and w.P >= 128
    passes = 2  # logit passes the kernel executes
    peak_tf = F32_PEAK_TFLOPS if w.dtype == "f32" else BF16_PEAK_TFLOPS
    stages = {
        "score_us": round(t_score, 2),
        "select_us": round(t_select, 2),
        "compact_us": round(t_compact, 2),
        "layer_us": round(ms_per_step / layers * 1e3, 2),
        "score_alg_GBps": round(ab["score"] / (t_score * 1e3), 1),
        "score_mfma_frac_alg": round(fl / (t_score * 1e-6) / (peak_tf * 1e12), 4),
        "score_mfma_frac_exec": round(passes * fl / (t_score * 1e-6) / (peak_tf * 1e12), 4),
        "select_alg_GBps": round(ab["select"] / (t_select * 1e3), 1),
        "compact_alg_GBps": round(ab["compact"] / (t_compact * 1e3), 1),
        "compact_hbm_frac": round(ab["compact"] / (t_compact * 1e3) / HBM_PEAK_GBS, 4),
        "select_compact_hbm_frac": round((ab["select"] + ab["compact"]) /
                                         ((t_select + t_compact) * 1e3) / HBM_PEAK_GBS, 4),
    }
    if t_pass2 is not None:
        stages["score_pass2_only_us"] = round(t_pass2, 2)
    log(f"[bench] stages {json.dumps(stages)}")

    # Dominant kernel: the score kernel.  Its roofline is HBM (algorithmic
    # intensity P flop/byte, below the bf16 ridge of ~312): algorithmic bytes
    # = K read once + proxy rows of Q + F written, per launch (one layer).
    kname = ("score_split_wide_kernel" if w.P >= 512 else "score_split_kernel") if split else "score_kernel"
    dom = {"kernel": kname, "bound": "hbm", "us": t_score,
           "achieved": ab["score"] / (t_score * 1e3), "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    traffic = None
    if MEASURED_TRAFFIC and MEASURED_TRAFFIC.get("workload") == w.name and \
            MEASURED_TRAFFIC.get("kernel") == dom["kernel"] and \
            MEASURED_TRAFFIC.get("source_sha") == _source_sha("paper_2408_03675_amd/csrc/score.hip"):
        traffic = MEASURED_TRAFFIC["bytes_per_launch"]
    roofline = {"bound": dom["bound"], "achieved": round(dom["achieved"], 1), "peak": dom["peak"],
                "unit": dom["unit"], "frac": round(dom["achieved"] / dom["peak"], 4),
                "traffic": traffic, "kernel": dom["kernel"], "avg_us": round(dom["us"], 2),
                "alg_bytes_per_launch": ab["score"]}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, data, args.cpu_seconds)
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
                   "protected": w.n_protect, "sampling": "softmax", "parallelism": "single GPU",
                   "streams": n_streams},
        "roofline": roofline,
        "stages": stages,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


def run_generation(name, m_steps=(16, 64, 256)):
    """Generation-phase eviction (Section 3; Algorithm 1, Generation) at decode
    shapes: the cache of one layer holds C kept entries per head plus m decoding
    steps; a round appends the m new K/V rows (nacl_append) and evicts the
    C + m cache back to C in place with the current token as the only proxy,
    in token order (nacl_evict) and in the slot form (nacl_evict_slots).
    Events around ten back-to-back rounds, median of three such runs; one JSON
    line per m."""
    import statistics
    import torch
    from paper_2408_03675_amd import nacl
    from synth import WORKLOADS

    w = WORKLOADS[name]
    dev = torch.device("cuda:0")
    nacl.load_library()
    g = torch.Generator(device=dev).manual_seed(5)
    dt = w.torch_dtype()
    for m in m_steps:
        L = w.C + m
        kc = torch.randn((w.B, w.H, L, w.D), generator=g, device=dev).to(dt)
        vc = torch.randn((w.B, w.H, L, w.D), generator=g, device=dev).to(dt)
        k_new = torch.randn((w.B, w.H, m, w.D), generator=g, device=dev).to(dt)
        v_new = torch.randn((w.B, w.H, m, w.D), generator=g, device=dev).to(dt)
        q_cur = torch.randn((w.B, w.H, 1, w.D), generator=g, device=dev).to(dt).expand(w.B, w.H, L, w.D)
        pos_dev = torch.tensor([L - 1], dtype=torch.int32, device=dev)
        prob = nacl.Problem.from_tensors(q_cur, kc, vc, [L - 1], n_protect=1, proxy_pos_dev=pos_dev)
        ws = nacl.workspace(prob, dev)
        F = torch.empty((w.B, w.H, L), dtype=torch.float32, device=dev)
        keep = torch.empty((w.B, w.H, w.C), dtype=torch.int32, device=dev)
        Cr = w.Cr
        stream = torch.cuda.current_stream(dev)

        def rnd(seed):
            nacl.append(prob, kc, vc, w.C, k_new, v_new)
            nacl.evict(prob, q_cur, kc, vc, w.C, Cr, nacl.SAMPLE_SOFTMAX, seed, 0, ws=ws, scores=F,
                       keep_idx=keep, in_place=True)

        def evict_only(seed):
            nacl.evict(prob, q_cur, kc, vc, w.C, Cr, nacl.SAMPLE_SOFTMAX, seed, 0, ws=ws, scores=F,
                       keep_idx=keep, in_place=True)

        # The slot form: kept rows stay in their slots, only the kept rows
        # among the m new ones move (nacl_evict_slots).
        slots = torch.empty((w.B, w.H, w.C), dtype=torch.int32, device=dev)

        def rnd_slots(seed):
            nacl.append(prob, kc, vc, w.C, k_new, v_new)
            nacl.evict_slots(prob, q_cur, kc, vc, w.C, Cr, nacl.SAMPLE_SOFTMAX, seed, 0, ws=ws, scores=F,
                             keep_idx=keep, slot_idx=slots)

        def evict_slots_only(seed):
            nacl.evict_slots(prob, q_cur, kc, vc, w.C, Cr, nacl.SAMPLE_SOFTMAX, seed, 0, ws=ws, scores=F,
                             keep_idx=keep, slot_idx=slots)

        def med(fn, reps=10, rounds=3):
            for i in range(3):
                fn(i)
            ts = []
            for r in range(rounds):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                torch.cuda.synchronize()
                e0.record(stream)
                for i in range(reps):
                    fn(100 + r * reps + i)
                e1.record(stream)
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1) * 1e3 / reps)
            return statistics.median(ts)
        t_round = med(rnd)
        t_evict = med(evict_only)
        t_round_s = med(rnd_slots)
        t_evict_s = med(evict_slots_only)
        if nacl.health(ws)[1]:
            raise RuntimeError("a kernel reported a health bit during the generation rounds")
        print(json.dumps({"metric": "generation-phase re-eviction round", "workload": name, "B": w.B, "H": w.H,
                          "D": w.D, "dtype": w.dtype, "C": w.C, "Cr": Cr, "m": m, "cache_rows": L,
                          "round_us": round(t_round, 2), "evict_in_place_us": round(t_evict, 2),
                          "append_us": round(t_round - t_evict, 2),
                          "us_per_decoding_step": round(t_round / m, 3),
                          "slot_form": {"round_us": round(t_round_s, 2), "evict_us": round(t_evict_s, 2),
                                        "us_per_decoding_step": round(t_round_s / m, 3)}}), flush=True)
        del kc, vc, k_new, v_new, F, keep, slots, ws
        torch.cuda.empty_cache()


def run_probe(which, w, prob, ws, layer0, out0):
    """Three launches of one kernel on layer 0, nothing else timed: the
    program rocprofv3 --pmc runs to read a kernel's HBM counters.  "copy" is
    the calibration: a plain 1 GiB device-to-device copy (1 GiB read, 1 GiB
    written per launch)."""
    import torch
    from paper_2408_03675_amd import nacl
    q, k, v = layer0
    F, keep, ko, vo = out0
    nacl.evict(prob, q, k, v, w.C, w.Cr, nacl.SAMPLE_SOFTMAX, w.rng_seed, 0, ws=ws, scores=F,
               keep_idx=keep, k_out=ko, v_out=vo)
    torch.cuda.synchronize()
    if which == "copy":
        src = torch.empty(1 << 30, dtype=torch.uint8, device=q.device)
        src.fill_(1)
        dst = torch.empty_like(src)
    for _ in range(3):
        if which == "score":
            nacl.score(prob, q, k, ws, out=F)
        elif which == "select":
            nacl.select(prob, F, w.C, w.Cr, nacl.SAMPLE_SOFTMAX, w.rng_seed, 0, ws=ws, out=keep)
        elif which == "compact":
            nacl.compact(prob, k, v, keep, k_out=ko, v_out=vo)
        else:
            dst.copy_(src)
    torch.cuda.synchronize()
    log(f"[bench] probe {which} done")


def run_prefill(name):
    """Appendix A.7's pipeline for one layer of a workload: nacl_attention
    (the causal prefill attention, which also returns each row's
    log-sum-exp and gathers the proxy rows'), then nacl_score with that
    log-sum-exp (the column reduction of Algorithm 2 alone: K read once),
    nacl_select and nacl_compact; beside it the eviction as the benchmark runs
    it (nacl_evict: two passes over K).  Events around three back-to-back
    calls, median of three such runs; one JSON line."""
    import statistics
    import torch
    from paper_2408_03675_amd import nacl
    from synth import WORKLOADS, make_layer

    w = WORKLOADS[name]
    dev = torch.device("cuda:0")
    nacl.load_library()
    q, k, v = make_layer(w, 0, device=dev)
    pos_dev = torch.tensor(w.proxy_pos, dtype=torch.int32, device=dev)
    prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos, n_protect=w.n_protect, sm_scale=w.scale,
                                     proxy_pos_dev=pos_dev)
    ws = nacl.workspace(prob, dev)
    Hq = w.H
    out = torch.empty_like(q)
    lse = torch.empty((w.B, Hq, w.L), dtype=torch.float32, device=dev)
    lp = torch.empty((w.B, Hq, w.P), dtype=torch.float32, device=dev)
    F = torch.empty((w.B, w.H, w.L), dtype=torch.float32, device=dev)
    keep = torch.empty((w.B, w.H, w.C), dtype=torch.int32, device=dev)
    ko = torch.empty((w.B, w.H, w.C, w.D), dtype=q.dtype, device=dev)
    vo = torch.empty_like(ko)

    def attention():
        nacl.attention(prob, q, k, v, out=out, lse=lse, lse_proxy=lp)

    def score_lse():
        nacl.score(prob, q, k, ws, lse=lp, out=F)

    def evict_lse():
        nacl.score(prob, q, k, ws, lse=lp, out=F)
        nacl.select(prob, F, w.C, w.Cr, nacl.SAMPLE_SOFTMAX, w.rng_seed, 0, ws=ws, out=keep)
        nacl.compact(prob, k, v, keep, k_out=ko, v_out=vo)

    def score_two_pass():
        nacl.score(prob, q, k, ws, out=F)

    def evict_two_pass():
        nacl.evict(prob, q, k, v, w.C, w.Cr, nacl.SAMPLE_SOFTMAX, w.rng_seed, 0, ws=ws, scores=F,
                   keep_idx=keep, k_out=ko, v_out=vo)

    def med(fn, reps=3, rounds=3):
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(rounds):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) / reps)
        return statistics.median(ts)

    t_att = med(attention)
    log(f"[prefill] attention {t_att:.3f} ms")
    t_sl, t_el = med(score_lse, 10), med(evict_lse, 10)
    t_s2, t_e2 = med(score_two_pass, 10), med(evict_two_pass, 10)
    flops = 4.0 * w.D * (w.L * (w.L + 1) / 2) * w.B * Hq
    print(json.dumps({
        "workload": name, "B": w.B, "H": w.H, "L": w.L, "D": w.D, "P": w.P, "C": w.C, "Cr": w.Cr,
        "attention_ms": round(t_att, 3),
        "attention_tflops": round(flops / t_att / 1e9, 1),
        "attention_mfma_frac": round(flops / t_att / 1e9 / 2500.0, 3),
        "score_with_lse_us": round(t_sl * 1e3, 1), "evict_with_lse_us": round(t_el * 1e3, 1),
        "score_two_pass_us": round(t_s2 * 1e3, 1), "evict_two_pass_us": round(t_e2 * 1e3, 1),
    }), flush=True)


def run_configs(oracle_seconds=5.0):
    """One JSON line per parity workload: nacl_evict and nacl_score times (events around ten
    back-to-back calls on one layer, median of three such rounds), the score kernel against its roofline (HBM below the ridge of the
    input dtype, MFMA above it, executed flops of both passes), and the oracle on the host on as
    many heads of the same inputs as fit in about oracle_seconds (at least one), scaled to the
    whole layer."""
    import statistics
    import torch
    from paper_2408_03675_amd import nacl
    from synth import WORKLOADS, alg_bytes, alg_flops, make_layer, sweep_workloads
    from oracle import evict as o_evict

    dev = torch.device("cuda:0")
    nacl.load_library()
    works = [WORKLOADS["small_f32"], WORKLOADS["longbench_4k"]] + sweep_workloads() + \
        [WORKLOADS["long_128k"], WORKLOADS["h2o_4k"], WORKLOADS["prefill_32k"]]
    cache = {}
    for w in works:
        key = (w.B, w.H, w.L, w.D, w.dtype, w.data_seed, w.inject, w.P)
        if key not in cache:
            cache.clear()
            torch.cuda.empty_cache()
            cache[key] = make_layer(w, 0, device=dev)
        q, k, v = cache[key]
        pos_dev = torch.tensor(w.proxy_pos, dtype=torch.int32, device=dev)
        prob = nacl.Problem.from_tensors(q, k, v, w.proxy_pos, n_protect=w.n_protect, sm_scale=w.scale,
                                         proxy_pos_dev=pos_dev)
        ws = nacl.workspace(prob, dev)
        stream = torch.cuda.current_stream(dev)

        def med_us(fn, reps=10, rounds=3):
            # Back-to-back calls between two events (as the benchmark's stage
            # timing), median over rounds of the per-call average.
            for _ in range(3):
                fn()
            ts = []
            for _ in range(rounds):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                torch.cuda.synchronize()
                e0.record(stream)
                for _ in range(reps):
                    fn()
                e1.record(stream)
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1) * 1e3 / reps)
            return statistics.median(ts)
        F = torch.empty((w.B, w.H, w.L), dtype=torch.float32, device=dev)
        t_ev = med_us(lambda: nacl.evict(prob, q, k, v, w.C, w.Cr, nacl.SAMPLE_SOFTMAX, w.rng_seed, 0, ws=ws))
        t_sc = med_us(lambda: nacl.score(prob, q, k, ws, out=F))
        elt = 4 if w.dtype == "f32" else 2
        ridge = (F32_PEAK_TFLOPS if w.dtype == "f32" else BF16_PEAK_TFLOPS) * 1e12 / (HBM_PEAK_GBS * 1e9)
        intensity = 2 * w.P * w.D / (w.D * elt)
        if intensity < ridge:
            bound, frac = "hbm", alg_bytes(w)["score"] / (t_sc * 1e3) / HBM_PEAK_GBS
        else:
            peak = F32_PEAK_TFLOPS if w.dtype == "f32" else BF16_PEAK_TFLOPS
            bound, frac = "mfma", 2 * alg_flops(w) / (t_sc * 1e6) / peak
        # The oracle on heads of batch row 0 (host copies of the same inputs).
        qh, kh, vh = (t[:1].float().cpu().numpy() for t in (q, k, v))
        n, spent = 0, 0.0
        while n < w.H and spent < oracle_seconds:
            h = n
            t0 = time.perf_counter()
            o_evict(qh[:, h:h + 1], kh[:, h:h + 1], vh[:, h:h + 1], w.proxy_pos, w.n_protect, w.C, w.Cr, 0,
                    w.rng_seed, 0, w.scale)
            spent += time.perf_counter() - t0
            n += 1
        per_head = spent / n
        line = {"workload": w.name, "B": w.B, "H": w.H, "L": w.L, "D": w.D, "P": w.P, "dtype": w.dtype,
                "C": w.C, "Cr": w.Cr, "evict_us": round(t_ev, 1), "score_us": round(t_sc, 1),
                "tokens_per_s": round(w.B * w.L / (t_ev * 1e-6), 1),
                "score_roofline": {"bound": bound, "frac": round(frac, 4)},
                "oracle_tokens_per_s": round(w.B * w.L / (per_head * w.B * w.H), 1),
                "oracle_sample": f"{n} of {w.B * w.H} heads, {spent:.1f} s"}
        print(json.dumps(line), flush=True)
        del ws, F, qh, kh, vh


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(w, data, seconds):
    """The oracle, as it stands, on whole layers of the same workload (host
    copies of the GPU inputs), layer after layer until `seconds` have passed
    (at least one layer).  tokens/s = B * L * layers done / time, the same
    per-layer rate as the GPU figure.  Also a one-thread run of the 4k
    LongBench-shaped layer (a per-core figure)."""
    from threadpoolctl import threadpool_info, threadpool_limits
    from oracle import evict as o_evict
    from synth import WORKLOADS, make_layer

    done, spent = 0, 0.0
    for l, (q, k, v) in enumerate(data):
        qh, kh, vh = (t.float().cpu().numpy() for t in (q, k, v))
        t0 = time.perf_counter()
        o_evict(qh, kh, vh, w.proxy_pos, w.n_protect, w.C, w.Cr, 0, w.rng_seed, l, w.scale)
        spent += time.perf_counter() - t0
        done += 1
        del qh, kh, vh
        if spent >= seconds:
            break
    blas = [i.get("num_threads") for i in threadpool_info() if i.get("user_api") == "blas"]
    threads = max(blas) if blas else 1
    # One thread on the 4k LongBench-shaped layer: the per-core figure.
    w2 = WORKLOADS["longbench_4k"]
    q2, k2, v2 = (t.float().numpy() for t in make_layer(w2, 0, device="cpu"))
    with threadpool_limits(limits=1):
        t0 = time.perf_counter()
        o_evict(q2, k2, v2, w2.proxy_pos, w2.n_protect, w2.C, w2.Cr, 0, w2.rng_seed, 0, w2.scale)
        t1 = time.perf_counter() - t0
    return {"value": round(w.B * w.L * done / spent, 1), "unit": "tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{done} whole layer(s) of {w.name} (all {w.B * w.H} heads each), float64 NumPy "
                      f"oracle, {spent:.1f} s; BLAS on {threads} threads, elementwise work single-threaded",
            "cpu_model": _cpu_model(),
            "host_cpus": len(os.sched_getaffinity(0)),
            "one_thread": {"workload": w2.name, "value": round(w2.B * w2.L / t1, 1), "unit": "tokens/s",
                           "cores": 1, "seconds": round(t1, 2)}}


if __name__ == "__main__":
    main()
