#!/usr/bin/env python3
"""Benchmark of the decode-step A/F operators on one MI355X.

A step is one interleaved A/F layer step of the Mixtral-shaped pipeline
workload (B = 256 decode tokens, 32/8 heads, D = 128, paged bf16 KV with
lognormal contexts of median 4096; top-2 of 8 SwiGLU experts, H = 4096,
I = 14336; M = 4 microbatches on two HIP streams): every microbatch's paged
GQA attention and its MoE FFN. The JSON line reports tokens/s of that step,
the roofline of its dominant kernel (the grouped gate/up GEMM, HBM-bound),
the oracle's CPU rate on a bounded sample, and per-operator throughput on the
other workloads (Qwen3-32B attention and dense SwiGLU, Mixtral MoE).

    python bench.py [--steps K] [--warmup W] [--gpus 1]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_HBM = 8.0e12      # B/s, MI355X HBM3E
PEAK_BF16 = 2.5e15     # flop/s, dense bf16 MFMA
METRIC = "attn-decode HBM GB/s & FFN bf16 TFLOPS vs peak; A/F layer-step tokens/s"
DOMINANT = "gemm_gate_up"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_gate_up_af_pipeline_traffic.json")
KERNEL_SOURCES = ["gemm.h", "gemm_dispatch.hip", "ffn_plan.h", "moe.hip"]


def _code_only(text):
    """C++ source without comments and whitespace, so that a comment edit does
    not mark the stored counter readings as stale."""
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    return re.sub(r"\s+", "", text)


def kernel_hash():
    """Hash of the dominant kernel's sources (code only), recorded with the
    counter readings in TRAFFIC_FILE."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2608_01891_amd", "csrc", f)) as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def parse():
    p = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-operators", action="store_true", help="skip the per-operator section")
    p.add_argument("--counters-pass", action="store_true",
                   help="only warm-up + steps of the layer step and a 1 GiB copy (for rocprofv3 --pmc)")
    p.add_argument("--prefill-counters-pass", action="store_true",
                   help="only the causal prefill attention at 2 x 4096 Qwen3-32B tokens, for rocprofv3 --pmc")
    p.add_argument("--ffn-counters-pass", action="store_true",
                   help="only the MFMA-bound FFN shapes (Qwen3 SwiGLU T=512, Mixtral MoE T=2048), for rocprofv3 --pmc")
    return p.parse_args()


def timed(fn, reps, stream=None):
    """Average ms of fn() over reps, HIP events on the current stream."""
    import torch
    s = stream or torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(s)
    for _ in range(reps):
        fn()
    e1.record(s)
    e1.synchronize()
    return e0.elapsed_time(e1) / reps


def warm_up(fn, warmup=3, warm_ms=30.0):
    """At least `warmup` untimed calls and `warm_ms` of back-to-back calls. The
    GPU's clocks rise over the first 10-20 ms of sustained load after an idle
    gap (Mixtral MoE T = 256 after a 2 s pause: 531 us per call with a 3-call
    warm-up, 502 us after 30 calls, 500 us after 100 or more)."""
    import torch
    t0 = time.perf_counter()
    n = 0
    while n < warmup or (time.perf_counter() - t0) * 1e3 < warm_ms:
        fn()
        n += 1
        if n % 4 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()


def timed_kernels(fn, reps, names, aflex, warmup=3, windows=3):
    """(ms per call without profiling events: the median of `windows` windows of
    `reps` calls after the warm-up above, {kernel: avg ms} from a separate
    profiled pass)."""
    warm_up(fn, warmup)
    ms = sorted(timed(fn, reps) for _ in range(windows))[windows // 2]
    aflex.profile_start(names)
    for _ in range(max(3, reps // 3)):
        fn()
    kp = aflex.profile_stop()
    return ms, {kname: round(v[1] / v[0], 5) for kname, v in kp.items()}


_SMI = {}


def smi_handle():
    """The first GPU's amdsmi handle, or None. amdsmi is initialised once per
    process and shut down at interpreter exit."""
    if "h" not in _SMI:
        _SMI["h"] = None
        try:
            import amdsmi
            amdsmi.amdsmi_init()
            import atexit
            atexit.register(amdsmi.amdsmi_shut_down)
            _SMI["h"] = amdsmi.amdsmi_get_processor_handles()[0]
        except Exception:
            pass
    return _SMI["h"]


def energy_reader():
    """Callable returning (accumulated energy in J, the counter's own timestamp
    in s) for the GPU, or None. The counter advances in bursts, so energy is
    divided by the counter's timestamps, not by the host's clock."""
    h = smi_handle()
    if h is None:
        return None
    try:
        import amdsmi

        def read():
            e = amdsmi.amdsmi_get_energy_count(h)
            acc = e.get("energy_accumulator", e.get("power"))
            return float(acc) * float(e["counter_resolution"]) * 1e-6, float(e["timestamp"]) * 1e-9
        read()
        return read
    except Exception:
        return None


def steady_power(fn, read_energy, secs=4.0):
    """Average board power (W) while fn() is issued back to back: the energy
    counter is read twice inside the busy period, 1 s after its start and 1 s
    before its end, and the energy between the two readings is divided by the
    time between the counter's own timestamps. The host keeps at most ~40
    calls queued."""
    import torch
    ev, s0, s1, n = [], None, None, 0
    t0 = time.perf_counter()
    while True:
        fn()
        n += 1
        if n % 20 == 0:
            e = torch.cuda.Event()
            e.record()
            ev.append(e)
            if len(ev) > 2:
                ev.pop(0).synchronize()
        el = time.perf_counter() - t0
        if s0 is None and el >= 1.0:
            s0 = read_energy()
        if s1 is None and el >= secs - 1.0:
            s1 = read_energy()
        if el >= secs:
            break
    torch.cuda.synchronize()
    return (s1[0] - s0[0]) / (s1[1] - s0[1]) if s1[1] > s0[1] else float("nan")


def energy_of(fn, tokens, read_energy):
    """J/token and board power of fn() run back to back (tokens per call)."""
    ms_each = timed(fn, 10)
    watts = steady_power(fn, read_energy)
    return {"J_per_token": round(watts * ms_each * 1e-3 / tokens, 6),
            "avg_watts": round(watts, 1), "ms_per_call": round(ms_each, 4)}


def cpu_model():
    """The host CPU's model name (/proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def host_cores():
    """Logical CPUs this process may run on and the host's physical cores
    (distinct (socket, core) pairs in /proc/cpuinfo)."""
    out = {"logical_cpus_available": len(os.sched_getaffinity(0))}
    try:
        pairs, phys = set(), None
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("physical id"):
                    phys = line.split(":", 1)[1].strip()
                elif line.startswith("core id"):
                    pairs.add((phys, line.split(":", 1)[1].strip()))
        if pairs:
            out["physical_cores_host"] = len(pairs)
    except OSError:
        pass
    return out


def clock_reader():
    """Callable returning the graphics clock amdsmi reports, in MHz, or None."""
    h = smi_handle()
    if h is None:
        return None
    try:
        import amdsmi

        def read():
            c = amdsmi.amdsmi_get_clock_info(h, amdsmi.AmdSmiClkType.GFX)
            return float(c.get("clk", c.get("cur_clk")))
        read()
        return read
    except Exception:
        return None


def topk_ids_host(logits, k):
    import numpy as np
    return np.argsort(-logits, axis=1, kind="stable")[:, :k]


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the decode-step operators are built and timed on a "
              "single MI355X (run with --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_01891_amd import aflex, plan, synth

    aflex.load()  # fails loudly if the HIP library is not built
    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    dev = "cuda:0"
    torch.cuda.set_device(0)

    # ---------------- the headline step: interleaved A/F layer step ----------------
    wl = synth.af_pipeline(device=dev)
    a, f, logits = wl.attn, wl.ffn, wl.router_logits
    mbs = wl.microbatches
    B, H, I, k = a.B, f.H, f.I, wl.top_k
    y = torch.empty(B, H, dtype=torch.bfloat16, device=dev)
    sa, sf = aflex.pipeline_streams(dev)
    pws = aflex.Workspace()

    def step(m=mbs):
        aflex.af_pipeline_step(a, f, logits, k, m, y=y, stream_a=sa, stream_f=sf, ws=pws, join=False)

    if args.prefill_counters_pass:
        pw = synth.prefill_workload("qwen3-32b", 4096, 2, device=dev)
        outp = aflex.attn_prefill(pw)
        for _ in range(3):
            aflex.attn_prefill(pw, out=outp)
        torch.cuda.synchronize()
        print("prefill counters pass: 2 x 4096 done", flush=True)
        print(json.dumps({"prefill_counters_pass": True}))
        return

    if args.ffn_counters_pass:
        # Counter collection for the MFMA-bound FFN GEMMs: a few calls of each shape.
        wd = synth.make_ffn_weights(2, 5120, 25600, device=dev)
        w512 = synth.qwen3_swiglu(512, device=dev, weights=wd)
        for _ in range(3):
            aflex.ffn_swiglu(w512.x, wd)
        torch.cuda.synchronize()
        print("ffn counters pass: dense SwiGLU T=512 done", flush=True)
        del wd
        w2k = synth.mixtral_moe(device=dev, T=2048, seed=103, weights=f)
        for _ in range(3):
            aflex.moe_ffn(w2k.x, w2k.ffn, w2k.router_logits, 2)
        torch.cuda.synchronize()
        print("ffn counters pass: MoE T=2048 done", flush=True)
        print(json.dumps({"ffn_counters_pass": True}))
        return

    if args.counters_pass:
        # Counter collection serialises dispatches; it runs the FFN stage's kernels
        # at the pipeline's microbatch shape on one stream (no cross-stream waits),
        # then a 1 GiB device copy that calibrates the counters.
        ws1 = aflex.Workspace()
        out = torch.empty(a.B, a.Hq, a.D, dtype=torch.bfloat16, device=dev)
        off = 0
        for n in mbs:
            am = synth.AttnInputs(q=a.q[off:off + n], k_cache=a.k_cache, v_cache=a.v_cache,
                                  block_table=a.block_table[off:off + n],
                                  context_lens=a.context_lens[off:off + n], B=n, Hq=a.Hq,
                                  Hkv=a.Hkv, D=a.D, block_size=16, max_blocks=a.max_blocks,
                                  num_blocks=a.num_blocks, max_context_len=a.max_context_len)
            aflex.attn_decode(am, out=out[off:off + n], ws=ws1)
            for _ in range(args.steps):
                aflex.moe_ffn(out[off:off + n].view(n, H), f, logits[off:off + n], k,
                              y=y[off:off + n], ws=ws1)
            off += n
            print(f"counters pass: microbatch of {n} done", flush=True)
        src = torch.empty(1 << 29, dtype=torch.int16, device=dev)  # 1 GiB
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"counters_pass": True, "steps": args.steps, "copy_bytes": 2 * src.numel()}))
        return

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_step = (t1 - t0) * 1e3 / args.steps

    # same steps again with HIP events around the dominant kernel on its stream
    STAGE_A = ("attn_decode", "attn_merge")
    STAGE_F = ("moe_route", DOMINANT, "gemm_down", "moe_combine")
    aflex.profile_start(list(STAGE_A + STAGE_F))
    t2 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t3 = time.perf_counter()
    prof = aflex.profile_stop()
    ms_step_ev = (t3 - t2) * 1e3 / args.steps

    lg = logits.cpu().numpy()
    ctx = a.context_lens.cpu().numpy().astype(np.int64)
    kv_bytes_total = int(ctx.sum()) * a.Hkv * a.D * 2 * 2
    w_bytes_expert = 3 * I * H * 2
    # algorithmic bytes of the gate/up GEMM per launch: touched experts' W_g and
    # W_u, the microbatch's x rows, and the bf16 h rows it writes
    gate_bytes, gate_flops, step_bytes = [], [], kv_bytes_total
    off = 0
    for n in mbs:
        ids = topk_ids_host(lg[off:off + n], k)
        touched = len(np.unique(ids))
        gate_bytes.append(touched * 2 * I * H * 2 + n * H * 2 + n * k * I * 2)
        gate_flops.append(n * k * 2 * 2 * H * I)
        step_bytes += touched * w_bytes_expert + n * H * 2 * 2
        off += n
    n_launch, tot_ms, mn_ms, mx_ms = prof[DOMINANT]
    avg_ms = tot_ms / n_launch
    gate_avg_bytes = sum(gate_bytes) / len(gate_bytes)
    achieved = gate_avg_bytes / (avg_ms * 1e-3)

    # The same kernel at the same shapes with nothing else on the GPU: each
    # microbatch's FFN alone on one stream (what sharing HBM with the
    # attention stream costs the dominant kernel inside the step).
    alone_ws = aflex.Workspace()
    alone_y = torch.empty_like(y)

    def ffn_alone():
        o = 0
        for n in mbs:
            aflex.moe_ffn(y[o:o + n], f, logits[o:o + n], k, y=alone_y[o:o + n], ws=alone_ws)
            o += n

    ffn_alone()
    torch.cuda.synchronize()
    aflex.profile_start([DOMINANT])
    for _ in range(max(3, args.steps // 4)):
        ffn_alone()
    torch.cuda.synchronize()
    alone = aflex.profile_stop()[DOMINANT]
    alone_ms = alone[1] / alone[0]
    standalone = {"avg_launch_ms": round(alone_ms, 5),
                  "achieved": round(gate_avg_bytes / (alone_ms * 1e-3) / 1e9, 1),
                  "frac": round(gate_avg_bytes / (alone_ms * 1e-3) / PEAK_HBM, 4),
                  "note": "same kernel and microbatch shapes, each microbatch's FFN alone on one stream"}

    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as fh:
            tf = json.load(fh)
        if tf.get("kernel_hash") == kernel_hash():
            traffic = tf.get("bytes_per_launch")

    result = {
        "metric": METRIC,
        "value": round(B / (ms_step * 1e-3), 1),
        "unit": "tok/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "timing": "wall clock over the K timed steps between two device synchronisations, "
                  "after W untimed warm-up steps; value = 256 tokens x K / that time",
        "config": {"workload": "af-pipeline: Mixtral-8x7B-shaped decode layer step, B=256, "
                               "32/8 heads x 128, paged bf16 KV (block 16, lognormal ctx median 4096, "
                               "sum 1392790 tokens), top-2 of 8 SwiGLU experts H=4096 I=14336, "
                               "M=4 microbatches of 64 on 2 HIP streams, L=1",
                   "global_batch": B, "microbatches": mbs, "kv_bytes": kv_bytes_total,
                   "step_algorithmic_bytes": step_bytes,
                   "step_hbm_fraction": round(step_bytes / (ms_step * 1e-3) / PEAK_HBM, 4)},
        "roofline": {"kernel": DOMINANT, "bound": "hbm", "achieved": round(achieved / 1e9, 1),
                     "peak": PEAK_HBM / 1e9, "unit": "GB/s", "frac": round(achieved / PEAK_HBM, 4),
                     "traffic": traffic, "bytes_per_launch": int(gate_avg_bytes),
                     "avg_launch_ms": round(avg_ms, 5), "launches": n_launch,
                     "min_launch_ms": round(mn_ms, 5), "max_launch_ms": round(mx_ms, 5),
                     "ms_per_step_with_events": round(ms_step_ev, 4),
                     "kernel_hash": kernel_hash(), "standalone": standalone},
    }
    result["kernels_in_step"] = {kname: {"launches": v[0], "avg_ms": round(v[1] / v[0], 5)}
                                 for kname, v in prof.items()}
    # Busy fraction of each stage's stream over the step (kernel time per step /
    # step time measured with the same events): the single-GPU analogue of the
    # paper's A/F idle time (section 3.3), with both stages sharing one GPU.
    steps_ev = args.steps
    busy = {}
    for stage, names in (("attention_stream", STAGE_A), ("ffn_stream", STAGE_F)):
        ms_k = sum(prof[n][1] for n in names if n in prof) / steps_ev
        busy[stage] = {"kernel_ms_per_step": round(ms_k, 4), "busy_fraction": round(ms_k / ms_step_ev, 4)}
    result["stage_busy"] = busy

    # Plain device-to-device copy of 4 GiB (2 GiB read + 2 GiB written): the
    # achievable-HBM reference of this run, next to the 8 TB/s nameplate.
    src = torch.empty(1 << 30, dtype=torch.int16, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    ms_copy = timed(lambda: dst.copy_(src), 5)
    # A read-dominated reference: the vendor BLAS matrix-vector product over the
    # same 2 GiB viewed as a [262144, 4096] bf16 matrix.
    mat = src.view(torch.bfloat16).view(-1, 4096)
    vec = torch.ones(4096, dtype=torch.bfloat16, device=dev)
    torch.mv(mat, vec)
    ms_mv = timed(lambda: torch.mv(mat, vec), 5)
    result["hbm_reference"] = {"copy_GB_per_s": round(4 * (1 << 30) / (ms_copy * 1e-3) / 1e9, 1),
                               "gemv_read_GB_per_s": round(2 * (1 << 30) / (ms_mv * 1e-3) / 1e9, 1),
                               "note": "read + write bytes of a 2 GiB device copy / time; bytes of a "
                                       "2 GiB bf16 matrix read by torch.mv / time"}
    del src, dst, mat, vec

    # ---------------- energy per token (where the counter is readable) -------------
    read_energy = energy_reader()
    read_clock = clock_reader()
    if read_energy is not None:
        watts = steady_power(step, read_energy)
        clocks = []
        if read_clock is not None:  # sampled while queued steps run
            for _ in range(8):
                step()
            for _ in range(10):
                time.sleep(0.002)
                clocks.append(read_clock())
            torch.cuda.synchronize()
        result["energy"] = {"joules_per_token": round(watts * ms_step * 1e-3 / B, 6),
                            "avg_watts": round(watts, 1),
                            "method": "board power in steady state (energy counter and its timestamps "
                                      "read twice inside 4 s of back-to-back steps) x measured step "
                                      "time / tokens"}
        if clocks:
            # amdsmi reports the clock set for the graphics domain, not the
            # clock the CUs run at under this load; the counter-derived clock
            # (GRBM_GUI_ACTIVE cycles over kernel time) is in the profiles.
            result["energy"]["amdsmi_set_gfx_clock_mhz"] = {
                "min": min(clocks), "max": max(clocks), "mean": round(sum(clocks) / len(clocks), 1),
                "note": "set clock as amdsmi reports it; the counters measure 1.7-2.1 GHz under this load"}
    else:
        result["energy"] = "n/a (energy counter not readable)"

    # ---------------- pipeline variants and Eq. 2 comparison -------------------------
    if not args.no_operators:
        ops = {}
        # The Mixtral MoE T = 256 line's inputs and expert weights are allocated
        # here, before the operator lines allocate and free their own tensors:
        # the same weights allocated at the line itself, after that churn, ran
        # 5% slower (533 against 505-509 us per call in one run, the early copy
        # timed at three points of the run), as a serving process loads its
        # weights once at start.
        wm256 = synth.mixtral_moe(device=dev, T=256, seed=3)
        variants = {}
        for M in (1, 2, 4):
            m = plan.equal_microbatches(B, M)
            step(m)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(args.steps):
                step(m)
            torch.cuda.synchronize()
            ms = (time.perf_counter() - t0) * 1e3 / args.steps
            variants[f"M={M}"] = {"ms": round(ms, 4), "tok_per_s": round(B / (ms * 1e-3), 1)}
        # standalone stage times per microbatch (one stream, no overlap)
        t_a = t_f = 0.0
        off = 0
        x_mb = torch.empty(64, H, dtype=torch.bfloat16, device=dev)
        for n in mbs:
            am = synth.AttnInputs(q=a.q[off:off + n], k_cache=a.k_cache, v_cache=a.v_cache,
                                  block_table=a.block_table[off:off + n],
                                  context_lens=a.context_lens[off:off + n], B=n, Hq=a.Hq, Hkv=a.Hkv,
                                  D=a.D, block_size=16, max_blocks=a.max_blocks,
                                  num_blocks=a.num_blocks, max_context_len=a.max_context_len)
            out = torch.empty(n, a.Hq, a.D, dtype=torch.bfloat16, device=dev)
            warm_up(lambda: aflex.attn_decode(am, out=out))
            t_a += timed(lambda: aflex.attn_decode(am, out=out), 5)
            xm = out.view(n, H)
            lm = logits[off:off + n]
            warm_up(lambda: aflex.moe_ffn(xm, f, lm, k, y=x_mb[:n]))
            t_f += timed(lambda: aflex.moe_ffn(xm, f, lm, k, y=x_mb[:n]), 5)
            off += n
        variants["standalone_sum_ms"] = {"attention": round(t_a, 4), "ffn": round(t_f, 4),
                                         "serial": round(t_a + t_f, 4)}
        # energy per token of each operator alone (the last microbatch, back to
        # back for about a second each): the single-GPU view of DA against DF
        if read_energy is not None:
            variants["energy_per_operator"] = {
                "attention_microbatch": energy_of(lambda: aflex.attn_decode(am, out=out), n, read_energy),
                "moe_ffn_microbatch": energy_of(lambda: aflex.moe_ffn(xm, f, lm, k, y=x_mb[:n]), n, read_energy)}
        variants["eq2_ms"] = {"M=1": round(plan.eq2_layer_time(t_a, t_f, 0.0, 1), 4),
                              "M=4": round(plan.eq2_layer_time(t_a, t_f, 0.0, 4), 4)}
        variants["byte_roofline_ms"] = round(step_bytes / PEAK_HBM * 1e3, 4)
        # dynamic microbatch depth + adaptive request batching: Eq. 2 over the
        # stage curves profiled here, and the measured layer time of each split
        prof_a, prof_f = {}, {}

        def stage_times(n):
            if n not in prof_a:
                am = synth.AttnInputs(q=a.q[:n], k_cache=a.k_cache, v_cache=a.v_cache,
                                      block_table=a.block_table[:n], context_lens=a.context_lens[:n],
                                      B=n, Hq=a.Hq, Hkv=a.Hkv, D=a.D, block_size=16,
                                      max_blocks=a.max_blocks, num_blocks=a.num_blocks,
                                      max_context_len=a.max_context_len)
                o = torch.empty(n, a.Hq, a.D, dtype=torch.bfloat16, device=dev)
                warm_up(lambda: aflex.attn_decode(am, out=o))
                prof_a[n] = timed(lambda: aflex.attn_decode(am, out=o), 3)
                yv = torch.empty(n, H, dtype=torch.bfloat16, device=dev)
                warm_up(lambda: aflex.moe_ffn(o.view(n, H), f, logits[:n], k, y=yv))
                prof_f[n] = timed(lambda: aflex.moe_ffn(o.view(n, H), f, logits[:n], k, y=yv), 3)
            return prof_a[n], prof_f[n]

        def measured(m):
            step(m)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(5):
                step(m)
            torch.cuda.synchronize()
            return (time.perf_counter() - t0) * 1e3 / 5
        cands = plan.candidate_splits(B)
        eq2_best, eq2_ms = plan.choose_split(
            cands, lambda m: plan.eq2_predict(m, lambda n: stage_times(n)[0], lambda n: stage_times(n)[1]))
        meas = {tuple(m): measured(m) for m in cands}
        best = min(meas, key=meas.get)
        variants["planner"] = {
            "candidates_ms": {"+".join(map(str, m)): round(v, 4) for m, v in meas.items()},
            "eq2_choice": "+".join(map(str, eq2_best)), "eq2_predicted_ms": round(eq2_ms, 4),
            "eq2_choice_measured_ms": round(meas[tuple(eq2_best)], 4),
            "measured_choice": "+".join(map(str, best)), "measured_ms": round(meas[best], 4),
            "measured_tok_per_s": round(B / (meas[best] * 1e-3), 1)}
        variants["t_F_over_t_A"] = round(t_f / t_a, 3)
        # A and F pools on one GPU: the two stages' streams on disjoint CU sets
        pools = {}
        ppws = aflex.Workspace()  # used on the pool streams only, freed before they are released
        for acu in (64, 128, 192):
            pa, pf = aflex.pool_streams(acu, dev)
            for M in (2, 4):
                m = plan.equal_microbatches(B, M)

                def pstep():
                    aflex.af_pipeline_step(a, f, logits, k, m, y=y, stream_a=pa, stream_f=pf, ws=ppws, join=False)
                pstep()
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                for _ in range(5):
                    pstep()
                torch.cuda.synchronize()
                pms = (time.perf_counter() - t0) * 1e3 / 5
                pools[f"attn_cus={acu},M={M}"] = {"ms": round(pms, 4), "tok_per_s": round(B / (pms * 1e-3), 1)}
        variants["cu_pools"] = pools
        ppws.buf = None
        aflex.release_pool_streams()
        ops["af_pipeline"] = variants

        # The whole decode layer on the two streams (section 4.3): KV append,
        # attention and output projection (+ the layer input) on the attention
        # stream, RMSNorm, router, experts and residual on the FFN stream. The
        # append writes each sequence's new token into the workload's pools
        # (the same draws' shapes; later sections only time kernels on them).
        lw = synth.make_layer(40, B, a.Hq, a.Hkv, a.D, H, f.E, device=dev)
        ly = torch.empty(B, H, dtype=torch.bfloat16, device=dev)
        lws = aflex.Workspace()
        layer_ops = {}
        for M in (1, 4):
            m = plan.equal_microbatches(B, M)

            def lstep():
                aflex.af_layer_step(a, f, lw, k, m, y=ly, stream_a=sa, stream_f=sf, ws=lws, join=False)
            lstep()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(args.steps):
                lstep()
            torch.cuda.synchronize()
            ms = (time.perf_counter() - t0) * 1e3 / args.steps
            # algorithmic bytes: the pipeline step's, plus W_o once per
            # microbatch, the router and norm weights, the layer input, h and y
            lbytes = (step_bytes if M == 4 else kv_bytes_total + 8 * w_bytes_expert + B * H * 4) \
                + M * (lw.w_o.numel() * 2 + lw.router_weight.numel() * 2 + H * 2) + 3 * B * H * 2
            layer_ops[f"M={M}"] = {"ms": round(ms, 4), "tok_per_s": round(B / (ms * 1e-3), 1),
                                   "GB_per_s": round(lbytes / (ms * 1e-3) / 1e9, 1),
                                   "hbm_frac": round(lbytes / (ms * 1e-3) / PEAK_HBM, 4)}
        layer_ops["note"] = ("KV append, attention, o_proj [4096 x 4096] + layer input | RMSNorm, "
                             "router, top-2 MoE, residual; the pipeline workload's shapes")
        ops["af_decode_layer"] = layer_ops
        del lw, ly, lws

        # Tiny decoder layer (B=4, 8/2 heads x 64, SwiGLU 512 -> 1408): cache-resident,
        # so its lines are latencies
        wt = synth.tiny_layer(device=dev)
        ot = aflex.attn_decode(wt.attn)
        yt = aflex.ffn_swiglu(wt.x, wt.ffn)
        ms_a, kk_a = timed_kernels(lambda: aflex.attn_decode(wt.attn, out=ot), 50, ["attn_decode", "attn_merge"], aflex)
        ms_f, kk_f = timed_kernels(lambda: aflex.ffn_swiglu(wt.x, wt.ffn, y=yt), 50,
                                   ["gemm_gate_up", "gemm_down", "splitk_reduce"], aflex)
        ops["tiny_layer"] = {"attention_ms": round(ms_a, 5), "swiglu_ms": round(ms_f, 5),
                             "attention_kernels": kk_a, "swiglu_kernels": kk_f}
        del wt, ot, yt

        # Qwen3-32B decode attention, 3 KV-pool copies rotated so the 256 MB MALL cannot hold them
        wq = synth.qwen3_attention(device=dev).attn
        copies = [wq] + [synth.AttnInputs(**{**wq.__dict__, "k_cache": wq.k_cache.clone(),
                                            "v_cache": wq.v_cache.clone()}) for _ in range(2)]
        outq = torch.empty(wq.B, wq.Hq, wq.D, dtype=torch.bfloat16, device=dev)
        cq = wq.context_lens.cpu().numpy().astype(np.int64)
        abytes = (int(cq.sum()) * wq.Hkv * wq.D * 2 * 2 + 2 * wq.B * wq.Hq * wq.D * 2
                  + int(((cq + 15) // 16).sum()) * 4 + wq.B * 4)
        aflops = 4 * int(cq.sum()) * wq.Hq * wq.D
        it = [0]

        def run_attn():
            aflex.attn_decode(copies[it[0] % 3], out=outq)
            it[0] += 1
        for _ in range(3):
            run_attn()
        ms, kk = timed_kernels(run_attn, 30, ["attn_decode", "attn_merge"], aflex)
        ops["attention_qwen3_B64"] = {
            "ms": round(ms, 5), "GB_per_s": round(abytes / (ms * 1e-3) / 1e9, 1),
            "hbm_frac": round(abytes / (ms * 1e-3) / PEAK_HBM, 4), "bytes": abytes,
            "tflops": round(aflops / (ms * 1e-3) / 1e12, 2), "tok_per_s": round(wq.B / (ms * 1e-3), 1),
            "kernels": kk}
        # The whole attention stage of a Qwen3 decode layer: KV append of the new
        # token, attention, output projection [64, 8192] x [5120, 8192]^T.
        kn = synth.normal_tensor(1, 40, (wq.B, wq.Hkv, wq.D), device=dev)
        vn = synth.normal_tensor(1, 41, (wq.B, wq.Hkv, wq.D), device=dev)
        # three copies of W_o (84 MB each) rotate with the KV pools, so the 256 MB
        # last-level cache cannot serve the projection's weights from the previous call
        w_os = [synth.normal_tensor(1, 42, (5120, wq.Hq * wq.D), scale=0.02, device=dev) for _ in range(3)]
        w_o = w_os[0]
        y_o = torch.empty(wq.B, 5120, dtype=torch.bfloat16, device=dev)
        it[0] = 0

        def run_stage():
            c = copies[it[0] % 3]
            aflex.kv_append(c, kn, vn)
            aflex.attn_decode(c, out=outq)
            aflex.linear(outq.view(wq.B, -1), w_os[it[0] % 3], y=y_o)
            it[0] += 1
        for _ in range(3):
            run_stage()
        ms, kk = timed_kernels(run_stage, 30, ["kv_append", "attn_decode", "attn_merge", "gemm_down", "splitk_reduce"], aflex)
        sbytes = abytes + w_o.numel() * 2 + 2 * wq.B * 5120 * 2 + 2 * kn.numel() * 2
        ops["attention_stage_qwen3_B64"] = {
            "ms": round(ms, 5), "GB_per_s": round(sbytes / (ms * 1e-3) / 1e9, 1),
            "hbm_frac": round(sbytes / (ms * 1e-3) / PEAK_HBM, 4), "bytes": sbytes,
            "tok_per_s": round(wq.B / (ms * 1e-3), 1),
            "kernels": kk}
        del copies, wq, w_o, w_os

        # Full-batch long-context attention of the pipeline workload
        outl = torch.empty(B, a.Hq, a.D, dtype=torch.bfloat16, device=dev)
        warm_up(lambda: aflex.attn_decode(a, out=outl))
        ms = timed(lambda: aflex.attn_decode(a, out=outl), 10)
        lbytes = kv_bytes_total + 2 * B * a.Hq * a.D * 2
        ops["attention_longctx_B256"] = {"ms": round(ms, 5),
                                         "GB_per_s": round(lbytes / (ms * 1e-3) / 1e9, 1),
                                         "hbm_frac": round(lbytes / (ms * 1e-3) / PEAK_HBM, 4)}

        # Qwen3-32B dense SwiGLU, T in {32, 128, 256, 512}
        wd = synth.make_ffn_weights(2, 5120, 25600, device=dev)
        for T in (32, 128, 256, 512):
            wlT = synth.qwen3_swiglu(T, device=dev, weights=wd)
            yT = torch.empty(T, 5120, dtype=torch.bfloat16, device=dev)
            aflex.ffn_swiglu(wlT.x, wd, y=yT)
            ms, kk = timed_kernels(lambda: aflex.ffn_swiglu(wlT.x, wd, y=yT), 10, ["gemm_gate_up", "gemm_down", "splitk_reduce"], aflex)
            flops = 6 * T * 5120 * 25600
            byts = 3 * 5120 * 25600 * 2 + 2 * T * 5120 * 2
            att = min(PEAK_BF16, flops / byts * PEAK_HBM)
            ops[f"swiglu_qwen3_T{T}"] = {
                "ms": round(ms, 5), "tflops": round(flops / (ms * 1e-3) / 1e12, 1),
                "mfma_frac": round(flops / (ms * 1e-3) / PEAK_BF16, 4),
                "attainable_frac": round(flops / (ms * 1e-3) / att, 4),
                "GB_per_s": round(byts / (ms * 1e-3) / 1e9, 1),
                "hbm_frac": round(byts / (ms * 1e-3) / PEAK_HBM, 4),
                "tok_per_s": round(T / (ms * 1e-3), 1),
                "kernels": kk}
        del wd

        # Mixtral MoE, T = 256 (and T = 2048 supplementary)
        for T, seed in ((256, 3), (2048, 103)):
            wm = wm256 if T == 256 else synth.mixtral_moe(device=dev, T=T, seed=seed, weights=f)
            yT = torch.empty(T, H, dtype=torch.bfloat16, device=dev)
            aflex.moe_ffn(wm.x, wm.ffn, wm.router_logits, 2, y=yT)
            ms, kk = timed_kernels(lambda: aflex.moe_ffn(wm.x, wm.ffn, wm.router_logits, 2, y=yT), 10, None, aflex)
            ids = topk_ids_host(wm.router_logits.cpu().numpy(), 2)
            touched = len(np.unique(ids))
            flops = T * 2 * 6 * H * I
            byts = touched * w_bytes_expert + 2 * T * H * 2
            att = min(PEAK_BF16, flops / byts * PEAK_HBM)
            ops[f"moe_mixtral_T{T}"] = {
                "ms": round(ms, 5), "tflops": round(flops / (ms * 1e-3) / 1e12, 1),
                "mfma_frac": round(flops / (ms * 1e-3) / PEAK_BF16, 4),
                "attainable_frac": round(flops / (ms * 1e-3) / att, 4),
                "GB_per_s": round(byts / (ms * 1e-3) / 1e9, 1),
                "hbm_frac": round(byts / (ms * 1e-3) / PEAK_HBM, 4),
                "tok_per_s": round(T / (ms * 1e-3), 1),
                "kernels": kk}
            if T == 256:
                # the whole MoE FFN block: RMSNorm, router GEMM, experts, residual
                gamma = (1.0 + 0.1 * synth.normal_tensor(seed, 50, (H,), dtype=torch.float32,
                                                         device=dev)).to(torch.bfloat16)
                wr = synth.normal_tensor(seed, 51, (8, H), scale=0.02, device=dev)
                aflex.moe_block(wm.x, wm.ffn, gamma, wr, 2, residual=True, y=yT)
                ms_b, kk = timed_kernels(lambda: aflex.moe_block(wm.x, wm.ffn, gamma, wr, 2, residual=True,
                                                     y=yT), 10, ["rmsnorm_router"], aflex)
                ops["moe_block_mixtral_T256"] = {
                    "ms": round(ms_b, 5), "GB_per_s": round(byts / (ms_b * 1e-3) / 1e9, 1),
                    "hbm_frac": round(byts / (ms_b * 1e-3) / PEAK_HBM, 4),
                    "tok_per_s": round(T / (ms_b * 1e-3), 1),
                    "kernels": kk}
            del wm
        del wm256

        # Prefill (the paper's PA and PF operators, section 3.2), at its two prompt
        # lengths (128 and 4096 tokens, section 6.1): causal attention over packed
        # prompts, the KV-cache write of the prompts, and the FFNs over all
        # prompt tokens at once.
        for model, plen, nprompt in (("qwen3-32b", 4096, 2), ("qwen3-32b", 128, 32), ("mixtral-8x7b", 4096, 2)):
            pw = synth.prefill_workload(model, plen, nprompt, device=dev)
            outp = aflex.attn_prefill(pw)
            ms, kk = timed_kernels(lambda: aflex.attn_prefill(pw, out=outp), 10, ["attn_prefill"], aflex)
            pflops = sum(4.0 * n * (n + 1) / 2 * pw.Hq * pw.D for n in pw.lens)
            tag = f"prefill_attention_{model.split('-')[0]}_{nprompt}x{plen}"
            # bytes the kernel must move: q in and out once, K and V of each KV head once
            pbytes = 2 * pw.T * pw.Hq * pw.D * 2 + 2 * pw.T * pw.Hkv * pw.D * 2
            patt = min(PEAK_BF16, pflops / pbytes * PEAK_HBM)
            ops[tag] = {"ms": round(ms, 5), "tflops": round(pflops / (ms * 1e-3) / 1e12, 1),
                        "mfma_frac": round(pflops / (ms * 1e-3) / PEAK_BF16, 4),
                        "GB_per_s": round(pbytes / (ms * 1e-3) / 1e9, 1),
                        "attainable_frac": round(pflops / (ms * 1e-3) / patt, 4),
                        "tok_per_s": round(pw.T / (ms * 1e-3), 1),
                        "kernels": kk}
            if plen == 4096 and model == "qwen3-32b":
                pc = synth.custom_attention(5, nprompt, pw.Hq, pw.Hkv, pw.D, pw.lens).to(dev)
                aflex.kv_write(pc, pw.k, pw.v, pw.cu_seqlens, max_seqlen=plen)
                ms, kk = timed_kernels(lambda: aflex.kv_write(pc, pw.k, pw.v, pw.cu_seqlens, max_seqlen=plen), 10, ["kv_write"], aflex)
                kvb = 2 * 2 * pw.k.numel() * 2
                ops[f"kv_write_qwen3_{nprompt}x{plen}"] = {
                    "ms": round(ms, 5), "GB_per_s": round(kvb / (ms * 1e-3) / 1e9, 1),
                    "hbm_frac": round(kvb / (ms * 1e-3) / PEAK_HBM, 4), "bytes": kvb,
                    "kernels": kk}
                del pc
            del pw, outp
        Tp = 4096
        wd = synth.make_ffn_weights(2, 5120, 25600, device=dev)
        xp = synth.prefill_ffn_tokens(5120, Tp, device=dev)
        yp = torch.empty(Tp, 5120, dtype=torch.bfloat16, device=dev)
        aflex.ffn_swiglu(xp, wd, y=yp)
        ms, kk = timed_kernels(lambda: aflex.ffn_swiglu(xp, wd, y=yp), 5, ["gemm_gate_up", "gemm_down", "splitk_reduce"], aflex)
        flops = 6 * Tp * 5120 * 25600
        ops[f"prefill_swiglu_qwen3_T{Tp}"] = {
            "ms": round(ms, 5), "tflops": round(flops / (ms * 1e-3) / 1e12, 1),
            "mfma_frac": round(flops / (ms * 1e-3) / PEAK_BF16, 4), "tok_per_s": round(Tp / (ms * 1e-3), 1),
            "kernels": kk}
        del wd, xp, yp
        wm = synth.mixtral_moe(device=dev, T=Tp, seed=7, weights=f)
        yp = torch.empty(Tp, H, dtype=torch.bfloat16, device=dev)
        aflex.moe_ffn(wm.x, wm.ffn, wm.router_logits, 2, y=yp)
        ms, kk = timed_kernels(lambda: aflex.moe_ffn(wm.x, wm.ffn, wm.router_logits, 2, y=yp), 5, None, aflex)
        flops = Tp * 2 * 6 * H * I
        ops[f"prefill_moe_mixtral_T{Tp}"] = {
            "ms": round(ms, 5), "tflops": round(flops / (ms * 1e-3) / 1e12, 1),
            "mfma_frac": round(flops / (ms * 1e-3) / PEAK_BF16, 4), "tok_per_s": round(Tp / (ms * 1e-3), 1),
            "kernels": kk}
        del wm, yp
        # Resource sensitivity per operator: the same call on 64, 128, 192 and all
        # 256 CUs (CU-masked streams). The single-GPU analogue of the paper's
        # per-operator frequency sensitivity (section 3.2: decode attention gains
        # little from more GPU clock, the FFN a lot); reduction = 1 - t(256) / t(64).
        sens = {}
        wd = synth.make_ffn_weights(2, 5120, 25600, device=dev)
        wq = synth.qwen3_attention(device=dev).attn
        oq = torch.empty(wq.B, wq.Hq, wq.D, dtype=torch.bfloat16, device=dev)
        x32 = synth.qwen3_swiglu(32, device=dev, weights=wd).x
        x512 = synth.qwen3_swiglu(512, device=dev, weights=wd).x
        y32 = torch.empty(32, 5120, dtype=torch.bfloat16, device=dev)
        y512 = torch.empty(512, 5120, dtype=torch.bfloat16, device=dev)
        pw = synth.prefill_workload("qwen3-32b", 4096, 2, device=dev)
        op_ = torch.empty_like(pw.q)
        cases = {
            "decode_attention_qwen3_B64": lambda st: aflex.attn_decode(wq, out=oq, stream=st, ws=wss["a"]),
            "decode_swiglu_qwen3_T32": lambda st: aflex.ffn_swiglu(x32, wd, y=y32, stream=st, ws=wss["f"]),
            "decode_swiglu_qwen3_T512": lambda st: aflex.ffn_swiglu(x512, wd, y=y512, stream=st, ws=wss["f"]),
            "prefill_attention_qwen3_2x4096": lambda st: aflex.attn_prefill(pw, out=op_, stream=st),
        }
        wss = {"a": aflex.Workspace(), "f": aflex.Workspace()}
        for name, fn in cases.items():
            row = {}
            for cus in (64, 128, 192, 256):
                st = aflex.pool_streams(cus, dev)[0] if cus < 256 else torch.cuda.current_stream()
                st.wait_stream(torch.cuda.current_stream())
                fn(st)
                row[f"{cus}_cus_ms"] = round(timed(lambda: fn(st), 10, stream=st), 5)
                torch.cuda.current_stream().wait_stream(st)
            row["reduction_64_to_256"] = round(1 - row["256_cus_ms"] / row["64_cus_ms"], 3)
            sens[name] = row
        torch.cuda.synchronize()
        for w_ in wss.values():  # their buffers were used on the pool streams
            w_.buf = None
        aflex.release_pool_streams()
        ops["cu_sensitivity"] = sens
        if read_energy is not None:  # the same operators on the whole GPU: energy per token
            toks = {"decode_attention_qwen3_B64": wq.B, "decode_swiglu_qwen3_T32": 32,
                    "decode_swiglu_qwen3_T512": 512, "prefill_attention_qwen3_2x4096": pw.T}
            st = torch.cuda.current_stream()
            ops["energy_per_operator"] = {name: energy_of(lambda fn=fn: fn(st), toks[name], read_energy)
                                          for name, fn in cases.items()}
        del wd, wq, oq, x32, x512, y32, y512, pw, op_
        result["operators"] = ops

    # ---------------- CPU baseline: the oracle on a bounded sample -------------------
    if not args.no_cpu_baseline:
        import oracle

        def oracle_sample(n_seq):
            bt = a.block_table[:n_seq].cpu()
            cl = a.context_lens[:n_seq].cpu()
            phys, table = [], torch.full((n_seq, a.max_blocks), -1, dtype=torch.int32)
            for i in range(n_seq):
                nb = -(-int(cl[i]) // 16)
                table[i, :nb] = torch.arange(len(phys), len(phys) + nb, dtype=torch.int32)
                phys += bt[i, :nb].tolist()
            idx = torch.tensor(phys, device=dev)
            sub = synth.AttnInputs(q=a.q[:n_seq].cpu(), k_cache=a.k_cache[idx].cpu(),
                                   v_cache=a.v_cache[idx].cpu(), block_table=table, context_lens=cl,
                                   B=n_seq, Hq=a.Hq, Hkv=a.Hkv, D=a.D, block_size=16,
                                   max_blocks=a.max_blocks, num_blocks=len(phys),
                                   max_context_len=a.max_context_len)
            wts = synth.FFNWeights(f.w_gate.cpu(), f.w_up.cpu(), f.w_down.cpu(), H, I, f.E)
            lgs = logits[:n_seq].cpu()
            t0 = time.perf_counter()
            oracle.af_layer_steps(sub, wts, lgs, k, [n_seq], L=1)
            return time.perf_counter() - t0, int(cl.sum())

        n_seq = 8
        dt, ntok = oracle_sample(n_seq)
        for _ in range(2):  # grow the sample towards ~15 s of oracle work (at most the whole batch)
            if dt >= 10.0 or n_seq >= B:
                break
            n_seq = min(B, max(n_seq + 1, int(n_seq * 15.0 / max(dt, 1e-3))))
            dt, ntok = oracle_sample(n_seq)
        # The oracle on two more workloads, at one thread and at all of them:
        # the tiny layer (attention and SwiGLU) and the Qwen3-32B decode attention.
        nthreads = torch.get_num_threads()
        wt = synth.tiny_layer()
        wq = synth.qwen3_attention(device=dev).attn.to("cpu")
        per_config = {}
        for threads in (1, nthreads):
            torch.set_num_threads(threads)
            ta = wt.attn
            t0 = time.perf_counter()
            oracle.attention_decode(ta.q, ta.k_cache, ta.v_cache, ta.block_table, ta.context_lens)
            oracle.swiglu_ffn(wt.x, wt.ffn.w_gate, wt.ffn.w_up, wt.ffn.w_down)
            t1 = time.perf_counter()
            oracle.attention_decode(wq.q, wq.k_cache, wq.v_cache, wq.block_table, wq.context_lens)
            t2 = time.perf_counter()
            per_config.setdefault("tiny_layer_attention_and_swiglu_ms", {})[f"{threads}_threads"] = round((t1 - t0) * 1e3, 2)
            per_config.setdefault("qwen3_attention_B64_ms", {})[f"{threads}_threads"] = round((t2 - t1) * 1e3, 1)
        torch.set_num_threads(nthreads)
        del wq
        # The dense SwiGLU (Qwen3-32B weights) at each decode batch size and the
        # Mixtral MoE at 256 tokens, all threads: wall time and tokens/s.
        wg = synth.make_ffn_weights(2, 5120, 25600, device=dev)  # generated on the GPU, copied
        wq3 = synth.FFNWeights(wg.w_gate.cpu(), wg.w_up.cpu(), wg.w_down.cpu(), 5120, 25600, 0)
        x512c = synth.qwen3_swiglu(512, device=dev, weights=wg).x.cpu()
        del wg
        for T in (32, 128, 512):
            t0 = time.perf_counter()
            oracle.swiglu_ffn(x512c[:T], wq3.w_gate, wq3.w_up, wq3.w_down)
            t1 = time.perf_counter()
            per_config[f"qwen3_swiglu_T{T}"] = {"threads": nthreads, "ms": round((t1 - t0) * 1e3, 1),
                                               "tok_s": round(T / (t1 - t0), 2)}
        del wq3, x512c
        mc = synth.mixtral_moe(T=256, weights=synth.FFNWeights(f.w_gate.cpu(), f.w_up.cpu(), f.w_down.cpu(), H, I, f.E))
        t0 = time.perf_counter()
        oracle.moe_ffn(mc.x, mc.router_logits, mc.ffn.w_gate, mc.ffn.w_up, mc.ffn.w_down, 2)
        t1 = time.perf_counter()
        per_config["mixtral_moe_T256"] = {"threads": nthreads, "ms": round((t1 - t0) * 1e3, 1),
                                          "tok_s": round(256 / (t1 - t0), 2)}
        del mc
        result["cpu_baseline"] = {
            "value": round(n_seq / dt, 4), "unit": "tok/s", "cores": nthreads, "cpu_model": cpu_model(),
            "host": host_cores(),
            "cores_note": "cores = torch CPU threads the oracle ran on; host gives the logical CPUs "
                          "this process may use and the host's physical cores",
            "kind": "oracle",
            "sample": f"first {n_seq} of the 256 sequences of the pipeline workload ({ntok} cached "
                      f"tokens): their attention and top-2 MoE FFN in the float64 oracle, {dt:.1f} s",
            "per_config": per_config}

    print(json.dumps(result))


if __name__ == "__main__":
    main()
