"""Benchmark: prefix-shared attention fwd+bwd on one MI355X.

One step = the whole three-phase schedule over one prompt group with inputs
already resident in HBM: zero the gK/gV cache, Phase A prefix forward, Phase
B suffix forward + backward-with-cache-accumulation for every suffix
microbatch (one suffix per microbatch, the paper's timing choice), Phase C
prefix backward.  The suffix forwards run on a side stream beside the
in-order backwards (``DeviceGroup.run_schedule``); the per-phase times come
from one extra step in serial order.  The dense-recompute baseline (full causal fwd+bwd over
every [P||S(i)], one sequence at a time) is timed the same way on the same
GPU for the speedup.

The default workload is the long-context Llama3-8B attention group (GQA
32/8, d = 128, P = 28672, N = 8 suffixes of 128 tokens): the largest group
of the configurations that one GPU holds.  ``--workload`` selects another.

value = useful TFLOP/s = 14 d FLOP per visible (query row, key) pair per q
head that the schedule computes (4d forward + 10d backward), divided by the
mean step time; the median and minimum of the per-step times are reported
beside it.  The dense baseline's extra work is never counted.  The other
batching policy (all suffixes packed into one microbatch) is timed on the
same inputs and reported beside the headline's, against the dense baseline
under the same policy (the N materialized trajectories as one varlen launch
pair).

Also reported: per-phase times of one step, the standalone gK/gV cache
accumulate (G += g, HBM-bound) against 8 TB/s, and the 12d (no S recompute)
FLOP figure.  ``roofline`` is the dominant kernel timed with HIP events
around each of its launches over the same steps run again in serial order
(the kernel alone on the GPU); ``roofline.in_step`` is the same kernel in
the last timed step, where it shares the GPU with the suffix forwards.
``roofline.traffic`` is taken from the committed FETCH_SIZE /
WRITE_SIZE counter summary of the dominant kernel when that summary was made
from the kernel sources in the tree (else null); ``roofline.mfma_util`` is
the matrix-core utilisation (busy cycles over elapsed cycles of all SIMDs)
of its Phase B and Phase C launches, from the committed counter summary,
under the same condition and on the headline workload only.

Prints ONE JSON line.  ``--sweep c3|c4|c5attn|all`` instead prints one JSON
line per configuration of the speedup surface (schedule vs dense, no CPU
baseline); ``--moe-aux`` prints the MoE router aux-loss accounting line
(App. B: reuse accounting against the materialized prefix copies); ``--layer``
the long-context decoder layer through the schedule against the dense
layer; ``--stack`` the Phase-B HBM with and without dormant-prefix offload;
``--shard`` one GPU's kv-head share of the Qwen3-8B sweep groups.
``--gpus N`` with N > 1 exits: the path runs on one GPU.
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

METRIC = "prefix-shared attn fwd+bwd TFLOP/s (% MFMA peak) + speedup vs dense recompute"
# MI355X dense bf16 MFMA peak, the published 2.5 PFLOP/s at its clock:
# 256 CUs x 4096 flop per CU per clock x 2.4 GHz
BF16_PEAK_TFLOPS = 256 * 4096 * 2.4e9 / 1e12
HBM_PEAK_GBS = 8000.0
# algorithmic FLOP per visible (row, key) pair per q head of each matrix-core
# kernel: forward QK^T + PV (4d); backward S recompute, dP, dV, dK, dQ (10d,
# the usual flash-attention count: the backward kernel's second S/dP pass
# for dQ is implementation overhead and is not counted)
KERNEL_FLOP_PER_PAIR_PER_D = {"fwd_bf16": 4, "bwd_bf16": 10}
# the headline workload: the long-context Llama3-8B attention group (GQA
# 32/8, d = 128, P = 28672, N = 8 suffixes of 128), the largest group that
# the configurations put on one GPU
DEFAULT_WORKLOAD = "llama3_8b_p28672_n8_s128"


def traffic_summary(workload: str) -> str:
    """Committed counter summary of the dominant kernel's HBM traffic."""
    return os.path.join(ROOT, "profiles", f"bwd_bf16_traffic_{workload}.md")


def mfma_summary(workload: str) -> str:
    """Committed counter summary of the matrix-core utilisation."""
    return os.path.join(ROOT, "profiles", f"mfma_util_{workload}.md")

BWD_SOURCES = ["kernels_bf16_bwd.hip", "tile.hpp", "common.hpp", "spr_api.hip", "launch.hpp"]
SWEEPS = {
    "c3": [f"qwen3_8b_p{p}_n{n}" for p in (2048, 8192, 16384) for n in (4, 8, 16)],
    "c4": ["qwen3_moe_p8192_n16_ragged"],
    "c5attn": ["llama3_8b_p28672_n8_s128"],
}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def workload(name: str, seed: int):
    from synthetic import GroupShape, NAMED_SHAPES, make_group, qwen3_sweep_shape
    if name == "llama3_8b_p4096_n8_s512":
        return make_group(NAMED_SHAPES[name], seed=seed)
    if name == "qwen3_moe_p8192_n16_ragged":
        return make_group(NAMED_SHAPES[name], seed=seed, ragged=(128, 2048))
    if name == "llama3_8b_p28672_n8_s128":
        return make_group(NAMED_SHAPES[name], seed=seed)
    if name.startswith("qwen3_8b_p"):  # qwen3_8b_p{P}_n{N}
        p, n = name[len("qwen3_8b_p"):].split("_n")
        return make_group(qwen3_sweep_shape(int(p), int(n)), seed=seed)
    raise SystemExit(f"unknown workload {name}")


def pair_counts(shape):
    """Visible (row, key) pairs per q head: prefix causal, each suffix against
    the whole prefix plus its own causal part; and the dense baseline's."""
    p = shape.prefix_len
    pre = p * (p + 1) // 2
    suf = [s * p + s * (s + 1) // 2 for s in shape.suffix_lens]
    dense = [(p + s) * (p + s + 1) // 2 for s in shape.suffix_lens]
    return pre, suf, dense


def bwd_source_hash() -> str:
    h = hashlib.sha256()
    for f in BWD_SOURCES:
        with open(os.path.join(ROOT, "paper_2606_01143_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def committed_traffic(workload: str):
    """(bytes per launch, note) from the counter summary, or (None, why)."""
    path = traffic_summary(workload)
    if not os.path.exists(path):
        return None, "no counter summary for this workload"
    text = open(path).read()
    m_hash = re.search(r"kernel source hash: `([0-9a-f]+)`", text)
    m_val = re.search(r"HBM bytes per launch \(calibrated\): `([0-9.eE+]+)`", text)
    if not m_hash or not m_val:
        return None, "summary unreadable"
    if m_hash.group(1) != bwd_source_hash():
        return None, "kernel changed since the counters were taken"
    return float(m_val.group(1)), os.path.relpath(path, ROOT)


def committed_mfma_util(workload: str):
    """{"phase_b": %, "phase_c": %, "source": path} from the counter summary
    of the dominant kernel's matrix-core utilisation, or None."""
    path = mfma_summary(workload)
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_hash = re.search(r"kernel source hash: `([0-9a-f]+)`", text)
    m_val = re.search(r"MfmaUtil % per launch: Phase B `([0-9.]+)`, Phase C `([0-9.]+)`", text)
    if not m_hash or not m_val or m_hash.group(1) != bwd_source_hash():
        return None
    return {"phase_b_pct": float(m_val.group(1)), "phase_c_pct": float(m_val.group(2)),
            "counter": "SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE x 1024 SIMDs)",
            "source": os.path.relpath(path, ROOT)}


def phase_times(grp, mbs):
    """Per-phase milliseconds of one schedule step in serial order (events
    between phases; a mark implies the serial order)."""
    import torch
    marks = []

    def mark(name):
        e = torch.cuda.Event(enable_timing=True)
        e.record()
        marks.append((name, e))

    start = torch.cuda.Event(enable_timing=True)
    start.record()
    grp.run_schedule(mbs, mark=mark)
    torch.cuda.synchronize()
    out, prev = {}, start
    for name, e in marks:
        out[name] = out.get(name, 0.0) + prev.elapsed_time(e)
        prev = e
    return {k: round(v, 4) for k, v in out.items()}


def gkv_accumulate_rate(grp, reps: int = 20):
    """Standalone G_K += g_K, G_V += g_V: HBM GB/s (12 bytes per element per
    cache: read G, read g, write G)."""
    import torch
    from paper_2606_01143_amd import binding as B
    dgk, dgv = torch.randn_like(grp.gk), torch.randn_like(grp.gv)
    ms = time_steps(lambda: B.gkv_accumulate(grp.dims, grp.gk, grp.gv, dgk, dgv), reps, 2)
    nbytes = 12 * (grp.gk.numel() + grp.gv.numel())
    gbs = nbytes / (ms * 1e-3) / 1e9
    return {"GB/s": round(gbs, 1), "frac_of_8TB/s": round(gbs / HBM_PEAK_GBS, 4),
            "bytes_per_call": nbytes, "ms_per_call": round(ms, 4)}


def time_steps_stats(fn, steps: int, warmup: int):
    """Mean, median and minimum milliseconds per step: one event between
    consecutive steps on the current stream (the mean is the whole span over
    the steps)."""
    import statistics
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    ev[0].record()
    for i in range(steps):
        fn()
        ev[i + 1].record()
    torch.cuda.synchronize()
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]
    return {"mean": ev[0].elapsed_time(ev[-1]) / steps, "median": statistics.median(per),
            "min": min(per)}


def time_steps(fn, steps: int, warmup: int):
    return time_steps_stats(fn, steps, warmup)["mean"]


def host_facts():
    """Host cores the process may use, BLAS vendor and thread pool, CPU model."""
    facts = {"cores": len(os.sched_getaffinity(0)), "blas": "unknown", "blas_threads": None,
             "cpu_model": "unknown"}
    try:
        from threadpoolctl import threadpool_info
        blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if blas:
            facts["blas"] = f"{blas[0].get('internal_api')} {blas[0].get('version')}"
            facts["blas_threads"] = int(blas[0].get("num_threads", 1))
    except Exception:  # pragma: no cover
        pass
    try:
        import subprocess
        txt = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in txt.splitlines():
            if line.strip().startswith("Model name"):
                facts["cpu_model"] = line.split(":", 1)[1].strip()
                return facts
    except Exception:  # pragma: no cover
        pass
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    facts["cpu_model"] = line.split(":", 1)[1].strip()
                    break
    except OSError:  # pragma: no cover
        pass
    return facts


def gemm_bf16_rate(n: int = 8192, reps: int = 10):
    """A measured dense bf16 matrix-core rate on this GPU: an n x n x n
    torch.matmul (served by hipBLASLt), TFLOP/s, as a second denominator
    beside the published peak."""
    import torch
    g = torch.Generator(device="cuda").manual_seed(1)
    a = torch.randn(n, n, generator=g, device="cuda").to(torch.bfloat16)
    b = torch.randn(n, n, generator=g, device="cuda").to(torch.bfloat16)
    st = time_steps_stats(lambda: torch.matmul(a, b), reps, 3)
    tf = 2.0 * n ** 3 / (st["min"] * 1e-3) / 1e12
    return {"tflops": round(tf, 1), "shape": f"{n}x{n}x{n} bf16 (torch.matmul, hipBLASLt)",
            "ms_min": round(st["min"], 4), "frac_of_published_peak": round(tf / BF16_PEAK_TFLOPS, 4)}


def cpu_baseline(inp, shape, budget_s: float):
    """The fp64 oracle's three-phase reference on a bounded sample of the same
    group: one q head at a time with its kv head (heads are independent, so
    each is the same schedule on a one-head group), until the time budget is
    spent; the BLAS pool uses every core the process may run on."""
    from oracle import three_phase_reference
    from synthetic import GroupShape
    facts = host_facts()
    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(limits=facts["cores"], user_api="blas")
        facts["blas_threads"] = facts["cores"]
    except Exception:  # pragma: no cover
        limiter = None
    g = shape.group
    pre, suf, _ = pair_counts(shape)
    per_head_flops = 14 * shape.head_dim * (pre + sum(suf))
    done, t0 = 0, time.perf_counter()
    while True:
        h = done % shape.num_q_heads
        kv = h // g
        sub = dict(inp)
        for k in ("q_p", "q_s", "do_s", "g_y"):
            sub[k] = inp[k][:, h:h + 1]
        sub["do_p"] = inp["do_p"][:, :, h:h + 1]
        for k in ("k_p", "v_p", "k_s", "v_s"):
            sub[k] = inp[k][:, kv:kv + 1]
        sub["shape"] = GroupShape(1, 1, shape.head_dim, shape.prefix_len, shape.suffix_lens,
                                  shape.dtype)
        three_phase_reference(sub)
        done += 1
        el = time.perf_counter() - t0
        if el >= budget_s or done >= shape.num_q_heads:
            break
    if limiter is not None:
        limiter.restore_original_limits()
    return {"value": round(done * per_head_flops / el / 1e12, 6), "unit": "TFLOP/s",
            "cores": int(facts["blas_threads"] or facts["cores"]), "kind": "oracle",
            "sample": f"fp64 three-phase oracle (NumPy) on {done} of {shape.num_q_heads} q heads of "
                      f"the same group, each with its kv head, {el:.1f} s wall; "
                      f"value = those heads' 14d FLOP per visible pair / wall time",
            "host_cores": facts["cores"], "cpu_model": facts["cpu_model"], "blas": facts["blas"]}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--policy", choices=["per_suffix", "packed"], default="per_suffix")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--atomic-dq", action="store_true",
                    help="SPR_ATOMIC_DQ: dQ added by the key-outer blocks with fp32 atomics")
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="time budget of the CPU oracle baseline (0: skip it)")
    ap.add_argument("--sweep", choices=["c3", "c4", "c5attn", "all"], default=None)
    ap.add_argument("--layout", choices=["packed", "padded"], default="packed",
                    help="suffix layout of Phase B (padded: batch-plus-padding calls)")
    ap.add_argument("--layer", action="store_true",
                    help="a long-context Llama3-8B decoder layer through the schedule vs dense")
    ap.add_argument("--stack", action="store_true",
                    help="Phase-B HBM with and without dormant-prefix offload over a decoder-layer stack")
    ap.add_argument("--layers", type=int, default=16, help="decoder layers of --stack")
    ap.add_argument("--shard", action="store_true",
                    help="the Qwen3-8B sweep kernels on one GPU's kv-head share (Hkv = 8/g, g = 1, 2, 4, 8)")
    ap.add_argument("--moe-aux", action="store_true",
                    help="time the MoE router aux-loss accounting instead (one JSON line)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (--gpus {args.gpus} requested); the multi-GPU "
              "sharding of this path (by kv head, or by suffix with one cache reduce) is not built.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_01143_amd import binding as B
    from paper_2606_01143_amd.group import DeviceGroup

    B.lib()  # fails loudly without the HIP library
    if args.moe_aux:
        moe_aux_bench(args)
        return
    if args.stack:
        stack_bench(args)
        return
    if args.layer:
        layer_bench(args)
        return
    if args.shard:
        shard_bench(args)
        return
    if args.sweep:
        names = sum(SWEEPS.values(), []) if args.sweep == "all" else SWEEPS[args.sweep]
        for name in names:
            sweep_one(name, args)
        return
    log(f"generating {args.workload} (seed {args.seed})")
    inp = workload(args.workload, args.seed)
    shape = inp["shape"]
    n = shape.n
    per_suffix = [(i, i + 1) for i in range(n)]
    packed = [(0, n)]
    mbs = per_suffix if args.policy == "per_suffix" else packed
    grp = DeviceGroup(inp, device="cuda:0", dense=not args.no_dense,
                      microbatch_splits=[per_suffix, packed], layout=args.layout,
                      atomic_dq=args.atomic_dq)
    grp.prepare(mbs)
    torch.cuda.synchronize()

    pre, suf, dense_pairs = pair_counts(shape)
    hq, d = shape.num_q_heads, shape.head_dim
    sched_flops = 14 * d * hq * (pre + sum(suf))
    dense_flops = 14 * d * hq * sum(dense_pairs)
    tf = lambda flop, ms: flop / (ms * 1e-3) / 1e12

    log("schedule warmup")
    for _ in range(args.warmup):
        grp.run_schedule(mbs)
    torch.cuda.synchronize()
    # ---- one profiled step with every kernel bracketed: per-kernel times and
    # the dominant matrix-core kernel (untimed)
    B.profile_reset()
    B.profile_enable(True)
    grp.run_schedule(mbs)
    torch.cuda.synchronize()
    B.profile_enable(False)
    per_kernel = {k: round(B.profile_query(k)[0], 4) for k in B.profile_kernels()}
    dominant = max(KERNEL_FLOP_PER_PAIR_PER_D, key=lambda k: per_kernel.get(k, 0.0))

    # ---- the timed steps, HIP events around the dominant kernel only
    log("schedule timed steps")
    # HIP events bracket the dominant kernel's launches of the last timed
    # step only: each event is a packet on the stream, and around every
    # launch of every step they would cost a few percent of the step
    done = [0]

    def step():
        done[0] += 1
        if done[0] == args.steps:
            B.profile_enable(True, dominant)
        grp.run_schedule(mbs)

    B.profile_reset()
    st = time_steps_stats(step, args.steps, 0)
    ms_step = st["mean"]
    B.profile_enable(False)
    dom_ms, dom_count = B.profile_query(dominant)
    # algorithmic FLOP of all launches of the dominant kernel in one step:
    # its per-pair figure times every visible pair of the schedule (Phase A/C
    # prefix pairs + Phase B suffix pairs)
    dom_flops_per_step = KERNEL_FLOP_PER_PAIR_PER_D[dominant] * d * hq * (pre + sum(suf))
    dom_avg_ms = dom_ms / max(dom_count, 1)
    dom_achieved = dom_flops_per_step / (dom_ms * 1e-3) / 1e12 if dom_ms > 0 else 0.0
    value = tf(sched_flops, ms_step)
    log(f"schedule {ms_step:.3f} ms/step (median {st['median']:.3f}, min {st['min']:.3f}), "
        f"{value:.1f} TFLOP/s; {dominant} {dom_count} launches avg {dom_avg_ms:.3f} ms "
        f"-> {dom_achieved:.1f} TFLOP/s")

    # the same steps in serial order, events around every launch of the
    # dominant kernel: its own rate, alone on the GPU (the roofline)
    log("schedule timed steps, serial order")
    B.profile_reset()
    B.profile_enable(True, dominant)
    ms_serial = time_steps(lambda: grp.run_schedule(mbs, overlap=False), args.steps, 0)
    B.profile_enable(False)
    iso_ms, iso_count = B.profile_query(dominant)
    iso_achieved = dom_flops_per_step * args.steps / (iso_ms * 1e-3) / 1e12 if iso_ms > 0 else 0.0
    phases = phase_times(grp, mbs)
    # per-phase rates of the serial step: algorithmic FLOP of each phase over
    # its time (forward 4d, backward 10d per visible pair)
    sp = sum(suf)
    phase_flops = {"A": 4 * d * hq * pre, "B_fwd": 4 * d * hq * sp, "B_bwd": 10 * d * hq * sp,
                   "C": 10 * d * hq * pre}
    phase_rates = {k: {"tflops": round(tf(f, phases[k]), 1),
                       "pct_peak": round(100 * tf(f, phases[k]) / BF16_PEAK_TFLOPS, 2)}
                   for k, f in phase_flops.items() if phases.get(k, 0) > 0}
    gkv = gkv_accumulate_rate(grp)
    out = {
        "metric": METRIC, "value": round(value, 3), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "ms_per_step_median": round(st["median"], 4), "ms_per_step_min": round(st["min"], 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": args.workload, "num_q_heads": hq,
                   "num_kv_heads": shape.num_kv_heads, "head_dim": d,
                   "prefix_len": shape.prefix_len, "n_suffixes": n,
                   "suffix_lens": list(shape.suffix_lens) if len(set(shape.suffix_lens)) > 1
                   else shape.suffix_lens[0],
                   "microbatching": args.policy, "layout": args.layout,
                   "dq": "atomic" if args.atomic_dq else "query_outer"},
        "pct_mfma_peak": round(100 * value / BF16_PEAK_TFLOPS, 2),
        "value_at_median": round(tf(sched_flops, st["median"]), 3),
        "schedule_tflop_per_step": round(sched_flops / 1e12, 4),
        "kernel_ms_one_step": per_kernel,
        "phases_ms": phases,
        "phase_rates": phase_rates,
        "ms_per_step_serial_order": round(ms_serial, 4),
        "value_12d_tflops": round(value * 12 / 14, 3),
        "gkv_accumulate": gkv,
    }

    # the other batching policy on the same inputs: all suffixes packed into
    # one microbatch (policy (ii)) when the headline runs one per microbatch,
    # and the reverse
    other = packed if mbs is per_suffix else per_suffix
    other_name = "packed" if mbs is per_suffix else "per_suffix"
    grp.prepare(other)
    st_o = time_steps_stats(lambda: grp.run_schedule(other), args.steps, 1)
    out["policy_" + other_name] = {"ms_per_step": round(st_o["mean"], 4),
                                   "ms_per_step_median": round(st_o["median"], 4),
                                   "ms_per_step_min": round(st_o["min"], 4),
                                   "value": round(tf(sched_flops, st_o["mean"]), 3)}
    log(f"schedule, {other_name} microbatches: {st_o['mean']:.3f} ms/step")

    if not args.no_dense:
        log("dense baseline warmup + timed steps")
        st_d = time_steps_stats(lambda: grp.run_dense(), max(3, args.steps // 2), 1)
        ms_dense = st_d["mean"]
        out["dense_ms_per_step"] = round(ms_dense, 4)
        out["dense_ms_per_step_median"] = round(st_d["median"], 4)
        out["dense_ms_per_step_min"] = round(st_d["min"], 4)
        out["speedup_vs_dense"] = round(ms_dense / ms_step, 3)
        out["dense_equiv_tflops"] = round(tf(dense_flops, ms_dense), 3)
        out["flop_ratio_dense_over_schedule"] = round(dense_flops / sched_flops, 3)
        out["policy_" + other_name]["speedup_vs_dense"] = round(ms_dense / st_o["mean"], 3)
        out["dense_policy"] = "one trajectory per forward/backward call pair (the dense trainer's per-sequence order)"
        log(f"dense {ms_dense:.3f} ms/step, speedup {ms_dense / ms_step:.2f}x")
        # the dense baseline under the packed policy: the N materialized
        # trajectories as one varlen microbatch, one forward/backward call pair; compared
        # with the schedule's packed policy
        log("dense baseline, packed: warmup + timed steps")
        grp.prepare_dense_packed()
        st_dp = time_steps_stats(lambda: grp.run_dense_packed(), max(3, args.steps // 2), 1)
        grp.release_dense_packed()
        ms_pk = st_o["mean"] if mbs is per_suffix else ms_step
        out["dense_packed"] = {
            "ms_per_step": round(st_dp["mean"], 4), "ms_per_step_median": round(st_dp["median"], 4),
            "ms_per_step_min": round(st_dp["min"], 4),
            "speedup_of_schedule_packed": round(st_dp["mean"] / ms_pk, 3),
            "policy": "all N trajectories materialized as one packed varlen microbatch: one forward "
                      "and one backward call of causal attention over the N whole sequences; prefix "
                      "gradients per copy (the N-way sum is not timed)"}
        log(f"dense packed {st_dp['mean']:.3f} ms/step, schedule packed speedup "
            f"{st_dp['mean'] / ms_pk:.2f}x")

    traffic, traffic_src = (committed_traffic(args.workload) if dominant == "bwd_bf16"
                            else (None, "n/a"))
    out["roofline"] = {"bound": "mfma", "achieved": round(iso_achieved, 2),
                       "peak": round(BF16_PEAK_TFLOPS, 1), "unit": "TFLOP/s",
                       "frac": round(iso_achieved / BF16_PEAK_TFLOPS, 4), "traffic": traffic,
                       "traffic_unit": "HBM bytes per launch", "traffic_source": traffic_src,
                       "kernel": dominant,
                       "mfma_util": (committed_mfma_util(args.workload)
                                     if dominant == "bwd_bf16" else None),
                       "flop_per_pair": f"{KERNEL_FLOP_PER_PAIR_PER_D[dominant]}d",
                       "launches_per_step": iso_count // max(args.steps, 1),
                       "avg_launch_ms": round(iso_ms / max(iso_count, 1), 4),
                       "measured": f"HIP events around each launch, {args.steps} steps in serial order",
                       # in the timed (overlapped) steps a backward shares the GPU
                       # with the suffix forwards, so its launches last longer
                       "in_step": {"achieved": round(dom_achieved, 2),
                                   "frac": round(dom_achieved / BF16_PEAK_TFLOPS, 4),
                                   "avg_launch_ms": round(dom_avg_ms, 4),
                                   "measured": "HIP events around each launch of the last timed step"}}
    del grp
    torch.cuda.empty_cache()
    gemm = gemm_bf16_rate()
    out["gemm_bf16_measured"] = gemm
    out["roofline"]["frac_of_measured_gemm"] = round(iso_achieved / gemm["tflops"], 4)
    if args.cpu_seconds > 0:
        log("cpu baseline (oracle)")
        out["cpu_baseline"] = cpu_baseline(inp, shape, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def sweep_one(name: str, args):
    """One configuration of the speedup surface: schedule and dense baseline
    timed on the same GPU, one suffix per microbatch."""
    import torch
    from paper_2606_01143_amd.group import DeviceGroup
    log(f"sweep {name}: generating")
    inp = workload(name, args.seed)
    shape = inp["shape"]
    mbs = [(i, i + 1) for i in range(shape.n)]
    grp = DeviceGroup(inp, device="cuda:0", dense=True)
    del inp
    grp.prepare(mbs)
    pre, suf, dense_pairs = pair_counts(shape)
    hq, d = shape.num_q_heads, shape.head_dim
    sched_flops = 14 * d * hq * (pre + sum(suf))
    dense_flops = 14 * d * hq * sum(dense_pairs)
    steps = max(1, args.steps)
    ms = time_steps(lambda: grp.run_schedule(mbs), steps, max(1, args.warmup))
    phases = phase_times(grp, mbs)
    ms_dense = time_steps(lambda: grp.run_dense(), max(1, steps // 2), 1)
    # the packed policy on both sides: all suffixes in one microbatch, and
    # the N materialized trajectories as one varlen forward/backward call pair
    packed = [(0, shape.n)]
    grp.prepare(packed)
    ms_pk = time_steps(lambda: grp.run_schedule(packed), steps, 1)
    grp.prepare_dense_packed()
    ms_dense_pk = time_steps(lambda: grp.run_dense_packed(), max(1, steps // 2), 1)
    grp.release_dense_packed()
    value = sched_flops / (ms * 1e-3) / 1e12
    rec = {"workload": name, "num_q_heads": hq, "num_kv_heads": shape.num_kv_heads, "head_dim": d,
           "prefix_len": shape.prefix_len, "n_suffixes": shape.n,
           "total_suffix_tokens": int(sum(shape.suffix_lens)),
           "ms_per_step": round(ms, 4), "value_tflops": round(value, 3),
           "pct_mfma_peak": round(100 * value / BF16_PEAK_TFLOPS, 2),
           "dense_ms_per_step": round(ms_dense, 4), "speedup_vs_dense": round(ms_dense / ms, 3),
           "flop_ratio_dense_over_schedule": round(dense_flops / sched_flops, 3),
           "packed": {"ms_per_step": round(ms_pk, 4), "dense_ms_per_step": round(ms_dense_pk, 4),
                      "speedup_vs_dense": round(ms_dense_pk / ms_pk, 3)},
           "phases_ms": phases, "steps": steps, "dtype": "bf16", "data": "synthetic"}
    print(json.dumps(rec), flush=True)
    del grp
    torch.cuda.empty_cache()


def shard_bench(args):
    """One GPU's share of a kv-head-sharded group: the Qwen3-8B sweep shape
    (GQA 32/8, d 128, suffixes of 1024) with Hq = 32/g and Hkv = 8/g for
    g = 1, 2, 4, 8, i.e. what each of g GPUs would run.  One JSON line per
    (P, N, g): step time, TFLOP/s of the shard, its efficiency against the
    unsharded group (TFLOP/s ratio), and the speedup over the dense baseline
    on the same shard."""
    import torch
    from paper_2606_01143_amd.group import DeviceGroup
    from synthetic import GroupShape, make_group
    steps, warm = max(1, args.steps), max(1, args.warmup)
    for p, n in ((2048, 4), (8192, 8), (16384, 16)):
        base = None
        for g in (1, 2, 4, 8):
            shape = GroupShape(32 // g, 8 // g, 128, p, (1024,) * n, "bf16")
            log(f"shard P={p} N={n} g={g}: generating")
            inp = make_group(shape, seed=args.seed)
            mbs = [(i, i + 1) for i in range(n)]
            grp = DeviceGroup(inp, device="cuda:0", dense=True)
            del inp
            grp.prepare(mbs)
            pre, suf, _ = pair_counts(shape)
            flops = 14 * shape.head_dim * shape.num_q_heads * (pre + sum(suf))
            ms = time_steps(lambda: grp.run_schedule(mbs), steps, warm)
            ms_dense = time_steps(lambda: grp.run_dense(), max(1, steps // 4), 1)
            tf = flops / (ms * 1e-3) / 1e12
            base = tf if g == 1 else base
            rec = {"workload": f"qwen3_8b_p{p}_n{n}", "shard_g": g, "num_q_heads": shape.num_q_heads,
                   "num_kv_heads": shape.num_kv_heads, "ms_per_step": round(ms, 4),
                   "value_tflops": round(tf, 2), "pct_mfma_peak": round(100 * tf / BF16_PEAK_TFLOPS, 2),
                   "efficiency_vs_unsharded": round(tf / base, 3), "dense_ms_per_step": round(ms_dense, 4),
                   "speedup_vs_dense": round(ms_dense / ms, 3), "steps": steps, "dtype": "bf16",
                   "data": "synthetic"}
            print(json.dumps(rec), flush=True)
            del grp
            torch.cuda.empty_cache()


def layer_bench(args):
    """A long-context Llama3-8B decoder layer (hidden 4096, GQA 32/8, d 128,
    RoPE theta 5e5, SwiGLU 14336, RMSNorm; weights N(0, 0.02)) over a group
    with P = 28672 and N = 8 suffixes of 128: the three-phase schedule
    against the dense per-trajectory layer, forward and backward with weight
    gradients.  One JSON line."""
    import torch
    from paper_2606_01143_amd.layer import DecoderLayer
    from synthetic.layer import LAYER_SHAPES, make_layer_group
    name = "llama3_8b_layer_p28672_n8_s128"
    shp = LAYER_SHAPES[name]
    layer = DecoderLayer(make_layer_group(shp, seed=args.seed))
    steps, warm = max(1, min(args.steps, 5)), max(1, min(args.warmup, 2))
    ms = time_steps(layer.run_schedule, steps, warm)
    ms_dense = time_steps(layer.run_dense, max(1, steps // 2), 1)
    P, S, n = shp.prefix_len, shp.suffix_lens[0], shp.n
    per_tok = 2 * (shp.hidden * (shp.num_q_heads + 2 * shp.num_kv_heads) * shp.head_dim
                   + shp.num_q_heads * shp.head_dim * shp.hidden + 3 * shp.hidden * shp.intermediate)
    gemm = 3 * per_tok  # forward, input gradient, weight gradient
    d, hq = shp.head_dim, shp.num_q_heads
    pairs_sched = P * (P + 1) // 2 + n * (S * P + S * (S + 1) // 2)
    pairs_dense = n * (P + S) * (P + S + 1) // 2
    flop = gemm * (P + n * S) + 14 * d * hq * pairs_sched
    flop_dense = gemm * n * (P + S) + 14 * d * hq * pairs_dense
    out = {"metric": "decoder layer fwd+bwd through the schedule, useful TFLOP/s + speedup vs dense",
           "value": round(flop / (ms * 1e-3) / 1e12, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": steps,
           "warmup": warm, "ms_per_step": round(ms, 2), "higher_is_better": True, "dtype": "bf16",
           "data": "synthetic", "config": {"workload": name, "hidden": shp.hidden, "num_q_heads": hq,
                                           "num_kv_heads": shp.num_kv_heads, "head_dim": d,
                                           "intermediate": shp.intermediate, "prefix_len": P,
                                           "n_suffixes": n, "suffix_len": S},
           "dense_ms_per_step": round(ms_dense, 2), "speedup_vs_dense": round(ms_dense / ms, 3),
           "flop_ratio_dense_over_schedule": round(flop_dense / flop, 3),
           "schedule_tflop_per_step": round(flop / 1e12, 2),
           "dense_equiv_tflops": round(flop_dense / (ms_dense * 1e-3) / 1e12, 2)}
    print(json.dumps(out), flush=True)


def stack_bench(args):
    """Phase-B HBM with and without offloading the dormant prefix state (the
    measurement of the paper's Table 6, Sec. 5.5): a stack of Llama3-8B
    decoder layers (hidden 4096, GQA 32/8, d 128, SwiGLU 14336; weights and
    inputs drawn on the GPU), chained across layers, N = 16 suffixes, total
    length 12288 split between prefix and suffix.  One JSON line per split:
    the allocator's peak during Phase B, the step time, and the dormant
    bytes moved to pinned host memory."""
    import torch
    from paper_2606_01143_amd.stack import DecoderStack
    from synthetic.layer import LayerShape
    L = args.layers
    gib = float(1 << 30)
    for P, S in ((2048, 10240), (6144, 6144), (8192, 4096), (10240, 2048)):
        shape = LayerShape(4096, 32, 8, 128, 14336, P, (S,) * 16)
        rec = {"workload": f"llama3_8b_decoder_stack{L}_p{P}_s{S}_n16", "layers": L, "prefix_len": P,
               "suffix_len": S, "n_suffixes": 16, "dtype": "bf16", "data": "synthetic"}
        for offload in (False, True):
            log(f"stack P={P} S={S} offload={offload}")
            st = DecoderStack(shape=shape, layers=L, seed=args.seed, offload=offload, pool_factor=1.1)
            st.run_schedule()  # warm: allocator pools, pinned pool, kernels
            torch.cuda.synchronize()
            marks = {}

            def mark(name):
                e = torch.cuda.Event(enable_timing=True)
                e.record()
                marks[name] = e
                if name == "A":
                    torch.cuda.reset_peak_memory_stats()
                if name == "B":
                    marks["peak_b"] = torch.cuda.max_memory_allocated()

            start = torch.cuda.Event(enable_timing=True)
            start.record()
            out = st.run_schedule(on_phase=mark)
            torch.cuda.synchronize()
            del out
            key = "offload" if offload else "no_offload"
            rec[f"phase_b_peak_gib_{key}"] = round(marks["peak_b"] / gib, 3)
            rec[f"step_ms_{key}"] = round(start.elapsed_time(marks["C"]), 2)
            rec[f"phase_ms_{key}"] = {"A": round(start.elapsed_time(marks["A"]), 2),
                                      "B": round(marks["A"].elapsed_time(marks["B"]), 2),
                                      "C": round(marks["B"].elapsed_time(marks["C"]), 2)}
            if offload:
                rec["dormant_gib"] = round(st.dormant_bytes / gib, 3)
                rec["restores"] = {k: v for k, v in st.stats.items()}
            del st
            torch.cuda.empty_cache()
            # pinned host blocks go back to the driver too (the next split's
            # pool is larger and cannot reuse them)
            if hasattr(torch._C, "_host_emptyCache"):
                torch._C._host_emptyCache()
        red = rec["phase_b_peak_gib_no_offload"] - rec["phase_b_peak_gib_offload"]
        rec["reduction_gib"] = round(red, 3)
        rec["reduction_pct"] = round(100 * red / rec["phase_b_peak_gib_no_offload"], 1)
        print(json.dumps(rec), flush=True)


def moe_aux_bench(args):
    """MoE router aux-loss accounting (App. B) for one MoE layer of one prompt
    group: the reuse accounting (prefix tokens once with multiplicity N, then
    each suffix microbatch with multiplicity 1; loss; router gradients of
    the prefix and of each suffix microbatch) against the materialized batch
    (every prefix copy explicit: one accumulate and one gradient over all
    logical tokens).  One JSON line; value = logical router tokens per second
    of the reuse step."""
    import numpy as np
    import torch
    from paper_2606_01143_amd import binding as B
    from synthetic.moe import ROUTER_SHAPES, make_router_group
    name = "qwen3_moe_router_p8192_n16_ragged"
    inp = make_router_group(ROUTER_SHAPES[name], seed=args.seed, ragged=(128, 2048))
    shp = inp["shape"]
    E, k, n, P = shp.num_experts, shp.top_k, shp.n, shp.prefix_len
    dev = torch.device("cuda:0")
    up = lambda x, dt: torch.from_numpy(np.ascontiguousarray(x)).to(device=dev, dtype=dt)
    p_p, r_p = up(inp["p_p"], torch.float32), up(inp["r_p"], torch.int32)
    p_s, r_s = up(inp["p_s"], torch.float32), up(inp["r_s"], torch.int32)
    cu = [int(x) for x in inp["cu_seqlens"]]
    T = cu[-1]
    # materialized batch: N prefix copies then the suffix tokens
    p_m = torch.cat([p_p] * n + [p_s]).contiguous()
    r_m = torch.cat([r_p] * n + [r_s]).contiguous()
    stats = torch.empty(B.moe_stats_bytes(E), dtype=torch.uint8, device=dev)
    ws = torch.empty(B.moe_aux_workspace_size(E, p_m.shape[0]), dtype=torch.uint8, device=dev)
    f = torch.empty(E, dtype=torch.float64, device=dev)
    pe = torch.empty_like(f)
    loss = torch.empty(1, dtype=torch.float64, device=dev)
    dp_p, dp_s, dp_m = torch.empty_like(p_p), torch.empty_like(p_s), torch.empty_like(p_m)
    lam = 0.01
    spans = [(cu[i], cu[i + 1]) for i in range(n)]

    def reuse_step():
        B.moe_stats_zero(E, stats)
        B.moe_aux_accumulate(E, k, p_p, r_p, stats, multiplicity=n, ws=ws)
        for a, b in spans:
            B.moe_aux_accumulate(E, k, p_s[a:b], r_s[a:b], stats, multiplicity=1, ws=ws)
        B.moe_aux_loss(E, k, lam, stats, f, pe, loss)
        B.moe_aux_grad(E, k, lam, 1.0, stats, dp_p, multiplicity=n)
        for a, b in spans:
            B.moe_aux_grad(E, k, lam, 1.0, stats, dp_s[a:b], multiplicity=1)

    def reuse_step_packed():
        # the same accounting with the suffixes as one packed microbatch
        B.moe_stats_zero(E, stats)
        B.moe_aux_accumulate(E, k, p_p, r_p, stats, multiplicity=n, ws=ws)
        B.moe_aux_accumulate(E, k, p_s, r_s, stats, multiplicity=1, ws=ws)
        B.moe_aux_loss(E, k, lam, stats, f, pe, loss)
        B.moe_aux_grad(E, k, lam, 1.0, stats, dp_p, multiplicity=n)
        B.moe_aux_grad(E, k, lam, 1.0, stats, dp_s, multiplicity=1)

    def materialized_step():
        B.moe_stats_zero(E, stats)
        B.moe_aux_accumulate(E, k, p_m, r_m, stats, multiplicity=1, ws=ws)
        B.moe_aux_loss(E, k, lam, stats, f, pe, loss)
        B.moe_aux_grad(E, k, lam, 1.0, stats, dp_m, multiplicity=1)

    steps, warm = max(1, args.steps), max(1, args.warmup)
    # per-kernel times of one untimed step
    B.profile_reset()
    B.profile_enable(True)
    reuse_step()
    torch.cuda.synchronize()
    B.profile_enable(False)
    per_kernel = {kk: round(B.profile_query(kk)[0] * 1e3, 2) for kk in B.profile_kernels()
                  if B.profile_query(kk)[1]}
    dominant = max(("moe_partial", "moe_grad"), key=lambda kk: per_kernel.get(kk, 0.0))
    nb_bytes = lambda nt: B.moe_aux_workspace_size(E, nt)
    if dominant == "moe_partial":
        per_step_bytes = sum((nt * E * 4 + nt * k * 4 + nb_bytes(nt)) for nt in [P] + [b - a for a, b in spans])
    else:
        per_step_bytes = (P + T) * E * 4
    for _ in range(warm):
        reuse_step()
    B.profile_reset()
    B.profile_enable(True, dominant)
    ms_eager = time_steps(reuse_step, steps, 0)
    B.profile_enable(False)
    dom_ms, dom_n = B.profile_query(dominant)
    ms_mat_eager = time_steps(materialized_step, steps, warm)
    # the step is a few dozen short launches: capture each in a HIP graph and
    # time the replays (no host launch overhead)
    graphs = {}
    for key, fn in (("reuse", reuse_step), ("packed", reuse_step_packed), ("materialized", materialized_step)):
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn()
        torch.cuda.current_stream().wait_stream(side)
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn()
        graphs[key] = g
    ms = time_steps(graphs["reuse"].replay, steps, warm)
    ms_mat = time_steps(graphs["materialized"].replay, steps, warm)
    ms_packed = time_steps(graphs["packed"].replay, steps, warm)
    # algorithmic HBM bytes of a step: probabilities and expert ids read, the
    # gradient written (reuse: physical tokens; materialized: logical ones)
    step_bytes = lambda nt: nt * (E * 4 + k * 4 + E * 4)
    logical = n * P + T
    achieved = per_step_bytes * steps / (dom_ms * 1e-3) / 1e9 if dom_ms > 0 else 0.0
    # cpu baseline: the oracle's reuse accounting on the same inputs
    from oracle.moe_aux import reuse_reference
    t0 = time.perf_counter()
    reps = 0
    while True:
        reuse_reference(inp, lam)
        reps += 1
        el = time.perf_counter() - t0
        if el >= min(args.cpu_seconds, 5.0) or reps >= 50:
            break
    out = {"metric": "MoE router aux-loss accounting, logical tokens/s (one MoE layer of one group)",
           "value": round(logical / (ms * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1, "steps": steps,
           "warmup": warm, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "f32", "data": "synthetic",
           "config": {"workload": name, "num_experts": E, "top_k": k, "prefix_len": P, "n_suffixes": n,
                      "total_suffix_tokens": T, "microbatching": "per_suffix"},
           "timing": "HIP graph replay of the step",
           "eager_ms_per_step": round(ms_eager, 4), "materialized_eager_ms_per_step": round(ms_mat_eager, 4),
           "materialized_ms_per_step": round(ms_mat, 4), "speedup_vs_materialized": round(ms_mat / ms, 3),
           "packed_suffix_ms_per_step": round(ms_packed, 4),
           "packed_speedup_vs_materialized": round(ms_mat / ms_packed, 3),
           "step_hbm_bytes": {"reuse": step_bytes(P + T), "materialized": step_bytes(logical)},
           "token_ratio_materialized_over_reuse": round(logical / (P + T), 3),
           "kernel_us_one_step": per_kernel,
           "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                        "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None, "kernel": dominant,
                        "launches_per_step": dom_n // steps,
                        "avg_launch_us": round(dom_ms * 1e3 / max(dom_n, 1), 2),
                        "measured": "HIP events around each launch of the eager step"},
           "cpu_baseline": {"value": round(logical * reps / el, 1), "unit": "tokens/s", "cores": 1,
                            "kind": "oracle", "sample": f"fp64 reuse accounting of the same group, {reps} "
                                                        f"repetitions in {el:.1f} s"}}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
