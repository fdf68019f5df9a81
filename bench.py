"""Benchmark of one PACI pipeline stage on one MI355X.

A step is one full asynchronous 1F1B replay of the GPT-2-medium-shaped bf16
middle stage through the C ABI's schedule driver (paci_stage_run). The stage
has 6 pre-LN blocks, d 1024, 16 heads of 64, FFN 4096, seq 1024 and
micro-batch 8. A replay is 64 micro-batches with delay 3 and an AdamW update
every K = 8 backwards. That is 64 forwards, 64 backwards with fp32 gradient
accumulation and 8 updates. Inputs and output gradients are seeded synthetic
tensors already resident in HBM. Successive replays keep training from the
state the previous one left (only the counters are rewound).

Printed: one JSON line with stage tokens/s over the timed replays, the
stage's MFMA utilisation against the bf16 dense peak, the roofline of the
dominant kernel family (from as many replays again after the timed region,
with HIP events around every launch on the stage stream), and the CPU oracle
timed on a bounded sample.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "hbm_traffic_gpt2m_mid_bf16.md")
WORKLOAD_SHAPE = {"gpt2s_mid_bf16": "GPT-2-small-shaped", "gpt2m_mid_bf16": "GPT-2-medium-shaped",
                  "gpt2m_first_bf16": "GPT-2-medium-shaped", "gpt2m_last_bf16": "GPT-2-medium-shaped",
                  "gpt1p3b_pos0_bf16": "1.3B-class"}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def make_device_inputs(torch, c, M, seed):
    """Seeded stage inputs [M, T, d] (N(0,1); token ids uniform over the vocabulary
    for a first stage), output gradients [M, T, d] (N(0, 0.01^2); none for a
    last stage) and targets [M, T] (uniform; last stage only)."""
    T, d = c["micro_batch"] * c["seq"], c["d_model"]
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    dt = torch.bfloat16 if c["dtype"] == "bf16" else torch.float32
    if c["kind"] == "first":
        x = torch.randint(0, c["vocab"], (M, T), generator=g, device="cuda", dtype=torch.int32)
    else:
        x = torch.empty(M, T, d, dtype=dt, device="cuda")
        for i in range(M):
            x[i].copy_(torch.randn(T, d, generator=g, device="cuda"))
    dy = tgt = None
    if c["kind"] == "last":
        tgt = torch.randint(0, c["vocab"], (M, T), generator=g, device="cuda", dtype=torch.int32)
    else:
        dy = torch.empty(M, T, d, dtype=dt, device="cuda")
        for i in range(M):
            dy[i].copy_(torch.randn(T, d, generator=g, device="cuda") * 1e-2)
    return x, dy, tgt


def gemm_reference(torch, c, reps=20):
    """The vendor BLAS (torch's bf16 matmul) on this stage's GEMM shapes, as a yardstick.

    Plain products only: no bias, GELU or residual epilogue, no accumulation
    into G, and the weight gradients over one contiguous window of K * T rows.
    Returned per family in the stage's own units (ms per replay of M
    micro-batches over all blocks), to set beside the gemm_* kernel families.
    """
    T, d, f, KT = c["micro_batch"] * c["seq"], c["d_model"], c["d_ff"], c["K"] * c["micro_batch"] * c["seq"]
    fams = {"gemm_fwd": [(T, 3 * d, d), (T, d, d), (T, f, d), (T, d, f)],
            "gemm_dgrad": [(T, f, d), (T, d, f), (T, d, d), (T, d, 3 * d)],
            "gemm_wgrad_acc": [(3 * d, d, KT), (d, d, KT), (f, d, KT), (d, f, KT)]}
    per_mb = c["n_layers"] * c["M"]
    out = {}
    for fam, shapes in fams.items():
        us_total, flop = 0.0, 0.0
        for M_, N_, K_ in shapes:
            if fam == "gemm_wgrad_acc":   # dY^T X, both stored token-major
                a = torch.randn(K_, M_, device="cuda", dtype=torch.bfloat16)
                b = torch.randn(K_, N_, device="cuda", dtype=torch.bfloat16)
                fn = lambda: torch.matmul(a.t(), b)
            else:                         # X W^T with W stored [out, in]
                a = torch.randn(M_, K_, device="cuda", dtype=torch.bfloat16)
                b = torch.randn(N_, K_, device="cuda", dtype=torch.bfloat16)
                fn = lambda: torch.matmul(a, b.t())
            for _ in range(3):
                fn()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(reps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / reps
            us_total += us / (c["K"] if fam == "gemm_wgrad_acc" else 1)
            flop += 2.0 * M_ * N_ * K_ / (c["K"] if fam == "gemm_wgrad_acc" else 1)
            del a, b
        out[fam] = {"ms_per_step": round(us_total * per_mb / 1e3, 3),
                    "tflops": round(flop / (us_total * 1e-6) / 1e12, 1)}
    return out


def cpu_baseline(c, seed=0, budget_s=90.0):
    """The oracle (float64 NumPy) timed on the protocol's bounded sample: the
    first W = K + delay + 1 micro-batches of the canonical asynchronous 1F1B
    order, with accumulation into G and the AdamW update after the K-th
    backward, i.e. every event of the first window and every stale backward
    that crosses its update. It runs at one sequence per micro-batch and is
    scaled per sequence to the workload's micro-batch: the oracle's forward
    and backward work is a sum over sequences, while the update's is not, so
    the estimate is mu * (forward + backward time) + update time for W * mu *
    seq tokens. If the forwards and backwards would exceed ``budget_s``, the
    rest are extrapolated from the mean per event of each kind and the update
    is timed on its own. BLAS threads are set to the cores this process may
    run on. Returns the JSON object."""
    import numpy as np
    from oracle import stage as ostage
    from oracle.schedule import canonical_events
    from paper_2606_07881_amd import inputs
    cores = len(os.sched_getaffinity(0))
    blas = None
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threadpool_limits(cores)
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover - threadpoolctl is optional
        pass
    K, delay, mu = c["K"], c["delay"], c["micro_batch"]
    W = K + delay + 1
    one = dict(c)
    one["micro_batch"] = 1
    kind = c["kind"]
    params = {k: v.astype(np.float64) for k, v in inputs.make_params(c, seed).items()}
    st = ostage.Stage(one, params, K, delay)
    events = canonical_events(W, K, delay)
    t = {"F": 0.0, "B": 0.0, "S": 0.0}
    n = {"F": 0, "B": 0, "S": 0}
    t_start = time.perf_counter()
    done = True
    for kd, i in events:
        if kd in ("F", "B") and n["F"] and n["B"] and t["F"] + t["B"] > budget_s:
            done = False
            break
        if kd == "F":   # inputs are drawn outside the timed calls
            x = inputs.make_ids(one, seed, i) if kind == "first" else inputs.make_x(one, seed, i)[0].astype(np.float64)
            tgt = inputs.make_targets(one, seed, i) if kind == "last" else None
            t0 = time.perf_counter()
            st.forward(i, x, tgt)
        elif kd == "B":
            dy = None if kind == "last" else inputs.make_dy(one, seed, i)[0].astype(np.float64)
            t0 = time.perf_counter()
            st.backward(i, dy)
        else:
            t0 = time.perf_counter()
            st.step()
        t[kd] += time.perf_counter() - t0
        n[kd] += 1
    if not done:   # the update on its own: AdamW over every parameter, as Stage.step does it
        if n["S"] == 0:
            for name in st.names:
                st.G[name] = np.full_like(st.G[name], 1e-3)
            st.counters.c = K
            t0 = time.perf_counter()
            st.step()
            t["S"] = time.perf_counter() - t0
    elapsed = time.perf_counter() - t_start
    fwd_bwd = W * (t["F"] / max(n["F"], 1) + t["B"] / max(n["B"], 1))
    est = mu * fwd_bwd + t["S"]
    tokens = W * mu * c["seq"]
    how = ("every event timed" if done else
           f"{n['F']} forwards and {n['B']} backwards timed within the budget, the rest extrapolated "
           "from their means, the update timed on its own")
    return {"value": tokens / est, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "blas_threads": blas,
            "sample": f"oracle replay of the first W = K + delay + 1 = {W} micro-batches of the asynchronous 1F1B "
                      f"order (K {K}, delay {delay}: {W} forwards, {W} backwards accumulated into G, 1 AdamW update "
                      f"over {sum(v.size for v in params.values())} parameters) at 1 sequence of {c['seq']} tokens "
                      f"per micro-batch, scaled per sequence to micro-batch {mu}: {mu} x {fwd_bwd:.1f} s forward and "
                      f"backward + {t['S']:.1f} s update = {est:.1f} s for {tokens} tokens ({how}; {elapsed:.1f} s "
                      f"measured); float64 NumPy, dense masked attention (about 2x the causal attention FLOPs); "
                      f"{cores} cores in the affinity mask, BLAS threads {blas}"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default=None)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=90.0,
                    help="seconds of oracle forward and backward work before the rest is extrapolated")
    ap.add_argument("--recompute", action="store_true",
                    help="the activation-checkpointed stage: keep only stage inputs, recompute the forward "
                         "in each backward under the current parameters")
    ap.add_argument("--window", action="store_true",
                    help="windowed block weight gradients: K + delay activation slots instead of the paper's "
                         "delay + 1, one contraction per weight and window")
    ap.add_argument("--fused-head", action="store_true",
                    help="last stage: the fused LM head (no [T, V] logits kept; the backward recomputes them)")
    ap.add_argument("--dropout", type=float, default=0.0,
                    help="dropout rate at the embedding, attention-probability and residual-branch sites "
                         "(the paper trains with 0.1; the headline workload has none)")
    ap.add_argument("--micro-batch", type=int, default=0,
                    help="sequences per micro-batch instead of the workload's (the paper trains with 16 or 32)")
    ap.add_argument("--K", type=int, default=0, help="accumulation factor instead of the workload's")
    ap.add_argument("--gemm-reference", action="store_true",
                    help="time only the vendor BLAS on this stage's GEMM shapes (plain products) and exit")
    ap.add_argument("--copy-probe", action="store_true",
                    help="first copy a 256 MiB device buffer 3 times (a kernel of known traffic, for scaling "
                         "hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one pipeline stage on one GPU; --gpus {args.gpus} is not supported "
              "(stages on several GPUs exchange activations point to point; this benchmark runs one stage)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_07881_amd import binding, configs, inputs

    name = args.config or configs.BENCH_CONFIG
    over = {}
    if args.recompute:
        over["recompute"] = 1
    if args.fused_head:
        over["fused_head"] = 1
    if args.window:
        over["window"] = 1
    if args.dropout > 0:
        over["dropout"] = args.dropout
        over["dropout_seed"] = 2606
    if args.micro_batch > 0:
        over["micro_batch"] = args.micro_batch
    if args.K > 0:
        over["K"] = args.K
    c = configs.get(name, **over)
    name = c["name"]
    M, K, delay = c["M"], c["K"], c["delay"]
    T = c["micro_batch"] * c["seq"]
    log(f"bench: {name} M={M} K={K} delay={delay} T={T}")
    torch.cuda.set_device(0)
    if args.gemm_reference:
        print(json.dumps({"workload": name, "gemm_reference": gemm_reference(torch, c),
                          "what": "torch bf16 matmul on the stage's GEMM shapes; plain products, ms per step"}),
              flush=True)
        return
    st = binding.Stage(c)
    st.load_params(inputs.make_params(c, args.seed))
    x_all, dy_all, tgt_all = make_device_inputs(torch, c, M, args.seed)
    torch.cuda.synchronize()
    log("bench: inputs resident")
    if args.copy_probe:
        src = torch.ones(64 * 2 ** 20, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log("bench: copy probe done (3 x 256 MiB device-to-device)")

    def replay():
        st.reset_counters()
        stamps = st.run(M, x_all, dy_all, targets_all=tgt_all)
        return stamps

    for w in range(args.warmup):
        replay()
        torch.cuda.synchronize()
        log(f"bench: warmup {w + 1}/{args.warmup} done")

    # the timed region: K plain replays on the stage stream
    stream = torch.cuda.current_stream()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    start.record(stream)
    marks[0].record(stream)
    for s in range(args.steps):
        stamps = replay()
        marks[s + 1].record(stream)
    stop.record(stream)
    torch.cuda.synchronize()
    ms_total = start.elapsed_time(stop)
    per_replay = sorted(marks[s].elapsed_time(marks[s + 1]) for s in range(args.steps))
    log(f"bench: {args.steps} timed replays in {ms_total:.1f} ms")

    # after the timed region: the same number of replays with HIP events around every
    # launch, for the per-family split and the roofline of the dominant kernel
    st.set_timing(True)
    replay()                 # creates the event pool
    st.set_timing(False)
    st.set_timing(True)      # re-enabling clears the counters
    start.record(stream)
    for s in range(args.steps):
        replay()
    stop.record(stream)
    torch.cuda.synchronize()
    ms_instr = start.elapsed_time(stop) / args.steps
    st.set_timing(False)
    kt = st.kernel_times()
    log(f"bench: {args.steps} instrumented replays in {ms_instr * args.steps:.1f} ms")

    ms_step = ms_total / args.steps
    tokens_per_step = M * T
    flop_step = M * configs.algorithmic_flop_per_microbatch(c)
    value = tokens_per_step / (ms_step / 1e3)
    mfma_util = flop_step / (ms_step / 1e3) / (PEAK_BF16_TFLOPS * 1e12)

    # HBM bytes per launch from the committed counter summary, while the kernel sources are unchanged
    from paper_2606_07881_amd import profile_summary
    rec = profile_summary.read_record(TRAFFIC_PROFILE)
    traffic_ok = (rec is not None and name == configs.BENCH_CONFIG
                  and rec.get("sources_sha256") == profile_summary.sources_sha256())

    # dominant kernel family by device time; matrix families are priced in FLOP, streaming ones in bytes
    mfma_fams = {"gemm_fwd", "gemm_dgrad", "gemm_wgrad_acc", "attn_fwd", "attn_bwd"}
    fam = max(kt, key=lambda k: kt[k]["ms"])
    f = kt[fam]
    per_launch_work = f["work"] / max(f["launches"], 1)
    per_launch_ms = f["ms"] / max(f["launches"], 1)
    if fam in mfma_fams:
        achieved = per_launch_work / (per_launch_ms / 1e3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": None, "kernel": fam,
                "launches": f["launches"], "avg_launch_us": round(per_launch_ms * 1e3, 2)}
    else:
        achieved = per_launch_work / (per_launch_ms / 1e3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": None, "kernel": fam,
                "launches": f["launches"], "avg_launch_us": round(per_launch_ms * 1e3, 2)}
    if traffic_ok and fam in rec["bytes_per_launch"]:
        roof["traffic"] = rec["bytes_per_launch"][fam]
        roof["traffic_unit"] = "bytes per launch (HBM, FETCH_SIZE + WRITE_SIZE scaled by a copy kernel)"
        roof["traffic_source"] = os.path.relpath(TRAFFIC_PROFILE, ROOT)
    else:
        roof["traffic_source"] = "none: counters were taken on other kernel sources or another workload"
    families = {}
    kernel_ms = sum(v["ms"] for v in kt.values())
    for k, v in kt.items():
        if v["launches"] == 0:
            continue
        rate = v["work"] / (v["ms"] / 1e3) if v["ms"] > 0 else 0.0
        families[k] = {"ms_per_step": round(v["ms"] / args.steps, 3), "launches_per_step": v["launches"] // args.steps,
                       "share": round(v["ms"] / kernel_ms, 4),
                       ("TFLOP/s" if k in mfma_fams else "GB/s"): round(rate / (1e12 if k in mfma_fams else 1e9), 1)}

    out = {
        "metric": "stage tokens/s (fwd+bwd+accum+step) and MFMA util vs bf16 peak, 1 GPU",
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if c["dtype"] == "bf16" else "f32",
        "data": "synthetic (seeded N(0,1) stage inputs, N(0,0.01^2) output gradients, N(0,0.02^2) weights)",
        "config": {"workload": f"{name}: {WORKLOAD_SHAPE.get(name.split('+')[0], 'GPT-style')} {c['kind']} "
                               f"pipeline stage, {c['n_layers']} pre-LN blocks, "
                               f"d {c['d_model']}, {c['n_heads']}x{c['head_dim']} heads, FFN {c['d_ff']}, "
                               f"seq {c['seq']}, micro-batch {c['micro_batch']}; one step = async 1F1B replay of "
                               f"{M} micro-batches, delay {delay}, AdamW every K={K}"
                               + ("; activation-checkpointed (forward recomputed in each backward)"
                                  if c.get("recompute") else "")
                               + (f"; dropout {c['dropout']} at every site" if c.get("dropout") else "")
                               + ("; windowed weight gradients (K + delay activation slots)" if c.get("window")
                                  else "; weight gradients accumulated per backward (delay + 1 activation slots)")
                               + (f"; LM head over V={c['vocab']} with softmax cross-entropy"
                                  + (", fused (no logits kept)" if c.get("fused_head") else ", fp32 logits kept")
                                  if c["kind"] == "last" else ""),
                   "micro_batches_per_step": M, "tokens_per_step": tokens_per_step, "K": K, "delay": delay,
                   "parallelism": "single stage, 1 GPU"},
        "mfma_util": round(mfma_util, 4),
        "ms_per_step_median": round(per_replay[len(per_replay) // 2], 3),
        "ms_per_step_min_max": [round(per_replay[0], 3), round(per_replay[-1], 3)],
        "ms_per_step_with_launch_events": round(ms_instr, 3),
        "flop_per_step": flop_step,
        "stamps_delta_sum": int(stamps[:, 2].sum()),
        "arena_gib": round(binding.arena_bytes(c) / 2 ** 30, 2),
        "roofline": roof,
        "kernels": families,
    }
    if not args.no_cpu_baseline:
        log("bench: timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(c, args.seed, args.cpu_budget)
    st.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
