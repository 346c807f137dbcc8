#!/usr/bin/env python
"""Benchmark of one ReTrace speculative-decoding round on one MI355X.

A step is one round (conditioning, drafter, block verify, acceptance + rollback,
drafter context append) for every sequence of the workload, replayed from a HIP
graph with all inputs (weights, prompts' KV caches, carried state) resident in
HBM.  `value` is committed tokens per second over exactly `--steps` rounds after
`--warmup` rounds.  A profiled phase then times every kernel launch with HIP
events on the library's stream to give the per-stage breakdown and the roofline
of the dominant kernel (the fused gate|up projection GEMM).  The CPU baseline is the
float64 oracle, started from the GPU's state, timed on this host.  Last, the same
prompts are decoded target-only (one row per sequence per step, same kernels, graph
replay) for the speedup of speculative over target-only decoding.  --cond-mode runs
the component-ablation drafters (raw gated fusion, overwrite) or plain block drafting
in place of the method's conditioning.

Random-initialised weights and uniform-random prompts of the workload's shapes
stand in for the trained checkpoints and the benchmark prompts.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0            # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0        # dense bf16 MFMA
FP32_PEAK_TFLOPS = 157.3


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def build_engine(wl, W):
    from paper_2608_29748_amd import binding as B
    from paper_2608_29748_amd.engine import RoundEngine, config_from
    from workloads import weight_specs
    cfg = config_from(wl.target, dtype=wl.dtype, draft_layers=wl.draft_layers, cond_layers=wl.cond_layers,
                      block_size=wl.block_size, mask_token_id=wl.mask_token_id, max_batch=wl.batch,
                      max_seq_len=wl.max_seq_len, rope_theta=wl.rope_theta, rms_eps=wl.rms_eps, beta=wl.beta,
                      cond_mode=B.COND_MODES[wl.cond_mode], temperature=wl.temperature, top_k=wl.top_k,
                      top_p=wl.top_p, sample_seed=wl.sample_seed)
    return RoundEngine(cfg, [W[name] for name, _, _ in weight_specs(wl)])


DOMINANT = "gemm_gate_up"
REPLAY_KINDS = (0, 1, 2, 3, 4, 5, 6, 7, 10)   # GEMM classes, attention, merge, LM head


def dominant_desc(wl):
    """The dominant kernel's launch class at this workload's verify shape."""
    rows = wl.batch * wl.block_size
    kern = "gemm16_kernel" if rows <= 64 else "gemm_mid_kernel"
    # at most 16 bf16 rows, K <= 2560 and at least 16384 columns: the k-slab kernel with
    # the activation block staged in LDS (one slab)
    if rows <= 16 and wl.dtype == "bf16" and wl.target.hidden <= 2560 and 2 * wl.target.ffn >= 16384:
        kern = "gemm16_slab_kernel"
    return (f"gemm_gate_up: fused gate|up projection GEMM with SwiGLU epilogue ({kern}, {wl.dtype} MFMA, "
            f"{rows} rows x {2 * wl.target.ffn} columns x K {wl.target.hidden})")


GEMM_SOURCES = ("paper_2608_29748_amd/csrc/gemm.hip", "paper_2608_29748_amd/csrc/gemm.h",
                "paper_2608_29748_amd/csrc/common.h")
MID_SOURCES = GEMM_SOURCES + ("paper_2608_29748_amd/csrc/gemm_mid.hip",)


def traffic_sources(wl):
    """The sources a traffic record of the dominant GEMM depends on: the mid-size kernel
    (more than 64 rows per round) adds its own file."""
    return MID_SOURCES if wl.batch * wl.block_size > 64 else GEMM_SOURCES


def gemm_source_hash(sources=GEMM_SOURCES) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in sources:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(wl):
    """HBM bytes per launch of the dominant kernel from the committed counter summary
    (rocprofv3 FETCH_SIZE and WRITE_SIZE passes, each scaled by the same counter's
    reading for a plain copy of known size); None when that summary was taken on
    different kernel sources or is absent."""
    path = os.path.join(ROOT, "profiles", f"{DOMINANT}_{wl.name}_traffic.md")
    if not os.path.exists(path):
        return None
    rec = None
    with open(path) as fh:
        for line in fh:
            if line.startswith("traffic-json:"):
                rec = json.loads(line.split(":", 1)[1])
    if not rec or rec.get("source_sha256") != gemm_source_hash(traffic_sources(wl)):
        return None
    return rec["bytes_per_launch"]


def copy_calibration(nbytes: int = 1 << 30):
    """A plain device-to-device copy of known size, for scaling the HBM byte counters."""
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    log(f"copy calibration: 3 copies of {nbytes} bytes")


def cpu_baseline(eng, wl, W, prompts, seconds: float):
    """Oracle rounds for sequence 0, started from the GPU's KV caches and carried state
    (an oracle prefill of the full prompt is far outside the time budget)."""
    from threadpoolctl import threadpool_info
    from oracle import OracleModel, OracleRunner
    from paper_2608_29748_amd import binding as B
    s = wl.target
    # float64 copies of every weight up to the 4B shape; float32 copies (exact for bf16,
    # widened on use) beyond, so that the 8B / 14B shapes fit in host memory
    big = sum(v.nbytes for v in W.values()) > 12e9
    model = OracleModel(wl, W, cache="f32" if big else True)
    R = OracleRunner(model)
    st_arr = eng.read(B.RT_T_STATE, 0, (9,), np.int32)
    P = int(st_arr[0])
    st = model.new_state(prompts[0], wl.new_tokens)
    et = np.uint16 if wl.dtype == "bf16" else np.float32
    f64 = (lambda a: (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)) if wl.dtype == "bf16" \
        else (lambda a: a.astype(np.float64))
    shp = (P, s.n_kv_heads, s.head_dim)
    for l in range(s.n_layers):
        st.tgt_k[l, :P] = f64(eng.read(B.RT_T_TARGET_K + l, 0, shp, et))
        st.tgt_v[l, :P] = f64(eng.read(B.RT_T_TARGET_V + l, 0, shp, et))
    for l in range(wl.draft_layers):
        st.ctx_k[l, :P] = f64(eng.read(B.RT_T_DRAFT_K + l, 0, shp, et))
        st.ctx_v[l, :P] = f64(eng.read(B.RT_T_DRAFT_V + l, 0, shp, et))
    kd = np.float16 if wl.dtype == "bf16" else np.float32
    st.hD_prev = eng.read(B.RT_T_HD, 0, (wl.block_size, s.hidden), kd).astype(np.float64)
    st.hT_prev = eng.read(B.RT_T_HT, 0, (wl.block_size, s.hidden), kd).astype(np.float64)
    st.P, st.anchor, st.r, st.cond_len = P, int(st_arr[1]), int(st_arr[2]), int(st_arr[3])
    st.rnd = int(st_arr[8])
    st.generated = [0] * (wl.new_tokens - int(st_arr[4]))
    # one-time float64 conversion of the weights (the oracle's setup) outside the sample
    t0 = time.perf_counter()
    for name in W:
        model.W[name]
    log(f"oracle weight conversion {time.perf_counter() - t0:.1f}s")
    rounds, committed = 0, 0
    t0 = time.perf_counter()
    while True:
        rec = R.round(st)
        rounds += 1
        committed += len(rec.committed)
        el = time.perf_counter() - t0
        if el >= seconds or st.done:
            break
    blas = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    host = os.cpu_count() or 1
    usable = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else host
    used = min(blas, usable)
    return {"value": committed / el, "unit": "tokens/s", "cores": used, "kind": "oracle",
            "sample": f"{rounds} round(s) of sequence 0 at context {P}, started from the GPU's KV caches and "
                      f"carried state; {el:.1f}s of wall time; float64 numpy, {blas} BLAS threads on "
                      f"{usable} usable of {host} host CPUs",
            "host_cpus": host, "usable_cpus": usable, "blas_threads": blas,
            "seconds_per_round": el / rounds}


def target_only(eng, wl, prompts, steps: int, spec_value: float, warmup: int = 4):
    """Target-only greedy decoding of the same prompts on the same kernels, one row per
    sequence per step, graph-replayed: committed tokens per second over `steps` steps."""
    import torch
    steps = min(steps, wl.new_tokens - 1 - warmup)
    eng.prefill(prompts, wl.new_tokens)
    eng.ar_steps(warmup)
    torch.cuda.synchronize()
    done, left = 0, steps
    t0 = time.perf_counter()
    while left:
        c = min(left, 256)
        _, n = eng.ar_steps(c)
        done += int(n.sum())
        left -= c
    el = time.perf_counter() - t0
    tps = done / el
    return {"tokens_per_s": tps, "ms_per_step": el * 1e3 / steps, "steps": steps, "warmup": warmup,
            "speedup_of_speculative": spec_value / tps}


def stream_ceiling(nbytes: int, buf) -> dict:
    """Best plain-read time of nbytes (one kernel of non-temporal loads, 512, 1024 or 2048
    workgroups, 20 launches each, every launch on data the memory-side cache does not
    hold) on this GPU: the streaming ceiling of a single kernel of that size."""
    from paper_2608_29748_amd import binding as B
    n = max(16, int(nbytes) // 16 * 16)
    us = min(B.rt_stream_read(buf.data_ptr(), buf.numel(), n, g, 20) for g in (512, 1024, 2048))
    return {"bytes": n, "us": us, "GBs": n / (us * 1e-6) / 1e9}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="qwen3-4b-shape")
    ap.add_argument("--batch", type=int, default=None, help="override the workload's batch (concurrency sweep)")
    ap.add_argument("--profile-rounds", type=int, default=5)
    ap.add_argument("--replay-reps", type=int, default=20)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--ar-steps", type=int, default=64, help="timed target-only greedy steps (0: skip)")
    ap.add_argument("--cond-mode", choices=["retrace", "raw_gated", "overwrite", "lowrank", "off"], default="retrace",
                    help="drafter conditioning: the method, a component-ablation variant, or none")
    ap.add_argument("--temperature", type=float, default=0.0,
                    help="0: greedy; > 0: speculative sampling with the workload's top-k / top-p (20 / 0.95)")
    ap.add_argument("--prompt-len", type=int, default=None,
                    help="override every prompt's length (short prefills for counter runs; verify GEMM shapes "
                         "do not depend on it, attention does)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run plain 1 GiB copies (reference reading for the HBM byte counters)")
    ap.add_argument("--stream-probe", action="store_true",
                    help="also time a plain read of each replayed kernel's bytes per launch (the single-kernel "
                         "streaming ceiling of that size) and of 22 MB .. 1 GiB")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported (a round's state is "
              "per sequence, so batches shard by sequence across GPUs with no exchange during a round)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from workloads import get, make_prompts, make_weights

    over = {"cond_mode": args.cond_mode, "temperature": args.temperature}
    if args.batch is not None:
        over["batch"] = args.batch
    if args.prompt_len is not None:
        over["prompt_len"] = (args.prompt_len, args.prompt_len)
    wl = get(args.workload, **over)
    need = args.warmup + args.steps + args.profile_rounds + 2
    if need > wl.new_tokens - 1:
        raise SystemExit(f"{need} rounds exceed the workload's generation budget of {wl.new_tokens} tokens")
    t0 = time.perf_counter()
    W = make_weights(wl)
    prompts = make_prompts(wl)
    log(f"weights {sum(v.nbytes for v in W.values()) / 1e9:.2f} GB generated in {time.perf_counter() - t0:.1f}s")
    t0 = time.perf_counter()
    eng = build_engine(wl, W)
    log(f"engine init {time.perf_counter() - t0:.1f}s")
    t0 = time.perf_counter()
    eng.prefill(prompts, wl.new_tokens)
    torch.cuda.synchronize()
    prefill_s = time.perf_counter() - t0
    log(f"prefill {prefill_s:.2f}s")

    for _ in range(args.warmup):
        eng.spec_round()
    torch.cuda.synchronize()
    committed, accepted, per_round = 0, [], []
    t_start = time.perf_counter()
    for _ in range(args.steps):
        r0 = time.perf_counter()
        tok, n, a = eng.spec_round()
        per_round.append(time.perf_counter() - r0)
        committed += int(n.sum())
        accepted.extend(int(x) for x in a)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    value = committed / elapsed
    log(f"timed {args.steps} rounds: {elapsed * 1e3 / args.steps:.3f} ms/round, {value:.1f} tokens/s")

    # profiled rounds: a HIP-event pair on every launch (per-stage breakdown; a launch's
    # pair also spans its dispatch, so these times exceed the kernels' execution times)
    from paper_2608_29748_amd import binding as B
    kinds, stages = {}, []
    for _ in range(args.profile_rounds):
        stats, st_ms, tok, n, a = eng.profile_round()
        stages.append(st_ms)
        for s in stats:
            k = kinds.setdefault(s["kind"], {"launches": 0, "ms": 0.0, "bytes": 0.0, "flops": 0.0})
            for f in ("launches", "ms", "bytes", "flops"):
                k[f] += s[f]
    stage_med = {n: float(np.median([s[i] for s in stages])) for i, n in enumerate(B.STAGE_NAMES)}
    # kernel replay: each replayable class's launches of one round, back to back in a HIP
    # graph between two HIP events on the library's stream (their execution time)
    replay = {}
    for kind in REPLAY_KINDS:
        r = eng.time_kernel(kind, args.replay_reps)
        if r["launches"]:
            replay[r["kind"]] = r
    kernels = {}
    for name, v in kinds.items():
        if not v["launches"]:
            continue
        launches_per_round = v["launches"] / args.profile_rounds
        rec = {"launches_per_round": launches_per_round, "GB_per_launch": v["bytes"] / v["launches"] / 1e9,
               "us_per_launch_profiled_round": v["ms"] * 1e3 / v["launches"]}
        if name in replay:
            r = replay[name]
            us = r["ms"] * 1e3 / r["launches"]
            rec["us_per_launch"] = us
            rec["achieved_GBs"] = r["bytes"] / r["launches"] / (us * 1e-6) / 1e9
            rec["achieved_TFLOPs"] = r["flops"] / r["launches"] / (us * 1e-6) / 1e12
        kernels[name] = rec
    round_ms_p50 = float(np.median(per_round) * 1e3)
    # the timed loop's per-round wall times and its mean must describe the same rounds
    assert abs(round_ms_p50 - elapsed * 1e3 / args.steps) <= 0.25 * elapsed * 1e3 / args.steps, \
        (round_ms_p50, elapsed * 1e3 / args.steps)
    dom = replay[DOMINANT]
    per_launch_bytes = dom["bytes"] / dom["launches"]
    per_launch_flops = dom["flops"] / dom["launches"]
    per_launch_us = dom["ms"] * 1e3 / dom["launches"]
    rows = wl.batch * wl.block_size
    if rows <= 64:   # weight streaming: 16 flop/byte per 16 rows, far below the ridge
        bound, unit, peak = "hbm", "GB/s", HBM_PEAK_GBS
        achieved = per_launch_bytes / (per_launch_us * 1e-6) / 1e9
    else:            # 128..512 rows: the bf16 matrix cores bound the mid-size GEMM
        bound, unit, peak = "mfma", "TFLOP/s", BF16_PEAK_TFLOPS
        achieved = per_launch_flops / (per_launch_us * 1e-6) / 1e12
    stream = None
    if args.stream_probe:
        buf = torch.empty(2 << 30, dtype=torch.uint8, device="cuda")
        buf.fill_(1)
        torch.cuda.synchronize()
        stream = {"sizes": [stream_ceiling(mb << 20, buf) for mb in (22, 32, 51, 100, 400, 1024)]}
        for name, rec in kernels.items():
            if "us_per_launch" in rec and rec["GB_per_launch"] * 1e9 <= (1 << 30):
                c = stream_ceiling(rec["GB_per_launch"] * 1e9, buf)
                rec["stream_ceiling_GBs"] = c["GBs"]
                rec["frac_of_stream_ceiling"] = rec["achieved_GBs"] / c["GBs"]
        del buf
        log("stream probe: " + ", ".join(f"{r['bytes'] >> 20} MB {r['GBs']:.0f} GB/s" for r in stream["sizes"]))
    if args.copy_calibration:
        copy_calibration()

    out = {
        "metric": "committed tokens/s/GPU, Qwen3-4B shape b=1; verify-pass % MFMA/HBM roofline",
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic: seeded N(0,0.02) random-init weights, uniform-random prompt tokens",
        "config": {"workload": wl.name, "batch": wl.batch, "prompt_len": list(wl.prompt_len),
                   "block_size": wl.block_size, "new_tokens": wl.new_tokens, "hidden": wl.target.hidden,
                   "layers": wl.target.n_layers, "draft_layers": wl.draft_layers,
                   "cond_layers": list(wl.cond_layers), "cond_mode": wl.cond_mode, "temperature": wl.temperature,
                   "top_k": wl.top_k, "top_p": wl.top_p, "parallelism": "single GPU"},
        "roofline": {"bound": bound, "kernel": dominant_desc(wl),
                     "achieved": achieved, "peak": peak, "unit": unit, "frac": achieved / peak,
                     "traffic": measured_traffic(wl), "traffic_unit": "bytes per launch (HBM fetch + write)",
                     "algorithmic_bytes_per_launch": per_launch_bytes, "algorithmic_flops_per_launch": per_launch_flops,
                     "us_per_launch": per_launch_us,
                     "hbm_frac": per_launch_bytes / (per_launch_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                     "mfma_frac": per_launch_flops / (per_launch_us * 1e-6) / 1e12 / BF16_PEAK_TFLOPS,
                     "launches_per_round": dom["launches"],
                     "timing": f"HIP events around {args.replay_reps} graph replays of the round's "
                               f"{dom['launches']} launches of this kernel on the library's stream"},
        "stages_ms_median": stage_med,
        "kernels": kernels,
        "acceptance": {"mean_A": float(np.mean(accepted)) if accepted else None,
                       "mean_committed_per_round": committed / args.steps / wl.batch},
        "round_ms_p50": round_ms_p50,
        "prefill_s": prefill_s,
    }
    if stream is not None:
        out["stream_probe"] = stream
    if wl.dtype == "f32":
        out["roofline"]["note"] = ("cache-resident fp32 model (about 13 MB per round): rounds are latency-bound, "
                                   "the HBM fraction is not a meaningful bound")
    if not args.no_cpu_baseline:
        try:
            out["cpu_baseline"] = cpu_baseline(eng, wl, W, prompts, args.cpu_seconds)
        except MemoryError as e:   # pragma: no cover
            out["cpu_baseline"] = {"error": f"oracle did not fit in host memory: {e}"}
    if args.ar_steps > 0:
        out["target_only"] = target_only(eng, wl, prompts, args.ar_steps, value)
        log(f"target-only: {out['target_only']['ms_per_step']:.3f} ms/step, "
            f"{out['target_only']['tokens_per_s']:.1f} tokens/s, "
            f"speedup {out['target_only']['speedup_of_speculative']:.2f}x")
    eng.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
