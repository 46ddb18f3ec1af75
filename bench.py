"""Benchmark of the Jacobi-decoding hot path on one MI355X.

A step is one request through the whole path: prefill of a 512-token prompt, then Jacobi
decoding of 256 tokens in blocks of n = 16 on the LLaMA-2-7B shape (bf16, seeded random
weights). Guesses are the GPU's own greedy AR continuation with a fraction p = 0.3 of
positions corrupted and re-drawn after every iteration (emulating a consistency-trained model);
the block shrinks as in the paper's algorithm. value = generated tokens / second over the
timed steps (inputs resident on the device when timing starts).

--workload 7b_long (prompt 2048, n = 64, 512 new) and 7b_batched (16 sequences, prompts uniform
in [256, 1024], n = 32, 256 new each, corruption rates uniform in [0.1, 0.6], all decoded in one
batched loop; value = tokens of all sequences / second) measure the other configurations.
--workload 7b_loss times the CLLM training loss at the LLaMA-2-7B LM head (32000 x 4096 bf16):
a step is one forward + backward of the loss head over 16 teacher/student pairs (one n = 16
block) and 48 AR rows, on device arrays; value = loss rows / second.

Prints one JSON line. --gpus above 1 is refused: the path runs on one GPU.
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
TIMING_EVERY = 33  # kernel-timing sample stride (coprime with 32 layers)
METRIC = "Jacobi-step ms & accepted tokens/s, 7B-shape bf16 n=16; HBM GB/s vs peak"
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "traffic_gemm_gate_up_llama7b_n16.md")
LOSS_SUMMARY = os.path.join(ROOT, "profiles", "loss_head_llama7b.md")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


GEMM_SOURCES = ("gemm.hip", "gemm.h", "device.h")  # everything the streaming GEMM's code depends on


def kernel_source_hash(files=GEMM_SOURCES):
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2403_00835_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def stream_ceiling():
    """The measured streaming-read rate (GB/s) recorded in the GEMM traffic summary, or None."""
    if not os.path.exists(TRAFFIC_SUMMARY):
        return None
    m = re.search(r"stream_read_gbps:\s*([0-9.]+)", open(TRAFFIC_SUMMARY).read())
    return float(m.group(1)) if m else None


def measured_traffic(summary=TRAFFIC_SUMMARY, files=GEMM_SOURCES):
    """HBM bytes per launch of a kernel from a committed rocprofv3 counter summary, if it was
    taken on the current source of `files`; otherwise None."""
    if not os.path.exists(summary):
        return None
    text = open(summary).read()
    m_hash = re.search(r"kernel_source_hash:\s*([0-9a-f]+)", text)
    m_bytes = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m_hash or not m_bytes or m_hash.group(1) != kernel_source_hash(files):
        return None
    return float(m_bytes.group(1))


ORACLE_CONTEXT = 16  # prompt tokens of the oracle's iteration sample


def oracle_iteration_s(cfg, ws, n, reps=5):
    """Seconds of the oracle, as it stands, for one Jacobi iteration of n rows at this shape
    after a prefill of ORACLE_CONTEXT tokens (the timed workloads iterate at contexts of 512 and
    more; attention over 16 instead of several hundred keys is about 2% of the iteration's work at
    the 7B shape, and a 512-token prefill would cost the oracle about a minute): the median of
    `reps` evaluations of the block."""
    import oracle
    from paper_2403_00835_amd import workload
    log("[bench] cpu baseline: oracle on the host")
    tensors = [workload.as_f32(cfg, t) for t in ws]
    om = oracle.Model(cfg, tensors)
    st = oracle.State(om, ORACLE_CONTEXT + n + 1)
    prompt = workload.make_prompt(cfg, ORACLE_CONTEXT, seed=11)
    y0 = st.prefill(prompt)
    block = np.array([y0] + list(workload.make_prompt(cfg, n - 1, seed=12)), dtype=np.int32)
    times = []
    for _ in range(reps):
        t0 = time.perf_counter()
        st.eval_block(block)
        times.append(time.perf_counter() - t0)
    del om, tensors
    return float(np.median(times)), oracle.num_threads()


def cpu_baseline(cfg, ws, mean_accept, n):
    """The oracle's tokens/s: one n-row iteration, scaled by the GPU run's mean accepted length."""
    dt, cores = oracle_iteration_s(cfg, ws, n)
    return {"value": mean_accept / dt, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"one Jacobi iteration of {n} rows at the 7B shape at a context of {ORACLE_CONTEXT} keys "
                      f"(the workload's is 512-768) after a {ORACLE_CONTEXT}-token prefill (median of 5: "
                      f"{dt:.2f} s), scaled by the GPU run's mean accepted length {mean_accept:.2f}",
            "context": ORACLE_CONTEXT, "iteration_s": dt}


def calibration_copy():
    """One device-to-device copy of 1 GiB: a kernel of known traffic, for scaling hardware byte
    counters."""
    import torch
    src = torch.empty(1 << 28, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    log("[bench] calibration copy: 1073741824 bytes read, 1073741824 bytes written")
    del src, dst


def oracle_decodes():
    """The oracle's own greedy AR and Jacobi decoding rates (tokens/s, wall clock on the host
    threads): full decodes of the tiny and small workloads, and a shortened 7B decode (16-token
    prompt, 2 blocks of n = 16). Jacobi guesses are the oracle's AR continuation corrupted at
    p = 0.3 and re-drawn each iteration, as in the GPU benchmark; the outputs must equal."""
    import oracle
    from paper_2403_00835_amd import workload
    from paper_2403_00835_amd.configs import BLOCK_SHRINK, GUESS_STREAM_REINJECT, LLAMA7B, SMALL, TINY
    out = {}
    for name, cfg, plen, n, max_new in (("tiny", TINY, 16, 8, 32), ("small", SMALL, 128, 16, 256),
                                        ("7b_2blocks", LLAMA7B, 16, 16, 32)):
        log(f"[bench] oracle decodes: {name}")
        ws = workload.make_weights(cfg)
        om = oracle.Model(cfg, [workload.as_f32(cfg, t) for t in ws])
        del ws
        prompt = workload.make_prompt(cfg, plen, seed=13)
        t0 = time.perf_counter()
        ar = om.ar_decode(prompt, max_new)
        t_ar = time.perf_counter() - t0
        spec = oracle.GuessSpec(GUESS_STREAM_REINJECT, BLOCK_SHRINK, ar, p=0.3, seed=3)
        t0 = time.perf_counter()
        jo, st = om.jacobi_decode(prompt, n, max_new, spec)
        t_j = time.perf_counter() - t0
        if not np.array_equal(jo, ar):
            raise RuntimeError(f"oracle Jacobi output differs from oracle AR ({name})")
        out[name] = {"prompt": plen, "n": n, "tokens": max_new, "ar_tokens_per_s": round(max_new / t_ar, 3),
                     "jacobi_tokens_per_s": round(max_new / t_j, 3), "jacobi_iterations": st["steps"],
                     "cores": oracle.num_threads()}
        del om
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="7b", choices=["7b", "small", "7b_long", "7b_batched", "7b_loss"])
    ap.add_argument("--p", type=float, default=0.3)
    ap.add_argument("--prefill-chunk", type=int, default=512,
                    help="prompt rows per prefill pass (prefill values do not depend on it)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--oracle-decode", action="store_true",
                    help="also time the oracle's AR and Jacobi decoding (tiny, small, shortened 7B; about "
                         "a minute of host time) and add it to the line as oracle_decode")
    ap.add_argument("--sweep-n", action="store_true",
                    help="single-sequence workloads: after the timed steps, decode the same request once per "
                         "block size n in 1, 8, 16, 24, 32, 48, 64 with sliding blocks (every iteration carries "
                         "n rows) and add the iteration cost against n to the line as n_sweep")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="after the timed steps, copy 1 GiB device-to-device (a kernel of known traffic "
                         "for scaling hardware byte counters)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path (--gpus must be 1)",
              file=sys.stderr, flush=True)
        sys.exit(2)

    import torch
    from paper_2403_00835_amd import binding, workload
    from paper_2403_00835_amd.configs import BLOCK_SHRINK, GUESS_STREAM, GUESS_STREAM_REINJECT, WORKLOADS

    if args.workload == "7b_loss":
        return main_loss(args)
    wl = WORKLOADS[args.workload]
    if wl.batch > 1:
        return main_batched(args, wl)
    cfg = wl.model
    P, n, max_new = wl.prompt_len, wl.n, wl.max_new
    torch.cuda.init()
    stream = torch.cuda.current_stream()
    log(f"[bench] generating {cfg.streamed_params() / 1e9:.2f} B streamed parameters")
    t0 = time.time()
    ws = workload.make_weights(cfg)
    log(f"[bench] weights drawn in {time.time() - t0:.1f} s; uploading")
    model = binding.Model(cfg, max_ctx=P + max_new + n + 64, max_block=max(n, 16), max_new=max_new,
                          prefill_chunk=args.prefill_chunk,
                          stream=stream.cuda_stream, weights=ws)
    prompt = workload.make_prompt(cfg, P)
    log("[bench] GPU AR decode (guess stream and AR baseline)")
    ar, ar_stats = model.ar_decode(prompt, max_new)
    ar_tps = max_new / ((ar_stats["prefill_ms"] + ar_stats["decode_ms"]) / 1e3)

    def one_step():
        return model.jacobi_decode(prompt, n, max_new, policy=GUESS_STREAM_REINJECT, block_policy=BLOCK_SHRINK,
                                   stream=ar, p=args.p, seed=3)

    for _ in range(args.warmup):
        out, _ = one_step()
        if not np.array_equal(out, ar):
            raise RuntimeError("Jacobi output differs from greedy AR output")
    torch.cuda.synchronize()
    # iteration launches only (not prefill chunks); one launch in TIMING_EVERY is bracketed by
    # events, rotating over the layers (every bracket adds queue time to the timed decode)
    model.timing_enable("gate_up", max_rows=n, every=TIMING_EVERY)
    stats = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        out, st = one_step()
        stats.append(st)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    launches, gu_ms = model.timing_read()
    model.timing_enable(-1)
    if not np.array_equal(out, ar):
        raise RuntimeError("Jacobi output differs from greedy AR output")

    tokens = args.steps * max_new
    value = tokens / elapsed
    iters = sum(s["steps"] for s in stats)
    decode_ms = sum(s["decode_ms"] for s in stats)
    prefill_ms = sum(s["prefill_ms"] for s in stats) / len(stats)
    iter_ms = decode_ms / iters
    mean_accept = tokens / iters
    wbytes = model.streamed_weight_bytes()
    d, F = cfg.d_model, cfg.ffn_dim
    # gate/up launch: packed weights (2 * F_pad * d bf16) + operand rows read (hi and lo bf16
    # planes, 4 bytes per value) + SwiGLU rows written (4 bytes per value) + row-factor partials,
    # at the mean block rows of the timed iterations (the sampled launches rotate over layers and
    # iterations, whose blocks shrink)
    f_pad = (F + 31) // 32 * 32
    mean_rows = sum(s["rows"] for s in stats) / iters
    gu_bytes = round(2 * f_pad * d * 2 + mean_rows * (d * 4 + f_pad * 4 + (d // 16) * 4))
    gu_avg_s = gu_ms / 1e3 / max(launches, 1)
    achieved = gu_bytes / gu_avg_s / 1e9
    # the same launches against the bf16 MFMA peak: algorithmic flops 2 * rows * (2 F) * d per
    # launch at the mean block rows; the executed MFMA work is twice that (hi and lo planes)
    gu_tflops = 2.0 * mean_rows * 2 * f_pad * d / gu_avg_s / 1e12 if gu_ms > 0 else 0.0
    traffic = measured_traffic() if (args.workload == "7b" and n == 16) else None
    ceiling = stream_ceiling()
    mean_ctx = P + max_new / 2
    kv_bytes = cfg.n_layers * 2 * mean_ctx * d * 2
    step_gbps = (wbytes + kv_bytes) / (iter_ms / 1e3) / 1e9

    if args.calibrate_copy:
        calibration_copy()

    # trajectory profile of one more decode of the same request (outside the timed steps):
    # fast-forwarded and stationary token counts (the paper's profiling of Jacobi trajectories),
    # and the recording's cost: that decode's device time against the timed decodes' mean
    model.trace_enable(True)
    tr_out, tr_st = one_step()
    traj = model.trace_read()
    model.trace_enable(False)
    tc = binding.trace_count(traj, tr_out, n, BLOCK_SHRINK)
    if not np.array_equal(tr_out, ar):
        raise RuntimeError("traced Jacobi output differs from greedy AR output")

    # the printed algorithm's policy on the same request, outside the timed steps: the corrupted
    # stream initialises each block, then the model's own predictions iterate (shrink blocks)
    torch.cuda.synchronize()
    p0 = time.perf_counter()
    pp_out, pp_st = model.jacobi_decode(prompt, n, max_new, policy=GUESS_STREAM, block_policy=BLOCK_SHRINK,
                                        stream=ar, p=args.p, seed=3)
    torch.cuda.synchronize()
    pp_s = time.perf_counter() - p0
    if not np.array_equal(pp_out, ar):
        raise RuntimeError("Jacobi output (printed policy) differs from greedy AR output")
    printed = {"policy": f"guesses = GPU greedy continuation corrupted at p={args.p} for each block's initial "
                         f"state, then the model's own predictions (the printed algorithm), shrink blocks",
               "iterations": pp_st["steps"], "mean_accepted": round(max_new / pp_st["steps"], 3),
               "tokens_per_s": round(max_new / pp_s, 3),
               "decode_tokens_per_s": round(max_new / (pp_st["decode_ms"] / 1e3), 3),
               "iteration_ms": round(pp_st["decode_ms"] / pp_st["steps"], 4),
               "speedup_vs_ar": round(max_new / pp_s / ar_tps, 3)}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, ws, mean_accept, n)

    line = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if cfg.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: prompt {P}, n={n}, {max_new} new tokens, guesses = GPU greedy "
                               f"continuation corrupted at p={args.p} and re-drawn each iteration, shrink blocks",
                   "prompt_len": P, "n": n, "max_new": max_new, "p": args.p, "batch": 1,
                   "layers": cfg.n_layers, "d_model": cfg.d_model, "prefill_chunk": args.prefill_chunk},
        "jacobi_step_ms": round(iter_ms, 4),
        "iteration_ms": {"mean": round(iter_ms, 4),
                         "p10": round(float(np.median([x["iter_ms_p10"] for x in stats])), 4),
                         "p50": round(float(np.median([x["iter_ms_p50"] for x in stats])), 4),
                         "p90": round(float(np.median([x["iter_ms_p90"] for x in stats])), 4),
                         "full_block_p10": round(float(np.median([x["iter_ms_full_p10"] for x in stats])), 4),
                         "full_block_p50": round(float(np.median([x["iter_ms_full_p50"] for x in stats])), 4),
                         "full_block_p90": round(float(np.median([x["iter_ms_full_p90"] for x in stats])), 4)},
        "decode_tokens_per_s": round(tokens / (decode_ms / 1e3), 3),
        "iterations_per_step": iters / args.steps,
        "mean_accepted": round(mean_accept, 3),
        "prefill_ms": round(prefill_ms, 3),
        "ar_tokens_per_s": round(ar_tps, 3),
        "speedup_vs_ar": round(value / ar_tps, 3),
        "step_hbm_gbps": round(step_gbps, 1),
        "step_hbm_frac": round(step_gbps / HBM_PEAK_GBPS, 4),
        "printed_policy": printed,
        "trajectory": {"decode_ms_recorded": round(tr_st["decode_ms"], 3),
                       "decode_ms_unrecorded_mean": round(decode_ms / len(stats), 3),
                       "fast_forward_mean": round(tc["fast_forward_mean"], 4), "stationary": tc["stationary"],
                       "blocks": tc["windows"], "stationary_per_block": round(tc["stationary_per_window"], 4)},
        "roofline": {"bound": "hbm", "kernel": "gemm gate/up + SwiGLU (per layer)", "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": traffic, "algorithmic_bytes": gu_bytes, "avg_launch_us": round(gu_avg_s * 1e6, 2),
                     "launches": launches, "stream_read_gbps": ceiling,
                     "frac_of_stream_read": round(achieved / ceiling, 4) if ceiling else None},
        "roofline_mfma": {"bound": "mfma", "kernel": "gemm gate/up + SwiGLU (per layer)",
                          "achieved": round(gu_tflops, 2), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                          "frac": round(gu_tflops / BF16_PEAK_TFLOPS, 4),
                          "executed_mfma_tflops": round(2 * gu_tflops, 2), "mean_rows": round(mean_rows, 2)},
        "cpu_baseline": cpu,
    }
    if args.oracle_decode:
        line["oracle_decode"] = oracle_decodes()
    if args.sweep_n:
        model.close()
        line["n_sweep"] = sweep_n(cfg, ws, prompt, ar, max_new, args, stream, wbytes)
    print(json.dumps(line), flush=True)


def sweep_n(cfg, ws, prompt, ar, max_new, args, stream, wbytes):
    """Iteration cost against the block size n on one request (the cost side of the paper's
    ablation over n): sliding blocks, so every iteration has n rows; guesses re-drawn from the
    corrupted greedy continuation (the headline's emulation). n = 1 is greedy AR decoding."""
    import torch
    from paper_2403_00835_amd import binding
    from paper_2403_00835_amd.configs import BLOCK_SLIDE, GUESS_STREAM_REINJECT
    P = len(prompt)
    model = binding.Model(cfg, max_ctx=P + max_new + 128, max_block=64, max_new=max_new,
                          prefill_chunk=args.prefill_chunk, stream=stream.cuda_stream, weights=ws)
    out = []
    try:
        for n in (1, 8, 16, 24, 32, 48, 64):
            if n == 1:
                tok, st = model.ar_decode(prompt, max_new)
            else:
                tok, st = model.jacobi_decode(prompt, n, max_new, policy=GUESS_STREAM_REINJECT,
                                              block_policy=BLOCK_SLIDE, stream=ar, p=args.p, seed=3)
            torch.cuda.synchronize()
            if not np.array_equal(tok, ar):
                raise RuntimeError(f"n={n}: output differs from greedy AR output")
            it_ms = st["iter_ms_full_p50"]  # iterations with n rows (the last ones may have fewer)
            kv = cfg.n_layers * 2 * (P + max_new / 2) * cfg.d_model * 2
            out.append({"n": n, "iterations": st["steps"], "mean_accepted": round(max_new / st["steps"], 3),
                        "iteration_ms": round(it_ms, 4),
                        "decode_tokens_per_s": round(max_new / (st["decode_ms"] / 1e3), 3),
                        "step_hbm_gbps": round((wbytes + kv) / (it_ms / 1e3) / 1e9, 1),
                        "gemm_tflops": round(2.0 * cfg.streamed_params() * n / (it_ms / 1e3) / 1e12, 2)})
            log(f"[bench] n={n}: {out[-1]}")
    finally:
        model.close()
    return out


def main_batched(args, wl):
    """Batched ragged decoding: all sequences of the workload in one device-resident loop."""
    import torch
    from paper_2403_00835_amd import binding, workload
    from paper_2403_00835_amd.configs import BLOCK_SHRINK, GUESS_STREAM_REINJECT

    cfg = wl.model
    n, max_new = wl.n, wl.max_new
    prompts, ps = workload.make_batch(cfg, wl.batch, wl.prompt_len_range, wl.p_range)
    B = len(prompts)
    ids = list(range(B))
    torch.cuda.init()
    stream = torch.cuda.current_stream()
    log(f"[bench] generating {cfg.streamed_params() / 1e9:.2f} B streamed parameters")
    ws = workload.make_weights(cfg)
    model = binding.Model(cfg, max_ctx=wl.prompt_len_range[1] + max_new + n + 64, max_block=n, max_new=max_new,
                          max_batch=B, stream=stream.cuda_stream, weights=ws, prefill_chunk=args.prefill_chunk)
    log(f"[bench] batched GPU AR decode of {B} sequences (guess streams and AR baseline)")
    ar, ar_stats = model.jacobi_decode_batch(ids, prompts, 1, max_new)
    ar_tps = B * max_new / ((ar_stats[0]["prefill_ms"] + ar_stats[0]["decode_ms"]) / 1e3)
    specs = [dict(policy=GUESS_STREAM_REINJECT, block_policy=BLOCK_SHRINK, stream=ar[b], p=float(ps[b]), seed=3)
             for b in range(B)]

    def one_step():
        return model.jacobi_decode_batch(ids, prompts, n, max_new, specs=specs)

    for _ in range(args.warmup):
        out, _ = one_step()
        if not np.array_equal(out, ar):
            raise RuntimeError("batched Jacobi output differs from batched greedy AR output")
    torch.cuda.synchronize()
    model.timing_enable("gate_up", max_rows=64, every=TIMING_EVERY)  # iteration launches (row tiles of 64)
    stats = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        out, st = one_step()
        stats.append(st)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    launches, gu_ms = model.timing_read()
    model.timing_enable(-1)
    if not np.array_equal(out, ar):
        raise RuntimeError("batched Jacobi output differs from batched greedy AR output")

    # Algorithm 1's collection of the same batch (outside the timed steps): the batched decode
    # with trajectory recording, then each sequence's states, fixed points and augmented copies
    # (rate 0.5); its wall-clock rate in collected states per second
    from paper_2403_00835_amd import collect
    torch.cuda.synchronize()
    c0 = time.perf_counter()
    entries = collect.collect(model, prompts, n, max_new, specs=specs, rate=0.5, seed=7)
    coll_s = time.perf_counter() - c0
    n_states = sum(len(e["states"]) for e in entries)

    tokens = args.steps * B * max_new
    value = tokens / elapsed
    iters = [max(s["steps"] for s in st) for st in stats]  # batched iterations per step
    rows = sum(s["rows"] for st in stats for s in st)
    decode_ms = sum(st[0]["decode_ms"] for st in stats)
    prefill_ms = sum(st[0]["prefill_ms"] for st in stats) / len(stats)
    d, F = cfg.d_model, cfg.ffn_dim
    f_pad = (F + 31) // 32 * 32
    # gate/up: algorithmic flops 2 * rows * (2 F) * d per layer over the timed launches (executed
    # MFMA work is twice that: the activation's hi and lo planes)
    gu_flops = 2.0 * rows * 2 * f_pad * d * cfg.n_layers
    # the sampled launches rotate over layers and iterations: their mean duration against the
    # mean flops of a launch (all launches of the timed steps)
    gu_launch_flops = gu_flops / (cfg.n_layers * sum(iters))
    achieved = gu_launch_flops / (gu_ms / 1e3 / max(launches, 1)) / 1e12 if gu_ms > 0 else 0.0
    mean_rows = rows / sum(iters)
    cpu = None
    if not args.no_cpu_baseline:
        dt, cores = oracle_iteration_s(cfg, ws, n)
        tok_per_row = tokens / rows
        cpu = {"value": n / dt * tok_per_row, "unit": "tokens/s", "cores": cores, "kind": "oracle",
               "sample": f"one Jacobi iteration of {n} rows of one sequence at the 7B shape at a context of "
                         f"{ORACLE_CONTEXT} keys (median of 5) after a {ORACLE_CONTEXT}-token prefill ({dt:.2f} s), "
                         f"scaled to tokens by the GPU run's {tok_per_row:.3f} tokens per row",
               "context": ORACLE_CONTEXT, "iteration_s": dt}
    line = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: {B} sequences, prompts uniform in {list(wl.prompt_len_range)}, n={n}, "
                               f"{max_new} new tokens each, guesses = GPU greedy continuation corrupted at per-sequence "
                               f"p uniform in {list(wl.p_range)} and re-drawn each iteration, shrink blocks, one "
                               f"batched loop",
                   "batch": B, "n": n, "max_new": max_new, "layers": cfg.n_layers, "d_model": d,
                   "prefill_chunk": args.prefill_chunk},
        "batched_iterations_per_step": sum(iters) / len(iters),
        "mean_rows_per_iteration": round(mean_rows, 2),
        "batched_iteration_ms": round(decode_ms / sum(iters), 4),
        "iteration_ms": {"mean": round(decode_ms / sum(iters), 4),
                         "p10": round(float(np.median([st[0]["iter_ms_p10"] for st in stats])), 4),
                         "p50": round(float(np.median([st[0]["iter_ms_p50"] for st in stats])), 4),
                         "p90": round(float(np.median([st[0]["iter_ms_p90"] for st in stats])), 4)},
        "decode_tokens_per_s": round(tokens / (decode_ms / 1e3), 3),
        "prefill_ms": round(prefill_ms, 3),
        "ar_tokens_per_s": round(ar_tps, 3),
        "speedup_vs_ar": round(value / ar_tps, 3),
        "collection": {"blocks": len(entries), "states": n_states, "seconds": round(coll_s, 3),
                       "states_per_s": round(n_states / coll_s, 1)},
        "roofline": {"bound": "mfma", "kernel": "gemm gate/up + SwiGLU (per layer), row tiles of 64",
                     "achieved": round(achieved, 2), "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / BF16_PEAK_TFLOPS, 4), "traffic": None,
                     "executed_mfma_tflops": round(2 * achieved, 2), "algorithmic_flops": gu_launch_flops,
                     "avg_launch_us": round(gu_ms / max(launches, 1) * 1e3, 2), "launches": launches},
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


LOSS_PAIRS, LOSS_AR, LOSS_OMEGA = 16, 48, 1.0
LOSS_STEPS_PER_STEP = 20  # loss-head calls per timed step (one call is ~0.2 ms)


def main_loss(args):
    """The CLLM loss head (global consistency KL + omega AR loss, forward then backward) at the
    LLaMA-2-7B LM head. The model holds one decoder layer: the loss head touches no weight but
    the LM head's, which has the 7B shape. A step is LOSS_STEPS_PER_STEP calls of
    cllm_loss_head_device on arrays resident on the GPU (each call: 16 pairs + 48 AR rows, with
    the weight gradient)."""
    import dataclasses

    import torch
    from paper_2403_00835_amd import binding, workload
    from paper_2403_00835_amd.configs import LLAMA7B

    cfg = dataclasses.replace(LLAMA7B, n_layers=1)
    d, V = cfg.d_model, cfg.vocab
    P, A, omega = LOSS_PAIRS, LOSS_AR, LOSS_OMEGA
    torch.cuda.init()
    stream = torch.cuda.current_stream()
    ws = workload.make_weights(cfg)
    model = binding.Model(cfg, max_ctx=64, max_block=16, max_new=16, stream=stream.cuda_stream, weights=ws)
    t, s, ar, tg = workload.make_head_rows(cfg, P, A, seed=1)

    def dev(x):
        return torch.from_numpy(np.ascontiguousarray(x)).cuda()

    T, S, Ar, TG = dev(t), dev(s), dev(ar), dev(tg)
    kl, nll = torch.empty(P, device="cuda"), torch.empty(A, device="cuda")
    ds, da = torch.empty(P, d, device="cuda"), torch.empty(A, d, device="cuda")
    dw = torch.empty(V, d, device="cuda")
    loss = torch.empty(1, dtype=torch.float64, device="cuda")

    def one_call():
        model.loss_head_device(P, A, omega, T, S, Ar, TG, kl, nll, ds, da, dw, loss)

    def one_step():
        for _ in range(LOSS_STEPS_PER_STEP):
            one_call()

    torch.cuda.synchronize()
    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    # the device entry point must give the host entry point's results bit for bit
    one_call()
    torch.cuda.synchronize()
    h = model.loss_head(t, s, ar, tg, omega, want_dw=True)
    if not (np.array_equal(kl.cpu().numpy(), h["kl"]) and np.array_equal(dw.cpu().numpy(), h["d_W"]) and
            loss.item() == h["loss"]):
        raise RuntimeError("device loss head differs from the host entry point")
    del h
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        one_step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    calls = args.steps * LOSS_STEPS_PER_STEP

    # per-kernel durations: one pass of the same calls per kernel class, every launch timed
    R, Rg = 2 * P + A, P + A
    nch = (V + 1023) // 1024
    w_bytes = V * d * 2
    algo = {"loss_logits": w_bytes + R * d * 4 + R * V * 4,
            "loss_rows": R * V * 4 + Rg * V * 4 + A * 4,
            "loss_dh": w_bytes + Rg * V * 4 + nch * Rg * d * 4,
            "loss_dw": Rg * V * 4 + Rg * d * 4 + V * d * 4}
    kern = {}
    for cls in algo:
        model.timing_enable(cls, every=1)
        for _ in range(args.steps):
            one_step()
        torch.cuda.synchronize()
        n_l, ms = model.timing_read()
        model.timing_enable(-1)
        us = ms * 1e3 / max(n_l, 1)
        kern[cls] = {"avg_launch_us": round(us, 2), "launches": n_l, "algorithmic_bytes": algo[cls],
                     "achieved_gbps": round(algo[cls] / (us * 1e3), 1) if us > 0 else None}
    # the roofline kernel: dW, the largest single kernel of a call (the logits class is two GEMM
    # launches, one per 64-row tile, plus the operand packing; dH is a GEMM plus its split sum)
    dom = "loss_dw"
    ach = kern[dom]["achieved_gbps"] or 0.0
    if args.calibrate_copy:
        calibration_copy()

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        log("[bench] cpu baseline: oracle loss head on the host")
        Wf = workload.as_f32(cfg, ws[-1]).astype(np.float64)
        reps, t_cpu = 0, 0.0
        while t_cpu < 10.0 and reps < 20:
            c0 = time.perf_counter()
            oracle.loss_head(Wf, t, s, ar, tg, omega)
            t_cpu += time.perf_counter() - c0
            reps += 1
        cpu = {"value": round(reps * Rg / t_cpu, 3), "unit": "rows/s", "cores": oracle.num_threads(),
               "kind": "oracle", "sample": f"{reps} full loss-head calls ({P} pairs + {A} AR rows, with the "
                                           f"weight gradient) in {t_cpu:.2f} s"}
    line = {
        "metric": "CLLM loss head (LM-head forward + backward) rows/s, 7B-shape bf16",
        "value": round(calls * Rg / elapsed, 1),
        "unit": "rows/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"CLLM loss head at the LLaMA-2-7B LM head ({V} x {d} bf16): {P} teacher/student "
                               f"pairs + {A} AR rows per call, omega {omega}, weight gradient on, "
                               f"{LOSS_STEPS_PER_STEP} calls per step, rows and gradients resident on the GPU",
                   "pairs": P, "ar_rows": A, "calls_per_step": LOSS_STEPS_PER_STEP, "d_model": d, "vocab": V},
        "call_us": round(elapsed / calls * 1e6, 2),
        "kernels": kern,
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": ach, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(ach / HBM_PEAK_GBPS, 4),
                     "traffic": measured_traffic(LOSS_SUMMARY, ("loss.hip", "device.h", "launch.h")),
                     "algorithmic_bytes": algo[dom], "avg_launch_us": kern[dom]["avg_launch_us"],
                     "launches": kern[dom]["launches"]},
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
