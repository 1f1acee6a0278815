"""Benchmark of the streaming action-decode step on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu] [--no-others]

One "step" is one fv_decode_step (Algorithm 1, steady streaming): the full
velocity pass of the action expert over the K-chunk buffer, the Euler update,
emission, shift and noise refill, with inputs resident in HBM and the buffer
carried over from step to step.  W untimed steps, then K timed steps between
two device synchronisations; per-step latencies come from HIP events on the
stream the library launches on.  Prints one JSON line.

The headline workload is the pi0.5-shaped expert at batch 1 (18 layers,
width 1024, 8q/1kv heads of 256, GeGLU 4096, prefix 560 = 2 views x 256 + 48
text tokens, K = 10 chunks of 50 x 32 actions).  The other workloads (short
chunks, batch 64 with ragged prefixes, the sequential 10-pass baseline) are
measured in the same run and reported under "other_workloads".
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402

HBM_PEAK_GBS = 8000.0           # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFS = 2500.0     # dense bf16 MFMA, TFLOP/s
MFMA_FP32_PEAK_TFS = 157.3
METRIC = "action chunks/s + p50 decode-step latency (\u00b5s), \u03c00.5-shaped, batch 1 and 64"


# ---------------------------------------------------------------- accounting

def weight_bytes(w) -> int:
    """Bytes of every weight one step reads once, at storage precision."""
    e = 2 if w.dtype == synth.BF16 else 4
    W, L, F, A = w.width, w.n_layers, w.mlp_dim, w.action_dim
    qd, kd = w.n_q_heads * w.head_dim, w.n_kv_heads * w.head_dim
    ngu = 2 * F if w.mlp_gated else F
    mats = 2 * W * W + (6 * L + 2) * W * W
    mats += L * (W * (qd + 2 * kd) + qd * W + W * ngu + F * W)
    biases_f32 = 2 * W + (6 * L + 2) * W + W + A + A * W + W * A
    return mats * e + biases_f32 * 4


def step_bytes(w, lens) -> int:
    e = 2 if w.dtype == synth.BF16 else 4
    kv = 2 * int(np.sum(lens)) * w.n_kv_heads * w.head_dim * w.n_layers * e
    buf = w.batch * w.tokens * w.action_dim * 4
    io = 2 * buf + w.batch * w.chunk_len * w.action_dim * 4 + w.batch * w.n_chunks * 4
    return weight_bytes(w) + kv + io


def visible_pairs(w, P) -> int:
    """Query-key pairs one stream's query token sees, summed over tokens (per head)."""
    K, C = w.n_chunks, w.chunk_len
    return w.tokens * int(P) + C * C * K * (K + 1) // 2


def step_flops(w, lens):
    """(GEMM flops, attention flops) of one velocity pass over real rows."""
    W, L, F, A = w.width, w.n_layers, w.mlp_dim, w.action_dim
    qd, kd = w.n_q_heads * w.head_dim, w.n_kv_heads * w.head_dim
    ngu = 2 * F if w.mlp_gated else F
    rows_t, rows_k = w.batch * w.tokens, w.batch * w.n_chunks
    gemm = 2 * rows_k * W * W * 2 + 2 * rows_k * W * (6 * L + 2) * W
    gemm += 2 * rows_t * A * W * 2
    gemm += L * 2 * rows_t * (W * (qd + 2 * kd) + qd * W + W * ngu + F * W)
    attn = sum(4 * w.head_dim * w.n_q_heads * visible_pairs(w, p) * L for p in lens)
    return gemm, attn


# ---------------------------------------------------------------- GPU side

class Inputs:
    def __init__(self, w, seed=0):
        import torch
        self.w = w
        self.W = synth.make_weights(w, seed)
        k, v, self.lens = synth.make_prefix(w, seed)
        if w.dtype == synth.BF16:
            self.kd = torch.from_numpy(synth.bf16_bits(k).view(np.int16)).cuda()
            self.vd = torch.from_numpy(synth.bf16_bits(v).view(np.int16)).cuda()
        else:
            self.kd, self.vd = torch.from_numpy(k).cuda(), torch.from_numpy(v).cuda()
        self.host_k, self.host_v = k, v
        self.x = np.array(synth.make_buffer(w, seed))  # writable copies for torch
        self.t = np.array(synth.noise_levels_batched(w))


def _events(n):
    import torch
    return [torch.cuda.Event(enable_timing=True) for _ in range(n)]


def time_steps(fn, steps, warmup):
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    st, en = _events(steps), _events(steps)
    t0 = time.perf_counter()
    for i in range(steps):
        st[i].record()
        fn()
        en[i].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = [s.elapsed_time(e) for s, e in zip(st, en)]   # ms
    total_ms = st[0].elapsed_time(en[-1])
    return per, total_ms, wall


def time_stage(ex, stage, layer, reps=200):
    """Average duration (ms) of one launch of a stage, HIP events on its stream."""
    import torch
    ex.debug_stage(stage, layer, 10)
    torch.cuda.synchronize()
    s, e = _events(2)
    s.record()
    ex.debug_stage(stage, layer, reps)
    e.record()
    torch.cuda.synchronize()
    return s.elapsed_time(e) / reps


def pct(xs, q):
    return float(np.percentile(np.asarray(xs), q))


def film_bytes(w) -> int:
    """Bytes of the time-MLP and FiLM map weights (skipped by a cached schedule)."""
    e = 2 if w.dtype == synth.BF16 else 4
    W, L = w.width, w.n_layers
    return (2 * W * W + (6 * L + 2) * W * W) * e + (2 * W + (6 * L + 2) * W) * 4


def measure_streaming(w, steps, warmup, with_roofline, cached=False, mask=None):
    """Steady streaming steps.  cached: static-schedule FiLM cache (t == NULL);
    mask: attention mask mode name (default chunk-causal)."""
    import torch
    from paper_2608_27384_amd.flashvla import Expert
    inp = Inputs(w)
    ex = Expert(inp.W, w, w.batch, w.max_prefix, noise_seed=w.noise_seed)
    try:
        ex.set_prefix(inp.kd, inp.vd, inp.lens)
        if mask:
            ex.set_mask_mode(mask)
        xd = torch.from_numpy(inp.x).cuda()
        td = torch.from_numpy(inp.t).cuda()
        out = torch.empty((w.batch, w.chunk_len, w.action_dim), dtype=torch.float32,
                          device="cuda")
        if cached:
            ex.set_schedule(td)
        tt = None if cached else td
        per, total_ms, wall = time_steps(lambda: ex.decode_step(xd, tt, out), steps, warmup)
        assert bool(torch.isfinite(out).all()) and bool(torch.isfinite(xd).all()), \
            "non-finite decode output"
        ms = total_ms / steps
        gemm_f, attn_f = step_flops(w, inp.lens)
        nbytes = step_bytes(w, inp.lens) - (film_bytes(w) if cached else 0)
        res = {
            "workload": w.name, "batch": w.batch, "n_chunks": w.n_chunks,
            "variant": ("static-schedule cache; " if cached else "") + f"mask {mask or 'causal'}",
            "chunk_len": w.chunk_len, "action_dim": w.action_dim,
            "prefix_len": [int(inp.lens.min()), int(inp.lens.max())],
            "steps": steps, "warmup": warmup, "ms_per_step": ms,
            "chunks_per_s": w.batch / (ms / 1e3),
            "p50_us": pct(per, 50) * 1e3, "p90_us": pct(per, 90) * 1e3,
            "p99_us": pct(per, 99) * 1e3, "wall_s": wall,
            "alg_bytes": nbytes, "alg_flops": gemm_f + attn_f,
            "hbm_frac_step": nbytes / (ms / 1e3) / (HBM_PEAK_GBS * 1e9),
            "mfma_frac_step": (gemm_f + attn_f) / (ms / 1e3) / (MFMA_BF16_PEAK_TFS * 1e12),
        }
        if with_roofline:
            res["stages"] = stage_rooflines(ex, w, inp.lens)
        return res
    finally:
        ex.close()


# Timed stages: (debug-stage id, launches per step, kernel(s) it launches).
STAGES = {
    "film_maps": (0, "step", "gemm_kernel<..., EpiBiasF32> (all FiLM maps, one GEMM)"),
    "qkv_gemm": (1, "layer", "gemm_dma_kernel<..., EpiQkv> (QKV + rotary + K/V arena write)"),
    "attention": (4, "layer", "attn16d_kernel (chunk-causal + prefix attention, per-split partials)"),
    "attn_combine": (5, "layer", "attn_combine (merge of the key splits)"),
    "o_proj": (6, "layer", "split-K gemm_dma_kernel + resid_norm_kernel (O proj, gated residual, FiLM norm)"),
    "gate_up_gemm": (3, "layer", "gemm_dma_kernel<..., EpiGeglu> (gate/up + GeGLU)"),
    "down_proj": (7, "layer", "split-K gemm_dma_kernel + resid_norm_kernel (down proj, gated residual, FiLM norm)"),
}
# stages that are one kernel launch each (eligible for the roofline record)
SINGLE_KERNEL = {"film_maps": "gemm_kernel", "qkv_gemm": "gemm_dma_kernel",
                 "attention": "attn16d_kernel", "attn_combine": "attn_combine",
                 "gate_up_gemm": "gemm_dma_kernel"}  # bf16 kernels (fp32 attention: attn_kernel)


def stage_work(w, lens, n_split):
    """Algorithmic (flops, bytes) of one launch of each timed stage.

    Bytes count each operand once: weights, the activations a stage reads
    and the results it writes; for attention the queries, the visible keys
    and values (valid prefix + the buffer's own tokens) and the output.  The
    split partials of the attention are an implementation choice and count
    only for the combine stage, whose whole job they are."""
    e = 2 if w.dtype == synth.BF16 else 4
    W, F = w.width, w.mlp_dim
    qd, kd = w.n_q_heads * w.head_dim, w.n_kv_heads * w.head_dim
    ngu = 2 * F if w.mlp_gated else F
    rows_t, rows_k = w.batch * w.tokens, w.batch * w.n_chunks
    nmod = (6 * w.n_layers + 2) * W
    kv_bytes = 2 * (int(np.sum(lens)) + rows_t) * kd * e
    R = rows_t * w.n_q_heads
    comb_bytes = (n_split * R * (w.head_dim * e + 8) + R * w.head_dim * e) if n_split > 1 else 0
    return {
        "film_maps": (2 * rows_k * W * nmod, nmod * W * e + nmod * 4 + rows_k * (W * e + nmod * 4)),
        "qkv_gemm": (2 * rows_t * W * (qd + 2 * kd), W * (qd + 2 * kd) * e + rows_t * W * e
                     + rows_t * (qd + 2 * kd) * e),
        "attention": (sum(4 * w.head_dim * w.n_q_heads * visible_pairs(w, p) for p in lens),
                      rows_t * qd * e + kv_bytes + rows_t * qd * e),
        "attn_combine": (0, comb_bytes),
        "o_proj": (2 * rows_t * qd * W, qd * W * e + rows_t * qd * e + 2 * rows_t * W * 4
                   + rows_t * W * e),
        "gate_up_gemm": (2 * rows_t * W * ngu, W * ngu * e + rows_t * W * e + rows_t * F * e),
        "down_proj": (2 * rows_t * F * W, F * W * e + rows_t * F * e + 2 * rows_t * W * 4
                      + rows_t * W * e),
    }


def stage_rooflines(ex, w, lens):
    """Per-launch algorithmic work and live-timed (HIP events) duration of each stage."""
    peak = MFMA_BF16_PEAK_TFS if w.dtype == synth.BF16 else MFMA_FP32_PEAK_TFS
    work = stage_work(w, lens, ex.attn_split())
    out = {}
    for name, (stage, per, kern) in STAGES.items():
        flops, nbytes = work[name]
        if nbytes == 0:
            continue
        ms = time_stage(ex, stage, 0)
        n = 1 if per == "step" else w.n_layers
        out[name] = {"us": ms * 1e3, "launches_per_step": n, "us_per_step": ms * 1e3 * n,
                     "kernels": kern,
                     "tflops": flops / (ms / 1e3) / 1e12,
                     "gbs": nbytes / (ms / 1e3) / 1e9,
                     "mfma_frac": flops / (ms / 1e3) / (peak * 1e12),
                     "hbm_frac": nbytes / (ms / 1e3) / (HBM_PEAK_GBS * 1e9),
                     "flops": flops, "bytes": nbytes}
    return out


def measure_cold_start(w, episodes=20):
    """Episode start: fv_cold_start, then K steps until the first real chunk is
    emitted (the K-1 warm-up steps emit zeros).  HIP events on the stream."""
    import torch
    from paper_2608_27384_amd.flashvla import Expert
    inp = Inputs(w)
    ex = Expert(inp.W, w, w.batch, w.max_prefix, noise_seed=w.noise_seed)
    try:
        ex.set_prefix(inp.kd, inp.vd, inp.lens)
        xd = torch.from_numpy(inp.x).cuda()
        td = torch.from_numpy(inp.t).cuda()
        out = torch.empty((w.batch, w.chunk_len, w.action_dim), dtype=torch.float32,
                          device="cuda")

        def episode():
            ex.cold_start(xd)
            for _ in range(w.n_chunks):
                ex.decode_step(xd, td, out)

        episode()
        torch.cuda.synchronize()
        assert bool(torch.isfinite(out).all()) and float(out.abs().max()) > 0.0
        st, en = _events(episodes), _events(episodes)
        cs_ms = []
        for i in range(episodes):
            a = _events(1)[0]
            st[i].record()
            ex.cold_start(xd)
            a.record()
            for _ in range(w.n_chunks):
                ex.decode_step(xd, td, out)
            en[i].record()
            cs_ms.append((st[i], a))
        torch.cuda.synchronize()
        tta = [s_.elapsed_time(e_) for s_, e_ in zip(st, en)]
        cs = [s_.elapsed_time(e_) for s_, e_ in cs_ms]
        return {"workload": w.name, "episodes": episodes, "warmup_steps": w.n_chunks - 1,
                "cold_start_call_us": pct(cs, 50) * 1e3,
                "time_to_first_action_ms_p50": pct(tta, 50),
                "time_to_first_action_ms_p99": pct(tta, 99)}
    finally:
        ex.close()


def measure_multibuffer(w, reps=50, warmup=5):
    """Packed multi-buffer forward of one observation (Sec. 3.3): the K buffer
    configurations of cold start in one call."""
    import torch
    from paper_2608_27384_amd.flashvla import Expert
    inp = Inputs(w)
    K = w.n_chunks
    ex = Expert(inp.W, w, max(w.batch, K), w.max_prefix, noise_seed=w.noise_seed)
    try:
        bufs = np.stack([inp.x[0].copy() for _ in range(K)])
        for j in range(K):
            bufs[j, :K - 1 - j] = 0.0
        bd = torch.from_numpy(bufs).cuda()
        tdv = torch.from_numpy(np.broadcast_to(inp.t[0], (K, K)).copy()).cuda()
        kd, vd = inp.kd[:, 0].contiguous(), inp.vd[:, 0].contiguous()
        vout = torch.empty_like(bd)
        per, total_ms, _ = time_steps(
            lambda: ex.multibuffer_velocity(kd, vd, int(inp.lens[0]), bd, tdv, vout), reps, warmup)
        assert bool(torch.isfinite(vout[:, -1]).all())
        return {"workload": w.name, "configurations": K, "reps": reps,
                "ms_per_call": total_ms / reps, "p50_us": pct(per, 50) * 1e3,
                "note": "includes installing the shared prefix for all configurations"}
    finally:
        ex.close()


def measure_async_pipeline(w, steps=60, warmup=6, hz=30.0):
    """Control loop with a new observation every step (the VLM prefix forward
    itself is not part of this library): either the prefix is installed and
    then the step runs on one stream (serialized), or the next observation is
    installed on a second stream while the current step runs (overlapped,
    fv_set_prefix_async).  Also reports the time-to-first-action /
    time-to-react model of Sec. 4.3 for a 30 Hz executor that runs the
    emitted chunk (C actions): TTR = TTFA + 0.5 * C / hz."""
    import torch
    from paper_2608_27384_amd.flashvla import Expert
    inp = Inputs(w)
    obs = []
    for i in range(2):
        k, v, lens = synth.make_prefix(w, seed=200 + i)
        if w.dtype == synth.BF16:
            kd = torch.from_numpy(synth.bf16_bits(k).view(np.int16)).cuda()
            vd = torch.from_numpy(synth.bf16_bits(v).view(np.int16)).cuda()
        else:
            kd, vd = torch.from_numpy(k).cuda(), torch.from_numpy(v).cuda()
        obs.append((kd, vd, [int(x) for x in lens]))
    res = {"workload": w.name, "batch": w.batch, "steps": steps}
    for mode in ("serialized", "overlapped"):
        ex = Expert(inp.W, w, w.batch, w.max_prefix, noise_seed=w.noise_seed)
        try:
            xd = torch.from_numpy(inp.x).cuda()
            td = torch.from_numpy(inp.t).cuda()
            out = torch.empty((w.batch, w.chunk_len, w.action_dim), dtype=torch.float32,
                              device="cuda")
            cs = torch.cuda.Stream()
            kd, vd, lens = obs[0]
            ex.set_prefix(kd, vd, lens)
            state = {"i": 0}

            def control_step():
                i = state["i"]
                state["i"] += 1
                kd, vd, lens = obs[(i + 1) % 2]
                if mode == "serialized":
                    ex.decode_step(xd, td, out)
                    ex.set_prefix(kd, vd, lens)      # next observation, same stream
                else:
                    ex.decode_step(xd, td, out)
                    ex.set_prefix_async(kd, vd, lens, cs)

            per, total_ms, wall = time_steps(control_step, steps, warmup)
            torch.cuda.synchronize()
            res[mode] = {"ms_per_control_step": wall * 1e3 / steps, "p50_us": pct(per, 50) * 1e3}
        finally:
            ex.close()
    ttfa = res["overlapped"]["ms_per_control_step"]
    exec_ms = 1e3 * w.chunk_len / hz
    res["ttfa_ms"] = ttfa
    res["ttr_expected_ms"] = ttfa + 0.5 * exec_ms
    res["executor_hz"] = hz
    res["note"] = ("per control step: decode step + install of the next observation's prefix; "
                   "wall clock per step including host calls (serialized waits for each install)")
    return res


def measure_sequential(w, chunks, warmup):
    import torch
    from paper_2608_27384_amd.flashvla import Expert
    inp = Inputs(w)
    ex = Expert(inp.W, w, w.batch, w.max_prefix)
    try:
        ex.set_prefix(inp.kd, inp.vd, inp.lens)
        noise = torch.from_numpy(np.ascontiguousarray(inp.x[:, 0])).cuda()
        out = torch.empty_like(noise)
        per, total_ms, wall = time_steps(lambda: ex.sequential_decode(noise, w.seq_steps, out),
                                         chunks, warmup)
        ms = total_ms / chunks
        gemm_f, attn_f = step_flops(w, inp.lens)
        nbytes = w.seq_steps * step_bytes(w, inp.lens)
        return {"workload": w.name, "batch": w.batch, "passes_per_chunk": w.seq_steps,
                "chunks": chunks, "ms_per_chunk": ms, "chunks_per_s": w.batch / (ms / 1e3),
                "p50_us": pct(per, 50) * 1e3, "p99_us": pct(per, 99) * 1e3,
                "alg_bytes": nbytes, "alg_flops": w.seq_steps * (gemm_f + attn_f),
                "hbm_frac_step": nbytes / (ms / 1e3) / (HBM_PEAK_GBS * 1e9)}
    finally:
        ex.close()


def pmc_driver(w, stage):
    """One velocity pass, 20 launches of one stage, then a 256 MiB copy."""
    import torch
    from paper_2608_27384_amd.flashvla import Expert
    inp = Inputs(w)
    ex = Expert(inp.W, w, w.batch, w.max_prefix)
    try:
        ex.set_prefix(inp.kd, inp.vd, inp.lens)
        xd = torch.from_numpy(inp.x).cuda()
        td = torch.from_numpy(inp.t).cuda()
        vo = torch.empty_like(xd)
        ex.set_graph_mode(False)
        ex.velocity(xd, td, vo)
        ex.debug_stage(STAGES[stage][0], 0, 20)
        src = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print(f"pmc driver: {w.name} stage {stage} x20, copy 256 MiB", flush=True)
    finally:
        ex.close()


# ---------------------------------------------------------------- CPU side

def cpu_baseline(w, budget_s=20.0):
    """The CPU oracle (fp64) timed on this host on a bounded sample: decode
    steps of the same workload, repeated until about budget_s has passed."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    W = synth.make_weights(w)
    k, v, lens = synth.make_prefix(w)
    x = synth.make_buffer(w)
    t = synth.noise_levels_batched(w)
    n, t0 = 0, time.perf_counter()
    while True:
        x, _ = oracle.decode_step(x, t, k, v, lens, W, w, noise_seed=0, step=n)
        n += 1
        el = time.perf_counter() - t0
        if el > budget_s or n >= 50:
            break
    sec = el / n
    return {"value": w.batch / sec, "unit": "chunks/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{n} fp64 oracle decode steps of {w.name} (batch {w.batch}), "
                      f"{sec:.2f} s/step",
            "s_per_step": sec}


# ---------------------------------------------------------------- main

def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="pi05_b1")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-others", action="store_true")
    ap.add_argument("--pmc-driver", default=None, metavar="STAGE",
                    help="counter-run driver: one velocity pass, then 20 launches of the named "
                         "stage (one of " + "|".join(STAGES) + ") and a 256 MiB "
                         "device copy used to calibrate byte counters; prints no JSON")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the decode step runs on a single MI355X and "
              "independent streams shard without any exchange; run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)
    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)

    w = synth.workload(args.workload)
    if args.pmc_driver:
        pmc_driver(w, args.pmc_driver)
        return
    main_res = measure_streaming(w, args.steps, args.warmup, with_roofline=True)
    print(f"# {w.name}: {main_res['ms_per_step'] * 1e3:.1f} us/step, "
          f"p50 {main_res['p50_us']:.1f} us", file=sys.stderr, flush=True)

    others = {}
    if not args.no_others:
        for name, steps in (("short_chunk", 1000), ("batched64", 200)):
            if name != w.name:
                others[name] = measure_streaming(synth.workload(name), steps, 10, False)
                print(f"# {name}: {others[name]['ms_per_step'] * 1e3:.1f} us/step",
                      file=sys.stderr, flush=True)
        others["seq_baseline"] = measure_sequential(synth.workload("seq_baseline"), 100, 10)
        print(f"# seq_baseline: {others['seq_baseline']['ms_per_chunk'] * 1e3:.1f} us/chunk",
              file=sys.stderr, flush=True)
        for key, kw in (("pi05_b1_static_schedule", {"cached": True}),
                        ("pi05_b1_isolated_mask", {"mask": "isolated"})):
            others[key] = measure_streaming(synth.workload("pi05_b1"), 100, 10, False, **kw)
            print(f"# {key}: {others[key]['ms_per_step'] * 1e3:.1f} us/step",
                  file=sys.stderr, flush=True)
        others["pi05_b1_multibuffer"] = measure_multibuffer(synth.workload("pi05_b1"))
        print(f"# pi05_b1 multi-buffer forward: "
              f"{others['pi05_b1_multibuffer']['ms_per_call'] * 1e3:.1f} us/call",
              file=sys.stderr, flush=True)
        for name in ("pi05_b1", "batched64"):
            key = f"{name}_async_pipeline"
            others[key] = measure_async_pipeline(synth.workload(name))
            print(f"# {key}: serialized {others[key]['serialized']['ms_per_control_step']:.3f} ms, "
                  f"overlapped {others[key]['overlapped']['ms_per_control_step']:.3f} ms",
                  file=sys.stderr, flush=True)
        others["pi05_b1_cold_start"] = measure_cold_start(synth.workload("pi05_b1"))
        print(f"# pi05_b1 cold start: first action after "
              f"{others['pi05_b1_cold_start']['time_to_first_action_ms_p50']:.2f} ms",
              file=sys.stderr, flush=True)

    stages = main_res.pop("stages")
    # dominant kernel: the single-kernel stage with the largest time per step
    dom_name = max((k for k in stages if k in SINGLE_KERNEL),
                   key=lambda k: stages[k]["us_per_step"])
    dom = stages[dom_name]
    bound = "mfma" if dom["mfma_frac"] >= dom["hbm_frac"] else "hbm"
    peak = MFMA_BF16_PEAK_TFS if w.dtype == synth.BF16 else MFMA_FP32_PEAK_TFS
    from paper_2608_27384_amd import counters
    tr = counters.load_traffic(dom_name, w.name)
    roofline = {"bound": bound,
                "achieved": dom["tflops"] if bound == "mfma" else dom["gbs"],
                "peak": peak if bound == "mfma" else HBM_PEAK_GBS,
                "unit": "TFLOP/s" if bound == "mfma" else "GB/s",
                "frac": dom["mfma_frac"] if bound == "mfma" else dom["hbm_frac"],
                "traffic": tr["bytes"] if tr else None,
                "kernel": SINGLE_KERNEL[dom_name], "stage": dom_name,
                "us_per_launch": dom["us"], "launches_per_step": dom["launches_per_step"],
                "alg_flops_per_launch": dom["flops"], "alg_bytes_per_launch": dom["bytes"],
                "traffic_source": tr["source"] if tr else None}

    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(w)
        print(f"# cpu oracle: {cpu['sample']}", file=sys.stderr, flush=True)

    line = {
        "metric": METRIC,
        "value": main_res["chunks_per_s"], "unit": "chunks/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": main_res["ms_per_step"],
        "p50_us": main_res["p50_us"], "p90_us": main_res["p90_us"], "p99_us": main_res["p99_us"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if w.dtype == synth.BF16 else "fp32", "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "n_chunks": w.n_chunks,
                   "chunk_len": w.chunk_len, "action_dim": w.action_dim,
                   "prefix_len": main_res["prefix_len"], "layers": w.n_layers,
                   "width": w.width, "parallelism": "single-gpu"},
        "step_roofline": {"alg_bytes": main_res["alg_bytes"], "alg_flops": main_res["alg_flops"],
                          "hbm_frac": main_res["hbm_frac_step"],
                          "mfma_frac": main_res["mfma_frac_step"]},
        "roofline": roofline,
        "stages": stages,
        "cpu_baseline": cpu,
        "other_workloads": others,
    }
    print(json.dumps(line))


if __name__ == "__main__":
    main()
