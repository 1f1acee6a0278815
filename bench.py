"""Benchmark of the streaming action-decode step on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu]
                [--no-others] [--no-stages] [--pmc-driver WHAT]

One "step" is one fv_decode_step (Algorithm 1, steady streaming): the full
velocity pass of the action expert over the K-chunk buffer, the Euler update,
emission, shift and noise refill, with inputs resident in HBM and the buffer
carried over from step to step.  W untimed steps, then K timed steps between
two device synchronisations; per-step latencies come from HIP events on the
stream the library launches on.  Prints one JSON line.

The headline workload is the pi0.5-shaped expert at batch 1 (18 layers,
width 1024, 8q/1kv heads of 256, GeGLU 4096, prefix 560 = 2 views x 256 + 48
text tokens, K = 10 chunks of 50 x 32 actions).  The other workloads (short
chunks, batch 64 with ragged prefixes, the sequential 10-pass baseline, the
asynchronous pipeline, cold start, the multi-buffer forward) are measured in
the same run and reported under "other_workloads".

Roofline records: every kernel of a layer is timed alone (fv_debug_stage,
launches captured in a graph and cycling over the layers as a step does),
its algorithmic work per launch is counted, and the kernel with the largest
time per step is the record.  Counter-based evidence (HBM bytes per launch
and per step, MFMA utilisation) is read from the rocprofv3 summaries under
profiles/, each valid only while the sources it was taken from are unchanged.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
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
METRIC = "action chunks/s + p50 decode-step latency (µs), π0.5-shaped, batch 1 and 64"


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
    rows_t, rows_f = w.batch * w.tokens, film_rows(w)
    gemm = 2 * rows_f * W * W * 2 + 2 * rows_f * W * (6 * L + 2) * W
    gemm += 2 * rows_t * A * W * 2
    gemm += L * 2 * rows_t * (W * (qd + 2 * kd) + qd * W + W * ngu + F * W)
    attn = sum(4 * w.head_dim * w.n_q_heads * visible_pairs(w, p) * L for p in lens)
    return gemm, attn


def film_bytes(w) -> int:
    """Bytes of the time-MLP and FiLM map weights (skipped by a cached schedule)."""
    e = 2 if w.dtype == synth.BF16 else 4
    W, L = w.width, w.n_layers
    return (2 * W * W + (6 * L + 2) * W * W) * e + (2 * W + (6 * L + 2) * W) * 4


# fv_debug_stage ids of the stages a counter run can launch alone
DEBUG_STAGES = {"film_maps": 0, "qkv_gemm": 1, "gate_up_gemm": 3, "attention": 4,
                "attn_combine": 5, "o_proj_gemm": 8, "down_proj_gemm": 9, "o_proj_norm": 10,
                "down_proj_norm": 11}


def film_rows(w):
    """FiLM-map rows a step computes: with several streams whose noise levels
    are the same staircase (these inputs), stream 0's K rows serve them all."""
    return w.n_chunks if w.batch > 1 else w.batch * w.n_chunks


def stage_kernels(w, split_k: int, n_split: int):
    """Stage -> (kernel label, substring of the kernel's name in a rocprofv3
    trace).  Stages that launch the same kernel share a label."""
    bf16 = w.dtype == synth.BF16
    rows_k, rows_t = w.batch * w.n_chunks, w.batch * w.tokens
    rows_f = film_rows(w)
    if bf16:
        attn = ("attn16d_kernel" if w.head_dim in (128, 256) else "attn16_kernel")
    else:
        attn = "attn_kernel"
    proj = (("gemm_dma_kernel<..., EpiNone> (split-K partials, output and down projections)",
             "EpiNone") if split_k > 1 else
            ("gemm_dma_kernel<..., EpiGatedResid> (output and down projections)",
             "EpiGatedResid"))
    norm = (("resid_norm_kernel (split-K sum + gated residual + FiLM norm)", "resid_norm_kernel")
            if split_k > 1 else ("adarms_kernel (FiLM norm)", "adarms_kernel"))
    mlp = (("gemv_bias_silu_kernel (time-MLP)", "gemv_bias_silu_kernel") if rows_f <= 16 else
           ("gemm<..., EpiBiasSilu> (time-MLP)", "EpiBiasSilu"))
    many = rows_t >= 4096 and w.width <= 1024
    small_head = not many and w.width <= 1024 and w.action_dim <= 32 and w.action_dim % 4 == 0
    stream_film = bf16 and rows_f <= 16 and w.width in (512, 1024)
    out = {
        "time_embed": ("time_embed_kernel (fp64 sinusoidal embedding)", "time_embed_kernel"),
        "time_mlp1": mlp, "time_mlp2": mlp,
        "film_maps": (("stream_bias_f32_kernel (all FiLM maps, weights streamed)",
                       "stream_bias_f32_kernel") if stream_film else
                      ("gemm<..., EpiBiasF32> (all FiLM maps)", "EpiBiasF32")),
        "embed": ((embed := ("embed_adarms_rows_kernel" if many else
                             "embed_adarms_small_kernel" if small_head else
                             "embed_adarms_kernel")) + " (in-projection + first FiLM norm)", embed),
        "qkv_gemm": ("gemm_dma_kernel<..., EpiQkv> (QKV + rotary + arena)", "EpiQkv"),
        "attention": (f"{attn} (chunk-causal + prefix attention)", attn),
        "o_proj_gemm": proj, "down_proj_gemm": proj,
        "o_proj_norm": norm, "down_proj_norm": norm,
        "gate_up_gemm": ("gemm_dma_kernel<..., EpiGeglu> (gate/up + GeGLU)",
                         "EpiGeglu" if w.mlp_gated else "EpiGelu"),
        "head": ((head := ("final_rows_kernel" if many else
                           "final_small_kernel" if small_head else "final_kernel")) +
                 " (final FiLM norm + velocity head)", head),
        "euler_shift": (("final_small_kernel<true> (Euler + emit + shift + refill fused into "
                         "the velocity head)", "final_small_kernel<true>") if small_head else
                        ("euler_shift_kernel (Euler + emit + shift + refill)",
                         "euler_shift_kernel")),
    }
    if n_split > 1:
        out["attn_combine"] = ("attn_combine (merge of the key splits)", "attn_combine")
    return out


def stage_work(w, lens, n_split: int, split_k: int):
    """Algorithmic (flops, bytes) of one launch of each stage.

    Bytes count each operand once: weights, the activations a kernel reads
    and the results it writes; for attention the queries, the visible keys
    and values (valid prefix + the buffer's own tokens) and the output.  The
    split partials (attention key splits, split-K tiles) are an
    implementation choice: a split GEMM is charged its output once, as if
    unsplit, and the partials count only for the kernels whose whole job is
    to reduce them (the combine, the split-K residual norm)."""
    e = 2 if w.dtype == synth.BF16 else 4
    W, F = w.width, w.mlp_dim
    qd, kd = w.n_q_heads * w.head_dim, w.n_kv_heads * w.head_dim
    ngu = 2 * F if w.mlp_gated else F
    rows_t, rows_k = w.batch * w.tokens, w.batch * w.n_chunks
    rows_f = film_rows(w)
    nmod = (6 * w.n_layers + 2) * W
    kv_bytes = 2 * (int(np.sum(lens)) + rows_t) * kd * e
    R = rows_t * w.n_q_heads
    comb_bytes = (n_split * R * (w.head_dim * e + 8) + R * w.head_dim * e) if n_split > 1 else 0
    h_rw = 2 * rows_t * W * 4                       # fp32 residual read + write
    if split_k > 1:
        proj_out = rows_t * W * e                   # the product once, element type
        norm_bytes = split_k * rows_t * W * (2 if e == 2 else 4) + h_rw + rows_t * W * e
    else:
        proj_out = h_rw                             # gated residual in the epilogue
        norm_bytes = rows_t * W * 4 + rows_t * W * e
    A, C = w.action_dim, w.chunk_len
    buf = w.batch * w.tokens * A * 4
    return {
        "time_embed": (0, rows_k * 4 + rows_k * W * e),
        "time_mlp1": (2 * rows_f * W * W, W * W * e + W * 4 + 2 * rows_f * W * e),
        "time_mlp2": (2 * rows_f * W * W, W * W * e + W * 4 + 2 * rows_f * W * e),
        "embed": (2 * rows_t * A * W, buf + (A + 1) * W * 4 + rows_t * W * (4 + e)),
        "head": (2 * rows_t * W * A, rows_t * W * 4 + (W + 1) * A * 4 + buf),
        "euler_shift": (0, 3 * buf + w.batch * C * A * 4 + rows_k * 4),
        "film_maps": (2 * rows_f * W * nmod, nmod * W * e + nmod * 4 + rows_f * (W * e + nmod * 4)),
        "qkv_gemm": (2 * rows_t * W * (qd + 2 * kd), W * (qd + 2 * kd) * e + rows_t * W * e
                     + rows_t * (qd + 2 * kd) * e),
        "attention": (sum(4 * w.head_dim * w.n_q_heads * visible_pairs(w, p) for p in lens),
                      rows_t * qd * e + kv_bytes + rows_t * qd * e),
        "attn_combine": (0, comb_bytes),
        "o_proj_gemm": (2 * rows_t * qd * W, qd * W * e + rows_t * qd * e + proj_out),
        "o_proj_norm": (0, norm_bytes),
        "gate_up_gemm": (2 * rows_t * W * ngu, W * ngu * e + rows_t * W * e + rows_t * F * e),
        "down_proj_gemm": (2 * rows_t * F * W, F * W * e + rows_t * F * e + proj_out),
        "down_proj_norm": (0, norm_bytes),
    }


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


def pct(xs, q):
    return float(np.percentile(np.asarray(xs), q))


def measure_streaming(w, steps, warmup, with_roofline, cached=False, mask=None, inp=None):
    """Steady streaming steps.  cached: static-schedule FiLM cache (t == NULL);
    mask: attention mask mode name (default chunk-causal)."""
    import torch
    from paper_2608_27384_amd.flashvla import Expert
    inp = inp or Inputs(w)
    ex = Expert(inp.W, w, w.batch, w.max_prefix, noise_seed=w.noise_seed)
    try:
        ex.set_prefix(inp.kd, inp.vd, inp.lens)
        if mask:
            ex.set_mask_mode(mask)
        xd = torch.from_numpy(inp.x.copy()).cuda()
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
            res["stages"] = stage_timing(ex, w, inp.lens)
        return res
    finally:
        ex.close()


def time_stage(ex, stage, n_layers, rounds=3):
    """Mean duration (ms) of one launch of a kernel stage: 4 passes over the
    layers (launch r runs layer r mod L, as a step walks them) captured in one
    graph and replayed between HIP events on the stream it runs on, so each
    launch is dispatched as inside a step; the median of `rounds` replays."""
    import torch
    reps = 4 * n_layers
    ex.debug_stage(stage, -1, reps)          # capture + first replay
    torch.cuda.synchronize()
    res = []
    for _ in range(rounds):
        s, e = _events(2)
        s.record()
        ex.debug_stage(stage, -1, reps)
        e.record()
        torch.cuda.synchronize()
        res.append(s.elapsed_time(e) / reps)
    return statistics.median(res)


def stage_timing(ex, w, lens):
    """Live duration and algorithmic work per launch of every kernel of a
    layer and of the FiLM-map GEMM (the small per-step kernels -- time
    embedding, time-MLP, in-projection, head, Euler -- are not timed alone)."""
    peak = MFMA_BF16_PEAK_TFS if w.dtype == synth.BF16 else MFMA_FP32_PEAK_TFS
    n_split, split_k = ex.attn_split(), ex.out_proj_splits()
    kern = stage_kernels(w, split_k, n_split)
    work = stage_work(w, lens, n_split, split_k)
    out = {}
    for name, stage in DEBUG_STAGES.items():
        if name not in kern:
            continue
        flops, nbytes = work[name]
        us = time_stage(ex, stage, w.n_layers) * 1e3
        n = 1 if name == "film_maps" else w.n_layers
        out[name] = {"us": us, "launches_per_step": n, "us_per_step": us * n,
                     "kernel": kern[name][0], "trace_match": kern[name][1],
                     "tflops": flops / (us * 1e-6) / 1e12,
                     "gbs": nbytes / (us * 1e-6) / 1e9,
                     "mfma_frac": flops / (us * 1e-6) / (peak * 1e12),
                     "hbm_frac": nbytes / (us * 1e-6) / (HBM_PEAK_GBS * 1e9),
                     "flops": flops, "bytes": nbytes}
    return out


def dominant_kernel(stages, w):
    """The kernel with the largest time per step, over every stage that
    launches it: achieved = its algorithmic work per launch / its mean launch
    duration; the bound is the roofline whose floor (work at peak) is larger."""
    peak_t = MFMA_BF16_PEAK_TFS if w.dtype == synth.BF16 else MFMA_FP32_PEAK_TFS
    groups = {}
    for name, st in stages.items():
        groups.setdefault(st["trace_match"], []).append((name, st))
    per_step = {k: sum(st["us_per_step"] for _, st in v) for k, v in groups.items()}
    key = max(per_step, key=per_step.get)
    members = groups[key]
    n = sum(st["launches_per_step"] for _, st in members)
    flops = sum(st["flops"] * st["launches_per_step"] for _, st in members) / n
    nbytes = sum(st["bytes"] * st["launches_per_step"] for _, st in members) / n
    us = per_step[key] / n
    t_mfma = flops / (peak_t * 1e12)
    t_hbm = nbytes / (HBM_PEAK_GBS * 1e9)
    bound = "mfma" if t_mfma >= t_hbm else "hbm"
    achieved = flops / (us * 1e-6) / 1e12 if bound == "mfma" else nbytes / (us * 1e-6) / 1e9
    peak = peak_t if bound == "mfma" else HBM_PEAK_GBS
    from paper_2608_27384_amd import counters
    tr = counters.load_traffic(key, w.name)
    prof = counters.load_in_step(w.name)
    in_step = None
    if prof:
        hits = [v for k, v in prof["avg_us"].items() if key in k]
        if hits:
            us_p = sum(hits) / len(hits)
            ach_p = flops / (us_p * 1e-6) / 1e12 if bound == "mfma" else \
                nbytes / (us_p * 1e-6) / 1e9
            in_step = {"us_per_launch": us_p, "achieved": ach_p,
                       "frac": ach_p / (peak_t if bound == "mfma" else HBM_PEAK_GBS),
                       "current": prof["current"], "source": prof["source"]}
    return {"bound": bound, "achieved": achieved, "peak": peak,
            "unit": "TFLOP/s" if bound == "mfma" else "GB/s", "frac": achieved / peak,
            "traffic": tr["bytes"] if tr else None,
            "kernel": members[0][1]["kernel"], "trace_match": key,
            "stages": [name for name, _ in members],
            "us_per_launch": us, "launches_per_step": n, "us_per_step": per_step[key],
            "alg_flops_per_launch": flops, "alg_bytes_per_launch": nbytes,
            "other_frac": (nbytes / (us * 1e-6) / (HBM_PEAK_GBS * 1e9) if bound == "mfma"
                           else flops / (us * 1e-6) / (peak_t * 1e12)),
            "traffic_source": tr["source"] if tr else None,
            "in_step_profiled": in_step,
            "kernels_by_time_per_step_us": dict(sorted(per_step.items(),
                                                       key=lambda kv: -kv[1]))}


def measure_cold_start(w, episodes=20, inp=None):
    """Episode start: fv_cold_start, then K steps until the first real chunk is
    emitted (the K-1 warm-up steps emit zeros).  HIP events on the stream."""
    import torch
    from paper_2608_27384_amd.flashvla import Expert
    inp = inp or Inputs(w)
    ex = Expert(inp.W, w, w.batch, w.max_prefix, noise_seed=w.noise_seed)
    try:
        ex.set_prefix(inp.kd, inp.vd, inp.lens)
        xd = torch.from_numpy(inp.x.copy()).cuda()
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


def measure_multibuffer(w, reps=50, warmup=5, inp=None):
    """Packed multi-buffer forward of one observation (Sec. 3.3): the K buffer
    configurations of cold start.  Timed twice: the whole call (which also
    installs the shared prefix for all configurations, host-synchronously),
    and the forward alone (fv_velocity over the installed configurations),
    next to an ordinary decode step at batch K on the same handle."""
    import torch
    from paper_2608_27384_amd.flashvla import Expert
    inp = inp or Inputs(w)
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
        # the forward alone: the configurations stay installed (batch K,
        # valid slots 1..K); fv_velocity runs the same pass
        perf, total_f, _ = time_steps(lambda: ex.velocity(bd, tdv, vout), reps, warmup)
        # an ordinary decode step of K full buffers over the same prefix
        ex.set_valid_slots([K] * K)
        xb = torch.from_numpy(np.stack([inp.x[0].copy() for _ in range(K)])).cuda()
        out = torch.empty((K, w.chunk_len, w.action_dim), dtype=torch.float32, device="cuda")
        pers, total_s, _ = time_steps(lambda: ex.decode_step(xb, tdv, out), reps, warmup)
        return {"workload": w.name, "configurations": K, "reps": reps,
                "ms_per_call": total_ms / reps, "p50_us": pct(per, 50) * 1e3,
                "call_note": "fv_multibuffer_velocity: host-synchronous prefix install for all "
                             "configurations, then the forward",
                "forward_ms": total_f / reps, "forward_p50_us": pct(perf, 50) * 1e3,
                "batch_k_decode_step_ms": total_s / reps,
                "batch_k_decode_step_p50_us": pct(pers, 50) * 1e3}
    finally:
        ex.close()


def _observations(w, n, seed0=200):
    import torch
    obs = []
    for i in range(n):
        k, v, lens = synth.make_prefix(w, seed=seed0 + i)
        if w.dtype == synth.BF16:
            kd = torch.from_numpy(synth.bf16_bits(k).view(np.int16)).cuda()
            vd = torch.from_numpy(synth.bf16_bits(v).view(np.int16)).cuda()
        else:
            kd, vd = torch.from_numpy(k).cuda(), torch.from_numpy(v).cuda()
        obs.append((kd, vd, [int(x) for x in lens]))
    return obs


LOOP_MODES = ("serialized", "pipelined_same_stream", "pipelined_copy_stream")


def measure_async_pipeline(w, steps=60, warmup=6, hz=30.0, horizons=(16, 5, 2),
                           delays=(0, 1, 2), segments=8, inp=None, modes=LOOP_MODES,
                           timeline=True):
    """Asynchronous execution (Sec. 4.2) and reaction speed (Sec. 4.3).

    1. Back-to-back control loop (the highest control rate the GPU allows):
       every control step takes a new observation, whose prefix is installed
       before the step reads it, then one decode step emits a chunk.
       * serialized: fv_set_prefix (host-synchronous) then fv_decode_step;
       * pipelined, same stream: fv_set_prefix_async on the step's own
         stream, so the host never waits and the install runs in stream order
         between steps;
       * pipelined, copy stream: fv_set_prefix_async on a second stream, so
         the install of observation i+1 runs concurrently with step i.
       Wall clock per control step, host calls included.
    2. The paper's timeline with a synthetic executor at `hz`: each segment
       executes E actions of the emitted chunk (E in `horizons`: 16 is the
       execution horizon of the paper's RoboTwin and real-robot runs, 5 its
       LIBERO replanning interval, 2 the segment its reaction-speed figures
       imply: TTR - TTFA = 33 ms = 0.5 * 2 / 30 Hz); the inference for
       the next segment is launched after E - d actions and its chunk is
       executed after the current segment ends (d = 0: synchronous, the
       robot waits for it).  The executor is simulated on the host clock
       (sleeps), the inference is real: prefix install + decode step, its
       latency measured from launch to the chunk being on the host side of a
       synchronisation.  Reported per d: TTFA = inference latency (p50),
       stall per segment = max(0, latency - d / hz), actions/s, and the
       expected time to react of the Sec. 4.3 model, TTR = TTFA + 0.5 E / hz
       (a stimulus lands uniformly within one E-action execution segment)."""
    import torch
    from paper_2608_27384_amd.flashvla import Expert
    inp = inp or Inputs(w)
    obs = _observations(w, 2)
    res = {"workload": w.name, "batch": w.batch, "steps": steps, "executor_hz": hz,
           "horizons_E": list(horizons)}
    # The modes run interleaved, in rounds of steps / rounds control steps
    # with the order rotating from round to round, so that a drift of the
    # GPU's clock over the run does not favour the mode measured first.
    loop, ctl, handles = {}, {}, []
    try:
        main = torch.cuda.current_stream()
        for mode in modes:
            ex = Expert(inp.W, w, w.batch, w.max_prefix, noise_seed=w.noise_seed)
            handles.append(ex)
            xd = torch.from_numpy(inp.x.copy()).cuda()
            td = torch.from_numpy(inp.t).cuda()
            out = torch.empty((w.batch, w.chunk_len, w.action_dim), dtype=torch.float32,
                              device="cuda")
            cs = torch.cuda.Stream() if mode == "pipelined_copy_stream" else main
            kd, vd, lens = obs[0]
            ex.set_prefix(kd, vd, lens)

            def control_step(mode=mode, ex=ex, xd=xd, td=td, out=out, cs=cs, state={"i": 0}):
                i = state["i"]
                state["i"] += 1
                kd, vd, lens = obs[(i + 1) % 2]
                ex.decode_step(xd, td, out)
                if mode == "serialized":
                    ex.set_prefix(kd, vd, lens)           # next observation, host waits
                else:
                    ex.set_prefix_async(kd, vd, lens, cs)  # next observation, no wait

            ctl[mode] = control_step
            for _ in range(warmup):
                control_step()
            torch.cuda.synchronize()
            loop[mode] = {"ms_per_control_step": 0.0, "gpu_ms_per_control_step": 0.0}
        rounds = max(1, min(6, steps // 5))
        per_round = steps // rounds
        for r in range(rounds):
            k = r % len(modes)
            for mode in modes[k:] + modes[:k]:
                _, total_ms, wall = time_steps(ctl[mode], per_round, 0)
                loop[mode]["ms_per_control_step"] += wall * 1e3 / (per_round * rounds)
                loop[mode]["gpu_ms_per_control_step"] += total_ms / (per_round * rounds)
        torch.cuda.synchronize()
    finally:
        for ex in handles:
            ex.close()
    res["control_loop"] = loop
    if not timeline:
        return res

    # timeline of Sec. 4.2 with a synthetic executor
    ex = Expert(inp.W, w, w.batch, w.max_prefix, noise_seed=w.noise_seed)
    try:
        xd = torch.from_numpy(inp.x.copy()).cuda()
        td = torch.from_numpy(inp.t).cuda()
        out = torch.empty((w.batch, w.chunk_len, w.action_dim), dtype=torch.float32,
                          device="cuda")
        kd, vd, lens = obs[0]
        ex.set_prefix(kd, vd, lens)
        for _ in range(3):
            ex.decode_step(xd, td, out)
            ex.set_prefix_async(*obs[1], torch.cuda.current_stream())
        torch.cuda.synchronize()
        period = 1.0 / hz
        timeline = {}
        for horizon, d in [(E, d) for E in horizons for d in delays if d < E]:
            lat, stall = [], []
            t_seg = time.perf_counter()
            for n in range(segments):
                # inference for segment n+1 starts after E - d actions of segment n
                launch = t_seg + (horizon - d) * period
                while time.perf_counter() < launch:
                    time.sleep(min(0.002, max(0.0, launch - time.perf_counter())))
                t0 = time.perf_counter()
                kd, vd, lens = obs[n % 2]
                ex.set_prefix_async(kd, vd, lens, torch.cuda.current_stream())
                ex.decode_step(xd, td, out)
                torch.cuda.synchronize()
                t1 = time.perf_counter()
                lat.append(t1 - t0)
                seg_end = t_seg + horizon * period
                st = max(0.0, t1 - seg_end)            # robot waits past its segment
                stall.append(st)
                t_seg = seg_end + st
            ttfa = pct(lat, 50) * 1e3
            timeline[f"E{horizon}_d{d}"] = {"horizon_actions": horizon, "delay_actions": d,
                                 "ttfa_ms_p50": ttfa, "ttfa_ms_p99": pct(lat, 99) * 1e3,
                                 "stall_ms_per_segment": 1e3 * float(np.mean(stall)),
                                 "actions_per_s": horizon / (horizon * period +
                                                             float(np.mean(stall))),
                                 "ttr_expected_ms": ttfa + 0.5 * horizon * period * 1e3}
        res["timeline"] = timeline
        res["model"] = ("Sec. 4.3: E[dt_react] = dt_infer + 0.5 dt_exec with dt_exec = E / hz, "
                        "the execution time of one E-action segment; TTFA = dt_infer is the "
                        "prefix install + one decode step on the GPU, measured on the host")
    finally:
        ex.close()
    return res


def measure_sequential(w, chunks, warmup, inp=None):
    import torch
    from paper_2608_27384_amd.flashvla import Expert
    inp = inp or Inputs(w)
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


def pmc_driver(w, what, steps=4):
    """Counter-run driver (prints no JSON).  what = "step": one warm-up step,
    then `steps` decode steps; otherwise a comma-separated list of STAGES,
    each launched 20 times (layers cycling) after one velocity pass.  Then
    three 256 MiB calibration passes: a device copy, a read-only sum and a
    write-only fill."""
    import torch
    from paper_2608_27384_amd.flashvla import Expert
    inp = Inputs(w)
    ex = Expert(inp.W, w, w.batch, w.max_prefix)
    try:
        ex.set_prefix(inp.kd, inp.vd, inp.lens)
        xd = torch.from_numpy(inp.x.copy()).cuda()
        td = torch.from_numpy(inp.t).cuda()
        if what == "step":
            out = torch.empty((w.batch, w.chunk_len, w.action_dim), dtype=torch.float32,
                              device="cuda")
            for _ in range(1 + steps):
                ex.decode_step(xd, td, out)
            label = f"1 + {steps} decode steps"
        else:
            vo = torch.empty_like(xd)
            ex.velocity(xd, td, vo)
            for name in what.split(","):
                ex.debug_stage(DEBUG_STAGES[name], -1, 20)
            label = f"stages {what} x20"
        torch.cuda.synchronize()
        src = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        s = src.sum()
        dst.fill_(2.0)
        torch.cuda.synchronize()
        assert float(s) == float(64 << 20)
        print(f"pmc driver: {w.name} {label}; calibration copy, sum, fill of 256 MiB", flush=True)
    finally:
        ex.close()


# ---------------------------------------------------------------- CPU side

def _cpu_info():
    model = platform.processor() or ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return model, len(os.sched_getaffinity(0))


def cpu_baselines(workloads, inputs):
    """The CPU oracle (fp32 mode, as written; not tuned) timed on this host
    with BLAS threads set to every core this process may use, on a bounded
    sample of each workload: per decode step (or emitted chunk)."""
    model, ncores = _cpu_info()
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
    except ImportError:
        return _cpu_runs(workloads, inputs, model, ncores)
    with threadpool_limits(limits=ncores):
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        return _cpu_runs(workloads, inputs, model, threads)


def _cpu_runs(workloads, inputs, model, threads):
    import oracle
    out = {"cpu_model": model, "cores": int(threads), "dtype": "fp32", "configs": {}}
    # sample plan: (decode steps timed, warm-up steps, streams used)
    plan = {"tiny_fp32": (8, 0, None), "pi05_b1": (3, 1, None), "short_chunk": (20, 1, None),
            "seq_baseline": (1, 0, None), "batched64": (1, 0, 4)}
    for name in workloads:
        w = synth.workload(name)
        n, warm, nstreams = plan[name]
        inp = inputs.get(name)
        W = inp.W if inp is not None else synth.make_weights(w)
        if inp is not None:
            k, v, lens, x = inp.host_k, inp.host_v, inp.lens, inp.x
        else:
            k, v, lens = synth.make_prefix(w)
            x = synth.make_buffer(w)
        t = synth.noise_levels_batched(w)
        if nstreams:  # a sample of the streams; scaled to the whole batch below
            k, v, lens, x, t = k[:, :nstreams], v[:, :nstreams], lens[:nstreams], \
                x[:nstreams], t[:nstreams]
        if w.seq_steps:
            t0 = time.perf_counter()
            oracle.sequential_decode(x[:, 0], w.seq_steps, k, v, lens, W, w, dtype=np.float32)
            sec = (time.perf_counter() - t0) / n
            unit_note = f"emitted chunk(s) of {w.seq_steps} Euler passes each"
        else:
            xx = x
            for i in range(warm):
                xx, _ = oracle.decode_step(xx, t, k, v, lens, W, w, noise_seed=0, step=i,
                                           dtype=np.float32)
            t0 = time.perf_counter()
            for i in range(n):
                xx, _ = oracle.decode_step(xx, t, k, v, lens, W, w, noise_seed=0, step=warm + i,
                                           dtype=np.float32)
            sec = (time.perf_counter() - t0) / n
            unit_note = "decode steps"
        scale = w.batch / nstreams if nstreams else 1.0
        sec_full = sec * scale
        out["configs"][name] = {
            "s_per_step": sec_full, "chunks_per_s": w.batch / sec_full,
            "sample": (f"{n} {unit_note} after {warm} warm-up" +
                       (f", {nstreams} of {w.batch} streams, time scaled by {scale:g}"
                        if nstreams else ""))}
        print(f"# cpu oracle fp32 {name}: {sec_full:.3f} s/step", file=sys.stderr, flush=True)
    return out


# ---------------------------------------------------------------- main

def counter_evidence(workload):
    """Step-level counter summaries (profiles/) for a workload, when current."""
    from paper_2608_27384_amd import counters
    ev = {}
    st = counters.load_step_bytes(workload)
    if st:
        ev["step_hbm_bytes"] = st
    mf = counters.load_step_mfma(workload)
    if mf:
        ev["step_mfma"] = mf
    return ev or None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="pi05_b1")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-others", action="store_true")
    ap.add_argument("--no-stages", action="store_true",
                    help="skip the per-kernel stage timing (decode steps only)")
    ap.add_argument("--control-loop", default=None, choices=LOOP_MODES,
                    help="only the back-to-back control loop of the asynchronous pipeline in "
                         "this mode (for a kernel trace); prints its JSON")
    ap.add_argument("--pmc-driver", default=None, metavar="WHAT",
                    help="counter-run driver: 'step' (decode steps) or a comma-separated list "
                         "of stages (" + "|".join(DEBUG_STAGES) + "), then the 256 MiB "
                         "calibration passes; prints no JSON")
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
    if args.control_loop:
        print(json.dumps(measure_async_pipeline(w, steps=args.steps, warmup=args.warmup,
                                                modes=(args.control_loop,), timeline=False)))
        return
    inputs = {w.name: Inputs(w)}
    main_res = measure_streaming(w, args.steps, args.warmup, with_roofline=not args.no_stages,
                                 inp=inputs[w.name])
    print(f"# {w.name}: {main_res['ms_per_step'] * 1e3:.1f} us/step, "
          f"p50 {main_res['p50_us']:.1f} us", file=sys.stderr, flush=True)

    others = {}
    if not args.no_others:
        for name, steps in (("short_chunk", 1000), ("batched64", 200)):
            if name != w.name:
                wo = synth.workload(name)
                inputs[name] = Inputs(wo)
                others[name] = measure_streaming(wo, steps, 10, name == "batched64"
                                                 and not args.no_stages, inp=inputs[name])
                print(f"# {name}: {others[name]['ms_per_step'] * 1e3:.1f} us/step",
                      file=sys.stderr, flush=True)
        wseq = synth.workload("seq_baseline")
        inputs["seq_baseline"] = Inputs(wseq)
        others["seq_baseline"] = measure_sequential(wseq, 100, 10, inp=inputs["seq_baseline"])
        print(f"# seq_baseline: {others['seq_baseline']['ms_per_chunk'] * 1e3:.1f} us/chunk",
              file=sys.stderr, flush=True)
        wp = synth.workload("pi05_b1")
        ip = inputs.get("pi05_b1") or Inputs(wp)
        for key, kw in (("pi05_b1_static_schedule", {"cached": True}),
                        ("pi05_b1_isolated_mask", {"mask": "isolated"})):
            others[key] = measure_streaming(wp, 100, 10, False, inp=ip, **kw)
            print(f"# {key}: {others[key]['ms_per_step'] * 1e3:.1f} us/step",
                  file=sys.stderr, flush=True)
        others["pi05_b1_multibuffer"] = measure_multibuffer(wp, inp=ip)
        mb = others["pi05_b1_multibuffer"]
        print(f"# pi05_b1 multi-buffer: call {mb['ms_per_call'] * 1e3:.1f} us, forward "
              f"{mb['forward_ms'] * 1e3:.1f} us, batch-{wp.n_chunks} step "
              f"{mb['batch_k_decode_step_ms'] * 1e3:.1f} us", file=sys.stderr, flush=True)
        for name in ("pi05_b1", "batched64"):
            key = f"{name}_async_pipeline"
            others[key] = measure_async_pipeline(synth.workload(name), inp=inputs.get(name))
            cl = others[key]["control_loop"]
            print(f"# {key}: " + ", ".join(f"{m} {v['ms_per_control_step']:.3f} ms"
                                            for m, v in cl.items()), file=sys.stderr, flush=True)
        others["pi05_b1_cold_start"] = measure_cold_start(wp, inp=ip)
        print(f"# pi05_b1 cold start: first action after "
              f"{others['pi05_b1_cold_start']['time_to_first_action_ms_p50']:.2f} ms",
              file=sys.stderr, flush=True)

    roofline = None
    if "stages" in main_res:
        stages = main_res.pop("stages")
        roofline = dominant_kernel(stages, w)
        roofline["stage_table"] = stages
    roofline_b64 = None
    if "batched64" in others and "stages" in others["batched64"]:
        st64 = others["batched64"].pop("stages")
        roofline_b64 = dominant_kernel(st64, synth.workload("batched64"))
        roofline_b64["stage_table"] = st64

    cpu = None
    if not args.no_cpu:
        names = [w.name] + ([] if args.no_others else
                            [n for n in ("tiny_fp32", "short_chunk", "seq_baseline", "batched64")
                             if n != w.name])
        cb = cpu_baselines(names, inputs)
        head = cb["configs"][w.name]
        cpu = {"value": head["chunks_per_s"], "unit": "chunks/s", "cores": cb["cores"],
               "kind": "oracle",
               "sample": f"fp32 CPU oracle, {head['sample']} of {w.name}, "
                         f"{head['s_per_step']:.2f} s/step",
               "cpu_model": cb["cpu_model"], "dtype": cb["dtype"],
               "per_config": cb["configs"]}

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
        "roofline_batch64": roofline_b64,
        "counters": {w.name: counter_evidence(w.name),
                     "batched64": counter_evidence("batched64")},
        "cpu_baseline": cpu,
        "other_workloads": others,
    }
    print(json.dumps(line))


if __name__ == "__main__":
    main()
