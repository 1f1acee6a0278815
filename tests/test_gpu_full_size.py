"""GPU parity at the benchmark's full sizes, in the configuration bench.py times.

The oracle (fp64) computes sampled outputs: every chunk of one stream for the
batch-1 workloads; for the 64-stream workload every chunk of up to ten
streams (extreme prefix lengths, every prefix length mod 8) and chunk 0 of all
64 streams; and one emitted chunk of the sequential baseline.  Tolerance: max relative error 1e-2
per (stream, chunk) slice in bf16 mode.
"""
import sys
import time

import numpy as np
import pytest

import oracle
import synth
from tests.gpu_util import Case, dev, host, rel_err, tol

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("name", ["pi05_b1", "short_chunk"])
def test_velocity_parity_full_size(name):
    w = synth.workload(name)
    case = Case(w)
    try:
        t0 = time.time()
        v = case.gpu_velocity()
        ref = case.oracle_velocity(0)
        errs = [rel_err(v[0, k], ref[k]) for k in range(w.n_chunks)]
        _say(f"{name}: per-chunk rel err max {max(errs):.2e} ({time.time() - t0:.1f}s)")
        assert max(errs) < tol(w), errs
    finally:
        case.close()


def _f64_weights(W):
    """The weights as fp64 arrays, converted once for many oracle calls."""
    return {k: (None if a is None else [np.asarray(x, np.float64) for x in a]
                if isinstance(a, list) else np.asarray(a, np.float64)) for k, a in W.items()}


def test_velocity_parity_batched64_all_streams():
    """Every chunk of the shortest- and longest-prefix streams and of one
    stream per residue of the prefix length mod 8 (the arena row alignment
    and the rotary gap depend on it); chunk 0 of all 64 streams.  Chunk 0
    sees only the prefix and itself (Sec. 3.1 mask), so it equals the
    velocity of a one-chunk buffer holding it at the same noise level and
    positions, which the oracle computes cheaply."""
    w = synth.workload("batched64")
    case = Case(w)
    try:
        v = case.gpu_velocity()
        assert np.all(np.isfinite(v))
        W64 = _f64_weights(case.W)
        full = [int(np.argmin(case.lens)), int(np.argmax(case.lens))]
        for r in range(8):
            hit = [b for b in range(w.batch) if case.lens[b] % 8 == r and b not in full]
            full += hit[:1]
        for b in full:
            ref = oracle.velocity(case.x[b], case.t[b], case.k[:, b], case.v[:, b],
                                  int(case.lens[b]), W64, w)
            errs = [rel_err(v[b, k], ref[k]) for k in range(w.n_chunks)]
            _say(f"batched64 stream {b} (P={case.lens[b]}, P%8={case.lens[b] % 8}): "
                 f"max rel err {max(errs):.2e}")
            assert max(errs) < tol(w), (b, errs)
        worst = 0.0
        for b in range(w.batch):
            ref0 = oracle.velocity(case.x[b, :1], case.t[b, :1], case.k[:, b], case.v[:, b],
                                   int(case.lens[b]), W64, w)[0]
            e = rel_err(v[b, 0], ref0)
            worst = max(worst, e)
            assert e < tol(w), (b, e)
        _say(f"batched64 chunk 0 of all {w.batch} streams: max rel err {worst:.2e}")
    finally:
        case.close()


def test_velocity_parity_ragged_large_m():
    """9 streams of the batched workload: 4500 token rows, so the large-row
    GEMM tiles (256 rows) end in a partial tile of 148 rows, which belongs to
    the last stream.  Then one decode step, which at this many rows runs the
    velocity head and the queue update as separate kernels: buffer and emitted
    chunk bit for bit against the fp32 queue update of the GPU's own velocity,
    refill against the oracle's Philox draw."""
    w = synth.workload("batched64").replace(name="batched9", batch=9)
    case = Case(w)
    try:
        v = case.gpu_velocity()
        assert np.all(np.isfinite(v))
        for b in (w.batch - 1, int(np.argmin(case.lens))):
            ref = case.oracle_velocity(b)
            errs = [rel_err(v[b, k], ref[k]) for k in range(w.n_chunks)]
            _say(f"batched9 stream {b} (P={case.lens[b]}): max rel err {max(errs):.2e}")
            assert max(errs) < tol(w), (b, errs)
        case.ex.set_noise_state(0, 5)
        pre = host(case.xd).copy()
        case.ex.decode_step(case.xd, case.td, case.out)
        post, out = host(case.xd), host(case.out)
        mism = 0
        for b in range(w.batch):
            z = oracle.gaussian_chunk(b, 5, w.chunk_len, w.action_dim)
            new, ref_out = oracle.euler_emit_shift(pre[b], case.t[b], v[b], z, np.float32)
            assert np.array_equal(out[b], ref_out), b
            assert np.array_equal(post[b, :-1], new[:-1]), b
            mism += int(np.count_nonzero(post[b, -1] != z))
            assert np.max(np.abs(post[b, -1] - z)) <= 1e-6
        _say(f"batched9 decode step: refill values differing from the oracle's draw: {mism}")
        assert mism <= 2
    finally:
        case.close()


@pytest.mark.parametrize("B", [2, 4, 12, 16, 36])
def test_velocity_parity_mid_batches(B):
    """Batch sizes between the benchmarked ones take other GEMM plans: at
    2 streams (1000 rows) the output and down projections split k in two on
    64 x 128 tiles, at 4 (2000 rows) on 128 x 128 tiles; at 12 (6000 rows)
    they run unsplit on 128 x 128 tiles, two workgroups per CU, where
    256 x 256 tiles would leave most CUs idle; at 16 the QKV GEMM and at 36
    the output and down projections take 128 x 128 tiles where 256 x 256
    tiles would leave a second round mostly idle.  The first and last
    streams against the oracle."""
    w = synth.workload("batched64").replace(name=f"batched{B}", batch=B)
    case = Case(w)
    try:
        assert case.ex.out_proj_splits() == (2 if B <= 4 else 1)
        v = case.gpu_velocity()
        assert np.all(np.isfinite(v))
        for b in (0, B - 1):
            ref = case.oracle_velocity(b)
            errs = [rel_err(v[b, k], ref[k]) for k in range(w.n_chunks)]
            _say(f"batched{B} stream {b} (P={case.lens[b]}): max rel err {max(errs):.2e}")
            assert max(errs) < tol(w), (b, errs)
    finally:
        case.close()


def test_velocity_parity_many_short_streams():
    """90 streams of 50 tokens: 4500 rows take the 256-row GEMM tiles, whose
    128-row wave slabs span three or four streams, so the QKV epilogue looks
    every row's stream up instead of reading two prefix lengths."""
    w = synth.workload("short_chunk").replace(name="short_b90", batch=90)
    case = Case(w)
    try:
        v = case.gpu_velocity()
        assert np.all(np.isfinite(v))
        for b in (0, 45, w.batch - 1):
            ref = case.oracle_velocity(b)
            errs = [rel_err(v[b, k], ref[k]) for k in range(w.n_chunks)]
            _say(f"short_b90 stream {b} (P={case.lens[b]}): max rel err {max(errs):.2e}")
            assert max(errs) < tol(w), (b, errs)
    finally:
        case.close()


def test_decode_steps_lockstep_pi05():
    """Two steps of the headline workload: emitted chunk within tolerance of
    the oracle, shifted slots bit-exact against the fp32 queue update of the
    GPU's own velocity, refill equal to the oracle's Philox draw."""
    w = synth.workload("pi05_b1")
    case = Case(w, noise_seed=7)
    try:
        for s in range(2):
            pre = host(case.xd).copy()
            v = case.gpu_velocity(pre)
            case.ex.decode_step(case.xd, case.td, case.out)
            post, out = host(case.xd), host(case.out)
            z = oracle.gaussian_chunk(7, s, w.chunk_len, w.action_dim)
            new, ref_out = oracle.euler_emit_shift(pre[0], case.t[0], v[0], z, np.float32)
            assert np.array_equal(out[0], ref_out)
            assert np.array_equal(post[0, :-1], new[:-1])
            mism = int(np.count_nonzero(post[0, -1] != z))
            _say(f"pi05 step {s}: refill values differing from the oracle's draw: {mism} of {z.size}")
            assert mism <= 2 and np.max(np.abs(post[0, -1] - z)) <= 1e-6
            ref_v = oracle.velocity(pre[0], case.t[0], case.k[:, 0], case.v[:, 0],
                                    int(case.lens[0]), case.W, w)
            _, o_out = oracle.euler_emit_shift(pre[0], case.t[0], ref_v, z)
            err = rel_err(out[0], o_out)
            _say(f"pi05 step {s}: emitted chunk rel err {err:.2e}")
            assert err < tol(w)
    finally:
        case.close()


def test_sequential_baseline_parity():
    w = synth.workload("seq_baseline")
    case = Case(w)
    try:
        import torch
        noise = synth.make_buffer(w, 3)[:, 0]
        nd = dev(noise)
        out = torch.empty_like(nd)
        case.ex.sequential_decode(nd, w.seq_steps, out)
        got = host(out)
        ref = oracle.sequential_decode(noise, w.seq_steps, case.k, case.v, case.lens, case.W, w)
        err = rel_err(got[0], ref[0])
        _say(f"seq_baseline: emitted chunk rel err {err:.2e}")
        assert err < tol(w)
    finally:
        case.close()
