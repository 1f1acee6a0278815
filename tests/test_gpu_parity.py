"""GPU parity: the HIP path against the CPU oracle on the same seeded inputs.

Velocities and emitted chunks are compared per (stream, chunk) slice as
max|gpu - oracle| / max|oracle|, within 1e-4 in fp32 mode and 1e-2 in bf16
mode.  Buffer bookkeeping (slot shift, emission, noise refill) is compared
bit for bit against the oracle's fp32 replica of the queue update applied to
the GPU's own velocity.
"""
import numpy as np
import pytest

import oracle
import synth
from tests.gpu_util import Case, dev, host, rel_err, tol

pytestmark = pytest.mark.gpu

SMALL = ["tiny_fp32", "small_fp32_b2", "small_bf16", "small_bf16_b3"]


def _stage_report(case):
    """Per-stage errors (FiLM params, embedding, each layer) for diagnosis."""
    import torch
    w = case.w
    B, T, W, L = w.batch, w.tokens, w.width, w.n_layers
    lines = []
    hd = torch.empty((B, T, W), dtype=torch.float32, device="cuda")
    md = torch.empty((B, w.n_chunks, (6 * L + 2) * W), dtype=torch.float32, device="cuda")
    for b in range(B):
        tr = {}
        oracle.velocity(case.x[b], case.t[b], case.k[:, b], case.v[:, b], int(case.lens[b]),
                        case.W, w, trace=tr)
        case.ex.debug_forward(case.xd, case.td, 0, hd, md)
        mod = host(md)[b]
        for n in range(2 * L + 1):
            for j in range(3 if n < 2 * L else 2):
                got = mod[:, 3 * W * n + W * j: 3 * W * n + W * (j + 1)]
                ref = tr["mods"][n][j][::w.chunk_len]
                lines.append(f"b{b} mod n{n} j{j}: {rel_err(got, ref):.2e}")
        h0 = case.x[b].reshape(T, -1).astype(np.float64) @ case.W["w_in"] + case.W["b_in"]
        lines.append(f"b{b} embed: {rel_err(host(hd)[b], h0):.2e}")
        for l in range(L):
            case.ex.debug_forward(case.xd, case.td, l + 1, hd)
            lines.append(f"b{b} layer {l}: {rel_err(host(hd)[b], tr['h'][l]):.2e}")
    return "\n".join(lines)


@pytest.mark.parametrize("name", SMALL)
def test_velocity_parity_small(name):
    w = synth.workload(name)
    case = Case(w)
    try:
        v = case.gpu_velocity()
        errs = []
        for b in range(w.batch):
            ref = case.oracle_velocity(b)
            errs += [rel_err(v[b, k], ref[k]) for k in range(w.n_chunks)]
        if max(errs) > tol(w):
            pytest.fail(f"max rel err {max(errs):.3e} > {tol(w)}\n" + _stage_report(case))
        print(name, "max rel err", max(errs))
    finally:
        case.close()


@pytest.mark.parametrize("name,dh,gated", [("small_bf16", 192, False), ("small_bf16", 192, True),
                                           ("small_fp32_b2", 64, False),
                                           ("small_fp32_b2", 128, True),
                                           ("small_fp32_b2", 192, True),
                                           ("small_fp32_b2", 256, True)])
def test_velocity_parity_head_dim_and_plain_mlp(name, dh, gated):
    """Head dims 128-256 (bf16 192: the register-staged attention; fp32:
    every instance of its attention kernel) and the plain tanh-GELU MLP (the
    GELU GEMM epilogue) against the oracle."""
    base = synth.workload(name)
    w = base.replace(name=f"{name}_dh{dh}_{'glu' if gated else 'mlp'}", head_dim=dh,
                     n_q_heads=2 if dh == 192 else base.n_q_heads,
                     n_kv_heads=1 if dh == 192 else base.n_kv_heads, mlp_gated=gated)
    case = Case(w)
    try:
        v = case.gpu_velocity()
        errs = []
        for b in range(w.batch):
            ref = case.oracle_velocity(b)
            errs += [rel_err(v[b, k], ref[k]) for k in range(w.n_chunks)]
        print(w.name, "max rel err", max(errs))
        assert max(errs) < tol(w), errs
    finally:
        case.close()


@pytest.mark.parametrize("name", ["small_bf16", "small_fp32_b2"])
def test_max_width(name):
    """Width 2048, the largest accepted: two column groups per thread in the
    embedding and the split-K reduction, the generic velocity head and the
    separate queue update (the fused head takes widths up to 1024).
    Velocities against the oracle; one decode step, buffer and emitted chunk
    bit for bit against the fp32 queue update of the GPU's own velocity."""
    w = synth.workload(name).replace(name=f"{name}_w2048", width=2048, n_layers=1)
    case = Case(w, noise_seed=4)
    try:
        v = case.gpu_velocity()
        errs = []
        for b in range(w.batch):
            ref = case.oracle_velocity(b)
            errs += [rel_err(v[b, k], ref[k]) for k in range(w.n_chunks)]
        print(w.name, "max rel err", max(errs))
        assert max(errs) < tol(w), errs
        case.ex.set_noise_state(4, 0)
        pre = host(case.xd).copy()
        case.ex.decode_step(case.xd, case.td, case.out)
        post, out = host(case.xd), host(case.out)
        for b in range(w.batch):
            z = oracle.gaussian_chunk(4 + b, 0, w.chunk_len, w.action_dim)
            new, ref_out = oracle.euler_emit_shift(pre[b], case.t[b], v[b], z, np.float32)
            assert np.array_equal(out[b], ref_out), b
            assert np.array_equal(post[b, :-1], new[:-1]), b
            assert np.max(np.abs(post[b, -1] - z)) <= 1e-6
    finally:
        case.close()


@pytest.mark.parametrize("name", ["tiny_fp32", "small_bf16"])
def test_max_token_limits(name):
    """The largest buffer and arena the handle accepts: K = 256 chunks of 16
    actions (K * C = 4096 query rows) after a 28672-token prefix, so the arena
    holds max_prefix + K * C = 32768 rows and the last chunk attends to all of
    them.  Velocities of every chunk against the oracle; one decode step,
    buffer and emitted chunk bit for bit against the fp32 queue update of the
    GPU's own velocity."""
    w = synth.workload(name).replace(name=f"{name}_maxtok", n_layers=1, n_chunks=256,
                                     chunk_len=16, prefix_len=28672, batch=1)
    assert w.tokens == 4096 and w.max_prefix + w.tokens == 32768
    case = Case(w, noise_seed=6)
    try:
        v = case.gpu_velocity()
        ref = case.oracle_velocity(0)
        errs = [rel_err(v[0, k], ref[k]) for k in range(w.n_chunks)]
        print(w.name, "max rel err", max(errs), "at chunk", int(np.argmax(errs)))
        assert max(errs) < tol(w), errs
        case.ex.set_noise_state(6, 0)
        pre = host(case.xd).copy()
        case.ex.decode_step(case.xd, case.td, case.out)
        post, out = host(case.xd), host(case.out)
        z = oracle.gaussian_chunk(6, 0, w.chunk_len, w.action_dim)
        new, ref_out = oracle.euler_emit_shift(pre[0], case.t[0], v[0], z, np.float32)
        assert np.array_equal(out[0], ref_out)
        assert np.array_equal(post[0, :-1], new[:-1])
        assert np.max(np.abs(post[0, -1] - z)) <= 1e-6
    finally:
        case.close()


@pytest.mark.parametrize("name,plen", [("tiny_fp32", (0, 64)), ("small_bf16", (0, 70))])
def test_max_batch(name, plen):
    """4096 streams, the largest batch a handle accepts, with ragged prefixes
    (some empty).  The oracle runs on a seeded sample of streams (both ends
    and six inside); every stream's output must be finite; one decode step
    then matches the fp32 queue update of the GPU's own velocity bit for bit
    on every stream, and the refill matches the oracle's Philox draw on the
    sampled ones."""
    w = synth.workload(name).replace(name=f"{name}_b4096", n_layers=1, batch=4096,
                                     prefix_len=plen)
    case = Case(w, noise_seed=8)
    try:
        assert int(case.lens.min()) == 0
        v = case.gpu_velocity()
        assert np.isfinite(v).all()
        rng = np.random.default_rng(4096)
        sample = sorted({0, 1, w.batch - 1, *rng.integers(2, w.batch - 1, size=5).tolist()})
        errs = []
        for b in sample:
            ref = case.oracle_velocity(b)
            errs += [rel_err(v[b, k], ref[k]) for k in range(w.n_chunks)]
        print(w.name, "streams", sample, "max rel err", max(errs))
        assert max(errs) < tol(w), errs
        case.ex.set_noise_state(8, 0)
        pre = host(case.xd).copy()
        case.ex.decode_step(case.xd, case.td, case.out)
        post, out = host(case.xd), host(case.out)
        zero = np.zeros((w.chunk_len, w.action_dim), np.float32)
        for b in range(w.batch):
            new, ref_out = oracle.euler_emit_shift(pre[b], case.t[b], v[b], zero, np.float32)
            assert np.array_equal(out[b], ref_out), b
            assert np.array_equal(post[b, :-1], new[:-1]), b
        for b in sample:
            z = oracle.gaussian_chunk(8 + b, 0, w.chunk_len, w.action_dim)
            assert np.max(np.abs(post[b, -1] - z)) <= 1e-6, b
    finally:
        case.close()


@pytest.mark.parametrize("name,lens", [("small_bf16_b3", [0, 1, 90]),
                                       ("small_fp32_b2", [0, 40])])
def test_velocity_parity_edge_prefix_lengths(name, lens):
    """An empty prefix (a query then sees only its own and earlier chunks), a
    one-token prefix and the maximum prefix, in one ragged batch."""
    w = synth.workload(name)
    case = Case(w, lens=lens)
    try:
        v = case.gpu_velocity()
        for b in range(w.batch):
            ref = case.oracle_velocity(b)
            errs = [rel_err(v[b, k], ref[k]) for k in range(w.n_chunks)]
            print(name, "P =", lens[b], "max rel err", max(errs))
            assert max(errs) < tol(w), (b, errs)
    finally:
        case.close()


def test_decode_steps_lockstep_tiny():
    """Eight decode steps of the tiny fp32 config; each step the oracle takes
    the GPU's pre-step buffer, so errors do not compound."""
    w = synth.workload("tiny_fp32")
    case = Case(w, noise_seed=5)
    try:
        xd = case.xd
        for s in range(8):
            pre = host(xd).copy()
            case.ex.decode_step(xd, case.td, case.out)
            post, out = host(xd), host(case.out)
            new, ref_out = oracle.decode_step(pre, case.t, case.k, case.v, case.lens, case.W, w,
                                              noise_seed=5, step=s)
            assert rel_err(out[0], ref_out[0]) < tol(w), s
            for k in range(w.n_chunks - 1):
                assert rel_err(post[0, k], new[0, k]) < tol(w), (s, k)
            # fresh noise: same Philox draw as the oracle (fp64 Box-Muller on both sides)
            z = oracle.gaussian_chunk(5, s, w.chunk_len, w.action_dim)
            mism = int(np.count_nonzero(post[0, -1] != z))
            print(f"tiny step {s}: refill values differing from the oracle's draw: {mism}")
            assert mism <= 2 and np.max(np.abs(post[0, -1] - z)) <= 1e-6, s
        assert case.ex.noise_state == (5, 8)
    finally:
        case.close()


@pytest.mark.parametrize("name", ["tiny_fp32", "small_bf16_b3"])
def test_bookkeeping_bit_exact(name):
    """After a step the buffer and emitted chunk equal, bit for bit, the fp32
    queue update (rounded product, rounded difference, shift, refill) applied
    to the GPU's own velocity; the refill equals the oracle's Philox draw."""
    w = synth.workload(name)
    case = Case(w, noise_seed=123)
    try:
        case.ex.set_noise_state(123, 2**32 + 7)
        v = case.gpu_velocity()
        pre = case.x.copy()
        case.ex.decode_step(case.xd, case.td, case.out)
        post, out = host(case.xd), host(case.out)
        mism = 0
        for b in range(w.batch):
            z = oracle.gaussian_chunk(123 + b, 2**32 + 7, w.chunk_len, w.action_dim)
            new, ref_out = oracle.euler_emit_shift(pre[b], case.t[b], v[b], z, np.float32)
            assert np.array_equal(out[b], ref_out)
            assert np.array_equal(post[b, :-1], new[:-1])
            mism += int(np.count_nonzero(post[b, -1] != z))
            assert np.max(np.abs(post[b, -1] - z)) <= 1e-6
        total = w.batch * w.chunk_len * w.action_dim
        print(f"{name}: refill values differing from the oracle's draw: {mism} of {total}")
        assert mism <= 2  # fp64 libm ties only
        assert case.ex.noise_state == (123, 2**32 + 8)
    finally:
        case.close()


@pytest.mark.parametrize("name,K,C", [("tiny_fp32", 4, 8), ("small_bf16_b3", 3, 10),
                                      ("tiny_fp32", 256, 2), ("small_fp32_b2", 255, 1)])
def test_euler_shift_entry_point_bit_exact(name, K, C):
    """fv_euler_shift, the separate queue-update kernel that the many-row
    decode step also runs, on a caller-given velocity: the buffer and emitted
    chunk equal, bit for bit, the fp32 queue update; the refill equals the
    oracle's Philox draw; a stream still in cold start pops padding and emits
    zeros; the valid-slot counts and the step counter advance.  Buffer
    lengths K = 3 .. 256 (the queue-update blocks hold 256 / K element groups
    of every slot, down to one group at K = 256)."""
    w = synth.workload(name).replace(n_chunks=K, chunk_len=C)
    case = Case(w, noise_seed=55)
    try:
        K = w.n_chunks
        v = synth.perturbed(np.zeros_like(case.x), 5, "euler_v")
        case.ex.set_noise_state(55, 3)
        counts = [K - 1] + [K] * (w.batch - 1)
        case.ex.set_valid_slots(counts)
        pre = case.x.copy()
        case.ex.euler_shift(case.xd, case.td, dev(v), case.out)
        post, out = host(case.xd), host(case.out)
        mism = 0
        for b in range(w.batch):
            z = oracle.gaussian_chunk(55 + b, 3, w.chunk_len, w.action_dim)
            new, ref_out = oracle.euler_emit_shift(pre[b], case.t[b], v[b], z, np.float32)
            if counts[b] < K:
                assert not np.any(out[b]), "padding popped: nothing is emitted"
            else:
                assert np.array_equal(out[b], ref_out)
            assert np.array_equal(post[b, :-1], new[:-1])
            mism += int(np.count_nonzero(post[b, -1] != z))
            assert np.max(np.abs(post[b, -1] - z)) <= 1e-6
        print(f"{name}: refill values differing from the oracle's draw: {mism}")
        assert mism <= 2  # fp64 libm ties only
        assert case.ex.noise_state == (55, 4)
        assert case.ex.valid_slots() == [K] * w.batch
    finally:
        case.close()


def test_fp32_many_rows():
    """fp32 mode at 4800 token rows (24 streams of 10 chunks x 20 tokens,
    ragged prefixes): the large-row fp32 GEMM tiles (256 x 128, the last one
    partial), the many-row head and the separate queue update.  Velocities of
    three streams against the oracle within 1e-4; one decode step, buffer and
    emitted chunks bit for bit against the fp32 queue update of the GPU's own
    velocity for every stream."""
    w = synth.workload("small_fp32_b2").replace(name="fp32_rows", n_chunks=10, chunk_len=20,
                                                 batch=24)
    assert w.batch * w.tokens >= 4096
    case = Case(w, noise_seed=9)
    try:
        v = case.gpu_velocity()
        for b in (0, int(np.argmin(case.lens)), w.batch - 1):
            ref = case.oracle_velocity(b)
            errs = [rel_err(v[b, k], ref[k]) for k in range(w.n_chunks)]
            print("fp32_rows stream", b, "P =", case.lens[b], "max rel err", max(errs))
            assert max(errs) < tol(w), (b, errs)
        case.ex.set_noise_state(9, 1)
        pre = host(case.xd).copy()
        case.ex.decode_step(case.xd, case.td, case.out)
        post, out = host(case.xd), host(case.out)
        mism = 0
        for b in range(w.batch):
            z = oracle.gaussian_chunk(9 + b, 1, w.chunk_len, w.action_dim)
            new, ref_out = oracle.euler_emit_shift(pre[b], case.t[b], v[b], z, np.float32)
            assert np.array_equal(out[b], ref_out), b
            assert np.array_equal(post[b, :-1], new[:-1]), b
            mism += int(np.count_nonzero(post[b, -1] != z))
            assert np.max(np.abs(post[b, -1] - z)) <= 1e-6
        assert mism <= 2
    finally:
        case.close()


def test_causality_bit_exact_on_gpu():
    """Perturbing chunks after k leaves the velocity of chunks <= k unchanged, bitwise."""
    w = synth.workload("small_bf16")
    case = Case(w)
    try:
        base = case.gpu_velocity()
        for k in range(w.n_chunks - 1):
            x2 = case.x.copy()
            x2[:, k + 1:] = synth.perturbed(case.x[:, k + 1:], 9, f"gpu_causal{k}")
            v2 = case.gpu_velocity(x2)
            assert np.array_equal(v2[:, :k + 1], base[:, :k + 1]), k
            assert not np.array_equal(v2[:, k + 1:], base[:, k + 1:])
    finally:
        case.close()


def test_stream_isolation_and_determinism():
    w = synth.workload("small_bf16_b3")
    case = Case(w)
    try:
        v1 = case.gpu_velocity()
        v2 = case.gpu_velocity()
        assert np.array_equal(v1, v2)
        x2 = case.x.copy()
        x2[1] = synth.perturbed(case.x[1], 4, "iso")
        v3 = case.gpu_velocity(x2)
        assert np.array_equal(v3[0], v1[0]) and np.array_equal(v3[2], v1[2])
        assert not np.array_equal(v3[1], v1[1])
    finally:
        case.close()


def test_graph_and_eager_agree():
    w = synth.workload("small_bf16")
    case = Case(w)
    try:
        vg = case.gpu_velocity()
        case.ex.set_graph_mode(False)
        ve = case.gpu_velocity()
        assert np.array_equal(vg, ve)
    finally:
        case.close()


@pytest.mark.parametrize("name", ["tiny_fp32", "small_bf16"])
def test_sequential_decode_parity(name):
    w = synth.workload(name).replace(n_chunks=1)
    case = Case(w)
    try:
        import torch
        noise = synth.make_buffer(w, 17)[:, 0]
        nd = dev(noise)
        out = torch.empty_like(nd)
        case.ex.sequential_decode(nd, 10, out)
        got = host(out)
        ref = oracle.sequential_decode(noise, 10, case.k, case.v, case.lens, case.W, w)
        for b in range(w.batch):
            assert rel_err(got[b], ref[b]) < tol(w)
    finally:
        case.close()


@pytest.mark.parametrize("name", ["small_bf16_b3", "small_fp32_b2"])
def test_velocity_parity_per_stream_noise_levels(name):
    """FiLM rows are shared only when every stream's noise levels equal stream
    0's bit for bit.  Passes alternate between one differing slot in the last
    stream, the shared staircase, a different staircase per stream and the
    first case again, so rows left over from an earlier pass are caught."""
    w = synth.workload(name)
    case = Case(w)
    try:
        base = synth.noise_levels_batched(w).astype(np.float32)
        one = base.copy()
        one[-1, w.n_chunks // 2] *= np.float32(0.5)
        every = (base * (1.0 - 0.07 * np.arange(w.batch, dtype=np.float32))[:, None]).astype(
            np.float32)
        for label, t in (("one slot", one), ("shared", base), ("every stream", every),
                         ("one slot again", one)):
            case.t = np.ascontiguousarray(t)
            case.td = dev(case.t)
            v = case.gpu_velocity()
            errs = [rel_err(v[b, k], ref[k]) for b in range(w.batch)
                    for ref in [case.oracle_velocity(b)] for k in range(w.n_chunks)]
            print(name, label, "max rel err", max(errs))
            assert max(errs) < tol(w), (label, max(errs))
    finally:
        case.close()
