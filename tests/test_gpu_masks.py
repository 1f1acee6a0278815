"""GPU parity of the mask variants, cold start and the static-schedule cache.

* Every mask mode (chunk-causal, isolated chunks, bidirectional) against the
  oracle, with full buffers and with cold-start padding.
* Cold start (Algorithm 1): padding never reaches a valid chunk, nothing is
  emitted for K-1 steps, and with zero velocity the queue bookkeeping is bit
  exact against the oracle's Philox draws.
* The static-schedule cache gives results bit-identical to passing t.
Tolerances: max relative error per (stream, chunk) slice, 1e-4 fp32 / 1e-2 bf16.
"""
import numpy as np
import pytest

import oracle
import synth
from tests.gpu_util import Case, dev, host, rel_err, tol

pytestmark = pytest.mark.gpu

SMALL = ["small_fp32_b2", "small_bf16_b3", "tiny_fp32"]


def _oracle_v(case, b, x=None, mask="causal", first=0):
    x = case.x if x is None else x
    return oracle.velocity(x[b], case.t[b], case.k[:, b], case.v[:, b], int(case.lens[b]),
                           case.W, case.w, mask=mask, first_valid=first)


@pytest.mark.parametrize("mode", ["isolated", "bidirectional", "causal"])
@pytest.mark.parametrize("name", SMALL)
def test_mask_modes_velocity_parity(name, mode):
    w = synth.workload(name)
    case = Case(w)
    try:
        case.ex.set_mask_mode(mode)
        v = case.gpu_velocity()
        for b in range(w.batch):
            ref = _oracle_v(case, b, mask=mode)
            errs = [rel_err(v[b, k], ref[k]) for k in range(w.n_chunks)]
            print(name, mode, b, max(errs))
            assert max(errs) < tol(w), (mode, b, errs)
    finally:
        case.close()


@pytest.mark.parametrize("mode", ["causal", "isolated", "bidirectional"])
@pytest.mark.parametrize("name", ["small_fp32_b2", "small_bf16_b3"])
def test_padded_buffer_velocity_parity(name, mode):
    """After a cold start of some streams, valid chunks match the oracle with
    the same padding; padding contents do not change them at all."""
    w = synth.workload(name)
    case = Case(w, noise_seed=3)
    try:
        case.ex.set_mask_mode(mode)
        cold = list(range(1, w.batch))            # stream 0 stays in steady state
        case.ex.cold_start(case.xd, 1, w.batch - 1)
        nv = case.ex.valid_slots()
        assert nv == [w.n_chunks] + [1] * (w.batch - 1)
        x = host(case.xd).copy()
        for b in cold:
            assert np.all(x[b, :-1] == 0.0)
        v = case.gpu_velocity(x)
        for b in range(w.batch):
            first = w.n_chunks - nv[b]
            ref = _oracle_v(case, b, x, mode, first)
            errs = [rel_err(v[b, k], ref[k]) for k in range(first, w.n_chunks)]
            assert max(errs) < tol(w), (mode, b, errs)
        # padding contents never reach a valid chunk (bitwise)
        y = x.copy()
        for b in cold:
            y[b, :-1] = 7.0 * np.random.default_rng(b).standard_normal(y[b, :-1].shape)
        v2 = case.gpu_velocity(y)
        for b in cold:
            assert np.array_equal(v2[b, -1], v[b, -1])
    finally:
        case.close()


def _zero_out_weights(W):
    W = dict(W)
    W["w_out"] = np.zeros_like(W["w_out"])
    W["b_out"] = np.zeros_like(W["b_out"])
    return W


@pytest.mark.parametrize("name", ["tiny_fp32", "small_bf16_b3"])
def test_cold_start_bookkeeping_bit_exact(name):
    """v = 0: K-1 zero emissions, then exactly the chunks drawn at the cold
    start counter and after it; valid slot counts 1, 2, ..., K."""
    w = synth.workload(name)
    W = _zero_out_weights(synth.make_weights(w))
    case = Case(w, weights=W, noise_seed=9)
    try:
        K, C, A = w.n_chunks, w.chunk_len, w.action_dim
        seed, s0 = case.ex.noise_state
        case.ex.cold_start(case.xd)
        assert case.ex.noise_state == (seed, s0 + 1)
        x = host(case.xd)
        for b in range(w.batch):
            assert np.all(x[b, :K - 1] == 0.0)
            assert np.array_equal(x[b, K - 1], oracle.gaussian_chunk(seed + b, s0, C, A))
        for i in range(2 * K):
            case.ex.decode_step(case.xd, case.td, case.out)
            out = host(case.out)
            nv = case.ex.valid_slots()
            assert nv == [min(i + 2, K)] * w.batch
            for b in range(w.batch):
                if i < K - 1:
                    assert np.all(out[b] == 0.0), (i, b)
                else:
                    want = oracle.gaussian_chunk(seed + b, s0 + i - (K - 1), C, A)
                    assert np.array_equal(out[b], want), (i, b)
    finally:
        case.close()


def test_cold_start_lockstep_against_oracle():
    """Real weights: a cold-started tiny fp32 stream follows the oracle's
    cold-start trajectory step by step (emission zeros until full)."""
    w = synth.workload("tiny_fp32")
    case = Case(w, noise_seed=4)
    try:
        K = w.n_chunks
        seed, s0 = case.ex.noise_state
        case.ex.cold_start(case.xd)
        ref_buf = oracle.cold_start(case.x, [0], seed, s0)
        assert np.array_equal(host(case.xd), ref_buf)
        nv = np.array([1])
        for i in range(K + 2):
            pre = host(case.xd).copy()
            v = case.gpu_velocity(pre)
            case.ex.decode_step(case.xd, case.td, case.out)
            post, out = host(case.xd), host(case.out)
            first = K - int(nv[0])
            z = oracle.gaussian_chunk(seed, s0 + 1 + i, w.chunk_len, w.action_dim)
            new, ref_out = oracle.euler_emit_shift(pre[0], case.t[0], v[0], z, np.float32)
            if first > 0:
                ref_out = np.zeros_like(ref_out)
            assert np.array_equal(out[0], ref_out)          # bookkeeping: bit exact
            assert np.array_equal(post[0, :-1], new[:-1])
            ref_v = _oracle_v(case, 0, pre, "causal", first)
            errs = [rel_err(v[0, k], ref_v[k]) for k in range(first, K)]
            assert max(errs) < tol(w), (i, errs)
            nv = np.minimum(nv + 1, K)
    finally:
        case.close()


@pytest.mark.parametrize("name", ["small_bf16_b3", "tiny_fp32"])
def test_static_schedule_cache_is_bit_identical(name):
    import torch
    w = synth.workload(name)
    a, b = Case(w, noise_seed=2), Case(w, noise_seed=2)
    try:
        b.ex.set_schedule(b.td)
        for _ in range(3):
            a.ex.decode_step(a.xd, a.td, a.out)
            b.ex.decode_step(b.xd, None, b.out)
            assert torch.equal(a.xd, b.xd) and torch.equal(a.out, b.out)
        va = torch.empty_like(a.xd)
        vb = torch.empty_like(b.xd)
        a.ex.velocity(a.xd, a.td, va)
        b.ex.velocity(b.xd, None, vb)
        assert torch.equal(va, vb)
    finally:
        a.close()
        b.close()


def test_decode_without_schedule_is_rejected():
    from paper_2608_27384_amd.flashvla import FlashVLAError
    w = synth.workload("tiny_fp32")
    case = Case(w)
    try:
        with pytest.raises(FlashVLAError):
            case.ex.decode_step(case.xd, None, case.out)
    finally:
        case.close()


def test_isolated_mask_full_size_pi05():
    w = synth.workload("pi05_b1")
    case = Case(w)
    try:
        case.ex.set_mask_mode("isolated")
        v = case.gpu_velocity()
        ref = _oracle_v(case, 0, mask="isolated")
        errs = [rel_err(v[0, k], ref[k]) for k in range(w.n_chunks)]
        print("pi05 isolated: max rel err", max(errs))
        assert max(errs) < tol(w)
    finally:
        case.close()


def test_cold_start_padding_full_size_pi05():
    """pi0.5 shape right after a cold start: the one valid chunk (with nine
    padding slots in front) matches the oracle."""
    w = synth.workload("pi05_b1")
    case = Case(w, noise_seed=1)
    try:
        case.ex.cold_start(case.xd)
        x = host(case.xd).copy()
        v = case.gpu_velocity(x)
        ref = _oracle_v(case, 0, x, "causal", w.n_chunks - 1)
        err = rel_err(v[0, -1], ref[-1])
        print("pi05 cold start: valid chunk rel err", err)
        assert err < tol(w)
    finally:
        case.close()
