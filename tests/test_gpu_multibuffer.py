"""GPU parity of the packed multi-buffer forward (Sec. 3.3).

One observation, N = K buffer configurations (configuration j: N - j padding
chunks, then j real chunks), each isolated from the others.  Real chunks are
compared with the oracle's multi-buffer forward per (configuration, chunk)
slice: max relative error 1e-4 (fp32) / 1e-2 (bf16).
"""
import numpy as np
import pytest

import oracle
import synth
from tests.gpu_util import Case, dev, host, rel_err, tol

pytestmark = pytest.mark.gpu


def _configs(x):
    """[K, C, A] real chunks -> [N, K, C, A] packed configurations (zero padding)."""
    K = x.shape[0]
    bufs = np.stack([x.copy() for _ in range(K)])
    for j in range(K):
        bufs[j, :K - 1 - j] = 0.0
    return bufs


def _run(name, check=None, b=0):
    import torch
    w = synth.workload(name)
    K = w.n_chunks
    case = Case(w, max_batch=max(w.batch, K))
    try:
        bufs = _configs(case.x[b])
        t = np.broadcast_to(case.t[b], (K, K)).copy()
        kd, vd = case.kd[:, b].contiguous(), case.vd[:, b].contiguous()
        bd, tdv = dev(bufs), dev(t)
        vout = torch.empty_like(bd)
        case.ex.multibuffer_velocity(kd, vd, int(case.lens[b]), bd, tdv, vout)
        got = host(vout)
        assert case.ex.valid_slots(K) == list(range(1, K + 1))
        js = range(K) if check is None else check
        for j in js:
            ref = oracle.velocity(bufs[j], case.t[b], case.k[:, b], case.v[:, b],
                                  int(case.lens[b]), case.W, w, first_valid=K - 1 - j)
            errs = [rel_err(got[j, k], ref[k]) for k in range(K - 1 - j, K)]
            print(f"{name} configuration {j + 1}: max rel err {max(errs):.2e}")
            assert max(errs) < tol(w), (j, errs)
        return got
    finally:
        case.close()


@pytest.mark.parametrize("name", ["tiny_fp32", "small_bf16_b3", "small_fp32_b2"])
def test_multibuffer_velocity_parity_small(name):
    _run(name)


def test_multibuffer_full_configuration_equals_steady_state():
    """The last configuration is the steady-state buffer: same result as the
    ordinary velocity pass of that stream (within tolerance; the batch of
    configurations tiles differently)."""
    w = synth.workload("small_bf16_b3")
    got = _run("small_bf16_b3", check=[])
    case = Case(w)
    try:
        v = case.gpu_velocity()
        errs = [rel_err(got[-1, k], v[0, k]) for k in range(w.n_chunks)]
        assert max(errs) < tol(w), errs
    finally:
        case.close()


def test_multibuffer_velocity_full_size_pi05():
    # first, middle and last of the ten configurations
    _run("pi05_b1", check=[0, 4, 9])
