"""The C ABI driven from plain C: a C99 program (tests/c_client) builds an
fp32 handle from files, installs the prefix, runs one velocity pass and one
decode step.  Its velocity is compared with the oracle (fp32 tolerance 1e-4
per chunk slice), its emitted chunk and buffer bit for bit with the fp32
queue update of that velocity, and its refill with the oracle's Philox draw.
"""
import subprocess
import sys

import numpy as np
import pytest

import oracle
import synth
from tests.c_client.build import build_client
from tests.gpu_util import rel_err, tol

pytestmark = pytest.mark.gpu


def _weights_blob(W, w):
    L = w.n_layers
    parts = [W["w_in"], W["b_in"], W["w_t1"], W["b_t1"], W["w_t2"], W["b_t2"]]
    parts += list(W["w_mod"]) + list(W["b_mod"])
    for name in ("wq", "wk", "wv", "wo", "wg", "wu", "wd"):
        assert len(W[name]) == L
        parts += list(W[name])
    parts += [W["w_out"], W["b_out"]]
    return np.concatenate([np.asarray(p, np.float32).ravel() for p in parts])


def test_c_client_velocity_and_step(tmp_path):
    w = synth.workload("tiny_fp32")
    assert w.batch == 1 and w.mlp_gated and w.noise_seed == 0
    W = synth.make_weights(w, 0)
    k, v, lens = synth.make_prefix(w, 0)
    P = int(lens[0])
    x = synth.make_buffer(w, 0)
    t = synth.noise_levels_batched(w)
    _weights_blob(W, w).tofile(tmp_path / "weights.bin")
    np.ascontiguousarray(k[:, :1, :P], np.float32).tofile(tmp_path / "prefix_k.bin")
    np.ascontiguousarray(v[:, :1, :P], np.float32).tofile(tmp_path / "prefix_v.bin")
    np.ascontiguousarray(x, np.float32).tofile(tmp_path / "buffer.bin")
    np.ascontiguousarray(t, np.float32).tofile(tmp_path / "t.bin")

    exe = str(tmp_path / "decode_client")
    build_client(exe)
    args = [exe, str(tmp_path)] + [str(a) for a in (w.n_layers, w.width, w.n_q_heads,
                                                    w.n_kv_heads, w.head_dim, w.mlp_dim,
                                                    w.action_dim, w.chunk_len, w.n_chunks, P)]
    print("running", " ".join(args), flush=True)
    sys.stdout.flush()
    r = subprocess.run(args, capture_output=True, text=True, timeout=120)
    print(r.stdout, r.stderr)
    assert r.returncode == 0, r.stderr
    assert "noise step 1" in r.stdout

    shape = (w.n_chunks, w.chunk_len, w.action_dim)
    vel = np.fromfile(tmp_path / "v.bin", np.float32).reshape(shape)
    out = np.fromfile(tmp_path / "out.bin", np.float32).reshape(shape[1:])
    after = np.fromfile(tmp_path / "buffer_after.bin", np.float32).reshape(shape)
    ref = oracle.velocity(x[0], t[0], k[:, 0], v[:, 0], P, W, w)
    errs = [rel_err(vel[c], ref[c]) for c in range(w.n_chunks)]
    print("C client velocity: max rel err", max(errs))
    assert max(errs) < tol(w), errs
    z = oracle.gaussian_chunk(0, 0, w.chunk_len, w.action_dim)
    new, ref_out = oracle.euler_emit_shift(x[0], t[0], vel, z, np.float32)
    assert np.array_equal(out, ref_out)
    assert np.array_equal(after[:-1], new[:-1])
    assert int(np.count_nonzero(after[-1] != z)) <= 2
    assert np.max(np.abs(after[-1] - z)) <= 1e-6
