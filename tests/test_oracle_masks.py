"""Pins of the oracle's attention-mask variants and cold start.

* Mask variants (Sec. 3.1 chunk-wise causal mask; the no-causal ablation of
  Appendix "Ablations", where chunks do not attend to each other at all; a
  fully bidirectional buffer) are checked against a dense mask built token by
  token from the stated rule.
* Cold start (Sec. 3.2, Algorithm 1): the buffer starts as N-1 padding chunks
  and one Gaussian sample, padding is never attended to, nothing is emitted
  for N-1 steps, and the queue then carries the chunks drawn at the
  cold-start counter and after it.
"""
import math

import numpy as np
import pytest
from scipy import special

import oracle
import synth

PIN = synth.Workload("pinm", n_layers=2, width=32, n_q_heads=4, n_kv_heads=2, head_dim=8,
                     mlp_dim=64, action_dim=3, chunk_len=2, n_chunks=4, prefix_len=3,
                     batch=1, dtype=synth.FP32)


def _rule(i_chunk, j_chunk, first, mode):
    """Token-level visibility of buffer chunk j to a query of chunk i."""
    if i_chunk < first:             # padding query: only itself
        return j_chunk == i_chunk
    if j_chunk < first:             # padding is never a key of a valid chunk
        return False
    if mode == "causal":
        return j_chunk <= i_chunk
    if mode == "isolated":
        return j_chunk == i_chunk
    return True                      # bidirectional


def _dense(q, kb, vb, kp, vp, C, first, mode):
    T, Hq, dh = q.shape
    P, Hkv = kp.shape[0], kb.shape[1]
    keys, vals = np.concatenate([kp, kb]), np.concatenate([vp, vb])
    mask = np.zeros((T, P + T), bool)
    for i in range(T):
        for j in range(P + T):
            mask[i, j] = True if j < P else _rule(i // C, (j - P) // C, first, mode)
    out, probs = np.zeros_like(q), np.zeros((Hq, T, P + T))
    for h in range(Hq):
        g = h // (Hq // Hkv)
        s = np.where(mask, q[:, h] @ keys[:, g].T / math.sqrt(dh), -np.inf)
        p = special.softmax(s, axis=1)
        out[:, h], probs[h] = p @ vals[:, g], p
    return out, probs, mask


@pytest.mark.parametrize("mode", oracle.MASK_MODES)
@pytest.mark.parametrize("K,C,P,first", [(4, 2, 3, 0), (4, 3, 0, 2), (3, 2, 4, 1), (5, 1, 2, 4)])
def test_mask_modes_brute_force(mode, K, C, P, first):
    rng = np.random.default_rng(K * 1000 + C * 100 + P * 10 + first)
    Hq, Hkv, dh, T = 4, 2, 8, K * C
    q = rng.standard_normal((T, Hq, dh))
    kb, vb = rng.standard_normal((T, Hkv, dh)), rng.standard_normal((T, Hkv, dh))
    kp, vp = rng.standard_normal((P, Hkv, dh)), rng.standard_normal((P, Hkv, dh))
    o, probs = oracle.chunk_causal_attention(q, kb, vb, kp, vp, C, return_probs=True,
                                             mode=mode, first_valid=first)
    ob, pb, mask = _dense(q, kb, vb, kp, vp, C, first, mode)
    np.testing.assert_allclose(o, ob, rtol=0, atol=1e-12)
    np.testing.assert_allclose(probs, pb, rtol=0, atol=1e-12)
    np.testing.assert_allclose(probs.sum(-1), 1.0, rtol=0, atol=1e-12)
    assert np.all(probs[:, ~mask] == 0.0)
    # padding columns are never attended to by valid rows
    if first > 0:
        assert np.all(probs[:, first * C:, P:P + first * C] == 0.0)


def _setup(seed=0):
    W = synth.make_weights(PIN, seed)
    k, v, lens = synth.make_prefix(PIN, seed)
    x = synth.make_buffer(PIN, seed)[0]
    t = synth.noise_levels(PIN)
    return W, k[:, 0], v[:, 0], int(lens[0]), x, t


def _vel(x, t, k, v, P, W, mask="causal", first=0):
    return oracle.velocity(x, t, k, v, P, W, PIN, mask=mask, first_valid=first)


def test_isolated_chunks_ignore_every_other_chunk():
    W, k, v, P, x, t = _setup()
    base = _vel(x, t, k, v, P, W, "isolated")
    for kk in range(PIN.n_chunks):
        y = x.copy()
        others = [j for j in range(PIN.n_chunks) if j != kk]
        y[others] += 1.7
        assert np.array_equal(_vel(y, t, k, v, P, W, "isolated")[kk], base[kk])
    # ...but the causal mask does couple a later chunk to an earlier one
    y = x.copy()
    y[0] += 1.7
    assert not np.array_equal(_vel(y, t, k, v, P, W)[1], _vel(x, t, k, v, P, W)[1])


def test_modes_agree_where_their_visible_sets_agree():
    W, k, v, P, x, t = _setup(1)
    K = PIN.n_chunks
    causal = _vel(x, t, k, v, P, W, "causal")
    bidir = _vel(x, t, k, v, P, W, "bidirectional")
    iso = _vel(x, t, k, v, P, W, "isolated")
    # In one layer the visible sets decide the result: the last chunk sees
    # every chunk under both the causal and the bidirectional mask, and chunk
    # 0 sees only itself under both the causal and the isolated mask.  (With
    # more layers the other chunks' hidden states already differ.)
    one = synth.Workload(**{**PIN.__dict__, "n_layers": 1})
    W1 = {kk: (vv[:1] if isinstance(vv, list) and kk not in ("w_mod", "b_mod") else vv)
          for kk, vv in W.items()}
    W1["w_mod"], W1["b_mod"] = W["w_mod"][:3], W["b_mod"][:3]
    c1 = oracle.velocity(x, t, k[:1], v[:1], P, W1, one, mask="causal")
    b1 = oracle.velocity(x, t, k[:1], v[:1], P, W1, one, mask="bidirectional")
    i1 = oracle.velocity(x, t, k[:1], v[:1], P, W1, one, mask="isolated")
    assert np.array_equal(c1[K - 1], b1[K - 1])
    assert np.array_equal(c1[0], i1[0])
    assert not np.array_equal(c1[0], b1[0])
    # with several layers the modes genuinely differ
    assert not np.allclose(causal, bidir) and not np.allclose(causal, iso)


@pytest.mark.parametrize("mode", oracle.MASK_MODES)
def test_padding_contents_never_reach_valid_chunks(mode):
    W, k, v, P, x, t = _setup(2)
    for first in (1, 2, 3):
        base = _vel(x, t, k, v, P, W, mode, first)
        y = x.copy()
        y[:first] = 100.0 * np.random.default_rng(first).standard_normal(y[:first].shape)
        got = _vel(y, t, k, v, P, W, mode, first)
        assert np.array_equal(got[first:], base[first:])


def _zero_velocity(W):
    W = dict(W)
    W["w_out"] = np.zeros_like(W["w_out"])
    W["b_out"] = np.zeros_like(W["b_out"])
    return W


def test_cold_start_queue_with_zero_velocity():
    """v = 0: nothing is emitted for K-1 steps, then the chunk drawn at the
    cold-start counter, then the chunks drawn at each later step."""
    W, k, v, P, x, t = _setup(3)
    W = _zero_velocity(W)
    K, C, A = PIN.n_chunks, PIN.chunk_len, PIN.action_dim
    seed, s0 = 11, 40
    buf = oracle.cold_start(x[None], [0], seed, s0)
    assert np.all(buf[0, :K - 1] == 0.0)
    assert np.array_equal(buf[0, K - 1], oracle.gaussian_chunk(seed, s0, C, A))
    nv = np.array([1])
    emitted = []
    for i in range(2 * K):
        buf, out, nv = oracle.decode_step(buf, t, k[:, None], v[:, None], [P], W, PIN,
                                          seed, s0 + 1 + i, n_valid=nv)
        emitted.append(out[0])
    for i in range(K - 1):
        assert np.all(emitted[i] == 0.0)
    for i in range(K - 1, 2 * K):
        assert np.array_equal(emitted[i], oracle.gaussian_chunk(seed, s0 + i - (K - 1), C, A))
    assert nv[0] == K


def test_cold_start_with_constant_velocity_emits_z_minus_c():
    """v = c: the first chunk leaves as z - sum_k dt_k c = z - c (t_{K-1} = 1)."""
    W, k, v, P, x, t = _setup(4)
    W = _zero_velocity(W)
    c = np.array([0.25, -0.5, 1.0])
    W["b_out"] = c
    K, C, A = PIN.n_chunks, PIN.chunk_len, PIN.action_dim
    buf = oracle.cold_start(x[None], [0], 5, 0)
    z = buf[0, K - 1].copy()
    nv = np.array([1])
    for i in range(K):
        buf, out, nv = oracle.decode_step(buf, t, k[:, None], v[:, None], [P], W, PIN, 5, 1 + i,
                                          n_valid=nv)
    np.testing.assert_allclose(out[0], z - c, rtol=0, atol=2e-6)


def test_cold_start_leaves_other_streams_alone():
    x = np.random.default_rng(0).standard_normal((3, 4, 2, 3)).astype(np.float32)
    new = oracle.cold_start(x, [1], 0, 0)
    assert np.array_equal(new[0], x[0]) and np.array_equal(new[2], x[2])
    assert not np.array_equal(new[1], x[1])


def test_packed_multibuffer_attention_equals_isolated_configurations():
    """Sec. 3.3 packs all N buffer configurations of one observation into one
    sequence whose attention mask isolates the configurations.  A dense
    attention over that packed sequence (mask written out token by token)
    equals the per-configuration attention with padding used by the
    multi-buffer forward."""
    rng = np.random.default_rng(7)
    N, C, P, Hq, Hkv, dh = 3, 2, 4, 2, 1, 8
    T = N * C
    q = rng.standard_normal((N, T, Hq, dh))
    kb, vb = rng.standard_normal((N, T, Hkv, dh)), rng.standard_normal((N, T, Hkv, dh))
    kp, vp = rng.standard_normal((P, Hkv, dh)), rng.standard_normal((P, Hkv, dh))
    # packed sequence: [prefix ; config 1 tokens ; ... ; config N tokens]
    keys = np.concatenate([kp] + [kb[j] for j in range(N)])
    vals = np.concatenate([vp] + [vb[j] for j in range(N)])
    out_packed = np.zeros((N, T, Hq, dh))
    for j in range(N):
        first = N - 1 - j                      # configuration j+1 has j+1 real chunks
        for i in range(T):
            vis = np.zeros(P + N * T, bool)
            vis[:P] = True
            for jj in range(N):
                for tk in range(T):
                    if jj == j:                # other configurations are invisible
                        vis[P + jj * T + tk] = _rule(i // C, tk // C, first, "causal")
            for h in range(Hq):
                g = h // (Hq // Hkv)
                sc = np.where(vis, keys[:, g] @ q[j, i, h] / math.sqrt(dh), -np.inf)
                out_packed[j, i, h] = special.softmax(sc) @ vals[:, g]
    for j in range(N):
        o = oracle.chunk_causal_attention(q[j], kb[j], vb[j], kp, vp, C, first_valid=N - 1 - j)
        np.testing.assert_allclose(o, out_packed[j], rtol=0, atol=1e-12)


def test_multibuffer_forward_is_the_cold_start_sequence_of_buffer_states():
    """Configuration j of the packed forward is exactly the buffer state a
    cold-started stream has after j-1 steps (same padding, same slots)."""
    W, k, v, P, x, t = _setup(5)
    N = PIN.n_chunks
    bufs = np.stack([x.copy() for _ in range(N)])
    for j in range(N):
        bufs[j, :N - 1 - j] = 0.0
    got = oracle.multibuffer_velocity(bufs, t, k, v, P, W, PIN)
    for j in range(N):
        ref = oracle.velocity(bufs[j], t, k, v, P, W, PIN, first_valid=N - 1 - j)
        assert np.array_equal(got[j], ref)
    # the full configuration is the steady-state buffer
    assert np.array_equal(got[N - 1], oracle.velocity(x, t, k, v, P, W, PIN))
