"""Pins of the CPU oracle against facts the paper and the mathematics fix.

Each test checks the oracle against something other than itself: brute
force on tiny inputs, closed forms, invariants and special cases that reduce
to a textbook computation.  Together they are chosen so that a plausible
mistake anywhere in the oracle (a dropped term, a wrong sign or index, a
transposed mask, a wrong slot shift) fails at least one of them.
"""
import math
import os

import numpy as np
import pytest
from scipy import special, stats

import oracle
import synth

PIN = synth.Workload("pin", n_layers=2, width=32, n_q_heads=4, n_kv_heads=2, head_dim=8,
                     mlp_dim=48, action_dim=3, chunk_len=3, n_chunks=3, prefix_len=5,
                     batch=1, dtype=synth.FP32, weight_std=0.2)


def _inputs(w, seed=0):
    W = synth.make_weights(w, seed)
    k, v, lens = synth.make_prefix(w, seed)
    x = synth.make_buffer(w, seed)
    t = synth.noise_levels(w)
    return W, k, v, lens, x, t


def _v(w, W, k, v, lens, x, t, b=0, dtype=np.float64):
    return oracle.velocity(x[b], t, k[:, b], v[:, b], int(lens[b]), W, w, dtype)


# --------------------------------------------------------------------- P1/P2


def _brute_force_attention(q, k_buf, v_buf, k_pre, v_pre, C):
    """Dense masked attention; the mask is built token by token from the
    visibility rule: a query of chunk i sees every prefix token and every
    buffer token of chunk j <= i."""
    T, Hq, dh = q.shape
    P = k_pre.shape[0]
    Hkv = k_buf.shape[1]
    keys = np.concatenate([k_pre, k_buf], axis=0)
    vals = np.concatenate([v_pre, v_buf], axis=0)
    mask = np.zeros((T, P + T), dtype=bool)
    for i in range(T):
        for j in range(P + T):
            if j < P:
                mask[i, j] = True
            else:
                mask[i, j] = (j - P) // C <= i // C
    out = np.zeros_like(q)
    probs = np.zeros((Hq, T, P + T))
    for h in range(Hq):
        g = h // (Hq // Hkv)
        s = q[:, h] @ keys[:, g].T / math.sqrt(dh)
        s = np.where(mask, s, -np.inf)
        p = special.softmax(s, axis=1)
        out[:, h] = p @ vals[:, g]
        probs[h] = p
    return out, probs, mask


@pytest.mark.parametrize("K,C,P,Hq,Hkv", [(3, 4, 5, 2, 1), (2, 3, 0, 4, 2), (3, 1, 2, 2, 2),
                                          (1, 4, 3, 2, 1)])
def test_p1_attention_brute_force(K, C, P, Hq, Hkv):
    rng = np.random.default_rng(K * 100 + C * 10 + P)
    dh, T = 8, K * C
    q = rng.standard_normal((T, Hq, dh))
    kb, vb = rng.standard_normal((T, Hkv, dh)), rng.standard_normal((T, Hkv, dh))
    kp, vp = rng.standard_normal((P, Hkv, dh)), rng.standard_normal((P, Hkv, dh))
    o, probs = oracle.chunk_causal_attention(q, kb, vb, kp, vp, C, return_probs=True)
    ob, pb, mask = _brute_force_attention(q, kb, vb, kp, vp, C)
    np.testing.assert_allclose(o, ob, rtol=0, atol=1e-12)
    np.testing.assert_allclose(probs, pb, rtol=0, atol=1e-12)
    # P2: rows sum to one; invisible keys get exactly zero probability.
    np.testing.assert_allclose(probs.sum(-1), 1.0, rtol=0, atol=1e-12)
    assert np.all(probs[:, ~mask] == 0.0)
    # Earlier chunks never see later ones (the mask is not transposed).
    if K > 1:
        assert np.all(probs[:, :C, P + C:] == 0.0)
        assert np.all(probs[:, T - C:, P:] > 0.0)


# ------------------------------------------------------------------------ P3


def test_p3_single_visible_key_returns_its_value():
    rng = np.random.default_rng(1)
    q = rng.standard_normal((1, 2, 8))
    kb, vb = rng.standard_normal((1, 1, 8)), rng.standard_normal((1, 1, 8))
    e = np.zeros((0, 1, 8))
    o = oracle.chunk_causal_attention(q, kb, vb, e, e, 1)
    np.testing.assert_allclose(o[0, 0], vb[0, 0], atol=1e-15)
    np.testing.assert_allclose(o[0, 1], vb[0, 0], atol=1e-15)


def test_p3_identical_keys_average_visible_values():
    rng = np.random.default_rng(2)
    K, C, P, dh = 3, 2, 4, 8
    T = K * C
    q = rng.standard_normal((T, 2, dh))
    key = rng.standard_normal(dh)
    kb = np.broadcast_to(key, (T, 1, dh)).copy()
    kp = np.broadcast_to(key, (P, 1, dh)).copy()
    vb, vp = rng.standard_normal((T, 1, dh)), rng.standard_normal((P, 1, dh))
    o = oracle.chunk_causal_attention(q, kb, vb, kp, vp, C)
    for k in range(K):
        vis = np.concatenate([vp[:, 0], vb[:(k + 1) * C, 0]])
        for c in range(C):
            np.testing.assert_allclose(o[k * C + c, 1], vis.mean(0), atol=1e-13)


def test_p3_gqa_equals_mha_with_replicated_kv():
    rng = np.random.default_rng(3)
    K, C, P, dh, Hq, Hkv = 2, 3, 4, 8, 4, 2
    T = K * C
    q = rng.standard_normal((T, Hq, dh))
    kb, vb = rng.standard_normal((T, Hkv, dh)), rng.standard_normal((T, Hkv, dh))
    kp, vp = rng.standard_normal((P, Hkv, dh)), rng.standard_normal((P, Hkv, dh))
    o = oracle.chunk_causal_attention(q, kb, vb, kp, vp, C)
    rep = lambda a: np.repeat(a, Hq // Hkv, axis=1)   # head h <- kv head h // group
    o_mha = oracle.chunk_causal_attention(q, rep(kb), rep(vb), rep(kp), rep(vp), C)
    np.testing.assert_allclose(o, o_mha, atol=1e-14)


def test_softmax_scale_is_inverse_sqrt_head_dim():
    # Two visible keys: o = sigma((s1 - s2)/sqrt(dh)) v1 + (1 - sigma) v2.
    rng = np.random.default_rng(4)
    dh = 16
    q = rng.standard_normal((1, 1, dh))
    kp, vp = rng.standard_normal((1, 1, dh)), rng.standard_normal((1, 1, dh))
    kb, vb = rng.standard_normal((1, 1, dh)), rng.standard_normal((1, 1, dh))
    o = oracle.chunk_causal_attention(q, kb, vb, kp, vp, 1)
    s1, s2 = q[0, 0] @ kp[0, 0], q[0, 0] @ kb[0, 0]
    a = 1.0 / (1.0 + math.exp(-(s1 - s2) / math.sqrt(dh)))
    np.testing.assert_allclose(o[0, 0], a * vp[0, 0] + (1 - a) * vb[0, 0], atol=1e-14)


# ------------------------------------------------------------------------ P4


def test_p4_rope_properties():
    rng = np.random.default_rng(5)
    dh, n = 16, 7
    x = rng.standard_normal((n, dh))
    pos = rng.integers(0, 1000, n)
    np.testing.assert_allclose(oracle.rope(x, np.zeros(n, int), 1e4), x, atol=0)
    r = oracle.rope(x, pos, 1e4)
    np.testing.assert_allclose(np.linalg.norm(r, axis=1), np.linalg.norm(x, axis=1), rtol=1e-13)
    # q.k depends only on the position difference.
    q, k = rng.standard_normal((1, dh)), rng.standard_normal((1, dh))
    d1 = oracle.rope(q, [37], 1e4) @ oracle.rope(k, [12], 1e4).T
    d2 = oracle.rope(q, [537], 1e4) @ oracle.rope(k, [512], 1e4).T
    np.testing.assert_allclose(d1, d2, rtol=1e-11)
    # Half-split pairing: e_i rotates into e_{i + dh/2} at angle pos*theta^(-2i/dh).
    for i in (0, 3):
        e = np.zeros((1, dh))
        e[0, i] = 1.0
        r = oracle.rope(e, [5], 1e4)[0]
        ang = 5 * 1e4 ** (-2.0 * i / dh)
        expect = np.zeros(dh)
        expect[i], expect[i + dh // 2] = math.cos(ang), math.sin(ang)
        np.testing.assert_allclose(r, expect, atol=1e-15)


# ------------------------------------------------------------------- P5/P6


def test_p5_causality_later_chunks_do_not_touch_earlier_velocities():
    W, k, v, lens, x, t = _inputs(PIN)
    base = _v(PIN, W, k, v, lens, x, t)
    for kk in range(PIN.n_chunks - 1):
        x2 = x.copy()
        x2[0, kk + 1:] = synth.perturbed(x[0, kk + 1:], 7, f"p5_{kk}")
        pert = _v(PIN, W, k, v, lens, x2, t)
        assert np.array_equal(pert[:kk + 1], base[:kk + 1]), kk
        assert not np.allclose(pert[kk + 1:], base[kk + 1:])


def test_p6_chunk0_alone_matches_full_buffer():
    W, k, v, lens, x, t = _inputs(PIN)
    full = _v(PIN, W, k, v, lens, x, t)
    alone = oracle.velocity(x[0, :1], t[:1], k[:, 0], v[:, 0], int(lens[0]), W, PIN)
    np.testing.assert_allclose(alone[0], full[0], rtol=0, atol=1e-13)


# ------------------------------------------------------------------- P7/P8


def test_p7_zero_modulation_makes_every_block_the_identity():
    W, k, v, lens, x, t = _inputs(PIN)
    W["w_mod"] = [np.zeros_like(a) for a in W["w_mod"]]
    W["b_mod"] = [np.zeros_like(a) for a in W["b_mod"]]
    got = _v(PIN, W, k, v, lens, x, t)
    h = x[0].reshape(-1, PIN.action_dim).astype(np.float64) @ W["w_in"] + W["b_in"]
    u = h / np.sqrt(np.mean(h * h, axis=1, keepdims=True) + PIN.rms_eps)
    expect = (u @ W["w_out"] + W["b_out"]).reshape(got.shape)
    np.testing.assert_allclose(got, expect, rtol=0, atol=1e-13)


def _textbook_prenorm_transformer(x, W, k_pre, v_pre, P, w):
    """Standard pre-norm transformer written token by token: weightless
    RMSNorm, rotary multi-query attention under the chunk-causal mask with
    the prefix, GeGLU MLP (w.mlp_gated) or a two-layer tanh-GELU MLP, plain
    residuals, and an output head."""
    K, C, A = x.shape
    T, Hq, Hkv, dh = K * C, w.n_q_heads, w.n_kv_heads, w.head_dim
    rms = lambda r: r / math.sqrt(float(np.dot(r, r)) / r.size + w.rms_eps)

    def rot(vec, p):
        out = vec.copy()
        for i in range(dh // 2):
            a = p * w.rope_theta ** (-2.0 * i / dh)
            out[i] = vec[i] * math.cos(a) - vec[i + dh // 2] * math.sin(a)
            out[i + dh // 2] = vec[i + dh // 2] * math.cos(a) + vec[i] * math.sin(a)
        return out

    gelu = lambda z: 0.5 * z * (1 + np.tanh(math.sqrt(2 / math.pi) * (z + 0.044715 * z ** 3)))
    hs = [x.reshape(T, A)[i].astype(np.float64) @ W["w_in"] + W["b_in"] for i in range(T)]
    for l in range(w.n_layers):
        us = [rms(hs[i]) for i in range(T)]
        qs = [(us[i] @ W["wq"][l]).reshape(Hq, dh) for i in range(T)]
        ks = [(us[i] @ W["wk"][l]).reshape(Hkv, dh) for i in range(T)]
        vs = [(us[i] @ W["wv"][l]).reshape(Hkv, dh) for i in range(T)]
        qs = [np.stack([rot(qs[i][h], P + i) for h in range(Hq)]) for i in range(T)]
        ks = [np.stack([rot(ks[i][g], P + i) for g in range(Hkv)]) for i in range(T)]
        new = []
        for i in range(T):
            heads = []
            for h in range(Hq):
                g = h * Hkv // Hq
                keys = [k_pre[l, j, g] for j in range(P)]
                vals = [v_pre[l, j, g] for j in range(P)]
                for j in range(T):
                    if j // C <= i // C:
                        keys.append(ks[j][g])
                        vals.append(vs[j][g])
                sc = np.array([qs[i][h] @ kj for kj in keys]) / math.sqrt(dh)
                pr = np.exp(sc - sc.max())
                pr /= pr.sum()
                heads.append(sum(pr[j] * vals[j] for j in range(len(vals))))
            new.append(hs[i] + np.concatenate(heads) @ W["wo"][l])
        hs = new
        for i in range(T):
            u2 = rms(hs[i])
            if w.mlp_gated:
                hs[i] = hs[i] + (gelu(u2 @ W["wg"][l]) * (u2 @ W["wu"][l])) @ W["wd"][l]
            else:
                hs[i] = hs[i] + gelu(u2 @ W["wu"][l]) @ W["wd"][l]
    return np.stack([rms(hs[i]) @ W["w_out"] + W["b_out"] for i in range(T)]).reshape(K, C, A)


@pytest.mark.parametrize("gated", [True, False])
def test_p8_unit_gates_reduce_to_textbook_prenorm_transformer(gated):
    w = PIN.replace(mlp_gated=gated)
    W, k, v, lens, x, t = _inputs(w)
    Wd = w.width
    W["w_mod"] = [np.zeros_like(a) for a in W["w_mod"]]
    W["b_mod"] = [np.concatenate([np.zeros(2 * Wd), np.ones(Wd)]).astype(np.float32)
                  for _ in W["b_mod"]]
    got = _v(w, W, k, v, lens, x, t)
    P = int(lens[0])
    expect = _textbook_prenorm_transformer(x[0], W, k[:, 0].astype(np.float64),
                                           v[:, 0].astype(np.float64), P, w)
    np.testing.assert_allclose(got, expect, rtol=0, atol=1e-11)


def test_film_scale_shift_gate_order():
    # cond @ M + m split as [scale | shift | gate] and applied as
    # rmsnorm(h) * (1 + scale) + shift: with a single active bias entry in
    # each third the effect is visible in exactly one place.
    W = 6
    cond = np.zeros(W)
    b = np.zeros(3 * W)
    b[1], b[W + 2], b[2 * W + 3] = 0.5, -2.0, 3.0
    s, sh, g = oracle.film(cond, np.zeros((W, 3 * W)), b)
    h = np.arange(1.0, W + 1)
    y = oracle.adaptive_rmsnorm(h, s, sh, 0.0)
    r = h / math.sqrt(np.mean(h * h))
    expect = r.copy()
    expect[1] *= 1.5
    expect[2] -= 2.0
    np.testing.assert_allclose(y, expect, rtol=1e-14)
    assert g[3] == 3.0 and np.count_nonzero(g) == 1


# ------------------------------------------------------------------------ P9


def test_p9_time_embedding():
    W = 64
    e0 = oracle.timestep_embedding(0.0, W)
    assert np.all(e0[:W // 2] == 0.0) and np.all(e0[W // 2:] == 1.0)
    for t in (0.1, 0.5, 0.93):
        e = oracle.timestep_embedding(t, W)
        np.testing.assert_allclose(np.sum(e * e), W / 2, rtol=1e-14)
        # Shortest period 4e-3 in the first pair, longest 4.0 in the last.
        np.testing.assert_allclose(e[0], math.sin(2 * math.pi * t / 4e-3), atol=1e-12)
        np.testing.assert_allclose(e[W // 2 - 1], math.sin(2 * math.pi * t / 4.0), atol=1e-15)
        np.testing.assert_allclose(e[W - 1], math.cos(2 * math.pi * t / 4.0), atol=1e-15)


def test_rmsnorm_unit_rms_and_gelu_close_to_exact_gelu():
    rng = np.random.default_rng(6)
    h = rng.standard_normal((5, 64)) * 3.0
    r = oracle.rmsnorm(h, 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(r * r, axis=1)), 1.0, rtol=1e-14)
    z = np.linspace(-6, 6, 2001)
    exact = z * 0.5 * (1 + special.erf(z / math.sqrt(2)))
    assert np.max(np.abs(oracle.gelu_tanh(z) - exact)) < 1e-3
    np.testing.assert_allclose(oracle.silu(z), z * special.expit(z), rtol=1e-13)


# ----------------------------------------------------------- P10/P11/P12 (queue)


def _run_queue(x0, t, velocity_fn, n_steps, tails):
    """Steady-streaming queue driven by a stub velocity; returns emitted chunks."""
    x, outs = x0.copy(), []
    for s in range(n_steps):
        v = velocity_fn(x, t)
        x, out = oracle.euler_emit_shift(x, t, v, tails[s])
        outs.append(out)
    return x, outs


def test_p10_constant_velocity_closed_form():
    K, C, A = 5, 4, 3
    rng = np.random.default_rng(8)
    t = (np.arange(1, K + 1) / K).astype(np.float32)
    c = rng.standard_normal((C, A))
    tails = [rng.standard_normal((C, A)).astype(np.float32) for _ in range(3 * K)]
    x0 = rng.standard_normal((K, C, A)).astype(np.float32)
    x, outs = _run_queue(x0, t, lambda x, t: np.broadcast_to(c, x.shape), 3 * K, tails)
    # A chunk pushed as z at step s leaves K steps later as z - t_{K-1} c = z - c.
    for s in range(K, 3 * K):
        np.testing.assert_allclose(outs[s], tails[s - K] - c, rtol=0, atol=2e-6)
    # Every slot k holds z - (1 - t_k) c: the noisiest slot is pure noise.
    for k in range(K):
        np.testing.assert_allclose(x[k], tails[3 * K - K + k] - (1 - t[k]) * c, atol=2e-6)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_p11_straight_line_flow_emits_the_target(seed):
    # v*(x, tau) = (x - a)/tau is the exact flow of Eq. 1 for a point mass at a.
    # Each step maps x - a to (x - a) t_{k-1}/t_k, so every chunk leaves the
    # buffer at exactly a, for any increasing staircase.
    K, C, A = 6, 3, 2
    rng = np.random.default_rng(seed)
    t = np.sort(rng.uniform(0.05, 1.0, K)).astype(np.float32)
    a = rng.standard_normal((C, A))
    stub = lambda x, tt: (x.astype(np.float64) - a) / tt.astype(np.float64)[:, None, None]
    tails = [rng.standard_normal((C, A)).astype(np.float32) for _ in range(3 * K)]
    x0 = rng.standard_normal((K, C, A)).astype(np.float32)
    _, outs = _run_queue(x0, t, stub, 3 * K, tails)
    for s in range(3 * K):
        np.testing.assert_allclose(outs[s], a, rtol=0, atol=1e-5)


def test_p11_wrong_sign_or_dt_would_fail():
    # The same straight-line flow through x + dt v, or dt = t_k, does not emit a.
    K, C, A = 4, 2, 2
    rng = np.random.default_rng(3)
    t = (np.arange(1, K + 1) / K).astype(np.float32)
    a = rng.standard_normal((C, A))
    x = rng.standard_normal((K, C, A))
    v = (x - a) / t[:, None, None]
    dt_wrong = t[:, None, None]
    assert not np.allclose((x - dt_wrong * v)[1], a + (x[1] - a) * t[0] / t[1])
    new, out = oracle.euler_emit_shift(x.astype(np.float32), t, v, np.zeros((C, A)))
    np.testing.assert_allclose(out, a, atol=1e-6)
    np.testing.assert_allclose(new[0], a + (x[1] - a) * t[0] / t[1], atol=1e-6)


def test_p12_zero_velocity_is_pure_bookkeeping():
    K, C, A = 4, 3, 2
    rng = np.random.default_rng(9)
    t = (np.arange(1, K + 1) / K).astype(np.float32)
    tails = [rng.standard_normal((C, A)).astype(np.float32) for _ in range(3 * K)]
    x0 = rng.standard_normal((K, C, A)).astype(np.float32)
    for arith in (np.float64, np.float32):
        x, outs = x0.copy(), []
        for s in range(3 * K):
            x, out = oracle.euler_emit_shift(x, t, np.zeros_like(x), tails[s], arith)
            outs.append(out)
        for s in range(K):
            assert np.array_equal(outs[s], x0[s])
        for s in range(K, 3 * K):
            assert np.array_equal(outs[s], tails[s - K])
        assert np.array_equal(x, np.stack(tails[2 * K:3 * K]))


def test_euler_fp32_replica_rounds_product_then_difference():
    x = np.array([[[1.0000001]]], np.float32)
    v = np.array([[[3.0000002]]], np.float32)
    t = np.array([0.3], np.float32)
    new, out = oracle.euler_emit_shift(x, t, v, np.zeros((1, 1), np.float32), np.float32)
    p = np.float32(np.float32(0.3) * np.float32(3.0000002))
    assert out[0, 0] == np.float32(np.float32(1.0000001) - p)


def test_dt_is_staircase_difference():
    t = np.array([0.1, 0.25, 0.7, 1.0], np.float32)
    dt = oracle.euler_steps(t)
    assert dt.dtype == np.float32
    np.testing.assert_array_equal(dt, np.array([t[0], t[1] - t[0], t[2] - t[1], t[3] - t[2]],
                                               np.float32))
    assert np.sum(dt.astype(np.float64)) == pytest.approx(1.0, abs=1e-7)


# ----------------------------------------------------------------------- P14


def test_p14_philox_known_answer_vectors():
    """Published Philox4x32-10 known answers (tests/golden/philox4x32_10_kat.txt)."""
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                        "philox4x32_10_kat.txt")
    n = 0
    for line in open(path):
        if line.startswith("#") or not line.strip():
            continue
        words = [int(x, 16) for x in line.split()]
        ctr, key, want = words[:4], words[4:6], words[6:]
        got = oracle.philox4x32_10(np.array(ctr, dtype=np.uint64), np.array(key, dtype=np.uint64))
        assert [int(x) for x in got] == want
        n += 1
    assert n == 3


def test_p14_philox_uniform_and_normal_statistics():
    words = np.concatenate([oracle.noise_words(seed, s, 4096) for seed in (0, 1, 2**40 + 3)
                            for s in range(0, 80, 7)])
    counts = np.bincount((words >> 24).astype(np.int64), minlength=256)
    chi2 = stats.chisquare(counts)
    assert chi2.pvalue > 1e-4
    z = np.concatenate([oracle.gaussian_chunk(seed, s, 500, 200).ravel()
                        for seed in range(2) for s in range(6)])
    n = z.size
    assert n >= 1_000_000
    assert abs(z.mean()) < 5 / math.sqrt(n)
    assert abs(z.var() - 1.0) < 5 * math.sqrt(2.0 / n)
    assert stats.kstest(z[:200000], "norm").pvalue > 1e-4


def test_p14_philox_no_counter_reuse_and_distinct_streams():
    a = oracle.noise_words(5, 3, 400).reshape(-1, 4)
    b = oracle.noise_words(5, 4, 400).reshape(-1, 4)
    c = oracle.noise_words(6, 3, 400).reshape(-1, 4)
    rows = {tuple(r) for r in np.concatenate([a, b, c])}
    assert len(rows) == 300
    # Step counters above 2^32 use the high counter word.
    d = oracle.noise_words(5, 3 + 2**32, 400)
    assert not np.array_equal(d, oracle.noise_words(5, 3, 400))


def test_p14_box_muller_maps_quadrants():
    # u0 -> radius, u1 -> angle: r with u1 = 1/4 gives (0, rad) up to rounding.
    r = np.array([2**31, 2**30], np.uint64)
    z = oracle.box_muller(r)
    u0 = (2**31 + 0.5) / 2**32
    rad = math.sqrt(-2 * math.log(u0))
    u1 = (2**30 + 0.5) / 2**32
    np.testing.assert_allclose(z, [rad * math.cos(2 * math.pi * u1), rad * math.sin(2 * math.pi * u1)],
                               rtol=1e-15)
    assert abs(z[0]) < 1e-8 * rad + 1e-8


# ----------------------------------------------------------------------- P16


def test_p16_fp32_oracle_agrees_with_fp64():
    w = synth.workload("tiny_fp32")
    W, k, v, lens, x, t = _inputs(w)
    v64 = _v(w, W, k, v, lens, x, t)
    v32 = _v(w, W, k, v, lens, x, t, dtype=np.float32)
    assert v32.dtype == np.float32
    for kk in range(w.n_chunks):
        assert np.max(np.abs(v32[kk] - v64[kk])) / np.max(np.abs(v64[kk])) < 1e-5


# ------------------------------------------------------------------- steps


def test_decode_step_stream_isolation_and_batch():
    w = synth.workload("small_fp32_b2")
    W, k, v, lens, x, t = _inputs(w)
    new, out = oracle.decode_step(x, t, k, v, lens, W, w, noise_seed=11, step=4)
    x2 = x.copy()
    x2[1] = synth.perturbed(x[1], 3, "iso")
    new2, out2 = oracle.decode_step(x2, t, k, v, lens, W, w, noise_seed=11, step=4)
    assert np.array_equal(new[0], new2[0]) and np.array_equal(out[0], out2[0])
    assert not np.array_equal(out[1], out2[1])
    # The tail of stream b is its own Philox draw (seed noise_seed + b).
    for b in range(w.batch):
        assert np.array_equal(new[b, -1], oracle.gaussian_chunk(11 + b, 4, w.chunk_len,
                                                                 w.action_dim))


def test_sequential_decode_constant_velocity():
    # v == c: ten Euler steps with sum(dt) = t_0 - t_n = 1 give noise - c.
    w = synth.workload("tiny_fp32").replace(n_chunks=1)
    W, k, v, lens, _, _ = _inputs(w)
    c = np.linspace(-1, 1, w.action_dim).astype(np.float32)
    W["w_out"] = np.zeros_like(W["w_out"])
    W["b_out"] = c
    noise = synth.make_buffer(w.replace(n_chunks=1), 3)[:, 0]
    out = oracle.sequential_decode(noise, 10, k, v, lens, W, w)
    np.testing.assert_allclose(out, noise - c, atol=1e-6)
    tj = oracle.sequential_levels(10)
    assert tj[0] == 1.0 and tj[-1] == 0.0 and np.all(np.diff(tj) < 0)


def test_time_mlp_with_diagonal_weights_is_elementwise():
    # With diagonal W_t1 = diag(a), W_t2 = diag(c) the time-MLP acts per
    # element: cond_i = s(c_i s(a_i e_i + b1_i) + b2_i), s(x) = x expit(x).
    W = 16
    rng = np.random.default_rng(12)
    a, c = rng.uniform(0.5, 2.0, W), rng.uniform(-2.0, 2.0, W)
    b1, b2 = rng.standard_normal(W), rng.standard_normal(W)
    w = {"w_t1": np.diag(a), "b_t1": b1, "w_t2": np.diag(c), "b_t2": b2}
    s = lambda x: x * special.expit(x)
    for t in (0.0, 0.3, 1.0):
        e = oracle.timestep_embedding(t, W)
        np.testing.assert_allclose(oracle.time_condition(t, w, W), s(c * s(a * e + b1) + b2),
                                   rtol=1e-13, atol=1e-15)
