"""CPU oracle for FlashVLA's streaming action-decode step (test infrastructure).

This file is test infrastructure, not product code.  Only the test suite, the
smoke check and the CPU-baseline leg of the benchmark import it; the HIP
library never calls it, and it shares no code, tables or constants with the
HIP library.

It is a plain, slow, step-by-step numpy implementation of what one decode
step computes, in fp64 by default (``dtype=np.float32`` gives the fp32 mode
used as a precision cross-check and as a CPU timing baseline).  It follows,
in the paper's order:

* Sec. 3.1, Eq. 1 -- the flow-matching interpolant x_tau = (1-tau) a + tau z,
  with velocity dx/dtau = z - a; tau = 1 is pure noise, tau = 0 a clean
  action, so an Euler step towards clean actions is x <- x - dt * v.
* Sec. 3.1, Eq. 2 -- the buffer of N chunks at a monotone staircase of noise
  levels tau_1 < ... < tau_N; slot position = denoising progress = execution
  order.
* Sec. 3.1 (chunk-wise causal mask) -- a noisier (later) chunk attends to the
  cleaner (earlier) chunks; never the reverse; granularity is the chunk.
* Appendix "Model architecture" -- FiLM: scale, shift and gate generated
  from the timestep embedding (via a time-MLP) condition every norm of the
  action expert, per chunk.
* Sec. 3.2 and Algorithm 1 (steady streaming) -- one pass advances every
  chunk; the cleanest chunk is popped and executed; the rest shift forward;
  a fresh N(0, I) chunk is pushed at the tail.

Where the paper is silent the oracle takes these readings (each is listed,
with its reason, in the design notes of the repository):

* R1 inference noise levels are caller inputs (the workloads use
  t_k = (k+1)/K); R2 dt_k = t_k - t_{k-1} with t_{-1} = 0, in fp32;
* R3 inside a chunk attention is bidirectional; a chunk sees itself, all
  earlier chunks and every valid prefix token; the prefix never sees actions;
* R4 FiLM is an adaptive RMSNorm per norm instance, u = rmsnorm(h)(1+s)+b,
  with a gated residual h += g * block(u); each norm n (2 per layer plus the
  final one) has its own linear map cond -> [s | b | g]; the final gate is
  unused;
* R5 the timestep embedding is [sin(2 pi t/p_i), cos(2 pi t/p_i)] with
  geometric periods p_i from 4e-3 to 4, followed by a 2-layer SiLU time-MLP,
  cond = silu(silu(e W1 + b1) W2 + b2);
* R6 RMSNorm eps = 1e-6 with no separate learned scale;
* R7 the MLP is GeGLU with the tanh GELU (or a plain tanh-GELU MLP);
* R8 RoPE with theta = 1e4 and half-split pairs (i, i + dh/2) on action
  queries and keys at positions P_b + k*C + c; prefix keys arrive rotated;
* R9 softmax scale 1/sqrt(dh);
* R10 fresh noise is Philox4x32-10 (Salmon et al., SC'11) keyed by
  seed_b = noise_seed + b with counter (j, lo32(s), hi32(s), 0) for the j-th
  group of 4 values of the row-major [C][A] chunk, mapped to (0,1) as
  (r + 0.5) 2^-32 and to N(0,1) by Box-Muller in fp64, then rounded to fp32.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

# ---------------------------------------------------------------------------
# Elementary functions
# ---------------------------------------------------------------------------


def silu(x: np.ndarray) -> np.ndarray:
    """x * sigmoid(x)."""
    return x / (1.0 + np.exp(-x))


def gelu_tanh(x: np.ndarray) -> np.ndarray:
    """Tanh-approximate GELU, 0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))."""
    c = math.sqrt(2.0 / math.pi)
    return 0.5 * x * (1.0 + np.tanh(c * (x + 0.044715 * x * x * x)))


def rmsnorm(h: np.ndarray, eps: float) -> np.ndarray:
    """h / sqrt(mean(h^2) + eps) over the last axis (reading R6)."""
    return h / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + eps)


def _as(a, dtype) -> np.ndarray:
    """``a`` as an array of ``dtype`` (no copy when it already is one)."""
    return np.asarray(a, dtype=dtype)


def softmax_rows(s: np.ndarray) -> np.ndarray:
    """Row softmax over the last axis."""
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


# ---------------------------------------------------------------------------
# Time conditioning (Appendix "Model architecture"; readings R4, R5)
# ---------------------------------------------------------------------------


def timestep_embedding(t: float, width: int, dtype=np.float64,
                       min_period: float = 4e-3, max_period: float = 4.0) -> np.ndarray:
    """Sinusoidal embedding of one noise level: [sin(2 pi t/p_i) | cos(2 pi t/p_i)].

    p_i = min_period * (max_period/min_period)^(i/(W/2-1)), i < W/2.
    """
    half = width // 2
    frac = np.arange(half, dtype=np.float64) / (half - 1)
    period = min_period * (max_period / min_period) ** frac
    ang = 2.0 * np.pi * np.float64(t) / period
    return np.concatenate([np.sin(ang), np.cos(ang)]).astype(dtype)


def time_condition(t: float, w: Dict, width: int, dtype=np.float64) -> np.ndarray:
    """cond = silu(silu(e W_t1 + b_t1) W_t2 + b_t2) for one chunk's noise level."""
    e = timestep_embedding(t, width, dtype)
    hid = silu(e @ _as(w["w_t1"], dtype) + _as(w["b_t1"], dtype))
    return silu(hid @ _as(w["w_t2"], dtype) + _as(w["b_t2"], dtype))


def film(cond: np.ndarray, w_mod: np.ndarray, b_mod: np.ndarray,
         dtype=np.float64) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """One norm's FiLM parameters: [scale | shift | gate] = cond M_n + m_n."""
    W = cond.shape[-1]
    y = cond @ _as(w_mod, dtype) + _as(b_mod, dtype)
    return y[:W], y[W:2 * W], y[2 * W:3 * W]


def adaptive_rmsnorm(h: np.ndarray, scale: np.ndarray, shift: np.ndarray,
                     eps: float) -> np.ndarray:
    """FiLM-conditioned RMSNorm: rmsnorm(h) * (1 + scale) + shift (reading R4)."""
    return rmsnorm(h, eps) * (1.0 + scale) + shift


# ---------------------------------------------------------------------------
# Rotary position embedding (reading R8)
# ---------------------------------------------------------------------------


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate x [..., n, dh] at integer positions pos [n] with half-split pairs.

    Pair (i, i + dh/2) is rotated by the angle pos * theta^(-2i/dh).
    """
    dh = x.shape[-1]
    half = dh // 2
    inv = theta ** (-np.arange(half, dtype=np.float64) * 2.0 / dh)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]      # [n, half]
    shape = (1,) * (x.ndim - 2) + ang.shape
    c = np.cos(ang).reshape(shape).astype(x.dtype)
    s = np.sin(ang).reshape(shape).astype(x.dtype)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def rope_tokens(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """rope() for a [T, H, dh] token-major tensor."""
    return np.swapaxes(rope(np.swapaxes(x, 0, 1), pos, theta), 0, 1)


# ---------------------------------------------------------------------------
# Chunk-wise causal attention over [prefix ; buffer] (Sec. 3.1; readings R3, R9)
# ---------------------------------------------------------------------------


MASK_MODES = ("causal", "isolated", "bidirectional")


def visible_chunks(chunk: int, n_chunks: int, first_valid: int = 0,
                   mode: str = "causal") -> Tuple[int, int]:
    """Buffer chunks [lo, hi) that the queries of ``chunk`` attend to.

    * "causal" (Sec. 3.1): the chunk itself and every cleaner (earlier) valid
      chunk, never a noisier one;
    * "isolated" (the no-causal ablation of Appendix "Ablations"): no chunk
      attends to another chunk, only to itself;
    * "bidirectional": every valid chunk.
    Slots before ``first_valid`` hold cold-start padding (Algorithm 1): they are
    never keys of a valid chunk; a padding chunk's own queries see only
    itself (their outputs are never used).  Every query also sees all valid
    prefix tokens (reading R3).
    """
    if mode not in MASK_MODES:
        raise ValueError(mode)
    if chunk < first_valid or mode == "isolated":
        return chunk, chunk + 1
    if mode == "causal":
        return first_valid, chunk + 1
    return first_valid, n_chunks


def chunk_causal_attention(q: np.ndarray, k_buf: np.ndarray, v_buf: np.ndarray,
                           k_pre: np.ndarray, v_pre: np.ndarray, chunk_len: int,
                           return_probs: bool = False, mode: str = "causal",
                           first_valid: int = 0):
    """Attention of one stream's action queries.

    q [T, Hq, dh]; k_buf, v_buf [T, Hkv, dh]; k_pre, v_pre [P, Hkv, dh] (the
    valid prefix only).  Query head h reads kv head h // (Hq/Hkv).  The buffer
    keys a chunk sees follow ``visible_chunks(mode, first_valid)``.  Returns o
    [T, Hq, dh] and, if asked, the probabilities [Hq, T, P + T] with exact
    zeros on invisible keys.
    """
    T, Hq, dh = q.shape
    Hkv = k_buf.shape[1]
    P = k_pre.shape[0]
    K = T // chunk_len
    group = Hq // Hkv
    o = np.zeros_like(q)
    probs = np.zeros((Hq, T, P + T), dtype=q.dtype) if return_probs else None
    scale = 1.0 / math.sqrt(dh)
    for k in range(K):
        rows = slice(k * chunk_len, (k + 1) * chunk_len)
        lo, hi = visible_chunks(k, K, first_valid, mode)
        buf = slice(lo * chunk_len, hi * chunk_len)
        for h in range(Hq):
            g = h // group
            keys = np.concatenate([k_pre[:, g], k_buf[buf, g]], axis=0)
            vals = np.concatenate([v_pre[:, g], v_buf[buf, g]], axis=0)
            p = softmax_rows((q[rows, h] @ keys.T) * scale)
            o[rows, h] = p @ vals
            if return_probs:
                probs[h, rows, :P] = p[:, :P]
                probs[h, rows, P + lo * chunk_len:P + hi * chunk_len] = p[:, P:]
    return (o, probs) if return_probs else o


# ---------------------------------------------------------------------------
# One forward of the action expert (the velocity v_theta of Eq. 1)
# ---------------------------------------------------------------------------


def _chunk_broadcast(per_chunk: np.ndarray, chunk_len: int) -> np.ndarray:
    """[K, W] per-chunk rows -> [K*C, W] per-token rows."""
    return np.repeat(per_chunk, chunk_len, axis=0)


def velocity(x: np.ndarray, t: np.ndarray, prefix_k: np.ndarray, prefix_v: np.ndarray,
             prefix_len: int, w: Dict, cfg, dtype=np.float64,
             trace: Optional[Dict] = None, mask: str = "causal",
             first_valid: int = 0) -> np.ndarray:
    """Velocity v_theta of every chunk in one stream's buffer.

    x [K, C, A] buffer; t [K] per-chunk noise levels; prefix_k, prefix_v
    [L, P_max, Hkv, dh] this stream's cached observation K/V (rows < prefix_len
    valid).  ``cfg`` supplies n_layers, width, n_q_heads, n_kv_heads,
    head_dim, mlp_dim, action_dim, rms_eps, rope_theta, mlp_gated.  ``mask``
    and ``first_valid`` select the attention mask and the first non-padding
    slot (see ``visible_chunks``).  Returns v [K, C, A] in ``dtype``.
    ``trace``, if given, receives intermediate values.
    """
    K, C, A = x.shape
    L, W = cfg.n_layers, cfg.width
    Hq, Hkv, dh = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    eps = cfg.rms_eps
    T = K * C
    f = lambda a: _as(a, dtype)

    # Time conditioning: one condition vector per chunk, and per norm the
    # FiLM [scale | shift | gate] triple of every chunk.
    cond = np.stack([time_condition(float(t[k]), w, W, dtype) for k in range(K)])
    mods = []
    for n in range(2 * L + 1):
        trip = [film(cond[k], w["w_mod"][n], w["b_mod"][n], dtype) for k in range(K)]
        mods.append(tuple(_chunk_broadcast(np.stack([tr[j] for tr in trip]), C)
                          for j in range(3)))
    if trace is not None:
        trace["cond"] = cond
        trace["mods"] = mods

    # Embed action tokens.
    h = f(x).reshape(T, A) @ f(w["w_in"]) + f(w["b_in"])
    pos = int(prefix_len) + np.arange(T)

    for l in range(L):
        s1, b1, g1 = mods[2 * l]
        u = adaptive_rmsnorm(h, s1, b1, eps)
        q = (u @ f(w["wq"][l])).reshape(T, Hq, dh)
        kk = (u @ f(w["wk"][l])).reshape(T, Hkv, dh)
        vv = (u @ f(w["wv"][l])).reshape(T, Hkv, dh)
        q = rope_tokens(q, pos, cfg.rope_theta)
        kk = rope_tokens(kk, pos, cfg.rope_theta)
        o = chunk_causal_attention(q, kk, vv, f(prefix_k[l, :prefix_len]),
                                   f(prefix_v[l, :prefix_len]), C, mode=mask,
                                   first_valid=first_valid)
        h = h + g1 * (o.reshape(T, Hq * dh) @ f(w["wo"][l]))

        s2, b2, g2 = mods[2 * l + 1]
        u2 = adaptive_rmsnorm(h, s2, b2, eps)
        if cfg.mlp_gated:
            m = gelu_tanh(u2 @ f(w["wg"][l])) * (u2 @ f(w["wu"][l]))
        else:
            m = gelu_tanh(u2 @ f(w["wu"][l]))
        h = h + g2 * (m @ f(w["wd"][l]))
        if trace is not None:
            trace.setdefault("h", []).append(h.copy())

    sf, bf, _unused_gate = mods[2 * L]
    uf = adaptive_rmsnorm(h, sf, bf, eps)
    v = uf @ f(w["w_out"]) + f(w["b_out"])
    return v.reshape(K, C, A)


# ---------------------------------------------------------------------------
# Euler update, emission and shift (Eq. 1; Sec. 3.2 and Algorithm 1)
# ---------------------------------------------------------------------------


def euler_steps(t: np.ndarray) -> np.ndarray:
    """dt_k = t_k - t_{k-1} with t_{-1} = 0, evaluated in fp32 (reading R2)."""
    t = np.asarray(t, dtype=np.float32)
    prev = np.concatenate([np.zeros(1, np.float32), t[:-1]])
    return (t - prev).astype(np.float32)


def euler_emit_shift(x: np.ndarray, t: np.ndarray, v: np.ndarray, tail: np.ndarray,
                     arith=np.float64) -> Tuple[np.ndarray, np.ndarray]:
    """One steady-streaming queue update of one stream.

    Every chunk takes x'_k = x_k - dt_k v_k; the cleanest chunk x'_0 is popped
    (emitted), the others move one slot forward and ``tail`` (fresh noise)
    is pushed into the last slot.  With ``arith=np.float32`` the update is
    done as the fp32 sequence p = fl(dt*v), x' = fl(x - p) (no fused
    multiply-add).  Returns (new buffer [K,C,A] fp32, out chunk [C,A] fp32).
    """
    dt = euler_steps(t)[:, None, None]
    if arith == np.float32:
        p = (dt.astype(np.float32) * np.asarray(v, np.float32)).astype(np.float32)
        xn = (np.asarray(x, np.float32) - p).astype(np.float32)
    else:
        xn = (np.asarray(x, np.float64) - dt.astype(np.float64) * np.asarray(v, np.float64))
        xn = xn.astype(np.float32)
    out = xn[0].copy()
    new = np.empty_like(xn)
    new[:-1] = xn[1:]
    new[-1] = tail
    return new, out


# ---------------------------------------------------------------------------
# Fresh Gaussian noise: Philox4x32-10 + Box-Muller (reading R10)
# ---------------------------------------------------------------------------

_PHILOX_M0 = np.uint64(0xD2511F53)
_PHILOX_M1 = np.uint64(0xCD9E8D57)
_PHILOX_W0 = np.uint64(0x9E3779B9)
_PHILOX_W1 = np.uint64(0xBB67AE85)
_MASK32 = np.uint64(0xFFFFFFFF)


def philox4x32_10(counter: np.ndarray, key: np.ndarray) -> np.ndarray:
    """Philox4x32 with 10 rounds (Salmon, Moraes, Dror, Shaw, SC'11).

    counter [..., 4] and key [..., 2] as unsigned 32-bit words; returns
    [..., 4] uint32.  Each round multiplies words 0 and 2 by the Philox
    multipliers, forms (hi1^c1^k0, lo1, hi0^c3^k1, lo0), and between rounds
    the key is bumped by the Weyl constants.
    """
    c = np.asarray(counter, dtype=np.uint64) & _MASK32
    k = np.asarray(key, dtype=np.uint64) & _MASK32
    c0, c1, c2, c3 = (c[..., i].copy() for i in range(4))
    k0, k1 = k[..., 0].copy(), k[..., 1].copy()
    for rnd in range(10):
        if rnd > 0:
            k0 = (k0 + _PHILOX_W0) & _MASK32
            k1 = (k1 + _PHILOX_W1) & _MASK32
        p0 = _PHILOX_M0 * c0          # < 2^64, exact in uint64
        p1 = _PHILOX_M1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & _MASK32
        hi1, lo1 = p1 >> np.uint64(32), p1 & _MASK32
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return np.stack([c0, c1, c2, c3], axis=-1).astype(np.uint32)


def noise_words(seed: int, step: int, n_values: int) -> np.ndarray:
    """Raw Philox words for one chunk: uint32 [ceil(n/4)*4]."""
    groups = (n_values + 3) // 4
    j = np.arange(groups, dtype=np.uint64)
    s = np.uint64(step)
    ctr = np.stack([j, np.full_like(j, s & _MASK32), np.full_like(j, s >> np.uint64(32)),
                    np.zeros_like(j)], axis=-1)
    sd = np.uint64(seed)
    key = np.array([sd & _MASK32, sd >> np.uint64(32)], dtype=np.uint64)
    return philox4x32_10(ctr, np.broadcast_to(key, (groups, 2))).reshape(-1)


def box_muller(r: np.ndarray) -> np.ndarray:
    """uint32 words (even count) -> standard normals (fp64), pairwise.

    u = (r + 0.5) 2^-32 in (0, 1); (u0, u1) -> (rad cos(2 pi u1), rad sin(2 pi u1))
    with rad = sqrt(-2 ln u0).
    """
    u = (r.astype(np.float64) + 0.5) * 2.0 ** -32
    u0, u1 = u[0::2], u[1::2]
    rad = np.sqrt(-2.0 * np.log(u0))
    out = np.empty_like(u)
    out[0::2] = rad * np.cos(2.0 * np.pi * u1)
    out[1::2] = rad * np.sin(2.0 * np.pi * u1)
    return out


def gaussian_chunk(seed: int, step: int, chunk_len: int, action_dim: int) -> np.ndarray:
    """Fresh N(0, I) chunk [C, A] fp32 for one stream at one step (reading R10)."""
    n = chunk_len * action_dim
    z = box_muller(noise_words(seed, step, n))[:n]
    return z.astype(np.float32).reshape(chunk_len, action_dim)


# ---------------------------------------------------------------------------
# Whole steps
# ---------------------------------------------------------------------------


def decode_step(buffer: np.ndarray, t: np.ndarray, prefix_k: np.ndarray, prefix_v: np.ndarray,
                prefix_len: Sequence[int], w: Dict, cfg, noise_seed: int, step: int,
                dtype=np.float64, v_out: Optional[List] = None, n_valid=None,
                mask: str = "causal"):
    """One streaming step for a batch of independent streams (Algorithm 1).

    buffer [B, K, C, A] fp32; t [B, K] (or [K]) fp32; prefix_k/v
    [L, B, P_max, Hkv, dh]; prefix_len [B].  Stream b draws its tail from
    seed noise_seed + b at counter ``step``.  ``n_valid`` [B] counts the
    non-padding slots of each stream (the last n_valid slots; default K, the
    steady state).  A stream whose buffer is full emits its cleanest chunk;
    during cold start (n_valid < K) the slot popped is padding, nothing is
    emitted (zeros: the caller executes its safe default action) and the
    stream gains one valid slot.  Returns (new buffer, out [B, C, A]) fp32,
    plus the new n_valid when ``n_valid`` was given.
    """
    B, K, C, A = buffer.shape
    t = np.broadcast_to(np.asarray(t, np.float32), (B, K))
    nv = np.full(B, K, np.int64) if n_valid is None else np.asarray(n_valid, np.int64)
    new = np.empty_like(buffer)
    out = np.empty((B, C, A), np.float32)
    for b in range(B):
        first = K - int(nv[b])
        v = velocity(buffer[b], t[b], prefix_k[:, b], prefix_v[:, b], int(prefix_len[b]),
                     w, cfg, dtype, mask=mask, first_valid=first)
        if v_out is not None:
            v_out.append(v)
        tail = gaussian_chunk(noise_seed + b, step, C, A)
        new[b], out[b] = euler_emit_shift(buffer[b], t[b], v, tail)
        if first > 0:
            out[b] = 0.0
    if n_valid is None:
        return new, out
    return new, out, np.minimum(nv + 1, K)


def cold_start(buffer: np.ndarray, streams: Sequence[int], noise_seed: int,
               step: int) -> np.ndarray:
    """Cold start of Algorithm 1 for the given streams: slots 0..K-2 become
    padding (zeros) and slot K-1 a fresh N(0, I) chunk drawn at counter
    ``step``; those streams then have one valid slot.  Returns the new
    buffer (other streams unchanged)."""
    new = np.array(buffer, dtype=np.float32, copy=True)
    K, C, A = new.shape[1:]
    for b in streams:
        new[b, :K - 1] = 0.0
        new[b, K - 1] = gaussian_chunk(noise_seed + b, step, C, A)
    return new


def multibuffer_velocity(buffers: np.ndarray, t: np.ndarray, prefix_k: np.ndarray,
                         prefix_v: np.ndarray, prefix_len: int, w: Dict, cfg,
                         dtype=np.float64, mask: str = "causal") -> np.ndarray:
    """Forward of the packed multi-buffer sample of Sec. 3.3 for one observation.

    buffers [N, N, C, A]: configuration j = 1..N is buffers[j-1], whose slots
    0..N-j-1 hold padding and slots N-j..N-1 the j real (noised) chunks; t
    [N] (or [N, N]) the slot noise levels; prefix_k/v [L, P_max, Hkv, dh] the
    one shared observation.  Every configuration attends to the same prefix
    and is isolated from the others, so the packed forward is the velocity of
    each configuration with its own padding.  Returns v [N, N, C, A]; entries
    of padding slots are the padding queries' outputs (never used).
    """
    N = buffers.shape[0]
    t = np.broadcast_to(np.asarray(t, np.float32), (N, N))
    return np.stack([velocity(buffers[j], t[j], prefix_k, prefix_v, prefix_len, w, cfg, dtype,
                              mask=mask, first_valid=N - 1 - j) for j in range(N)])


def sequential_levels(n_steps: int) -> np.ndarray:
    """Sequential decode schedule t_j = fl32((n - j)/n), j = 0..n (t_n = 0)."""
    return (np.arange(n_steps, -1, -1, dtype=np.float64) / n_steps).astype(np.float32)


def sequential_decode(noise: np.ndarray, n_steps: int, prefix_k: np.ndarray,
                      prefix_v: np.ndarray, prefix_len: Sequence[int], w: Dict, cfg,
                      dtype=np.float64) -> np.ndarray:
    """The isolated per-chunk decode of Sec. 3.1: n_steps Euler passes of one chunk.

    noise [B, C, A]: every pass conditions on the same observation, the chunk
    attends only to itself and the prefix, and x <- x - (t_j - t_{j+1}) v(x, t_j)
    for t_j = (n - j)/n.  Returns the final chunk [B, C, A] fp32.
    """
    B, C, A = noise.shape
    tj = sequential_levels(n_steps)
    dt = (tj[:-1] - tj[1:]).astype(np.float32)
    out = np.empty((B, C, A), np.float32)
    for b in range(B):
        x = noise[b].astype(dtype)[None]
        for j in range(n_steps):
            v = velocity(x, tj[j:j + 1], prefix_k[:, b], prefix_v[:, b], int(prefix_len[b]),
                         w, cfg, dtype)
            x = x - dtype(dt[j]) * v
        out[b] = x[0].astype(np.float32)
    return out
