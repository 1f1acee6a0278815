"""Seeded synthetic inputs for the streaming action-decode step.

This module draws the inputs that both the CPU oracle and the HIP path
consume: expert weights, the cached observation prefix K/V, the initial
action buffer and the per-slot noise levels.  It holds none of the method's
arithmetic; it only fixes shapes, value distributions and seeds.

Every named tensor gets its own generator,
``default_rng(SeedSequence([seed, crc32(name)]))``, so a tensor's values do
not depend on the order in which tensors are generated.  Draws are fp64
normals, scaled and cast to fp32.  In bf16 mode every weight and prefix
value is rounded to the nearest bf16 (ties to even) before it is handed out,
so the oracle (which upcasts to fp64) and the GPU library (which stores
bf16) see exactly the same numbers.

Workloads follow the paper's shapes: a pi0.5-style action expert (Sec. 4.1
setup; Appendix "Model architecture"), observation prefixes of 2 or 3 camera
views of 256 tokens plus 48 text tokens (the 2- and 3-view latency study,
Table 2), buffers of N chunks of C actions (Sec. 3.1, Eq. 2) and the
noise-level staircase of Eq. 2 read as t_k = (k+1)/K at inference.
"""
from __future__ import annotations

import dataclasses
import zlib
from typing import Dict, List, Optional, Tuple

import numpy as np

FP32 = "fp32"
BF16 = "bf16"


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape of one synthetic workload.

    ``prefix_len`` is either an int (every stream) or a (lo, hi) range from
    which per-stream lengths are drawn uniformly (inclusive).
    """

    name: str
    n_layers: int
    width: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    mlp_dim: int
    action_dim: int
    chunk_len: int
    n_chunks: int
    prefix_len: object
    batch: int
    dtype: str
    mlp_gated: bool = True
    rms_eps: float = 1e-6
    rope_theta: float = 10000.0
    weight_std: float = 0.02
    noise_seed: int = 0
    seq_steps: int = 0  # >0: sequential flow-matching decode with this many Euler steps

    @property
    def tokens(self) -> int:
        return self.n_chunks * self.chunk_len

    @property
    def max_prefix(self) -> int:
        if isinstance(self.prefix_len, tuple):
            return int(self.prefix_len[1])
        return int(self.prefix_len)

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


_PI05 = dict(n_layers=18, width=1024, n_q_heads=8, n_kv_heads=1, head_dim=256,
             mlp_dim=4096, action_dim=32)

WORKLOADS: Dict[str, Workload] = {
    # Tiny fp32 expert: 2 layers, width 128, 2q/1kv heads of 64, MLP 512, A=8,
    # 64 prefix tokens, K=4 chunks of 8 actions, 8 decode steps.
    "tiny_fp32": Workload("tiny_fp32", 2, 128, 2, 1, 64, 512, 8, 8, 4, 64, 1, FP32),
    # pi0.5-shaped expert, 2-view prefix (2x256 image + 48 text), K=10 x 50.
    "pi05_b1": Workload("pi05_b1", chunk_len=50, n_chunks=10, prefix_len=560,
                        batch=1, dtype=BF16, **_PI05),
    # Sequential baseline: one chunk of 50, 10 Euler steps, same expert/prefix.
    "seq_baseline": Workload("seq_baseline", chunk_len=50, n_chunks=1,
                             prefix_len=560, batch=1, dtype=BF16, seq_steps=10,
                             **_PI05),
    # Short chunks, 3-view prefix (3x256 + 48), K=5 x 10.
    "short_chunk": Workload("short_chunk", chunk_len=10, n_chunks=5,
                            prefix_len=816, batch=1, dtype=BF16, **_PI05),
    # 64 independent streams, ragged prefixes in [300, 816].
    "batched64": Workload("batched64", chunk_len=50, n_chunks=10,
                          prefix_len=(300, 816), batch=64, dtype=BF16, **_PI05),
    # Small bf16 shapes for parity tests: several tiles and ragged tails.
    "small_bf16": Workload("small_bf16", 2, 256, 4, 1, 64, 512, 32, 12, 4, 70, 1, BF16),
    "small_bf16_b3": Workload("small_bf16_b3", 2, 256, 4, 2, 128, 768, 32, 10, 3,
                              (0, 90), 3, BF16),
    "small_fp32_b2": Workload("small_fp32_b2", 2, 128, 4, 2, 64, 256, 8, 6, 5,
                              (3, 40), 2, FP32),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


def _rng(seed: int, name: str) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, zlib.crc32(name.encode())]))


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Nearest bf16 value (ties to even) of each fp32 element, returned as fp32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    bits = x.view(np.uint32).astype(np.uint64)
    bits = (bits + 0x7FFF + ((bits >> 16) & 1)) & 0xFFFF0000
    return bits.astype(np.uint32).view(np.float32).reshape(x.shape)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Upper 16 bits of bf16-representable fp32 values (the bf16 encoding)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)


def _normal(seed: int, name: str, shape, std: float, dtype: str) -> np.ndarray:
    a = (_rng(seed, name).standard_normal(size=shape) * std).astype(np.float32)
    return round_to_bf16(a) if dtype == BF16 else a


def make_weights(w: Workload, seed: int = 0) -> Dict[str, object]:
    """Expert weights, all ~N(0, weight_std), in the y = x @ W ([in, out]) layout.

    Keys: w_in [A,W], b_in [W], w_t1 [W,W], b_t1, w_t2 [W,W], b_t2,
    w_mod / b_mod: lists of 2L+1 arrays [W,3W] / [3W] (norm n = 2l before
    attention, 2l+1 before the MLP, 2L the final norm),
    wq/wk/wv/wo/wg/wu/wd: lists of L arrays, w_out [W,A], b_out [A].
    ``wg`` is None for the plain (ungated) GELU MLP.
    """
    W, A, L = w.width, w.action_dim, w.n_layers
    qd, kd = w.n_q_heads * w.head_dim, w.n_kv_heads * w.head_dim
    s, d = w.weight_std, w.dtype
    out: Dict[str, object] = {
        "w_in": _normal(seed, "w_in", (A, W), s, d),
        "b_in": _normal(seed, "b_in", (W,), s, d),
        "w_t1": _normal(seed, "w_t1", (W, W), s, d),
        "b_t1": _normal(seed, "b_t1", (W,), s, d),
        "w_t2": _normal(seed, "w_t2", (W, W), s, d),
        "b_t2": _normal(seed, "b_t2", (W,), s, d),
        "w_out": _normal(seed, "w_out", (W, A), s, d),
        "b_out": _normal(seed, "b_out", (A,), s, d),
        "w_mod": [_normal(seed, f"w_mod{n}", (W, 3 * W), s, d) for n in range(2 * L + 1)],
        "b_mod": [_normal(seed, f"b_mod{n}", (3 * W,), s, d) for n in range(2 * L + 1)],
        "wq": [_normal(seed, f"wq{l}", (W, qd), s, d) for l in range(L)],
        "wk": [_normal(seed, f"wk{l}", (W, kd), s, d) for l in range(L)],
        "wv": [_normal(seed, f"wv{l}", (W, kd), s, d) for l in range(L)],
        "wo": [_normal(seed, f"wo{l}", (qd, W), s, d) for l in range(L)],
        "wu": [_normal(seed, f"wu{l}", (W, w.mlp_dim), s, d) for l in range(L)],
        "wd": [_normal(seed, f"wd{l}", (w.mlp_dim, W), s, d) for l in range(L)],
        "wg": ([_normal(seed, f"wg{l}", (W, w.mlp_dim), s, d) for l in range(L)]
               if w.mlp_gated else None),
    }
    return out


def prefix_lengths(w: Workload, seed: int = 0) -> np.ndarray:
    """Valid prefix length per stream (int32 [B])."""
    if isinstance(w.prefix_len, tuple):
        lo, hi = w.prefix_len
        return _rng(seed, "plen").integers(lo, hi + 1, size=w.batch).astype(np.int32)
    return np.full((w.batch,), int(w.prefix_len), dtype=np.int32)


def make_prefix(w: Workload, seed: int = 0) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Cached observation K/V per expert layer, ~N(0,1).

    Returns (k, v, lengths) with k, v fp32 [L, B, P_max, Hkv, dh] (bf16
    representable in bf16 mode) and lengths int32 [B].  Keys are taken as
    already position-encoded by the observation encoder; slots at or beyond a
    stream's length are zero and never read.
    """
    lens = prefix_lengths(w, seed)
    shape = (w.n_layers, w.batch, w.max_prefix, w.n_kv_heads, w.head_dim)
    k = _normal(seed, "prefix_k", shape, 1.0, w.dtype)
    v = _normal(seed, "prefix_v", shape, 1.0, w.dtype)
    for b, n in enumerate(lens):
        k[:, b, n:] = 0.0
        v[:, b, n:] = 0.0
    return k, v, lens


def make_buffer(w: Workload, seed: int = 0, tag: str = "buffer") -> np.ndarray:
    """Initial action buffer, fp32 [B, K, C, A] ~N(0,1)."""
    shape = (w.batch, w.n_chunks, w.chunk_len, w.action_dim)
    return _rng(seed, tag).standard_normal(size=shape).astype(np.float32)


def noise_levels(w: Workload) -> np.ndarray:
    """Per-slot noise levels t_k = (k+1)/K in fp32 ([K])."""
    K = w.n_chunks
    return (np.arange(1, K + 1, dtype=np.float64) / K).astype(np.float32)


def noise_levels_batched(w: Workload) -> np.ndarray:
    """The same staircase for every stream, fp32 [B, K]."""
    return np.ascontiguousarray(np.broadcast_to(noise_levels(w), (w.batch, w.n_chunks)))


def perturbed(x: np.ndarray, seed: int, tag: str, scale: float = 1.0) -> np.ndarray:
    """x plus seeded N(0, scale^2) noise, fp32 (for invariant tests)."""
    return (x + _rng(seed, tag).standard_normal(size=x.shape) * scale).astype(np.float32)
