"""ctypes binding of libflashvla (the C ABI declared in include/flashvla.h).

Argument marshalling only: every step of the decode path runs in the HIP
library.  Device tensors are torch tensors (PyTorch provides device memory
and streams); the binding passes their data pointers and the current HIP
stream.  There is no fallback: if the library is missing the import of this
module's functions raises.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_float, c_int32, c_int64, c_uint64, c_void_p
from typing import Dict, Optional, Sequence

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libflashvla.so")

FV_OK, FV_ERR_INVALID_ARG, FV_ERR_STATE, FV_ERR_OOM, FV_ERR_HIP, FV_ERR_INTERNAL = range(6)
FV_BF16, FV_FP32 = 0, 1
FV_QUERY_ATTN_SPLITS, FV_QUERY_DEVICE_BYTES, FV_QUERY_NOALLOC_SCRATCH_BYTES = 1, 2, 3
FV_QUERY_OUT_PROJ_SPLITS = 4
FV_NOALLOC_SCRATCH_BYTES = 24 << 20
FV_MASK_CHUNK_CAUSAL, FV_MASK_ISOLATED, FV_MASK_BIDIRECTIONAL = 0, 1, 2
MASK_MODES = {"causal": FV_MASK_CHUNK_CAUSAL, "isolated": FV_MASK_ISOLATED,
              "bidirectional": FV_MASK_BIDIRECTIONAL}

EXPORTED = (
    "fv_create", "fv_set_prefix", "fv_decode_step", "fv_velocity", "fv_euler_shift",
    "fv_sequential_decode", "fv_get_noise_state", "fv_set_noise_state", "fv_set_graph_mode",
    "fv_destroy", "fv_status_string", "fv_last_error", "fv_abi_version", "fv_debug_forward",
    "fv_debug_stage", "fv_query", "fv_set_mask_mode", "fv_set_schedule", "fv_cold_start",
    "fv_get_valid_slots", "fv_set_valid_slots", "fv_multibuffer_velocity", "fv_set_prefix_async",
    "fv_decode_step_noalloc",
)


class FvCfg(ctypes.Structure):
    _fields_ = [(n, c_int32) for n in (
        "n_layers", "width", "n_q_heads", "n_kv_heads", "head_dim", "mlp_dim", "action_dim",
        "chunk_len", "n_chunks", "max_prefix", "max_batch", "dtype", "mlp_gated")] + [
        ("rms_eps", c_float), ("rope_theta", c_float), ("noise_seed", c_uint64)]


class FvWeights(ctypes.Structure):
    _fields_ = [(n, c_void_p) for n in ("w_in", "b_in", "w_t1", "b_t1", "w_t2", "b_t2")] + [
        (n, POINTER(c_void_p)) for n in ("w_mod", "b_mod", "wq", "wk", "wv", "wo", "wg", "wu",
                                         "wd")] + [("w_out", c_void_p), ("b_out", c_void_p)]


class FlashVLAError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{message} (status {status})")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    """Loads libflashvla.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"libflashvla.so not built at {LIB_PATH}; run "
                              "python -m paper_2608_27384_amd.build")
        L = ctypes.CDLL(LIB_PATH)
        H, S = c_void_p, c_int32
        sig = {
            "fv_create": ([POINTER(FvWeights), POINTER(FvCfg), POINTER(c_void_p)], S),
            "fv_set_prefix": ([H, c_void_p, c_void_p, POINTER(c_int32), c_int32, c_int32, c_void_p], S),
            "fv_decode_step": ([H, c_void_p, c_void_p, c_void_p, c_void_p], S),
            "fv_decode_step_noalloc": ([H, c_void_p, c_void_p, c_void_p, c_void_p], S),
            "fv_velocity": ([H, c_void_p, c_void_p, c_void_p, c_void_p], S),
            "fv_euler_shift": ([H, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p], S),
            "fv_sequential_decode": ([H, c_void_p, c_int32, c_void_p, c_void_p], S),
            "fv_get_noise_state": ([H, POINTER(c_uint64), POINTER(c_uint64)], S),
            "fv_set_noise_state": ([H, c_uint64, c_uint64], S),
            "fv_set_graph_mode": ([H, c_int32], S),
            "fv_destroy": ([H], S),
            "fv_status_string": ([S], c_char_p),
            "fv_last_error": ([H], c_char_p),
            "fv_abi_version": ([], c_int32),
            "fv_debug_forward": ([H, c_void_p, c_void_p, c_int32, c_void_p, c_void_p, c_void_p], S),
            "fv_debug_stage": ([H, c_int32, c_int32, c_int32, c_void_p], S),
            "fv_query": ([H, c_int32, c_int32, POINTER(c_int64)], S),
            "fv_set_mask_mode": ([H, c_int32], S),
            "fv_set_schedule": ([H, c_void_p, c_void_p], S),
            "fv_cold_start": ([H, c_void_p, c_int32, c_int32, c_void_p], S),
            "fv_get_valid_slots": ([H, POINTER(c_int32), c_int32], S),
            "fv_set_valid_slots": ([H, POINTER(c_int32), c_int32], S),
            "fv_set_prefix_async": ([H, c_void_p, c_void_p, POINTER(c_int32), c_int32, c_int32,
                                     c_void_p], S),
            "fv_multibuffer_velocity": ([H, c_void_p, c_void_p, c_int32, c_int32, c_void_p,
                                         c_void_p, c_void_p, c_void_p], S),
        }
        for name, (args, res) in sig.items():
            fn = getattr(L, name)
            fn.argtypes, fn.restype = args, res
        _lib = L
    return _lib


def _check(handle, status: int, what: str) -> None:
    if status != FV_OK:
        msg = lib().fv_last_error(handle) if handle else b""
        txt = lib().fv_status_string(status).decode()
        raise FlashVLAError(status, f"{what}: {txt}: {(msg or b'').decode()}")


def _ptr(x) -> Optional[int]:
    """Device pointer of a torch tensor (or None)."""
    if x is None:
        return None
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is not None:
        return int(getattr(stream, "cuda_stream", stream))
    import torch
    return int(torch.cuda.current_stream().cuda_stream)


def make_cfg(shape, max_batch: int, max_prefix: int, noise_seed: int = 0) -> FvCfg:
    """fv_cfg from a shape object (attributes named as in fv_cfg)."""
    return FvCfg(n_layers=shape.n_layers, width=shape.width, n_q_heads=shape.n_q_heads,
                 n_kv_heads=shape.n_kv_heads, head_dim=shape.head_dim, mlp_dim=shape.mlp_dim,
                 action_dim=shape.action_dim, chunk_len=shape.chunk_len,
                 n_chunks=shape.n_chunks, max_prefix=max_prefix, max_batch=max_batch,
                 dtype=FV_BF16 if shape.dtype == "bf16" else FV_FP32,
                 mlp_gated=1 if shape.mlp_gated else 0, rms_eps=shape.rms_eps,
                 rope_theta=shape.rope_theta, noise_seed=noise_seed)


class _HostWeights:
    """Keeps contiguous fp32 host arrays alive while fv_create copies them."""

    def __init__(self, w: Dict):
        self.keep = []
        self.s = FvWeights()

        def one(a):
            a = np.ascontiguousarray(a, dtype=np.float32)
            self.keep.append(a)
            return a.ctypes.data

        def many(lst):
            if lst is None:
                return None
            arr = (c_void_p * len(lst))(*[one(a) for a in lst])
            self.keep.append(arr)
            return ctypes.cast(arr, POINTER(c_void_p))

        for k in ("w_in", "b_in", "w_t1", "b_t1", "w_t2", "b_t2", "w_out", "b_out"):
            setattr(self.s, k, one(w[k]))
        for k in ("w_mod", "b_mod", "wq", "wk", "wv", "wo", "wg", "wu", "wd"):
            p = many(w.get(k))
            if p is not None:
                setattr(self.s, k, p)


# ------------------------------------------------------------- C-ABI names

def fv_create(weights: Dict, cfg: FvCfg) -> int:
    hw = _HostWeights(weights)
    h = c_void_p()
    st = lib().fv_create(ctypes.byref(hw.s), ctypes.byref(cfg), ctypes.byref(h))
    if st != FV_OK:
        raise FlashVLAError(st, "fv_create: " + lib().fv_status_string(st).decode())
    return h.value


def fv_set_prefix(h, k, v, lengths: Sequence[int], ld: int, stream=None) -> None:
    lens = (c_int32 * len(lengths))(*[int(x) for x in lengths])
    _check(h, lib().fv_set_prefix(h, _ptr(k), _ptr(v), lens, len(lengths), ld, _stream(stream)),
           "fv_set_prefix")


def fv_set_prefix_async(h, k, v, lengths: Sequence[int], ld: int, copy_stream) -> None:
    lens = (c_int32 * len(lengths))(*[int(x) for x in lengths])
    _check(h, lib().fv_set_prefix_async(h, _ptr(k), _ptr(v), lens, len(lengths), ld,
                                        _stream(copy_stream)), "fv_set_prefix_async")


def fv_decode_step(h, buffer, t, out_chunk, stream=None) -> None:
    _check(h, lib().fv_decode_step(h, _ptr(buffer), _ptr(t), _ptr(out_chunk), _stream(stream)),
           "fv_decode_step")


def fv_decode_step_noalloc(h, buffer, t, out_chunk, stream=None) -> None:
    _check(h, lib().fv_decode_step_noalloc(h, _ptr(buffer), _ptr(t), _ptr(out_chunk),
                                           _stream(stream)), "fv_decode_step_noalloc")


def fv_velocity(h, buffer, t, v_out, stream=None) -> None:
    _check(h, lib().fv_velocity(h, _ptr(buffer), _ptr(t), _ptr(v_out), _stream(stream)),
           "fv_velocity")


def fv_euler_shift(h, buffer, t, v, out_chunk, stream=None) -> None:
    _check(h, lib().fv_euler_shift(h, _ptr(buffer), _ptr(t), _ptr(v), _ptr(out_chunk),
                                   _stream(stream)), "fv_euler_shift")


def fv_sequential_decode(h, noise, n_steps: int, out_chunk, stream=None) -> None:
    _check(h, lib().fv_sequential_decode(h, _ptr(noise), n_steps, _ptr(out_chunk),
                                         _stream(stream)), "fv_sequential_decode")


def fv_get_noise_state(h):
    seed, step = c_uint64(), c_uint64()
    _check(h, lib().fv_get_noise_state(h, ctypes.byref(seed), ctypes.byref(step)),
           "fv_get_noise_state")
    return seed.value, step.value


def fv_set_noise_state(h, seed: int, step: int) -> None:
    _check(h, lib().fv_set_noise_state(h, seed, step), "fv_set_noise_state")


def fv_set_graph_mode(h, enabled: bool) -> None:
    _check(h, lib().fv_set_graph_mode(h, 1 if enabled else 0), "fv_set_graph_mode")


def fv_debug_forward(h, buffer, t, n_layers_run: int, h_out, mod_out=None, stream=None) -> None:
    _check(h, lib().fv_debug_forward(h, _ptr(buffer), _ptr(t), n_layers_run, _ptr(h_out),
                                     _ptr(mod_out), _stream(stream)), "fv_debug_forward")


def fv_set_mask_mode(h, mode: int) -> None:
    _check(h, lib().fv_set_mask_mode(h, mode), "fv_set_mask_mode")


def fv_set_schedule(h, t, stream=None) -> None:
    _check(h, lib().fv_set_schedule(h, _ptr(t), _stream(stream)), "fv_set_schedule")


def fv_cold_start(h, buffer, first_stream: int, n_streams: int, stream=None) -> None:
    _check(h, lib().fv_cold_start(h, _ptr(buffer), first_stream, n_streams, _stream(stream)),
           "fv_cold_start")


def fv_get_valid_slots(h, count: int):
    arr = (c_int32 * count)()
    _check(h, lib().fv_get_valid_slots(h, arr, count), "fv_get_valid_slots")
    return [int(x) for x in arr]


def fv_set_valid_slots(h, counts: Sequence[int]) -> None:
    arr = (c_int32 * len(counts))(*[int(c) for c in counts])
    _check(h, lib().fv_set_valid_slots(h, arr, len(counts)), "fv_set_valid_slots")


def fv_multibuffer_velocity(h, k, v, prefix_len: int, ld: int, buffers, t, v_out,
                            stream=None) -> None:
    _check(h, lib().fv_multibuffer_velocity(h, _ptr(k), _ptr(v), prefix_len, ld, _ptr(buffers),
                                            _ptr(t), _ptr(v_out), _stream(stream)),
           "fv_multibuffer_velocity")


def fv_query(h, what: int, batch: int = 1) -> int:
    val = c_int64(0)
    _check(h, lib().fv_query(h, what, batch, ctypes.byref(val)), "fv_query")
    return int(val.value)


def fv_debug_stage(h, stage: int, layer: int, reps: int, stream=None) -> None:
    _check(h, lib().fv_debug_stage(h, stage, layer, reps, _stream(stream)), "fv_debug_stage")


def fv_destroy(h) -> None:
    if h:
        lib().fv_destroy(h)


# ------------------------------------------------------------- convenience

class Expert:
    """One fv_handle: the action expert on one GPU plus its decode state."""

    def __init__(self, weights: Dict, shape, max_batch: int, max_prefix: int,
                 noise_seed: int = 0):
        self.shape = shape
        self.cfg = make_cfg(shape, max_batch, max_prefix, noise_seed)
        self.handle = fv_create(weights, self.cfg)
        self.batch = max_batch

    def set_prefix(self, k, v, lengths, stream=None):
        fv_set_prefix(self.handle, k, v, lengths, k.shape[2], stream)
        self.batch = len(lengths)

    def set_prefix_async(self, k, v, lengths, copy_stream):
        fv_set_prefix_async(self.handle, k, v, lengths, k.shape[2], copy_stream)

    def decode_step(self, buffer, t, out_chunk, stream=None):
        fv_decode_step(self.handle, buffer, t, out_chunk, stream)

    def decode_step_noalloc(self, buffer, t, out_chunk, stream=None):
        fv_decode_step_noalloc(self.handle, buffer, t, out_chunk, stream)

    def noalloc_scratch_bytes(self, batch=None) -> int:
        return fv_query(self.handle, FV_QUERY_NOALLOC_SCRATCH_BYTES,
                        self.batch if batch is None else batch)

    def velocity(self, buffer, t, v_out, stream=None):
        fv_velocity(self.handle, buffer, t, v_out, stream)

    def euler_shift(self, buffer, t, v, out_chunk, stream=None):
        fv_euler_shift(self.handle, buffer, t, v, out_chunk, stream)

    def sequential_decode(self, noise, n_steps, out_chunk, stream=None):
        fv_sequential_decode(self.handle, noise, n_steps, out_chunk, stream)

    @property
    def noise_state(self):
        return fv_get_noise_state(self.handle)

    def set_noise_state(self, seed: int, step: int):
        fv_set_noise_state(self.handle, seed, step)

    def set_graph_mode(self, enabled: bool):
        fv_set_graph_mode(self.handle, enabled)

    def debug_forward(self, buffer, t, n_layers_run, h_out, mod_out=None, stream=None):
        fv_debug_forward(self.handle, buffer, t, n_layers_run, h_out, mod_out, stream)

    def set_mask_mode(self, mode):
        fv_set_mask_mode(self.handle, MASK_MODES[mode] if isinstance(mode, str) else mode)

    def set_schedule(self, t, stream=None):
        fv_set_schedule(self.handle, t, stream)

    def cold_start(self, buffer, first_stream=0, n_streams=None, stream=None):
        n = self.batch - first_stream if n_streams is None else n_streams
        fv_cold_start(self.handle, buffer, first_stream, n, stream)

    def set_valid_slots(self, counts):
        fv_set_valid_slots(self.handle, counts)

    def multibuffer_velocity(self, k, v, prefix_len, buffers, t, v_out, stream=None):
        fv_multibuffer_velocity(self.handle, k, v, prefix_len, k.shape[1], buffers, t, v_out,
                                stream)
        self.batch = self.cfg.n_chunks

    def valid_slots(self, count=None):
        return fv_get_valid_slots(self.handle, self.batch if count is None else count)

    def attn_split(self, batch=None) -> int:
        return fv_query(self.handle, FV_QUERY_ATTN_SPLITS, self.batch if batch is None else batch)

    def out_proj_splits(self, batch=None) -> int:
        return fv_query(self.handle, FV_QUERY_OUT_PROJ_SPLITS,
                        self.batch if batch is None else batch)

    def device_bytes(self) -> int:
        return fv_query(self.handle, FV_QUERY_DEVICE_BYTES)

    def debug_stage(self, stage, layer, reps, stream=None):
        fv_debug_stage(self.handle, stage, layer, reps, stream)

    def close(self):
        if self.handle:
            fv_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
