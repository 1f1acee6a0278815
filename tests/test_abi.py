"""The C-ABI library loads and exports every entry point include/flashvla.h
declares; argument validation that happens before any device work is
checked here without a GPU."""
import ctypes
import os
import re
import subprocess

import pytest

import synth
from paper_2608_27384_amd import flashvla as fvb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    txt = open(os.path.join(ROOT, "include", "flashvla.h")).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(fv_[a-z_]+)\s*\(", txt)))


def test_header_declares_the_bound_entry_points():
    assert _declared() == sorted(fvb.EXPORTED)


def test_library_exports_every_declared_symbol():
    L = fvb.lib()
    for name in _declared():
        assert hasattr(L, name), name
    assert L.fv_abi_version() == 2


def test_status_strings():
    L = fvb.lib()
    assert L.fv_status_string(0) == b"ok"
    assert L.fv_status_string(1) == b"invalid argument"
    assert L.fv_status_string(4) == b"HIP runtime error"
    assert L.fv_last_error(None) == b""


def test_null_handle_and_null_arguments_are_rejected():
    L = fvb.lib()
    assert L.fv_decode_step(None, None, None, None, None) == fvb.FV_ERR_INVALID_ARG
    assert L.fv_velocity(None, None, None, None, None) == fvb.FV_ERR_INVALID_ARG
    assert L.fv_destroy(None) == fvb.FV_ERR_INVALID_ARG
    assert L.fv_set_noise_state(None, 0, 0) == fvb.FV_ERR_INVALID_ARG
    assert L.fv_query(None, fvb.FV_QUERY_ATTN_SPLITS, 1, None) == fvb.FV_ERR_INVALID_ARG
    assert L.fv_debug_stage(None, 0, 0, 1, None) == fvb.FV_ERR_INVALID_ARG
    assert L.fv_set_mask_mode(None, 0) == fvb.FV_ERR_INVALID_ARG
    assert L.fv_set_schedule(None, None, None) == fvb.FV_ERR_INVALID_ARG
    assert L.fv_cold_start(None, None, 0, 1, None) == fvb.FV_ERR_INVALID_ARG
    assert L.fv_get_valid_slots(None, None, 1) == fvb.FV_ERR_INVALID_ARG
    assert L.fv_set_valid_slots(None, None, 1) == fvb.FV_ERR_INVALID_ARG
    assert L.fv_set_prefix_async(None, None, None, None, 1, 0, None) == fvb.FV_ERR_INVALID_ARG
    assert L.fv_multibuffer_velocity(None, None, None, 0, 0, None, None, None,
                                     None) == fvb.FV_ERR_INVALID_ARG
    out = ctypes.c_void_p()
    assert L.fv_create(None, None, ctypes.byref(out)) == fvb.FV_ERR_INVALID_ARG
    assert out.value is None


@pytest.mark.parametrize("field,value", [
    ("n_kv_heads", 3), ("width", 96), ("head_dim", 48), ("head_dim", 512), ("mlp_dim", 100),
    ("action_dim", 65), ("n_chunks", 0), ("n_chunks", 257), ("max_batch", 0), ("dtype", 7),
    ("mlp_gated", 2),
])
def test_invalid_config_rejected_before_device_work(field, value):
    w = synth.workload("tiny_fp32")
    cfg = fvb.make_cfg(w, 1, 64)
    setattr(cfg, field, value)
    hw = fvb._HostWeights(synth.make_weights(w))
    out = ctypes.c_void_p()
    st = fvb.lib().fv_create(ctypes.byref(hw.s), ctypes.byref(cfg), ctypes.byref(out))
    assert st == fvb.FV_ERR_INVALID_ARG
    assert out.value is None


def test_header_is_plain_c99():
    """The public header compiles as C99 on its own, pedantic, no warnings."""
    r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror",
                        "-fsyntax-only", "-x", "c", os.path.join(ROOT, "include", "flashvla.h")],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_c_client_builds_and_links(tmp_path):
    """A plain C99 program that drives the library compiles with gcc and links
    against the built libflashvla.so (it runs in the GPU tests)."""
    from tests.c_client.build import build_client
    fvb.lib()  # the library is built
    out = str(tmp_path / "decode_client")
    build_client(out)
    assert os.path.exists(out)
