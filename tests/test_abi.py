"""C-ABI contract checks that need no GPU: the library loads, exports every
symbol declared in include/termezo.h, and rejects bad arguments or a missing
device cleanly (no compute calls are made here)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "termezo.h")


def _declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(termezo_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_four_hot_path_calls():
    syms = _declared_symbols()
    for name in ("termezo_build_mask", "termezo_perturb", "termezo_bitlinear_forward",
                 "termezo_update"):
        assert name in syms


def test_library_exports_every_declared_symbol():
    from paper_2609_33548_amd import termezo
    lib = ctypes.CDLL(termezo.LIB_PATH)
    missing = [s for s in _declared_symbols() if not hasattr(lib, s)]
    assert not missing, missing


def test_create_validates_arguments_before_touching_a_device():
    from paper_2609_33548_amd import termezo as T
    out = ctypes.c_void_p()
    L = T.Layer
    # null layer table / non-positive count
    assert T.lib.termezo_create(None, 1, T.F32, None, ctypes.byref(out)) == T.ERR_INVALID_ARG
    arr = (L * 1)(L(16, 4, 32))
    assert T.lib.termezo_create(arr, 0, T.F32, None, ctypes.byref(out)) == T.ERR_INVALID_ARG
    # d_in not a multiple of 16
    arr = (L * 1)(L(4096, 4, 24))
    assert T.lib.termezo_create(arr, 1, T.F32, None, ctypes.byref(out)) == T.ERR_INVALID_ARG
    # misaligned latent pointer
    arr = (L * 1)(L(4096 + 4, 4, 32))
    assert T.lib.termezo_create(arr, 1, T.F32, None, ctypes.byref(out)) == T.ERR_INVALID_ARG
    # layer above 2^25 weights (fixed-point bound)
    arr = (L * 1)(L(4096, (1 << 25) // 32 + 1, 32))
    assert T.lib.termezo_create(arr, 1, T.F32, None, ctypes.byref(out)) == T.ERR_INVALID_ARG
    # unsupported latent dtype
    arr = (L * 1)(L(4096, 4, 32))
    assert T.lib.termezo_create(arr, 1, T.I8, None, ctypes.byref(out)) == T.ERR_INVALID_ARG
    assert out.value is None


def test_create_without_device_reports_device_error():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    from paper_2609_33548_amd import termezo as T
    out = ctypes.c_void_p()
    arr = (T.Layer * 1)(T.Layer(4096, 4, 32))
    assert T.lib.termezo_create(arr, 1, T.F32, None, ctypes.byref(out)) == T.ERR_DEVICE
    assert out.value is None


def test_null_context_calls_are_rejected():
    from paper_2609_33548_amd import termezo as T
    assert T.lib.termezo_perturb(None, 1, 1e-3, 1) == T.ERR_INVALID_ARG
    assert T.lib.termezo_update(None, 1.0, 1e-3, None) == T.ERR_INVALID_ARG
    assert T.lib.termezo_build_mask(None, 0.1, 1e-5, 0, None, None) == T.ERR_INVALID_ARG
    assert T.lib.termezo_bitlinear_forward(None, 0, None, 0, 1, None, 0, None, None, None) \
        == T.ERR_INVALID_ARG
    T.lib.termezo_destroy(None)


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one MI355X: --gpus above 1 exits with status 2 and says so,
    before importing torch or touching a device."""
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_bench_cpu_baseline_legs_are_combined_by_direction():
    """The two oracle legs (one thread, all host cores) are both reported with their
    thread counts; the headline value is the faster one (higher rate, or lower time for
    time-like units); nested results are left to the caller."""
    import bench
    calls = []

    def rate(value):
        calls.append(value)
        return {"value": value, "unit": "steps/s", "sample": "s", "_fwd": 1.0}

    out, st, mt = bench.two_legs(rate, {"value": 2.0}, {"value": 5.0})
    assert out["value"] == 5.0 and out["cores"] == bench.all_cores()
    assert out["single_thread"]["cores"] == 1 and out["all_cores"]["value"] == 5.0
    assert "_fwd" not in out and st["_fwd"] == 1.0
    t = bench.combine_legs({"value": 3.0, "unit": "us"}, {"value": 7.0, "unit": "us"}, 16)
    assert t["value"] == 3.0 and t["cores"] == 1 and t["all_cores"]["cores"] == 16
    nested, a, b = bench.two_legs(lambda: {"perturb": {"value": 1.0, "unit": "GB/s"}}, {}, {})
    assert nested is None and a["perturb"]["value"] == 1.0
