"""Host-side checks of the HIP library that need no GPU: it loads, exports
every symbol its headers declare, sizes workspaces, and rejects bad
arguments before touching the device."""
import ctypes
import os
import re

import pytest

from paper_2503_12450_amd import binding as B
from paper_2503_12450_amd.workload import WORKLOADS, MarDims

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for h in ("mar_cache.h", "mar_kernels.h", "mar_head.h"):
        text = open(os.path.join(ROOT, "include", h)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b(mar_[a-z_]+)\s*\(", text))
    return names


def test_library_exports_every_declared_symbol():
    lib = B.load()
    declared = _declared()
    assert declared == set(B.EXPORTED)
    for name in declared:
        assert getattr(lib, name) is not None


def test_workspace_bytes_for_every_workload():
    for key, w in WORKLOADS.items():
        n = B.workspace_bytes(w.dims)
        d = w.dims
        es = 2 if d.dtype == "bf16" else 4
        cache = (d.n_layers - d.full_prefix) * 2 * d.max_slots * d.seq_len * d.d_model * es
        assert n > cache, key
        assert n % 256 == 0


@pytest.mark.parametrize("bad", [
    dict(d_model=100), dict(n_heads=7), dict(d_mlp=100), dict(seq_len=0), dict(seq_len=5000),
    dict(max_slots=0), dict(full_prefix=4), dict(full_prefix=-1), dict(n_layers=0),
    dict(d_model=1152, n_heads=8),   # d_head 144 > 128
    dict(d_model=192, n_heads=16),   # d_head 12 not a multiple of 16
])
def test_workspace_rejects_unsupported_dims(bad):
    base = dict(n_layers=4, d_model=256, n_heads=4, d_mlp=1024, seq_len=64, max_slots=2,
                full_prefix=2, dtype="bf16")
    base.update(bad)
    with pytest.raises(B.MarError) as e:
        B.workspace_bytes(MarDims(**base))
    assert e.value.status == B.MAR_E_SHAPE


@pytest.mark.parametrize("slots,ok", [(256, True), (327, True), (328, False), (330, False)])
def test_workspace_rejects_dims_past_32_bit_offsets(slots, ok):
    """Every product addresses its operands and outputs with 32-bit byte
    offsets.  The sizing call refuses any dims for which one launch of a
    step would pass 2 GiB: fc1 on every row of a full step writes
    max_slots * seq_len * d_mlp values, counted at 4 bytes.  So no accepted
    dims can make a step fail after it has started enqueueing work."""
    from dataclasses import replace
    d = replace(WORKLOADS["mar-h"].dims, max_slots=slots)
    assert (d.max_slots * d.seq_len * max(3 * d.d_model, d.d_mlp) * 4 < 2 ** 31) == ok
    if ok:
        assert B.workspace_bytes(d) > 0
        return
    with pytest.raises(B.MarError) as e:
        B.workspace_bytes(d)
    assert e.value.status == B.MAR_E_SHAPE
    assert "2 GiB" in str(e.value)


def test_host_checks_run_before_any_device_call():
    lib = B.load()
    d = B.dims_c(WORKLOADS["block-f32"].dims)
    h = ctypes.c_void_p()
    assert lib.mar_cache_init(ctypes.byref(d), None, None, 0, None, ctypes.byref(h)) == B.MAR_E_ARG
    assert b"blocks" in lib.mar_last_error()
    assert lib.mar_step(None, None, None, 0, 1, 0, 0, None, None) == B.MAR_E_ARG
    assert lib.mar_cfg_combine(None, None, None, 0, 1, 0, 1.0, None, None, None) == B.MAR_E_ARG
    assert lib.mar_k_select(None, 1, 8, 2, None, None) == B.MAR_E_ARG
    assert lib.mar_k_attention(1, 16, 16, 16, 16, 1, 1, 8, 24, 8, None) == B.MAR_E_SHAPE
    assert lib.mar_cache_destroy(None) == B.MAR_OK
    assert lib.mar_output(None) is None


@pytest.mark.parametrize("field,value", [("score_source", 2), ("score_source", -1), ("fresh_kv", 2),
                                         ("fresh_kv", -1)])
def test_workspace_rejects_unknown_method_options(field, value):
    lib = B.load()
    d = B.dims_c(WORKLOADS["block-f32"].dims)
    setattr(d, field, value)
    assert lib.mar_workspace_bytes(ctypes.byref(d)) == 0
    assert field.encode() in lib.mar_last_error()


def test_feature_reference_is_sized_by_its_precision():
    """The feature score source keeps one reference row per token: the step
    input's storage type when no block is always computed, else the fp32
    residual stream; the value source needs no such buffer."""
    from dataclasses import replace
    for P, dtype, es in ((0, "bf16", 2), (2, "bf16", 4), (0, "f32", 4)):
        d = MarDims(4, 256, 4, 1024, 64, 3, P, dtype)
        extra = B.workspace_bytes(replace(d, score_source="features")) - B.workspace_bytes(d)
        need = d.max_slots * d.seq_len * d.d_model * es
        assert need <= extra < need + 1024, (P, dtype)
        assert B.workspace_bytes(replace(d, fresh_kv=True)) == B.workspace_bytes(d)


def test_headers_are_plain_c_and_host_entry_points_answer(tmp_path):
    """tests/abi_check.c is compiled as C99 against include/*.h only and
    linked to the library; it checks sizing, option validation and the
    argument checks that precede any device call."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    B.load()  # the library is built
    libdir = os.path.dirname(B.LIB_PATH)
    exe = str(tmp_path / "abi_check")
    build = subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic",
                            "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "abi_check.c"),
                            "-L", libdir, "-lmarcache", "-Wl,-rpath," + libdir, "-o", exe],
                           capture_output=True, text=True)
    assert build.returncode == 0, build.stderr
    run = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "abi check: ok" in run.stdout


def test_head_sizing_and_checks():
    """The diffusion head's sizing refuses unsupported shapes and checks its
    arguments on the host before any device call."""
    from dataclasses import replace
    from paper_2503_12450_amd.workload import HEADS
    lib = B.load()
    hd = replace(HEADS["mar-l"], max_rows=1024)
    n = B.head_workspace_bytes(hd)
    w, nm = hd.width, hd.n_mod
    assert n > 2 * hd.max_rows * nm * w * 2 + nm * w * w * 2
    assert n % 256 == 0
    for bad in (dict(width=100), dict(depth=0), dict(token_dim=0), dict(token_dim=65), dict(steps=0),
                dict(train_steps=50), dict(freq_dim=100), dict(dtype="f32"), dict(beta_end=1.0),
                dict(max_rows=0), dict(max_rows=16384)):
        with pytest.raises(B.MarError):
            B.head_workspace_bytes(replace(hd, **bad))
    d = B.head_dims_c(hd)
    h = ctypes.c_void_p(1)
    assert lib.mar_head_init(ctypes.byref(d), None, None, 0, None, ctypes.byref(h)) == B.MAR_E_ARG
    assert h.value is None
    assert lib.mar_head_sample(None, None, None, 1, None, None, 1, None, None, 1.0, None, None, None,
                               None) == B.MAR_E_ARG
    assert lib.mar_head_destroy(None) == B.MAR_OK
