"""ctypes binding of libmarcache.so (argument marshalling only).

Every function here forwards to the C ABI declared in include/mar_cache.h,
include/mar_kernels.h and include/mar_head.h; every step of the computation runs in the HIP
library.  PyTorch supplies device memory and the current stream.  There is
no fallback: if the library is missing or fails to load, an ImportError /
OSError is raised.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmarcache.so")

MAR_OK, MAR_E_ARG, MAR_E_SHAPE, MAR_E_STATE, MAR_E_WORKSPACE, MAR_E_DEVICE, MAR_E_HOST = 0, -1, -2, -3, -4, -5, -6
MAR_F32, MAR_BF16 = 0, 1
MAR_FULL, MAR_TOKEN_CACHED, MAR_TOKEN_GIVEN, MAR_TOKEN_CACHED_MOST_SIMILAR = 0, 1, 2, 3
MAR_CFG_STORE, MAR_CFG_REUSE = 0, 1
MAR_SCORE_VALUES, MAR_SCORE_FEATURES = 0, 1
PROF_KINDS = ("qkv", "proj", "fc1", "fc2", "attention", "layernorm", "scores", "select", "cfg")

STATUS_NAMES = {0: "MAR_OK", -1: "MAR_E_ARG", -2: "MAR_E_SHAPE", -3: "MAR_E_STATE",
                -4: "MAR_E_WORKSPACE", -5: "MAR_E_DEVICE", -6: "MAR_E_HOST"}

# every symbol the headers declare (checked by the CPU tests)
EXPORTED = (
    "mar_workspace_bytes", "mar_cache_init", "mar_step", "mar_cfg_combine", "mar_output",
    "mar_cache_destroy", "mar_last_error", "mar_profile_start", "mar_profile_stop",
    "mar_k_layernorm", "mar_k_linear", "mar_k_linear_residual", "mar_k_qkv",
    "mar_k_attention", "mar_k_scores", "mar_k_select", "mar_k_select_most_similar",
    "mar_k_gemm_variant",
    "mar_head_workspace_bytes", "mar_head_init", "mar_head_sample", "mar_head_destroy",
    "mar_head_sample_noalloc",
)
GEMM_VARIANTS = 16


class MarError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class MarDimsC(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("d_mlp", ctypes.c_int32),
                ("seq_len", ctypes.c_int32), ("max_slots", ctypes.c_int32),
                ("full_prefix", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("ln_eps", ctypes.c_float), ("score_source", ctypes.c_int32),
                ("fresh_kv", ctypes.c_int32)]


WEIGHT_FIELDS = ("ln1_w", "ln1_b", "qkv_w", "qkv_b", "proj_w", "proj_b",
                 "ln2_w", "ln2_b", "fc1_w", "fc1_b", "fc2_w", "fc2_b")


class MarBlockWeightsC(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in WEIGHT_FIELDS]


class MarHeadDimsC(ctypes.Structure):
    _fields_ = [("width", ctypes.c_int32), ("depth", ctypes.c_int32), ("cond_dim", ctypes.c_int32),
                ("token_dim", ctypes.c_int32), ("steps", ctypes.c_int32), ("train_steps", ctypes.c_int32),
                ("freq_dim", ctypes.c_int32), ("max_rows", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("beta_start", ctypes.c_float), ("beta_end", ctypes.c_float), ("ln_eps", ctypes.c_float)]


HEAD_WEIGHT_FIELDS = ("z_w", "z_b", "t1_w", "t1_b", "t2_w", "t2_b", "in_w", "in_b", "ada_w", "ada_b",
                      "fc1_w", "fc1_b", "fc2_w", "fc2_b", "out_w", "out_b")


class MarHeadWeightsC(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in HEAD_WEIGHT_FIELDS]


_vp, _i32, _f32, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t
_SIGNATURES = {
    "mar_workspace_bytes": (_sz, [ctypes.POINTER(MarDimsC)]),
    "mar_cache_init": (_i32, [ctypes.POINTER(MarDimsC), ctypes.POINTER(MarBlockWeightsC), _vp, _sz, _vp,
                              ctypes.POINTER(_vp)]),
    "mar_step": (_i32, [_vp, _vp, _vp, _i32, _i32, _i32, _i32, _vp, _vp]),
    "mar_cfg_combine": (_i32, [_vp, _vp, _vp, _i32, _i32, _i32, _f32, _vp, _vp, _vp]),
    "mar_output": (_vp, [_vp]),
    "mar_cache_destroy": (_i32, [_vp]),
    "mar_last_error": (ctypes.c_char_p, []),
    "mar_profile_start": (_i32, [_vp, _i32]),
    "mar_profile_stop": (_i32, [_vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64),
                                ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]),
    "mar_k_layernorm": (_i32, [_i32, _vp, _i32, _vp, _i32, _i32, _i32, _i32, _vp, _vp, _f32, _vp, _vp, _vp]),
    "mar_k_linear": (_i32, [_i32, _i32, _vp, _vp, _vp, _i32, _i32, _i32, _vp, _vp]),
    "mar_k_linear_residual": (_i32, [_i32, _vp, _vp, _vp, _i32, _i32, _i32, _vp, _vp, _vp, _i32, _i32,
                                     _vp, _vp]),
    "mar_k_qkv": (_i32, [_i32, _vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp,
                         _vp, _vp, _vp]),
    "mar_k_attention": (_i32, [_i32, _vp, _vp, _vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp]),
    "mar_k_scores": (_i32, [_i32, _vp, _vp, _i32, _i32, _i32, _i32, _vp, _i32, _vp]),
    "mar_k_select": (_i32, [_vp, _i32, _i32, _i32, _vp, _vp]),
    "mar_k_select_most_similar": (_i32, [_vp, _i32, _i32, _i32, _vp, _vp]),
    "mar_k_gemm_variant": (_i32, [_i32]),
    "mar_head_workspace_bytes": (_sz, [ctypes.POINTER(MarHeadDimsC)]),
    "mar_head_init": (_i32, [ctypes.POINTER(MarHeadDimsC), ctypes.POINTER(MarHeadWeightsC), _vp, _sz, _vp,
                             ctypes.POINTER(_vp)]),
    "mar_head_sample": (_i32, [_vp, _vp, _vp, _i32, _vp, _vp, _i32, _vp, _vp, _f32, _vp, _vp, _vp, _vp]),
    "mar_head_destroy": (_i32, [_vp]),
    "mar_head_sample_noalloc": (_i32, [_vp, _vp, _vp, _i32, _vp, _vp, _i32, _vp, _vp, _f32, _vp, _vp, _vp,
                                       _vp]),
}

_lib: Optional[ctypes.CDLL] = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the HIP library (raises if it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built: run `python -m paper_2503_12450_amd.build`")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int) -> None:
    if status != MAR_OK:
        raise MarError(status, load().mar_last_error().decode())


def dtype_code(dtype: str) -> int:
    return {"f32": MAR_F32, "bf16": MAR_BF16}[dtype]


SCORE_SOURCES = {"values": MAR_SCORE_VALUES, "features": MAR_SCORE_FEATURES}


def dims_c(dims) -> MarDimsC:
    return MarDimsC(dims.n_layers, dims.d_model, dims.n_heads, dims.d_mlp, dims.seq_len,
                    dims.max_slots, dims.full_prefix, dtype_code(dims.dtype), dims.ln_eps,
                    SCORE_SOURCES[getattr(dims, "score_source", "values")],
                    1 if getattr(dims, "fresh_kv", False) else 0)


# --------------------------------------------------------------------------
# torch plumbing
# --------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream=None) -> int:
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def workspace_bytes(dims) -> int:
    d = dims_c(dims)
    n = load().mar_workspace_bytes(ctypes.byref(d))
    if n == 0:
        raise MarError(MAR_E_SHAPE, load().mar_last_error().decode())
    return n


class MarCache:
    """Handle over a workspace tensor; the library copies the weights in."""

    def __init__(self, dims, blocks: Sequence[Dict[str, "object"]], device="cuda", stream=None):
        torch = _torch()
        self.dims = dims
        self.lib = load()
        nbytes = workspace_bytes(dims)
        self.workspace = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
        off = (-self.workspace.data_ptr()) % 256
        self._ws = self.workspace[off:off + nbytes]
        arr = (MarBlockWeightsC * dims.n_layers)()
        for i, blk in enumerate(blocks):
            for f in WEIGHT_FIELDS:
                setattr(arr[i], f, blk[f].data_ptr())
        self._blocks = blocks  # kept alive until the copies are done
        handle = ctypes.c_void_p()
        d = dims_c(dims)
        _check(self.lib.mar_cache_init(ctypes.byref(d), arr, self._ws.data_ptr(), nbytes,
                                       _stream(stream), ctypes.byref(handle)))
        self.handle = handle

    def close(self) -> None:
        if getattr(self, "handle", None):
            self.lib.mar_cache_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def step(self, x, mode: int, n_recompute: int = 0, slot0: int = 0, y=None, sel_idx=None,
             stream=None) -> None:
        n_slots = x.shape[0]
        if mode == MAR_TOKEN_GIVEN and sel_idx is not None:
            import numpy as np
            host = np.ascontiguousarray(sel_idx, dtype=np.int32)
            self._given = host  # stays alive while the upload is in flight
            idx_ptr = host.ctypes.data
        else:
            idx_ptr = _ptr(sel_idx)
        _check(self.lib.mar_step(self.handle, x.data_ptr(), _ptr(y), slot0, n_slots, mode,
                                 n_recompute, idx_ptr, _stream(stream)))

    def cfg_combine(self, op: int, y_cond, y_uncond, scale: float, guided, uncond_out=None,
                    pair0: int = 0, stream=None) -> None:
        n_pairs = y_cond.shape[0]
        _check(self.lib.mar_cfg_combine(self.handle, y_cond.data_ptr(), _ptr(y_uncond), pair0, n_pairs,
                                        op, float(scale), guided.data_ptr(), _ptr(uncond_out),
                                        _stream(stream)))

    def profile_start(self, kind: str) -> None:
        _check(self.lib.mar_profile_start(self.handle, PROF_KINDS.index(kind)))

    def profile_stop(self):
        """(ms_total, launches, flops, bytes) of the launches timed since start."""
        ms, n = ctypes.c_double(), ctypes.c_int64()
        fl, by = ctypes.c_double(), ctypes.c_double()
        _check(self.lib.mar_profile_stop(self.handle, ctypes.byref(ms), ctypes.byref(n), ctypes.byref(fl),
                                         ctypes.byref(by)))
        return ms.value, n.value, fl.value, by.value

    def output(self):
        """The output cache [max_slots, S, D] fp32 as a view of the workspace."""
        torch = _torch()
        p = self.lib.mar_output(self.handle)
        off = p - self._ws.data_ptr()
        d = self.dims
        n = d.max_slots * d.seq_len * d.d_model
        return self._ws[off:off + 4 * n].view(torch.float32).view(d.max_slots, d.seq_len, d.d_model)


# --------------------------------------------------------------------------
# per-kernel entry points
# --------------------------------------------------------------------------

def k_layernorm(dtype: str, src, w, b, eps: float, out, idx=None, per_slot=None, seq=None,
                copy_f32=None, m=None, stream=None) -> None:
    torch = _torch()
    d = src.shape[-1]
    src_f32 = 1 if src.dtype == torch.float32 else 0
    if m is None:
        m = out.shape[0]
    if per_slot is None:
        per_slot = m if idx is None else idx.shape[-1]
    if seq is None:
        seq = per_slot
    _check(load().mar_k_layernorm(dtype_code(dtype), src.data_ptr(), src_f32, _ptr(idx), per_slot, seq, m, d,
                                  w.data_ptr(), b.data_ptr(), float(eps), _ptr(copy_f32), out.data_ptr(),
                                  _stream(stream)))


def k_linear(dtype: str, a, w, bias, out, gelu: bool = False, stream=None) -> None:
    m, k = a.shape
    n = w.shape[0]
    _check(load().mar_k_linear(dtype_code(dtype), 1 if gelu else 0, a.data_ptr(), w.data_ptr(),
                               bias.data_ptr(), m, n, k, out.data_ptr(), _stream(stream)))


def k_linear_residual(dtype: str, a, w, bias, resid, out, out_idx=None, per_slot=0, seq=0,
                      resid_copy=None, stream=None) -> None:
    m, k = a.shape
    n = w.shape[0]
    _check(load().mar_k_linear_residual(dtype_code(dtype), a.data_ptr(), w.data_ptr(), bias.data_ptr(), m,
                                        n, k, resid.data_ptr(), out.data_ptr(), _ptr(out_idx), per_slot,
                                        seq, _ptr(resid_copy), _stream(stream)))


def k_qkv(dtype: str, a, w, bias, d_model: int, n_heads: int, seq: int, per_slot: int,
          q_out=None, k_cache=None, v_cache=None, v_copy=None, idx=None, n_offset: int = 0,
          n_cols: Optional[int] = None, stream=None) -> None:
    m = a.shape[0]
    if n_cols is None:
        n_cols = w.shape[0]
    _check(load().mar_k_qkv(dtype_code(dtype), a.data_ptr(), w.data_ptr(), bias.data_ptr(), m, n_cols,
                            n_offset, d_model, n_heads, seq, per_slot, _ptr(idx), _ptr(q_out),
                            _ptr(k_cache), _ptr(v_cache), _ptr(v_copy), _stream(stream)))


def k_attention(dtype: str, q, k, v, out, n_slots: int, n_heads: int, seq: int, d_head: int,
                per_slot: int, stream=None) -> None:
    _check(load().mar_k_attention(dtype_code(dtype), q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                  out.data_ptr(), n_slots, n_heads, seq, d_head, per_slot, _stream(stream)))


def k_scores(dtype: str, v_cur, v_ref, scores, update_ref: bool = False, stream=None) -> None:
    n_slots, n_heads, seq, d_head = v_cur.shape
    _check(load().mar_k_scores(dtype_code(dtype), v_cur.data_ptr(), v_ref.data_ptr(), n_slots, n_heads,
                               seq, d_head, scores.data_ptr(), 1 if update_ref else 0, _stream(stream)))


def k_select(scores, n: int, idx, stream=None, most_similar: bool = False) -> None:
    n_slots, seq = scores.shape
    fn = load().mar_k_select_most_similar if most_similar else load().mar_k_select
    _check(fn(scores.data_ptr(), n_slots, seq, n, idx.data_ptr(), _stream(stream)))


def k_gemm_variant(variant: int) -> None:
    """Force a tile configuration of the matrix products (-1: by shape)."""
    _check(load().mar_k_gemm_variant(variant))


# --------------------------------------------------------------------------
# the diffusion head (include/mar_head.h)
# --------------------------------------------------------------------------

def head_dims_c(hd) -> MarHeadDimsC:
    return MarHeadDimsC(hd.width, hd.depth, hd.cond_dim, hd.token_dim, hd.steps, hd.train_steps, hd.freq_dim,
                        hd.max_rows, dtype_code(hd.dtype), hd.beta_start, hd.beta_end, hd.ln_eps)


def head_workspace_bytes(hd) -> int:
    d = head_dims_c(hd)
    n = load().mar_head_workspace_bytes(ctypes.byref(d))
    if n == 0:
        raise MarError(MAR_E_SHAPE, load().mar_last_error().decode())
    return n


class MarHead:
    """Handle over a workspace tensor; the library copies the head's weights
    in and computes its time embeddings."""

    def __init__(self, hd, weights: Dict[str, "object"], device="cuda", stream=None):
        torch = _torch()
        self.dims = hd
        self.lib = load()
        nbytes = head_workspace_bytes(hd)
        self.workspace = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
        off = (-self.workspace.data_ptr()) % 256
        self._ws = self.workspace[off:off + nbytes]
        w = MarHeadWeightsC(*[weights[f].data_ptr() for f in HEAD_WEIGHT_FIELDS])
        self._weights = weights
        handle = ctypes.c_void_p()
        d = head_dims_c(hd)
        _check(self.lib.mar_head_init(ctypes.byref(d), ctypes.byref(w), self._ws.data_ptr(), nbytes,
                                      _stream(stream), ctypes.byref(handle)))
        self.handle = handle

    def close(self) -> None:
        if getattr(self, "handle", None):
            self.lib.mar_head_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def sample(self, y_cond, y_uncond, row_cond, row_uncond, x_init, xi, scale: float, x_out,
               trajectory=None, eps_out=None, stream=None, noalloc: bool = False) -> None:
        """y_cond, y_uncond: [y_rows, cond_dim] fp32 (any leading shape
        flattened); row_*: int32 [rows]; x_init [rows, T]; xi [steps, rows, T].
        noalloc: the entry point whose scratch is the library's static array."""
        y_rows = y_cond.numel() // self.dims.cond_dim
        fn = self.lib.mar_head_sample_noalloc if noalloc else self.lib.mar_head_sample
        _check(fn(self.handle, y_cond.data_ptr(), y_uncond.data_ptr(), y_rows,
                                        row_cond.data_ptr(), row_uncond.data_ptr(), row_cond.shape[0],
                                        x_init.data_ptr(), xi.data_ptr(), float(scale), x_out.data_ptr(),
                                        _ptr(trajectory), _ptr(eps_out), _stream(stream)))
