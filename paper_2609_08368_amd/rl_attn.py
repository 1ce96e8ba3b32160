"""Thin ctypes binding over librlattn.so (argument marshalling only).

Every step of the attention runs in the HIP library; this module turns torch
tensors into the ABI's non-owning ``rl_tensor`` views and passes torch's
current stream. There is no fallback: if the library is missing or a call
fails, an exception is raised.
"""

from __future__ import annotations

import ctypes
import os
import re
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
# RL_ATTN_LIB selects another build of the library (A/B comparisons of builds)
LIB_PATH = os.environ.get("RL_ATTN_LIB", os.path.join(_PKG, "librlattn.so"))
INCLUDE = os.path.join(os.path.dirname(_PKG), "include")
HEADER = os.path.join(INCLUDE, "rl_attn.h")

RL_BF16, RL_F32, RL_I32, RL_FP8_E4M3 = 1, 2, 3, 4
RL_PREFIX_AUTO, RL_PREFIX_OFF = 0, 1
STATUS = {
    0: "RL_OK", -1: "RL_ERR_INVALID_ARG", -2: "RL_ERR_SHAPE", -3: "RL_ERR_DTYPE", -4: "RL_ERR_UNSUPPORTED",
    -5: "RL_ERR_WORKSPACE", -6: "RL_ERR_HIP", -7: "RL_ERR_DEVICE",
}
CODES = {v: k for k, v in STATUS.items()}


class RlTensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("shape", ctypes.c_int64 * 4), ("strides", ctypes.c_int64 * 4)]


class RlOpts(ctypes.Structure):
    _fields_ = [("split_tokens", ctypes.c_int32), ("prefix_share", ctypes.c_int32),
                ("validate", ctypes.c_int32), ("deterministic", ctypes.c_int32), ("reserved", ctypes.c_int32 * 4)]


class RlAttnError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"{STATUS.get(code, code)}: {message}")
        self.code = code
        self.status = STATUS.get(code, str(code))


_lib = None


def lib() -> ctypes.CDLL:
    """Load librlattn.so (built by ``python -m paper_2609_08368_amd.build``)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER(RlTensor)
        vp = ctypes.c_void_p
        L.rl_attn_decode.argtypes = [P, P, P, P, P, ctypes.c_float, P, vp]
        L.rl_attn_extend.argtypes = [P, P, P, P, P, P, ctypes.c_float, P, vp]
        L.rl_attn_decode_ex.argtypes = [P, P, P, P, P, ctypes.c_float, P, P, ctypes.POINTER(RlOpts), vp]
        L.rl_attn_extend_ex.argtypes = [P, P, P, P, P, P, ctypes.c_float, P, P, ctypes.POINTER(RlOpts), vp]
        L.rl_attn_decode_noalloc.argtypes = [P, P, P, P, P, ctypes.c_float, P, P, ctypes.POINTER(RlOpts), vp]
        L.rl_attn_decode_fp8.argtypes = [P, P, P, P, P, P, P, ctypes.c_float, P, P, ctypes.POINTER(RlOpts), vp]
        L.rl_attn_extend_fp8.argtypes = [P, P, P, P, P, P, P, P, ctypes.c_float, P, P, ctypes.POINTER(RlOpts), vp]
        L.rl_attn_append_kv.argtypes = [P, P, P, P, P, P, P, vp]
        L.rl_attn_append_kv_fp8.argtypes = [P, P, P, P, P, P, P, P, P, vp]
        L.rl_attn_merge.argtypes = [P, P, P, P, P, vp]
        L.rl_attn_last_error.restype = ctypes.c_char_p
        L.rl_attn_check_device_errors.argtypes = [vp]
        L.rl_attn_reserve_workspace.argtypes = [ctypes.c_size_t, vp]
        L.rl_attn_decode_workspace_size.argtypes = [ctypes.c_int64] * 6 + [ctypes.c_int32]
        L.rl_attn_decode_workspace_size.restype = ctypes.c_size_t
        L.rl_attn_extend_workspace_size.argtypes = [ctypes.c_int64] * 6
        L.rl_attn_extend_workspace_size.restype = ctypes.c_size_t
        L.rl_attn_release.restype = None
        L.rl_attn_profile_enable.argtypes = [ctypes.c_int]
        L.rl_attn_profile_read.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_int), ctypes.POINTER(ctypes.c_double)]
        dp = ctypes.POINTER(ctypes.c_double)
        L.rl_attn_diag_read_bandwidth.argtypes = [vp, ctypes.c_int64, ctypes.c_int32, dp, vp]
        L.rl_attn_diag_mfma_bf16.argtypes = [ctypes.c_int64, dp, vp]
        i64p = ctypes.POINTER(ctypes.c_int64)
        L.rl_attn_diag_decode_capacity.argtypes = [ctypes.c_int64] * 6 + [ctypes.c_int32] * 4 + [i64p]
        L.rl_attn_diag_extend_capacity.argtypes = [ctypes.c_int64] * 4 + [i64p]
        for name in ("rl_attn_decode", "rl_attn_extend", "rl_attn_decode_ex", "rl_attn_extend_ex",
                     "rl_attn_decode_noalloc",
                     "rl_attn_decode_fp8", "rl_attn_extend_fp8", "rl_attn_append_kv", "rl_attn_append_kv_fp8",
                     "rl_attn_merge", "rl_attn_check_device_errors", "rl_attn_reserve_workspace",
                     "rl_attn_profile_enable", "rl_attn_profile_read", "rl_attn_diag_read_bandwidth",
                     "rl_attn_diag_mfma_bf16", "rl_attn_diag_decode_capacity", "rl_attn_diag_extend_capacity"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def header_functions() -> list:
    """Names of the functions the headers under ``include/`` declare."""
    names = set()
    for fn in sorted(os.listdir(INCLUDE)):
        if fn.endswith(".h"):
            with open(os.path.join(INCLUDE, fn)) as f:
                text = re.sub(r"/\*.*?\*/", "", f.read(), flags=re.S)
            names.update(re.findall(r"\b(rl_attn_\w+)\s*\(", text))
    return sorted(names)


def last_error() -> str:
    return lib().rl_attn_last_error().decode()


def _check(rc: int):
    if rc != 0:
        raise RlAttnError(rc, last_error())


_DTYPES = {torch.bfloat16: RL_BF16, torch.float32: RL_F32, torch.int32: RL_I32,
           torch.float8_e4m3fn: RL_FP8_E4M3}


def view(t: Optional[torch.Tensor]):
    """An ``rl_tensor`` describing ``t`` (no copy); None -> NULL.

    The library dereferences the pointers on the current HIP device, so every
    tensor must live there (a host pointer would reach a kernel)."""
    if t is None:
        return None
    if not t.is_cuda or t.device.index != torch.cuda.current_device():
        raise ValueError(f"tensor on {t.device}: the library reads and writes tensors on the current device "
                         f"(cuda:{torch.cuda.current_device() if torch.cuda.is_available() else '?'})")
    if t.dim() > 4:
        raise ValueError("rl_tensor holds at most 4 dimensions")
    v = RlTensor()
    v.data = t.data_ptr() if t.numel() else (t.data_ptr() or None)
    v.dtype = _DTYPES.get(t.dtype, 0)
    v.ndim = t.dim()
    for i in range(t.dim()):
        v.shape[i] = t.shape[i]
        v.strides[i] = t.stride(i)
    return v


def _ref(v):
    return ctypes.byref(v) if v is not None else None


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def _opts(split_tokens=0, prefix_share=True, validate=False, deterministic=False):
    o = RlOpts()
    o.split_tokens = int(split_tokens)
    o.prefix_share = RL_PREFIX_AUTO if prefix_share else RL_PREFIX_OFF
    o.validate = int(bool(validate))
    o.deterministic = int(bool(deterministic))
    return o


def decode(q, k_pages, v_pages, block_table, seq_lens, scale, out=None, lse=None, *, split_tokens=0,
           prefix_share=True, validate=False, deterministic=False, stream=None):
    """``rl_attn_decode_ex``: returns ``out`` (and fills ``lse`` if given)."""
    if out is None:
        out = torch.empty_like(q)
    o = _opts(split_tokens, prefix_share, validate, deterministic)
    _check(lib().rl_attn_decode_ex(_ref(view(q)), _ref(view(k_pages)), _ref(view(v_pages)),
                                   _ref(view(block_table)), _ref(view(seq_lens)), ctypes.c_float(scale),
                                   _ref(view(out)), _ref(view(lse)), ctypes.byref(o), _stream(stream)))
    return out


def decode_noalloc(q, k_pages, v_pages, block_table, seq_lens, scale, out=None, lse=None, *, split_tokens=0,
                   prefix_share=True, deterministic=False, stream=None):
    """``rl_attn_decode_noalloc``: decode with the library's static scratch array as workspace
    (``out`` must be given by a caller that cannot allocate)."""
    if out is None:
        out = torch.empty_like(q)
    o = _opts(split_tokens, prefix_share, False, deterministic)
    _check(lib().rl_attn_decode_noalloc(_ref(view(q)), _ref(view(k_pages)), _ref(view(v_pages)),
                                        _ref(view(block_table)), _ref(view(seq_lens)), ctypes.c_float(scale),
                                        _ref(view(out)), _ref(view(lse)), ctypes.byref(o), _stream(stream)))
    return out


def decode_plain(q, k_pages, v_pages, block_table, seq_lens, scale, out=None, stream=None):
    """``rl_attn_decode`` (the fixed signature, no options)."""
    if out is None:
        out = torch.empty_like(q)
    _check(lib().rl_attn_decode(_ref(view(q)), _ref(view(k_pages)), _ref(view(v_pages)),
                                _ref(view(block_table)), _ref(view(seq_lens)), ctypes.c_float(scale),
                                _ref(view(out)), _stream(stream)))
    return out


def extend(q, qo_indptr, k_pages, v_pages, block_table, kv_lens, scale, out=None, lse=None, *,
           validate=False, stream=None):
    """``rl_attn_extend_ex``: returns ``out`` (and fills ``lse`` if given)."""
    if out is None:
        out = torch.empty_like(q)
    o = _opts(0, True, validate)
    _check(lib().rl_attn_extend_ex(_ref(view(q)), _ref(view(qo_indptr)), _ref(view(k_pages)),
                                   _ref(view(v_pages)), _ref(view(block_table)), _ref(view(kv_lens)),
                                   ctypes.c_float(scale), _ref(view(out)), _ref(view(lse)), ctypes.byref(o),
                                   _stream(stream)))
    return out


def extend_plain(q, qo_indptr, k_pages, v_pages, block_table, kv_lens, scale, out=None, stream=None):
    """``rl_attn_extend`` (the fixed signature)."""
    if out is None:
        out = torch.empty_like(q)
    _check(lib().rl_attn_extend(_ref(view(q)), _ref(view(qo_indptr)), _ref(view(k_pages)), _ref(view(v_pages)),
                                _ref(view(block_table)), _ref(view(kv_lens)), ctypes.c_float(scale),
                                _ref(view(out)), _stream(stream)))
    return out


def decode_fp8(q, k_pages, v_pages, k_scale, v_scale, block_table, seq_lens, scale, out=None, lse=None, *,
               split_tokens=0, prefix_share=True, validate=False, deterministic=False, stream=None):
    """``rl_attn_decode_fp8``: pages are ``torch.float8_e4m3fn``, scales ``[Hkv]`` float32."""
    if out is None:
        out = torch.empty_like(q)
    o = _opts(split_tokens, prefix_share, validate, deterministic)
    _check(lib().rl_attn_decode_fp8(_ref(view(q)), _ref(view(k_pages)), _ref(view(v_pages)), _ref(view(k_scale)),
                                    _ref(view(v_scale)), _ref(view(block_table)), _ref(view(seq_lens)),
                                    ctypes.c_float(scale), _ref(view(out)), _ref(view(lse)), ctypes.byref(o),
                                    _stream(stream)))
    return out


def extend_fp8(q, qo_indptr, k_pages, v_pages, k_scale, v_scale, block_table, kv_lens, scale, out=None, lse=None,
               *, validate=False, stream=None):
    """``rl_attn_extend_fp8``: pages are ``torch.float8_e4m3fn``, scales ``[Hkv]`` float32."""
    if out is None:
        out = torch.empty_like(q)
    o = _opts(0, True, validate)
    _check(lib().rl_attn_extend_fp8(_ref(view(q)), _ref(view(qo_indptr)), _ref(view(k_pages)), _ref(view(v_pages)),
                                    _ref(view(k_scale)), _ref(view(v_scale)), _ref(view(block_table)),
                                    _ref(view(kv_lens)), ctypes.c_float(scale), _ref(view(out)), _ref(view(lse)),
                                    ctypes.byref(o), _stream(stream)))
    return out


def append_kv(k_new, v_new, qo_indptr, block_table, kv_lens, k_pages, v_pages, stream=None):
    """``rl_attn_append_kv``: writes the new rows into ``k_pages``/``v_pages`` (in place)."""
    _check(lib().rl_attn_append_kv(_ref(view(k_new)), _ref(view(v_new)), _ref(view(qo_indptr)),
                                   _ref(view(block_table)), _ref(view(kv_lens)), _ref(view(k_pages)),
                                   _ref(view(v_pages)), _stream(stream)))


def append_kv_fp8(k_new, v_new, qo_indptr, block_table, kv_lens, k_pages, v_pages, k_scale, v_scale, stream=None):
    """``rl_attn_append_kv_fp8``: bf16 rows quantised into ``torch.float8_e4m3fn`` pages (in place)."""
    _check(lib().rl_attn_append_kv_fp8(_ref(view(k_new)), _ref(view(v_new)), _ref(view(qo_indptr)),
                                       _ref(view(block_table)), _ref(view(kv_lens)), _ref(view(k_pages)),
                                       _ref(view(v_pages)), _ref(view(k_scale)), _ref(view(v_scale)),
                                       _stream(stream)))


def merge(o_parts, lse_parts, num_parts, out=None, lse=None, stream=None):
    """``rl_attn_merge``: log-sum-exp merge of partial results."""
    n, _, h, d = o_parts.shape
    if out is None:
        out = torch.empty((n, h, d), dtype=torch.float32, device=o_parts.device)
    _check(lib().rl_attn_merge(_ref(view(o_parts)), _ref(view(lse_parts)), _ref(view(num_parts)),
                               _ref(view(out)), _ref(view(lse)), _stream(stream)))
    return out


def check_device_errors(stream=None):
    _check(lib().rl_attn_check_device_errors(_stream(stream)))


def reserve_workspace(nbytes: int, stream=None):
    _check(lib().rl_attn_reserve_workspace(ctypes.c_size_t(nbytes), _stream(stream)))


def decode_workspace_size(batch: int, num_q_heads: int, num_kv_heads: int, max_pages: int, page_size: int,
                          query_tokens: int = 1, split_tokens: int = 0) -> int:
    """Workspace bytes a decode call may need (``query_tokens`` per sequence, the call's ``split_tokens``)."""
    return int(lib().rl_attn_decode_workspace_size(batch, num_q_heads, num_kv_heads, max_pages, page_size,
                                                   query_tokens, split_tokens))


def extend_workspace_size(batch: int, total_q: int, num_q_heads: int, num_kv_heads: int, max_pages: int,
                          page_size: int) -> int:
    return int(lib().rl_attn_extend_workspace_size(batch, total_q, num_q_heads, num_kv_heads, max_pages, page_size))


def profile_enable(on: bool = True):
    _check(lib().rl_attn_profile_enable(int(bool(on))))


def profile_read(kind: str):
    """(launches, mean ms) of the main kernel timed since the last read; kind 'decode', 'extend' or 'append'."""
    n = ctypes.c_int()
    ms = ctypes.c_double()
    _check(lib().rl_attn_profile_read({"decode": 0, "extend": 1, "append": 2}[kind], ctypes.byref(n),
                                      ctypes.byref(ms)))
    return n.value, ms.value


def release():
    lib().rl_attn_release()


def diag_read_bandwidth(buf: torch.Tensor, reps: int = 10, stream=None) -> float:
    """HBM read rate (GB/s) of streaming ``buf`` (a device tensor) ``reps`` times."""
    r = ctypes.c_double(0.0)
    _check(lib().rl_attn_diag_read_bandwidth(ctypes.c_void_p(buf.data_ptr()), buf.numel() * buf.element_size(),
                                            reps, ctypes.byref(r), _stream(stream)))
    return r.value


def diag_mfma_bf16(iters: int = 20000, stream=None) -> float:
    """TFLOP/s of a register-only bf16 MFMA loop on every CU."""
    t = ctypes.c_double(0.0)
    _check(lib().rl_attn_diag_mfma_bf16(iters, ctypes.byref(t), _stream(stream)))
    return t.value


def diag_decode_capacity(batch, num_q_heads, num_kv_heads, max_pages, page_size, query_tokens=1, split_tokens=0,
                         prefix_share=True, cus=256, workers_per_cu=1) -> dict:
    """Workspace capacities a decode call would be given (host arithmetic only)."""
    out = (ctypes.c_int64 * 7)()
    _check(lib().rl_attn_diag_decode_capacity(batch, num_q_heads, num_kv_heads, max_pages, page_size, query_tokens,
                                              split_tokens, int(bool(prefix_share)), cus, workers_per_cu, out))
    keys = ("max_items", "max_slots", "max_workers", "group_cap", "target_items", "prefix_grid", "bytes")
    return dict(zip(keys, (int(x) for x in out)))


def diag_extend_capacity(batch, total_q, num_q_heads, num_kv_heads) -> dict:
    """Work-unit capacity of an extend call (host arithmetic only)."""
    out = (ctypes.c_int64 * 4)()
    _check(lib().rl_attn_diag_extend_capacity(batch, total_q, num_q_heads, num_kv_heads, out))
    return dict(zip(("max_items", "rows_head", "tile_tokens", "head_blocks"), (int(x) for x in out)))
