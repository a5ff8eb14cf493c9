"""Python binding of ``libheterofold.so`` (argument marshalling only).

Every function here has the name of the C entry point it wraps
(``include/heterofold.h``) and does no arithmetic of the method: it checks
Python-side types, allocates outputs and workspaces with torch when the caller
does not pass them, hands raw pointers and the current HIP stream to the
library, and raises ``HeteroFoldError`` on a negative status.

The library is loaded on first use; if it has not been built the call raises
(there is no fallback path).
"""

from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libheterofold.so")

HF_OK = 0
HF_ERR_SHAPE, HF_ERR_MODE = -2, -4
STATUS = {0: "HF_OK", -1: "HF_ERR_NULL", -2: "HF_ERR_SHAPE", -3: "HF_ERR_OFFSETS",
          -4: "HF_ERR_MODE", -5: "HF_ERR_DTYPE", -6: "HF_ERR_CAPACITY", -7: "HF_ERR_HIP",
          -8: "HF_ERR_UNSUPPORTED"}
HF_ALIGN_OVERLAP, HF_ALIGN_TA = 0, 1
HF_LAYERS_INTERP2 = 0
HF_F32, HF_BF16 = 0, 1
HF_KERNEL_TRANSFER, HF_KERNEL_ROPE_TABLES, HF_KERNEL_ALIGNMENT, HF_KERNEL_PACK = 0, 1, 2, 3
HF_KERNEL_MOMENTS_STATS, HF_KERNEL_MOMENTS_COV, HF_KERNEL_RECOLOR_SOLVE, HF_KERNEL_FOLD = 4, 5, 6, 7
HF_KERNEL_TRANSFER_STAGE = 8
HF_KERNEL_STAGED_BUILD, HF_KERNEL_STAGED_GEMM = 9, 10
HF_MAX_BATCH = 64
ALIGN_MODES = {"overlap": HF_ALIGN_OVERLAP, "ta": HF_ALIGN_TA}


class HeteroFoldError(RuntimeError):
    def __init__(self, status: int, where: str, message: str):
        super().__init__(f"{where}: {STATUS.get(status, status)}: {message}")
        self.status = status


class hf_kv_desc(C.Structure):
    _fields_ = [("ptr", C.c_void_p), ("dtype", C.c_int32), ("L", C.c_int32), ("H", C.c_int32),
                ("d_h", C.c_int32), ("T_cap", C.c_int32), ("stride_b", C.c_int64),
                ("stride_l", C.c_int64), ("stride_c", C.c_int64), ("stride_h", C.c_int64),
                ("stride_t", C.c_int64)]


class hf_rope(C.Structure):
    _fields_ = [("theta_s", C.c_double), ("theta_r", C.c_double),
                ("unrotate_sender_k", C.c_int32), ("rotate_receiver_k", C.c_int32),
                ("pos0_s", C.POINTER(C.c_int32)), ("pos0_r", C.POINTER(C.c_int32))]


class hf_transfer_opts(C.Structure):
    _fields_ = [("inv_r", C.c_void_p), ("k_norm", C.c_void_p), ("k_norm_eps", C.c_float)]


class hf_recolor_info(C.Structure):
    _fields_ = [("iterations", C.c_int32 * 3), ("converged", C.c_int32 * 3),
                ("residual", C.c_double * 3)]


_I32P = C.POINTER(C.c_int32)
_SIGNATURES = {
    "hf_last_error": (C.c_char_p, []),
    "hf_version": (C.c_int32, []),
    "hf_alignment_nnz_capacity": (C.c_int64, [C.c_int32, _I32P, _I32P, C.c_int32]),
    "hf_alignment_workspace_bytes": (C.c_size_t, [C.c_int32, _I32P]),
    "hf_build_alignment": (C.c_int32, [C.c_int32, _I32P, _I32P, C.c_void_p, C.c_void_p,
                                       C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p,
                                       C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64,
                                       C.c_void_p, C.c_size_t, C.c_void_p]),
    "hf_validate_offsets_host": (C.c_int32, [C.c_int32, _I32P, _I32P]),
    "hf_build_layer_map": (C.c_int32, [C.c_int32, C.c_int32, C.c_int32, _I32P, _I32P, _I32P,
                                       _I32P]),
    "hf_build_layer_taps": (C.c_int32, [C.c_int32, C.c_int32, _I32P]),
    "hf_packed_maps_bytes": (C.c_size_t, [C.c_int32, C.c_int32, C.c_int32, C.c_int32]),
    "hf_pack_maps": (C.c_int32, [C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.c_void_p,
                                 C.c_void_p, C.c_void_p]),
    "hf_transfer_workspace_bytes": (C.c_size_t, [C.c_int32, _I32P, _I32P, C.POINTER(hf_kv_desc),
                                                 C.POINTER(hf_kv_desc), C.POINTER(hf_rope)]),
    "hf_transfer_staged_workspace_bytes": (C.c_size_t, [C.c_int32, _I32P, _I32P,
                                                        C.POINTER(hf_kv_desc), C.POINTER(hf_kv_desc),
                                                        C.POINTER(hf_rope), C.c_int32]),
    "hf_transfer_kv": (C.c_int32, [C.c_int32, _I32P, _I32P, C.c_void_p, C.c_void_p, C.c_void_p,
                                   C.c_void_p, _I32P, _I32P, _I32P, _I32P,
                                   C.POINTER(hf_kv_desc), C.POINTER(hf_kv_desc), C.c_void_p,
                                   C.c_size_t, C.c_void_p, C.POINTER(hf_rope),
                                   C.POINTER(hf_transfer_opts), C.c_void_p, C.c_size_t,
                                   C.c_void_p]),
    "hf_transfer_kv_noalloc": (C.c_int32, [C.c_int32, _I32P, _I32P, C.c_void_p, C.c_void_p,
                                           C.c_void_p, C.c_void_p, _I32P, _I32P, _I32P, _I32P,
                                           C.POINTER(hf_kv_desc), C.POINTER(hf_kv_desc),
                                           C.c_void_p, C.c_size_t, C.c_void_p,
                                           C.POINTER(hf_rope), C.POINTER(hf_transfer_opts),
                                           C.c_void_p]),
    "hf_transfer_kv_taps": (C.c_int32, [C.c_int32, _I32P, _I32P, C.c_void_p, C.c_void_p,
                                        C.c_void_p, C.c_void_p, C.c_int32, _I32P,
                                        C.POINTER(hf_kv_desc), C.POINTER(hf_kv_desc), C.c_void_p,
                                        C.c_size_t, C.c_void_p, C.POINTER(hf_rope),
                                        C.POINTER(hf_transfer_opts), C.c_void_p, C.c_size_t,
                                        C.c_void_p]),
    "hf_recolor_moments_workspace_bytes": (C.c_size_t, [C.c_int64, C.c_int32, C.c_int32]),
    "hf_recolor_moments": (C.c_int32, [C.c_int64, C.c_int32, C.c_int32, C.c_int32, C.c_void_p,
                                       C.c_int64, C.c_void_p, C.c_int64, C.c_void_p, C.c_void_p,
                                       C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t,
                                       C.c_void_p]),
    "hf_recolor_solve_workspace_bytes": (C.c_size_t, [C.c_int32, C.c_int32]),
    "hf_recolor_solve": (C.c_int32, [C.c_int32, C.c_int32, C.c_void_p, C.c_void_p, C.c_double,
                                     C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t,
                                     C.c_void_p]),
    "hf_fold_workspace_bytes": (C.c_size_t, [C.c_int32, C.c_int32]),
    "hf_fold_map": (C.c_int32, [C.c_int32, C.c_int32, C.c_int32, C.c_void_p, C.c_void_p,
                                C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                C.c_size_t, C.c_void_p]),
    "hf_gemm_f64": (C.c_int32, [C.c_int32, C.c_int32, C.c_int64, C.c_void_p, C.c_int64,
                                C.c_int32, C.c_void_p, C.c_int64, C.c_int32, C.c_void_p,
                                C.c_int64, C.c_double, C.c_double, C.c_void_p, C.c_int64,
                                C.c_double, C.c_void_p]),
    "hf_profiler_enable": (C.c_int32, [C.c_int32]),
    "hf_profiler_reset": (C.c_int32, []),
    "hf_profiler_query": (C.c_int32, [C.c_int32, C.POINTER(C.c_double), C.POINTER(C.c_int64)]),
    "hf_profiler_samples": (C.c_int32, [C.c_int32, C.POINTER(C.c_float), C.c_int64,
                                        C.POINTER(C.c_int64)]),
}

_lib = None


def lib() -> C.CDLL:
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2609_32259_amd.build`")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def exported_symbols() -> Sequence[str]:
    return list(_SIGNATURES)


def _check(status: int, where: str):
    if status != HF_OK:
        msg = lib().hf_last_error().decode(errors="replace")
        raise HeteroFoldError(status, where, msg)


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _p32(a: np.ndarray):
    return a.ctypes.data_as(_I32P)


def _torch():
    import torch
    return torch


def _stream(stream):
    torch = _torch()
    if stream is None:
        return C.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return C.c_void_p(stream)
    return C.c_void_p(stream.cuda_stream)


def _nbytes(t) -> int:
    return int(t.numel() * t.element_size())


def _dev_i32(t, name):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or t.dtype != torch.int32 or not t.is_cuda \
            or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous int32 CUDA tensor")
    return C.c_void_p(t.data_ptr())


def hf_version() -> int:
    return int(lib().hf_version())


# ---------------------------------------------------------------------------
# Alignment
# ---------------------------------------------------------------------------

def _mode_code(mode) -> int:
    return ALIGN_MODES[mode] if isinstance(mode, str) else int(mode)


def hf_alignment_nnz_capacity(s_len, r_len, mode="overlap") -> int:
    """s_len, r_len: per-sequence token counts [B]."""
    s_len, r_len = _i32(s_len), _i32(r_len)
    if s_len.size != r_len.size:
        raise ValueError("s_len and r_len differ in length")
    code = _mode_code(mode)
    n = lib().hf_alignment_nnz_capacity(s_len.size, _p32(s_len), _p32(r_len), code)
    if n < 0:
        msg = lib().hf_last_error().decode(errors="replace")
        st = HF_ERR_MODE if code not in ALIGN_MODES.values() else HF_ERR_SHAPE
        raise HeteroFoldError(st, "hf_alignment_nnz_capacity", msg)
    return int(n)


def hf_alignment_workspace_bytes(r_cu) -> int:
    r_cu = _i32(r_cu)
    return int(lib().hf_alignment_workspace_bytes(r_cu.size - 1, _p32(r_cu)))


@dataclass
class Alignment:
    row_ptr: "object"   # int32 [sum T_r + 1] device
    col: "object"       # int32 [capacity] device
    num: "object"       # int32 [capacity] device
    den: "object"       # int32 [sum T_r] device
    s_cu: np.ndarray
    r_cu: np.ndarray

    def nnz(self) -> int:
        return int(self.row_ptr[-1].item())


def hf_build_alignment(s_cu, r_cu, s_beg, s_end, r_beg, r_end, mode="overlap",
                       out: Optional[Alignment] = None, workspace=None, stream=None) -> Alignment:
    """Spans are int32 CUDA tensors (concatenated over the batch); s_cu, r_cu
    host prefix sums.  Returns the CSR table (allocated unless ``out``)."""
    torch = _torch()
    s_cu, r_cu = _i32(s_cu), _i32(r_cu)
    B = s_cu.size - 1
    dev = s_beg.device
    cap = hf_alignment_nnz_capacity(np.diff(s_cu), np.diff(r_cu), mode)
    nR = int(r_cu[-1])
    if out is None:
        out = Alignment(torch.empty(nR + 1, dtype=torch.int32, device=dev),
                        torch.empty(max(cap, 1), dtype=torch.int32, device=dev),
                        torch.empty(max(cap, 1), dtype=torch.int32, device=dev),
                        torch.empty(max(nR, 1), dtype=torch.int32, device=dev), s_cu, r_cu)
    wsb = hf_alignment_workspace_bytes(r_cu)
    if workspace is None:
        workspace = torch.empty(max(wsb, 16), dtype=torch.uint8, device=dev)
    st = lib().hf_build_alignment(
        B, _p32(s_cu), _p32(r_cu), _dev_i32(s_beg, "s_beg"), _dev_i32(s_end, "s_end"),
        _dev_i32(r_beg, "r_beg"), _dev_i32(r_end, "r_end"), _mode_code(mode),
        _dev_i32(out.row_ptr, "row_ptr"), _dev_i32(out.col, "col"), _dev_i32(out.num, "num"),
        _dev_i32(out.den, "den"), int(out.col.numel()), C.c_void_p(workspace.data_ptr()),
        int(workspace.numel() * workspace.element_size()), _stream(stream))
    _check(st, "hf_build_alignment")
    return out


def hf_validate_offsets_host(beg, end) -> None:
    beg, end = _i32(beg), _i32(end)
    if beg.size != end.size:
        raise ValueError("beg and end differ in length")
    _check(lib().hf_validate_offsets_host(beg.size, _p32(beg), _p32(end)), "hf_validate_offsets_host")


# ---------------------------------------------------------------------------
# Layer map
# ---------------------------------------------------------------------------

def hf_build_layer_map(L_s: int, L_r: int, mode: int = HF_LAYERS_INTERP2):
    """Host table (lo, hi, rem, den), int32 numpy arrays [L_r]."""
    out = [np.zeros(max(L_r, 1), dtype=np.int32) for _ in range(4)]
    _check(lib().hf_build_layer_map(int(L_s), int(L_r), int(mode), *[_p32(o) for o in out]),
           "hf_build_layer_map")
    return tuple(o[:L_r] for o in out)


def hf_build_layer_taps(L_s: int, L_r: int):
    """The paper's three-layer neighbourhood: host int32 numpy [L_r, 3]."""
    out = np.zeros((max(L_r, 1), 3), dtype=np.int32)
    _check(lib().hf_build_layer_taps(int(L_s), int(L_r), _p32(out)), "hf_build_layer_taps")
    return out[:L_r]


# ---------------------------------------------------------------------------
# Maps and transfer
# ---------------------------------------------------------------------------

def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return HF_BF16
    if t.dtype == torch.float32:
        return HF_F32
    raise TypeError(f"unsupported storage dtype {t.dtype}")


def hf_packed_maps_bytes(L_r, d_r, d_in, dtype) -> int:
    return int(lib().hf_packed_maps_bytes(L_r, d_r, d_in, dtype))


def hf_pack_maps(A, out=None, stream=None):
    """A: contiguous CUDA tensor [L_r, 2, d_r, d_in] (bf16 or fp32).  Returns
    the packed buffer (header + maps) as a flat uint8 tensor of
    hf_packed_maps_bytes bytes."""
    torch = _torch()
    if A.dim() != 4 or A.shape[1] != 2 or not A.is_contiguous() or not A.is_cuda:
        raise TypeError("A must be a contiguous CUDA tensor [L_r, 2, d_r, d_in]")
    L_r, _, d_r, d_in = A.shape
    code = _dtype_code(A)
    if out is None:
        out = torch.empty(hf_packed_maps_bytes(L_r, d_r, d_in, code), dtype=torch.uint8,
                          device=A.device)
    st = lib().hf_pack_maps(L_r, d_r, d_in, code, C.c_void_p(A.data_ptr()),
                            C.c_void_p(out.data_ptr()), _stream(stream))
    _check(st, "hf_pack_maps")
    return out


def kv_desc(t) -> hf_kv_desc:
    """Descriptor of a cache tensor [B, L, 2, H, T_cap, d_h] (channels contiguous)."""
    if t.dim() != 6 or t.stride(5) != 1:
        raise TypeError("cache must be [B, L, 2, H, T_cap, d_h] with contiguous channels")
    B, L, two, H, T, d = t.shape
    if two != 2:
        raise TypeError("cache dim 2 must be the K/V role (size 2)")
    s = t.stride()
    return hf_kv_desc(C.c_void_p(t.data_ptr()), _dtype_code(t), L, H, d, T, s[0], s[1], s[2],
                      s[3], s[4])


def make_rope(theta_s, theta_r, unrotate_sender_k=True, rotate_receiver_k=True,
              pos0_s=None, pos0_r=None):
    """An hf_rope plus the host arrays it points to (keep the tuple alive)."""
    ps = None if pos0_s is None else _i32(pos0_s)
    pr = None if pos0_r is None else _i32(pos0_r)
    r = hf_rope(float(theta_s), float(theta_r), int(bool(unrotate_sender_k)),
                int(bool(rotate_receiver_k)), _p32(ps) if ps is not None else None,
                _p32(pr) if pr is not None else None)
    return r, (ps, pr)


def _rope_struct(rope):
    if rope is None:
        return None, None
    return make_rope(rope["theta_s"], rope["theta_r"], rope.get("unrotate_sender_k", True),
                     rope.get("rotate_receiver_k", True), rope.get("pos0_s"), rope.get("pos0_r"))


def _opts_struct(opts):
    """opts: None or dict(inv_r=fp32 CUDA tensor [L_r, 2] or None,
    k_norm=fp32 CUDA tensor [L_r, d_h] or None, k_norm_eps=float)."""
    if opts is None:
        return None
    torch = _torch()
    ptrs = []
    for key in ("inv_r", "k_norm"):
        t = opts.get(key)
        if t is not None and (not t.is_cuda or t.dtype != torch.float32 or not t.is_contiguous()):
            raise TypeError(f"{key} must be a contiguous fp32 CUDA tensor")
        ptrs.append(C.c_void_p(t.data_ptr()) if t is not None else None)
    return hf_transfer_opts(ptrs[0], ptrs[1], float(opts.get("k_norm_eps", 1e-6)))


def hf_transfer_workspace_bytes(s_len, r_len, S, R, rope=None) -> int:
    s_len, r_len = _i32(s_len), _i32(r_len)
    sd, rd = kv_desc(S), kv_desc(R)
    rs, keep = _rope_struct(rope)
    return int(lib().hf_transfer_workspace_bytes(s_len.size, _p32(s_len), _p32(r_len),
                                                 C.byref(sd), C.byref(rd),
                                                 C.byref(rs) if rs is not None else None))


def hf_transfer_staged_workspace_bytes(s_len, r_len, S, R, rope=None, n_taps=0) -> int:
    """Workspace bytes that select the staged path (n_taps 0: hf_transfer_kv;
    1..3: hf_transfer_kv_taps); 0 where it does not apply."""
    s_len, r_len = _i32(s_len), _i32(r_len)
    sd, rd = kv_desc(S), kv_desc(R)
    rs, keep = _rope_struct(rope)
    return int(lib().hf_transfer_staged_workspace_bytes(s_len.size, _p32(s_len), _p32(r_len),
                                                        C.byref(sd), C.byref(rd),
                                                        C.byref(rs) if rs is not None else None,
                                                        int(n_taps)))


def hf_transfer_kv(s_len, r_len, alignment: Alignment, layer_map, S, R, A_packed, bias=None,
                   rope=None, workspace=None, stream=None, opts=None):
    """Map sender caches S [B, L_s, 2, H_s, T_cap, d_h] into receiver caches
    R [B, L_r, 2, H_r, T_cap, d_h] (written in place).  layer_map is the
    (lo, hi, rem, den) host table; rope a dict (theta_s, theta_r,
    unrotate_sender_k, rotate_receiver_k, pos0_s, pos0_r) or None; opts a
    dict (inv_r, k_norm, k_norm_eps) or None."""
    torch = _torch()
    s_len, r_len = _i32(s_len), _i32(r_len)
    lo, hi, rem, den_l = (_i32(x) for x in layer_map)
    sd, rd = kv_desc(S), kv_desc(R)
    rs, keep = _rope_struct(rope)
    os_ = _opts_struct(opts)
    wsb = hf_transfer_workspace_bytes(s_len, r_len, S, R, rope)
    if workspace is None and wsb > 0:
        workspace = torch.empty(wsb, dtype=torch.uint8, device=S.device)
    if bias is not None and (bias.dtype != torch.float32 or not bias.is_contiguous()):
        raise TypeError("bias must be a contiguous fp32 tensor [L_r, 2, d_r]")
    st = lib().hf_transfer_kv(
        s_len.size, _p32(s_len), _p32(r_len), _dev_i32(alignment.row_ptr, "row_ptr"),
        _dev_i32(alignment.col, "col"), _dev_i32(alignment.num, "num"),
        _dev_i32(alignment.den, "den"), _p32(lo), _p32(hi), _p32(rem), _p32(den_l),
        C.byref(sd), C.byref(rd), C.c_void_p(A_packed.data_ptr()), _nbytes(A_packed),
        C.c_void_p(bias.data_ptr()) if bias is not None else None,
        C.byref(rs) if rs is not None else None,
        C.byref(os_) if os_ is not None else None,
        C.c_void_p(workspace.data_ptr()) if workspace is not None else None,
        int(workspace.numel() * workspace.element_size()) if workspace is not None else 0,
        _stream(stream))
    _check(st, "hf_transfer_kv")
    return R


def hf_transfer_kv_noalloc(s_len, r_len, alignment: Alignment, layer_map, S, R, A_packed,
                           bias=None, rope=None, stream=None, opts=None):
    """hf_transfer_kv without a workspace: the library's own device scratch
    array holds it, and the call allocates nothing (arguments as
    hf_transfer_kv)."""
    torch = _torch()
    s_len, r_len = _i32(s_len), _i32(r_len)
    lo, hi, rem, den_l = (_i32(x) for x in layer_map)
    sd, rd = kv_desc(S), kv_desc(R)
    rs, keep = _rope_struct(rope)
    os_ = _opts_struct(opts)
    if bias is not None and (bias.dtype != torch.float32 or not bias.is_contiguous()):
        raise TypeError("bias must be a contiguous fp32 tensor [L_r, 2, d_r]")
    st = lib().hf_transfer_kv_noalloc(
        s_len.size, _p32(s_len), _p32(r_len), _dev_i32(alignment.row_ptr, "row_ptr"),
        _dev_i32(alignment.col, "col"), _dev_i32(alignment.num, "num"),
        _dev_i32(alignment.den, "den"), _p32(lo), _p32(hi), _p32(rem), _p32(den_l),
        C.byref(sd), C.byref(rd), C.c_void_p(A_packed.data_ptr()), _nbytes(A_packed),
        C.c_void_p(bias.data_ptr()) if bias is not None else None,
        C.byref(rs) if rs is not None else None,
        C.byref(os_) if os_ is not None else None, _stream(stream))
    _check(st, "hf_transfer_kv_noalloc")
    return R


def hf_transfer_kv_taps(s_len, r_len, alignment: Alignment, taps, S, R, A_packed, bias=None,
                        rope=None, workspace=None, stream=None, opts=None):
    """hf_transfer_kv with concatenated-tap maps: taps is the host table
    [L_r, n_taps] (e.g. hf_build_layer_taps) and A_packed packs maps of input
    size n_taps * H_s * d_h."""
    torch = _torch()
    s_len, r_len = _i32(s_len), _i32(r_len)
    taps = np.ascontiguousarray(np.asarray(taps, dtype=np.int32))
    if taps.ndim != 2:
        raise TypeError("taps must be a table [L_r, n_taps]")
    sd, rd = kv_desc(S), kv_desc(R)
    rs, keep = _rope_struct(rope)
    os_ = _opts_struct(opts)
    wsb = hf_transfer_workspace_bytes(s_len, r_len, S, R, rope)
    if workspace is None and wsb > 0:
        workspace = torch.empty(wsb, dtype=torch.uint8, device=S.device)
    if bias is not None and (bias.dtype != torch.float32 or not bias.is_contiguous()):
        raise TypeError("bias must be a contiguous fp32 tensor [L_r, 2, d_r]")
    st = lib().hf_transfer_kv_taps(
        s_len.size, _p32(s_len), _p32(r_len), _dev_i32(alignment.row_ptr, "row_ptr"),
        _dev_i32(alignment.col, "col"), _dev_i32(alignment.num, "num"),
        _dev_i32(alignment.den, "den"), int(taps.shape[1]), _p32(taps),
        C.byref(sd), C.byref(rd), C.c_void_p(A_packed.data_ptr()), _nbytes(A_packed),
        C.c_void_p(bias.data_ptr()) if bias is not None else None,
        C.byref(rs) if rs is not None else None,
        C.byref(os_) if os_ is not None else None,
        C.c_void_p(workspace.data_ptr()) if workspace is not None else None,
        int(workspace.numel() * workspace.element_size()) if workspace is not None else 0,
        _stream(stream))
    _check(st, "hf_transfer_kv_taps")
    return R


# ---------------------------------------------------------------------------
# Profiler
# ---------------------------------------------------------------------------

def hf_profiler_enable(on: bool = True):
    _check(lib().hf_profiler_enable(int(bool(on))), "hf_profiler_enable")


def hf_profiler_reset():
    _check(lib().hf_profiler_reset(), "hf_profiler_reset")


def hf_profiler_query(kernel_id: int):
    ms, n = C.c_double(0.0), C.c_int64(0)
    _check(lib().hf_profiler_query(int(kernel_id), C.byref(ms), C.byref(n)), "hf_profiler_query")
    return float(ms.value), int(n.value)


def hf_profiler_samples(kernel_id: int) -> np.ndarray:
    """Per-launch durations (ms) of one kernel since the last reset."""
    n = C.c_int64(0)
    _check(lib().hf_profiler_samples(int(kernel_id), None, 0, C.byref(n)), "hf_profiler_samples")
    out = np.zeros(max(n.value, 1), dtype=np.float32)
    _check(lib().hf_profiler_samples(int(kernel_id), out.ctypes.data_as(C.POINTER(C.c_float)),
                                     out.size, C.byref(n)), "hf_profiler_samples")
    return out[:n.value]


# ---------------------------------------------------------------------------
# Offline construction of the maps (fp64)
# ---------------------------------------------------------------------------

def _dev_f64(t, name, numel=None):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or t.dtype != torch.float64 or not t.is_cuda \
            or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous float64 CUDA tensor")
    if numel is not None and t.numel() != numel:
        raise TypeError(f"{name} must have {numel} elements")
    return C.c_void_p(t.data_ptr())


def _rows(t, name, width):
    """(pointer, leading dimension) of a [n, >=width] row-major CUDA tensor."""
    if t.dim() != 2 or t.stride(1) != 1 or t.shape[1] < width or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA tensor [n, {width}] with contiguous rows")
    return C.c_void_p(t.data_ptr()), int(t.stride(0))


def _workspace(ws, nbytes, dev):
    torch = _torch()
    if ws is None:
        return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=dev)
    return ws


def hf_recolor_moments_workspace_bytes(n: int, p: int, q: int) -> int:
    return int(lib().hf_recolor_moments_workspace_bytes(int(n), int(p), int(q)))


def hf_recolor_moments(x, y, w=None, workspace=None, stream=None):
    """x: [n, p], y: [n, q] CUDA tensors (fp32 or bf16, same dtype, contiguous
    rows); w: fp32 [n] or None.  Returns (r [1], mu [p+q], cov [p+q, p+q]) as
    float64 CUDA tensors (asynchronous)."""
    torch = _torch()
    if x.dtype != y.dtype or x.shape[0] != y.shape[0]:
        raise TypeError("x and y must have the same dtype and number of rows")
    n, p = int(x.shape[0]), int(x.shape[1])
    q = int(y.shape[1])
    xp, ldx = _rows(x, "x", p)
    yp, ldy = _rows(y, "y", q)
    wp = None
    if w is not None:
        if w.dtype != torch.float32 or not w.is_cuda or not w.is_contiguous() or w.numel() != n:
            raise TypeError("w must be a contiguous float32 CUDA tensor [n]")
        wp = C.c_void_p(w.data_ptr())
    dev = x.device
    r = torch.empty(1, dtype=torch.float64, device=dev)
    mu = torch.empty(p + q, dtype=torch.float64, device=dev)
    cov = torch.empty((p + q, p + q), dtype=torch.float64, device=dev)
    ws = _workspace(workspace, hf_recolor_moments_workspace_bytes(n, p, q), dev)
    st = lib().hf_recolor_moments(n, p, q, _dtype_code(x), xp, ldx, yp, ldy, wp,
                                  C.c_void_p(r.data_ptr()), C.c_void_p(mu.data_ptr()),
                                  C.c_void_p(cov.data_ptr()), C.c_void_p(ws.data_ptr()),
                                  int(ws.numel() * ws.element_size()), _stream(stream))
    _check(st, "hf_recolor_moments")
    return r, mu, cov


def hf_recolor_solve_workspace_bytes(p: int, q: int) -> int:
    return int(lib().hf_recolor_solve_workspace_bytes(int(p), int(q)))


def hf_recolor_solve(mu, cov, p: int, ridge: float = 0.0, workspace=None, stream=None):
    """Recolor map from moments.  Returns (A [q, p], b [q], info) where A and b
    are float64 CUDA tensors and info a CUDA byte tensor holding an
    ``hf_recolor_info`` (read it with ``recolor_info`` after the stream is
    done)."""
    torch = _torch()
    pq = int(mu.numel())
    p = int(p)
    q = pq - p
    if q < 1 or p < 1:
        raise ValueError("need 1 <= p < mu.numel()")
    dev = mu.device
    A = torch.empty((q, p), dtype=torch.float64, device=dev)
    b = torch.empty(q, dtype=torch.float64, device=dev)
    info = torch.zeros(C.sizeof(hf_recolor_info), dtype=torch.uint8, device=dev)
    ws = _workspace(workspace, hf_recolor_solve_workspace_bytes(p, q), dev)
    st = lib().hf_recolor_solve(p, q, _dev_f64(mu, "mu", pq), _dev_f64(cov, "cov", pq * pq),
                                float(ridge), C.c_void_p(A.data_ptr()), C.c_void_p(b.data_ptr()),
                                C.c_void_p(info.data_ptr()), C.c_void_p(ws.data_ptr()),
                                int(ws.numel() * ws.element_size()), _stream(stream))
    _check(st, "hf_recolor_solve")
    return A, b, info


def recolor_info(info) -> dict:
    """Host copy of an hf_recolor_info written by hf_recolor_solve (synchronizes)."""
    raw = bytes(info.cpu().numpy().tobytes())
    s = hf_recolor_info.from_buffer_copy(raw)
    return {"iterations": list(s.iterations), "converged": list(s.converged),
            "residual": list(s.residual)}


def hf_fold_workspace_bytes(p: int, rank: int) -> int:
    return int(lib().hf_fold_workspace_bytes(int(p), int(rank)))


def hf_fold_map(A, b, B, G, out=None, workspace=None, stream=None):
    """Fold y + (y B) G into the stored map: A [q, p], b [q], B [q, rank],
    G [rank, q] float64 CUDA tensors.  Returns (A_out, b_out) (``out`` may be
    ``(A, b)`` for in place)."""
    torch = _torch()
    q, p = int(A.shape[0]), int(A.shape[1])
    rank = int(B.shape[1]) if B.dim() == 2 else -1
    if B.dim() != 2 or B.shape[0] != q or G.dim() != 2 or tuple(G.shape) != (rank, q):
        raise TypeError("need B [q, rank] and G [rank, q]")
    if out is None:
        out = (torch.empty_like(A), torch.empty_like(b))
    ws = _workspace(workspace, hf_fold_workspace_bytes(p, rank), A.device)
    st = lib().hf_fold_map(p, q, rank, _dev_f64(A, "A", p * q), _dev_f64(b, "b", q),
                           _dev_f64(B, "B", q * rank), _dev_f64(G, "G", rank * q),
                           _dev_f64(out[0], "A_out", p * q), _dev_f64(out[1], "b_out", q),
                           C.c_void_p(ws.data_ptr()), int(ws.numel() * ws.element_size()),
                           _stream(stream))
    _check(st, "hf_fold_map")
    return out


def hf_gemm_f64(A, B, a_kmajor=False, b_kmajor=True, alpha=1.0, beta=0.0, C_in=None, gamma=0.0,
                out=None, stream=None):
    """D = alpha op(A) op(B) + beta C + gamma I on float64 CUDA tensors.
    a_kmajor: A is stored [k, m] (else [m, k]); b_kmajor: B is stored [k, n]
    (else [n, k])."""
    torch = _torch()
    if A.dim() != 2 or B.dim() != 2:
        raise TypeError("A and B must be 2-D")
    m, k = (A.shape[1], A.shape[0]) if a_kmajor else (A.shape[0], A.shape[1])
    kb, n = (B.shape[0], B.shape[1]) if b_kmajor else (B.shape[1], B.shape[0])
    if kb != k:
        raise TypeError("inner dimensions differ")
    if out is None:
        out = torch.empty((m, n), dtype=torch.float64, device=A.device)
    cp, ldc = (None, 0)
    if beta != 0.0:
        if C_in is None or tuple(C_in.shape) != (m, n):
            raise TypeError("C_in [m, n] needed when beta != 0")
        cp, ldc = _dev_f64(C_in, "C"), n
    st = lib().hf_gemm_f64(int(m), int(n), int(k), _dev_f64(A, "A"), int(A.shape[1]),
                           int(bool(a_kmajor)), _dev_f64(B, "B"), int(B.shape[1]),
                           int(bool(b_kmajor)), _dev_f64(out, "D", m * n), int(n), float(alpha),
                           float(beta), cp, int(ldc), float(gamma), _stream(stream))
    _check(st, "hf_gemm_f64")
    return out
