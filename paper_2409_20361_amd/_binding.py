"""ctypes marshalling for librrs.so (names follow include/rrs.h without the prefix)."""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "librrs.so")
_lib: Optional[ctypes.CDLL] = None

_vp = ctypes.c_void_p
_i = ctypes.c_int
_sz = ctypes.c_size_t

_SIGNATURES = {
    "rrs_status_string": (ctypes.c_char_p, [ctypes.c_int32]),
    "rrs_version": (_i, []),
    "rrs_workspace_bytes": (_sz, [_i, _i, _i]),
    "rrs_linear_workspace_bytes": (_sz, [_i, _i, _i]),
    "rrs_prepare_weight": (ctypes.c_int32, [_vp, _i, _i, _vp, _vp, _vp, _vp]),
    "rrs_rotate_smooth_quant": (ctypes.c_int32,
                                [_vp, _i, _i, _i, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "rrs_w4a4_gemm": (ctypes.c_int32, [_vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _vp, _vp]),
    "rrs_linear": (ctypes.c_int32, [_vp, _vp, _vp, _i, _i, _i, _i, _vp, _vp, _vp, _sz, _vp]),
    "rrs_w4a4_gemm_partials": (ctypes.c_int32, [_vp, _vp, _i, _i, _i, _i, _vp, _vp]),
    "rrs_linear_noalloc": (ctypes.c_int32, [_vp, _vp, _vp, _i, _i, _i, _i, _vp, _vp, _vp]),
    "rrs_test_quant_rows_wait": (ctypes.c_int32, [_vp, _i, _i, _i, _i, _i, _vp, _vp, _vp, _vp,
                                                  _sz, _vp, _vp]),
    "rrs_test_quant_reorder_wait": (ctypes.c_int32, [_vp, _i, _i, _i, _i, _i, _vp, _vp, _vp,
                                                     _vp, _vp, _sz, _vp, _vp]),
    "rrs_prepare_weight_ex": (ctypes.c_int32, [_vp, _i, _i, _vp, _i, _vp, _vp, _vp]),
    "rrs_rotate_smooth_quant_ex": (ctypes.c_int32,
                                   [_vp, _i, _i, _i, _vp, _i, _vp, _vp, _vp, _vp, _sz, _vp]),
    "rrs_w4a4_gemm_ex": (ctypes.c_int32,
                         [_vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _vp, _vp]),
    "rrs_linear_ex": (ctypes.c_int32,
                      [_vp, _vp, _vp, _i, _i, _i, _i, _vp, _i, _vp, _vp, _sz, _vp]),
    "rrs_quantize_sub_channel": (ctypes.c_int32, [_vp, _i, _i, _i, _i, _vp, _vp, _vp]),
    "rrs_prepare_weight_sub_channel": (ctypes.c_int32, [_vp, _i, _i, _i, _i, _vp, _vp, _vp]),
    "rrs_w4a4_gemm_per_channel": (ctypes.c_int32,
                                  [_vp, _vp, _vp, _vp, _i, _i, _i, _i, _vp, _vp]),
    "rrs_w4a4_gemm_scheme": (ctypes.c_int32,
                             [_i, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _vp, _vp]),
    "rrs_reorder_workspace_bytes": (_sz, [_i, _i, _i]),
    "rrs_linear_reorder_workspace_bytes": (_sz, [_i, _i, _i]),
    "rrs_rotate_smooth_quant_reorder": (ctypes.c_int32,
                                        [_vp, _i, _i, _i, _i, _vp, _vp, _vp, _vp, _vp, _sz,
                                         _vp]),
    "rrs_w4a4_gemm_reorder": (ctypes.c_int32,
                              [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _vp, _vp]),
    "rrs_linear_reorder": (ctypes.c_int32,
                           [_vp, _vp, _vp, _i, _i, _i, _i, _i, _vp, _vp, _sz, _vp]),
}

# Channels per block of the runtime reorder (include/rrs.h, RRS_REORDER_BLOCK).
REORDER_BLOCK = 32

# Scale schemes of the kernel comparison (include/rrs.h, RRS_SCHEME_*).
SCHEME_PER_CHANNEL = 0
SCHEME_RUNTIME_SMOOTH = 1
SCHEME_SUB_CHANNEL = 2

# Ablation switches (include/rrs.h): 0 is RRS itself.
SKIP_ROTATION = 1    # plain Runtime Smooth: no Hadamard rotation
SKIP_SMOOTHING = 2   # rotation + per-token quantization only (smoothing scales all 1)
WEIGHT_TILED = 4     # Wq in 16-row blocks of 1 KB tiles (layout switch, not an ablation)


class RRSError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {status_string(code)} (status {code})")


def lib_path() -> str:
    return _LIB_PATH


def lib() -> ctypes.CDLL:
    """Load librrs.so from the package directory (built by build.py)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(
                f"{_LIB_PATH} is missing: build it with `python -m paper_2409_20361_amd.build` "
                "(there is no non-HIP fallback)")
        handle = ctypes.CDLL(_LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def status_string(code: int) -> str:
    return lib().rrs_status_string(code).decode()


def version() -> int:
    return lib().rrs_version()


def workspace_bytes(M: int, K: int, g: int) -> int:
    return lib().rrs_workspace_bytes(M, K, g)


def linear_workspace_bytes(M: int, K: int, g: int) -> int:
    return lib().rrs_linear_workspace_bytes(M, K, g)


def _check(code: int, where: str) -> None:
    if code != 0:
        raise RRSError(code, where)


def _stream(device: torch.device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _dev(t: torch.Tensor, name: str, dtype: torch.dtype, shape: Tuple[int, ...]) -> int:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor, got {t.device}")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _perm_ptr(perm: Optional[torch.Tensor], K: int) -> Optional[int]:
    if perm is None:
        return None
    return _dev(perm, "perm", torch.int32, (K,))


def prepare_weight(W: torch.Tensor, perm: Optional[torch.Tensor] = None, flags: int = 0
                   ) -> Tuple[torch.Tensor, torch.Tensor]:
    """W: K x N fp16 (the transpose of nn.Linear's weight) -> (Wq N x K/2 uint8, w_scale N f32).

    Wq holds the packed codes row-major; with flags | WEIGHT_TILED in the tiled
    layout of include/rrs.h (16-row blocks of 1 KB tiles), which the GEMM calls
    then need the same flag for."""
    K, N = W.shape
    wp = _dev(W, "W", torch.float16, (K, N))
    Wq = torch.empty((N, K // 2), dtype=torch.uint8, device=W.device)
    ws = torch.empty((N,), dtype=torch.float32, device=W.device)
    _check(lib().rrs_prepare_weight_ex(wp, K, N, _perm_ptr(perm, K), flags, Wq.data_ptr(),
                                       ws.data_ptr(), _stream(W.device)), "rrs_prepare_weight")
    return Wq, ws


def rotate_smooth_quant(X: torch.Tensor, g: int, perm: Optional[torch.Tensor] = None,
                        workspace: Optional[torch.Tensor] = None, out=None, flags: int = 0):
    """X: M x K fp16 -> (Xq M x K/2 uint8, a_scale M f32, s_group K/g f32)."""
    M, K = X.shape
    xp = _dev(X, "X", torch.float16, (M, K))
    if out is None:
        Xq = torch.empty((M, K // 2), dtype=torch.uint8, device=X.device)
        a = torch.empty((M,), dtype=torch.float32, device=X.device)
        s = torch.empty((max(K // g, 1),), dtype=torch.float32, device=X.device)
    else:
        Xq, a, s = out
    nbytes = workspace_bytes(M, K, g)
    if workspace is None:
        workspace = torch.zeros((max(nbytes, 1),), dtype=torch.uint8, device=X.device)
    _check(lib().rrs_rotate_smooth_quant_ex(
        xp, M, K, g, _perm_ptr(perm, K), flags, Xq.data_ptr(), a.data_ptr(), s.data_ptr(),
        workspace.data_ptr(), workspace.numel() * workspace.element_size(), _stream(X.device)),
        "rrs_rotate_smooth_quant")
    return Xq, a, s


def w4a4_gemm(Xq: torch.Tensor, a_scale: torch.Tensor, s_group: torch.Tensor,
              Wq: torch.Tensor, w_scale: torch.Tensor, g: int,
              out: Optional[torch.Tensor] = None, flags: int = 0) -> torch.Tensor:
    """Y = fp16(a_i w_n / K * sum_b s_b P_b) (M x N; no 1/K with SKIP_ROTATION)."""
    M, Kh = Xq.shape
    K = 2 * Kh
    N = Wq.shape[0]
    args = (_dev(Xq, "Xq", torch.uint8, (M, Kh)), _dev(a_scale, "a_scale", torch.float32, (M,)),
            _dev(s_group, "s_group", torch.float32, (K // g,)),
            _dev(Wq, "Wq", torch.uint8, (N, Kh)), _dev(w_scale, "w_scale", torch.float32, (N,)))
    Y = out if out is not None else torch.empty((M, N), dtype=torch.float16, device=Xq.device)
    yp = _dev(Y, "Y", torch.float16, (M, N))
    _check(lib().rrs_w4a4_gemm_ex(*args, M, N, K, g, flags, yp, _stream(Xq.device)),
           "rrs_w4a4_gemm")
    return Y


def linear(X: torch.Tensor, Wq: torch.Tensor, w_scale: torch.Tensor, g: int,
           perm: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
           out: Optional[torch.Tensor] = None, flags: int = 0) -> torch.Tensor:
    """One RRS linear layer: X M x K fp16 -> Y M x N fp16."""
    M, K = X.shape
    N = Wq.shape[0]
    xp = _dev(X, "X", torch.float16, (M, K))
    wqp = _dev(Wq, "Wq", torch.uint8, (N, K // 2))
    wsp = _dev(w_scale, "w_scale", torch.float32, (N,))
    nbytes = linear_workspace_bytes(M, K, g)
    if workspace is None:
        workspace = torch.zeros((max(nbytes, 1),), dtype=torch.uint8, device=X.device)
    Y = out if out is not None else torch.empty((M, N), dtype=torch.float16, device=X.device)
    yp = _dev(Y, "Y", torch.float16, (M, N))
    _check(lib().rrs_linear_ex(xp, wqp, wsp, M, N, K, g, _perm_ptr(perm, K), flags, yp,
                               workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                               _stream(X.device)), "rrs_linear")
    return Y


def linear_noalloc(X: torch.Tensor, Wq: torch.Tensor, w_scale: torch.Tensor, g: int,
                   perm: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None
                   ) -> torch.Tensor:
    """rrs_linear with the library-held scratch instead of a workspace: the C call
    allocates nothing (for graph capture and serving loops). Only Y is
    allocated here, and only when `out` is not given."""
    M, K = X.shape
    N = Wq.shape[0]
    xp = _dev(X, "X", torch.float16, (M, K))
    wqp = _dev(Wq, "Wq", torch.uint8, (N, K // 2))
    wsp = _dev(w_scale, "w_scale", torch.float32, (N,))
    Y = out if out is not None else torch.empty((M, N), dtype=torch.float16, device=X.device)
    yp = _dev(Y, "Y", torch.float16, (M, N))
    _check(lib().rrs_linear_noalloc(xp, wqp, wsp, M, N, K, g, _perm_ptr(perm, K), yp,
                                    _stream(X.device)), "rrs_linear_noalloc")
    return Y


def w4a4_gemm_partials(Xq: torch.Tensor, Wq: torch.Tensor, g: int) -> torch.Tensor:
    """Exact int32 group partials P[b, i, n] (test hook) from the kernel that
    rrs_w4a4_gemm runs for this shape with row-major Wq."""
    M, Kh = Xq.shape
    K = 2 * Kh
    N = Wq.shape[0]
    xp = _dev(Xq, "Xq", torch.uint8, (M, Kh))
    wp = _dev(Wq, "Wq", torch.uint8, (N, Kh))
    P = torch.empty((K // g, M, N), dtype=torch.int32, device=Xq.device)
    _check(lib().rrs_w4a4_gemm_partials(xp, wp, M, N, K, g, P.data_ptr(), _stream(Xq.device)),
           "rrs_w4a4_gemm_partials")
    return P


def quant_rows_wait_hook(X: torch.Tensor, g: int, extra_rows: int, max_polls: int,
                         workspace: Optional[torch.Tensor] = None):
    """Test hook of the one-launch quantizers' bounded wait: runs the kernel
    rrs_rotate_smooth_quant would choose with the readers also waiting for
    extra_rows rows that nobody writes and at most max_polls polling rounds;
    returns (Xq, a_scale, s_group, failed)."""
    M, K = X.shape
    xp = _dev(X, "X", torch.float16, (M, K))
    Xq = torch.empty((M, K // 2), dtype=torch.uint8, device=X.device)
    a = torch.empty((M,), dtype=torch.float32, device=X.device)
    s = torch.empty((K // g,), dtype=torch.float32, device=X.device)
    if workspace is None:
        workspace = torch.zeros((max(workspace_bytes(M, K, g), 1),), dtype=torch.uint8,
                                device=X.device)
    n = ctypes.c_int32(-1)
    _check(lib().rrs_test_quant_rows_wait(
        xp, M, K, g, extra_rows, max_polls, Xq.data_ptr(), a.data_ptr(), s.data_ptr(),
        workspace.data_ptr(), workspace.numel() * workspace.element_size(), ctypes.byref(n),
        _stream(X.device)), "rrs_test_quant_rows_wait")
    return Xq, a, s, bool(n.value)


def quant_reorder_wait_hook(X: torch.Tensor, g: int, extra_rows: int, max_polls: int,
                            workspace: Optional[torch.Tensor] = None):
    """Test hook of the one-launch runtime-reorder quantizer's bounded wait (as
    quant_rows_wait_hook); returns (Xq, a_scale, s_group, block_order, failed)."""
    M, K = X.shape
    xp = _dev(X, "X", torch.float16, (M, K))
    Xq = torch.empty((M, K // 2), dtype=torch.uint8, device=X.device)
    a = torch.empty((M,), dtype=torch.float32, device=X.device)
    s = torch.empty((K // g,), dtype=torch.float32, device=X.device)
    order = torch.empty((K // REORDER_BLOCK,), dtype=torch.int32, device=X.device)
    if workspace is None:
        workspace = torch.zeros((max(reorder_workspace_bytes(M, K, g), 1),), dtype=torch.uint8,
                                device=X.device)
    n = ctypes.c_int32(-1)
    _check(lib().rrs_test_quant_reorder_wait(
        xp, M, K, g, extra_rows, max_polls, Xq.data_ptr(), a.data_ptr(), s.data_ptr(),
        order.data_ptr(), workspace.data_ptr(), workspace.numel() * workspace.element_size(),
        ctypes.byref(n), _stream(X.device)), "rrs_test_quant_reorder_wait")
    return Xq, a, s, order, bool(n.value)


def quantize_sub_channel(X: torch.Tensor, g: int, flags: int = 0
                         ) -> Tuple[torch.Tensor, torch.Tensor]:
    """X: M x K fp16 -> (Xq M x K/2 uint8, a_sub K/g x M f32), one scale per (token, group)."""
    M, K = X.shape
    xp = _dev(X, "X", torch.float16, (M, K))
    Xq = torch.empty((M, K // 2), dtype=torch.uint8, device=X.device)
    a = torch.empty((K // g, M), dtype=torch.float32, device=X.device)
    _check(lib().rrs_quantize_sub_channel(xp, M, K, g, flags, Xq.data_ptr(), a.data_ptr(),
                                          _stream(X.device)), "rrs_quantize_sub_channel")
    return Xq, a


def prepare_weight_sub_channel(W: torch.Tensor, g: int, flags: int = 0
                               ) -> Tuple[torch.Tensor, torch.Tensor]:
    """W: K x N fp16 -> (Wq N x K/2 uint8, w_sub K/g x N f32), one scale per (channel, group)."""
    K, N = W.shape
    wp = _dev(W, "W", torch.float16, (K, N))
    Wq = torch.empty((N, K // 2), dtype=torch.uint8, device=W.device)
    ws = torch.empty((K // g, N), dtype=torch.float32, device=W.device)
    _check(lib().rrs_prepare_weight_sub_channel(wp, K, N, g, flags, Wq.data_ptr(), ws.data_ptr(),
                                                _stream(W.device)),
           "rrs_prepare_weight_sub_channel")
    return Wq, ws


def w4a4_gemm_scheme(scheme: int, Xq: torch.Tensor, x_scale: torch.Tensor,
                     s_group: Optional[torch.Tensor], Wq: torch.Tensor, w_scale: torch.Tensor,
                     g: int, flags: int = 0, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """One scale scheme on the comparison skeleton -> Y M x N fp16.

    per-channel: x_scale (M,), w_scale (N,); Runtime Smooth: x_scale (M,), s_group (K/g,),
    w_scale (N,); sub-channel: x_scale (K/g, M), w_scale (K/g, N).
    """
    M, Kh = Xq.shape
    N = Wq.shape[0]
    K = 2 * Kh
    G = K // g
    xq = _dev(Xq, "Xq", torch.uint8, (M, Kh))
    wq = _dev(Wq, "Wq", torch.uint8, (N, Kh))
    if scheme == SCHEME_SUB_CHANNEL:
        xs = _dev(x_scale, "x_scale", torch.float32, (G, M))
        ws = _dev(w_scale, "w_scale", torch.float32, (G, N))
    else:
        xs = _dev(x_scale, "x_scale", torch.float32, (M,))
        ws = _dev(w_scale, "w_scale", torch.float32, (N,))
    sp = None
    if scheme == SCHEME_RUNTIME_SMOOTH:
        sp = _dev(s_group, "s_group", torch.float32, (G,))
    if out is None:
        out = torch.empty((M, N), dtype=torch.float16, device=Xq.device)
    yp = _dev(out, "Y", torch.float16, (M, N))
    _check(lib().rrs_w4a4_gemm_scheme(scheme, xq, xs, sp, wq, ws, M, N, K, g, flags, yp,
                                      _stream(Xq.device)), "rrs_w4a4_gemm_scheme")
    return out


def w4a4_gemm_per_channel(Xq: torch.Tensor, a_scale: torch.Tensor, Wq: torch.Tensor,
                          w_scale: torch.Tensor, flags: int = 0,
                          out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Per-channel A4W4 on the tuned main loop: Y = fp16(a_i w_n / K * sum_j q q)."""
    M, Kh = Xq.shape
    N = Wq.shape[0]
    K = 2 * Kh
    xq = _dev(Xq, "Xq", torch.uint8, (M, Kh))
    ap = _dev(a_scale, "a_scale", torch.float32, (M,))
    wq = _dev(Wq, "Wq", torch.uint8, (N, Kh))
    wp = _dev(w_scale, "w_scale", torch.float32, (N,))
    if out is None:
        out = torch.empty((M, N), dtype=torch.float16, device=Xq.device)
    yp = _dev(out, "Y", torch.float16, (M, N))
    _check(lib().rrs_w4a4_gemm_per_channel(xq, ap, wq, wp, M, N, K, flags, yp,
                                           _stream(Xq.device)), "rrs_w4a4_gemm_per_channel")
    return out


def reorder_workspace_bytes(M: int, K: int, g: int) -> int:
    return lib().rrs_reorder_workspace_bytes(M, K, g)


def linear_reorder_workspace_bytes(M: int, K: int, g: int) -> int:
    return lib().rrs_linear_reorder_workspace_bytes(M, K, g)


def rotate_smooth_quant_reorder(X: torch.Tensor, g: int, workspace: Optional[torch.Tensor] = None,
                                out=None, flags: int = 0):
    """Runtime reorder variant: X M x K fp16 -> (Xq, a_scale, s_group, block_order K/32 int32)."""
    M, K = X.shape
    xp = _dev(X, "X", torch.float16, (M, K))
    if out is None:
        Xq = torch.empty((M, K // 2), dtype=torch.uint8, device=X.device)
        a = torch.empty((M,), dtype=torch.float32, device=X.device)
        s = torch.empty((max(K // g, 1),), dtype=torch.float32, device=X.device)
        order = torch.empty((max(K // REORDER_BLOCK, 1),), dtype=torch.int32, device=X.device)
    else:
        Xq, a, s, order = out
    nbytes = reorder_workspace_bytes(M, K, g)
    if workspace is None:
        workspace = torch.zeros((max(nbytes, 1),), dtype=torch.uint8, device=X.device)
    _check(lib().rrs_rotate_smooth_quant_reorder(
        xp, M, K, g, flags, Xq.data_ptr(), a.data_ptr(), s.data_ptr(), order.data_ptr(),
        workspace.data_ptr(), workspace.numel() * workspace.element_size(), _stream(X.device)),
        "rrs_rotate_smooth_quant_reorder")
    return Xq, a, s, order


def w4a4_gemm_reorder(Xq: torch.Tensor, a_scale: torch.Tensor, s_group: torch.Tensor,
                      Wq: torch.Tensor, w_scale: torch.Tensor, block_order: torch.Tensor, g: int,
                      out: Optional[torch.Tensor] = None, flags: int = 0) -> torch.Tensor:
    """GEMM pairing position block p of Xq with block block_order[p] of every Wq row."""
    M, Kh = Xq.shape
    K = 2 * Kh
    N = Wq.shape[0]
    args = (_dev(Xq, "Xq", torch.uint8, (M, Kh)), _dev(a_scale, "a_scale", torch.float32, (M,)),
            _dev(s_group, "s_group", torch.float32, (K // g,)),
            _dev(Wq, "Wq", torch.uint8, (N, Kh)), _dev(w_scale, "w_scale", torch.float32, (N,)),
            _dev(block_order, "block_order", torch.int32, (K // REORDER_BLOCK,)))
    Y = out if out is not None else torch.empty((M, N), dtype=torch.float16, device=Xq.device)
    yp = _dev(Y, "Y", torch.float16, (M, N))
    _check(lib().rrs_w4a4_gemm_reorder(*args, M, N, K, g, flags, yp, _stream(Xq.device)),
           "rrs_w4a4_gemm_reorder")
    return Y


def linear_reorder(X: torch.Tensor, Wq: torch.Tensor, w_scale: torch.Tensor, g: int,
                   workspace: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                   flags: int = 0) -> torch.Tensor:
    """One RRS linear layer with the runtime reorder: X M x K fp16 -> Y M x N fp16."""
    M, K = X.shape
    N = Wq.shape[0]
    xp = _dev(X, "X", torch.float16, (M, K))
    wqp = _dev(Wq, "Wq", torch.uint8, (N, K // 2))
    wsp = _dev(w_scale, "w_scale", torch.float32, (N,))
    nbytes = linear_reorder_workspace_bytes(M, K, g)
    if workspace is None:
        workspace = torch.zeros((max(nbytes, 1),), dtype=torch.uint8, device=X.device)
    Y = out if out is not None else torch.empty((M, N), dtype=torch.float16, device=X.device)
    yp = _dev(Y, "Y", torch.float16, (M, N))
    _check(lib().rrs_linear_reorder(xp, wqp, wsp, M, N, K, g, flags, yp, workspace.data_ptr(),
                                    workspace.numel() * workspace.element_size(),
                                    _stream(X.device)), "rrs_linear_reorder")
    return Y
