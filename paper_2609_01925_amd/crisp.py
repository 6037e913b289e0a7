"""Python binding of libcrisp (include/crisp.h): argument marshalling only.

Every function takes torch tensors that already live on the GPU, passes their
device pointers and the current HIP stream to the C entry point of the same
name, and returns the output tensors it allocated.  All computation happens in
the HIP kernels of libcrisp.so; if the library is missing, importing this
module raises -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Tuple

import torch

# CRISP_DEBUG=1 in the environment loads the debug build, which also checks the inputs on
# the device (non-finite values, malformed caller lists) and waits for the stream to do so.
_LIB_DIR = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_LIB_DIR, "libcrisp_debug.so" if os.environ.get("CRISP_DEBUG") == "1" else "libcrisp.so")
DEBUG_LIB_PATH = os.path.join(_LIB_DIR, "libcrisp_debug.so")

CRISP_OK, CRISP_EINVAL, CRISP_EUNSUPPORTED, CRISP_EHIP = 0, 1, 2, 3
ROUTE_VS, ROUTE_PE = 0, 1


class CrispShape(ctypes.Structure):
    _fields_ = [("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32), ("seq_len", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("block", ctypes.c_int32)]


class CrispParams(ctypes.Structure):
    _fields_ = [("alpha", ctypes.c_float), ("tau_proxy", ctypes.c_float), ("gamma", ctypes.c_float),
                ("w_sink", ctypes.c_int32), ("w_local", ctypes.c_int32), ("k_min_blocks", ctypes.c_int32),
                ("softmax_scale", ctypes.c_float), ("route_mode", ctypes.c_int32), ("vs_mode", ctypes.c_int32),
                ("tau_jsd", ctypes.c_float), ("floor_mode", ctypes.c_int32), ("dense_below_len", ctypes.c_int32)]


class CrispError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} (status {status})")
        self.status = status


def _load(path: str = _LIB_PATH):
    if not os.path.exists(path):
        raise ImportError(f"libcrisp.so not built at {path}; run `python -m paper_2609_01925_amd.build`")
    lib = ctypes.CDLL(path)
    P, F, I32, I64, SZ = ctypes.c_void_p, ctypes.c_float, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    sh, pa = ctypes.POINTER(CrispShape), ctypes.POINTER(CrispParams)
    sig = {
        "crisp_params_default": (None, [pa]),
        "crisp_col_capacity": (I64, [sh]),
        "crisp_workspace_size": (ctypes.c_int, [sh, ctypes.POINTER(SZ)]),
        "crisp_prefill_workspace_size": (ctypes.c_int, [sh, ctypes.POINTER(SZ)]),
        "crisp_estimate": (ctypes.c_int, [sh, pa, P, P, P, P, P, P, SZ, P]),
        "crisp_jsd": (ctypes.c_int, [sh, pa, P, P, P, P, P, SZ, P]),
        "crisp_route_select": (ctypes.c_int, [sh, pa, P, P, P, P, P, P, P, P, I64, P, P, SZ, P]),
        "crisp_sparse_workspace_size": (ctypes.c_int, [sh, ctypes.POINTER(SZ)]),
        "crisp_sparse_attn": (ctypes.c_int, [sh, F, P, P, P, P, P, I64, P, P, SZ, P]),
        "crisp_sparse_attn_noalloc": (ctypes.c_int, [sh, F, P, P, P, P, P, I64, P, P]),
        "crisp_prefill_attn": (ctypes.c_int, [sh, pa, P, P, P, P, P, P, P, P, SZ, P]),
        "crisp_dense_attn": (ctypes.c_int, [sh, F, P, P, P, P, P]),
        "crisp_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "crisp_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load()
EXPORTED = ("crisp_params_default", "crisp_col_capacity", "crisp_workspace_size", "crisp_prefill_workspace_size",
            "crisp_sparse_workspace_size", "crisp_estimate", "crisp_jsd", "crisp_route_select", "crisp_sparse_attn",
            "crisp_sparse_attn_noalloc", "crisp_prefill_attn", "crisp_dense_attn", "crisp_status_string", "crisp_last_error")

# route_mode / vs_mode values (include/crisp.h)
ROUTE_BY_CSTRUCT, ROUTE_BY_JSD = 0, 1
VS_FLOOR, VS_GAMMA = 0, 1
FLOOR_MEAN, FLOOR_MEDIAN = 0, 1


def _check(status: int, what: str):
    if status != CRISP_OK:
        msg = lib.crisp_last_error().decode()
        raise CrispError(status, f"{what}: {lib.crisp_status_string(status).decode()}: {msg}")


def make_params(alpha=1.0, tau_proxy=0.2, gamma=0.95, w_sink=128, w_local=128, k_min_blocks=0,
                softmax_scale=0.0, route_mode=ROUTE_BY_CSTRUCT, vs_mode=VS_FLOOR, tau_jsd=0.1,
                floor_mode=FLOOR_MEAN, dense_below_len=0) -> CrispParams:
    return CrispParams(alpha, tau_proxy, gamma, w_sink, w_local, k_min_blocks, softmax_scale, route_mode, vs_mode,
                       tau_jsd, floor_mode, dense_below_len)


def flexprefill_params(gamma=0.95, tau_jsd=0.1, **kw) -> CrispParams:
    """The FlexPrefill comparator (App. A): JSD routing and gamma-coverage VS selection."""
    return make_params(gamma=gamma, tau_jsd=tau_jsd, route_mode=ROUTE_BY_JSD, vs_mode=VS_GAMMA, **kw)


def crisp_params_default() -> CrispParams:
    p = CrispParams()
    lib.crisp_params_default(ctypes.byref(p))
    return p


def shape_of(q: torch.Tensor, k: torch.Tensor, block: int) -> CrispShape:
    return CrispShape(q.shape[0], k.shape[0], q.shape[1], q.shape[2], block)


def n_blocks(n: int, block: int) -> int:
    return -(-n // block)


def crisp_col_capacity(shape: CrispShape) -> int:
    return int(lib.crisp_col_capacity(ctypes.byref(shape)))


def crisp_workspace_size(shape: CrispShape) -> int:
    b = ctypes.c_size_t()
    _check(lib.crisp_workspace_size(ctypes.byref(shape), ctypes.byref(b)), "crisp_workspace_size")
    return int(b.value)


def crisp_prefill_workspace_size(shape: CrispShape) -> int:
    b = ctypes.c_size_t()
    _check(lib.crisp_prefill_workspace_size(ctypes.byref(shape), ctypes.byref(b)), "crisp_prefill_workspace_size")
    return int(b.value)


def crisp_sparse_workspace_size(shape: CrispShape) -> int:
    b = ctypes.c_size_t()
    _check(lib.crisp_sparse_workspace_size(ctypes.byref(shape), ctypes.byref(b)), "crisp_sparse_workspace_size")
    return int(b.value)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _inputs(q: torch.Tensor, k: torch.Tensor, v: Optional[torch.Tensor] = None):
    """q [H_q, n, d], k and v [H_kv, n, d]: contiguous bf16 on one CUDA device.  The C ABI
    sees only pointers, so every size it will read is checked here."""
    ts = (q, k) if v is None else (q, k, v)
    for t in ts:
        if not (t.is_cuda and t.dtype == torch.bfloat16 and t.is_contiguous() and t.dim() == 3):
            raise ValueError("q, k, v must be contiguous 3-d bf16 CUDA tensors [heads, seq, head_dim]")
        if t.device != q.device:
            raise ValueError("q, k, v must be on one device")
    if k.shape[1:] != q.shape[1:]:
        raise ValueError(f"k {tuple(k.shape)} does not match q {tuple(q.shape)} in seq_len and head_dim")
    if v is not None and v.shape != k.shape:
        raise ValueError(f"v {tuple(v.shape)} must have k's shape {tuple(k.shape)}")


def _tensor(t: torch.Tensor, name: str, dtype, shape, device):
    """A caller-given buffer: contiguous, of the given dtype and shape (None: any size in that
    dimension) on the given device."""
    ok = t.is_cuda and t.device == device and t.dtype == dtype and t.is_contiguous() and t.dim() == len(shape)
    ok = ok and all(w is None or t.shape[i] == w for i, w in enumerate(shape))
    if not ok:
        raise ValueError(f"{name} must be a contiguous {dtype} CUDA tensor of shape {shape} on {device}, "
                         f"got {t.dtype} {tuple(t.shape)} on {t.device}")


def _tensor_out(out: torch.Tensor, q: torch.Tensor) -> torch.Tensor:
    _tensor(out, "out", torch.bfloat16, tuple(q.shape), q.device)
    return out


def _ws(ws: torch.Tensor, device) -> torch.Tensor:
    _tensor(ws, "ws", torch.uint8, (None,), device)
    return ws


def workspace(shape: CrispShape, device, prefill: bool = False) -> torch.Tensor:
    nbytes = crisp_prefill_workspace_size(shape) if prefill else crisp_workspace_size(shape)
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)


def crisp_estimate(q: torch.Tensor, k: torch.Tensor, params: CrispParams, block: int = 128,
                   ws: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """Stages 1-2 -> (c_struct [H_q], p_v [H_q, N_b], p_s [H_q, N_b]) float32."""
    _inputs(q, k)
    sh = shape_of(q, k, block)
    nb = n_blocks(q.shape[1], block)
    dev = q.device
    cs = torch.empty(q.shape[0], dtype=torch.float32, device=dev)
    pv = torch.empty(q.shape[0], nb, dtype=torch.float32, device=dev)
    ps = torch.empty(q.shape[0], nb, dtype=torch.float32, device=dev)
    ws = workspace(sh, dev) if ws is None else _ws(ws, dev)
    _check(lib.crisp_estimate(ctypes.byref(sh), ctypes.byref(params), _ptr(q), _ptr(k), _ptr(cs), _ptr(pv), _ptr(ps),
                              _ptr(ws), ws.numel(), _stream(dev)), "crisp_estimate")
    return cs, pv, ps


def crisp_jsd(q: torch.Tensor, k: torch.Tensor, p_v: torch.Tensor, params: CrispParams, block: int = 128,
              ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """FlexPrefill's pattern search (App. A) -> D_JS per query head, float32 [H_q]."""
    _inputs(q, k)
    sh = shape_of(q, k, block)
    dev = q.device
    _tensor(p_v, "p_v", torch.float32, (q.shape[0], n_blocks(q.shape[1], block)), dev)
    jsd = torch.empty(q.shape[0], dtype=torch.float32, device=dev)
    ws = workspace(sh, dev) if ws is None else _ws(ws, dev)
    _check(lib.crisp_jsd(ctypes.byref(sh), ctypes.byref(params), _ptr(q), _ptr(k), _ptr(p_v), _ptr(jsd), _ptr(ws),
                         ws.numel(), _stream(dev)), "crisp_jsd")
    return jsd


def crisp_route_select(q: torch.Tensor, k: torch.Tensor, c_struct: torch.Tensor, p_v: torch.Tensor,
                       p_s: torch.Tensor, params: CrispParams, block: int = 128, want_mask: bool = True,
                       ws: Optional[torch.Tensor] = None):
    """Stage 3 -> (route int8 [H_q], row_ptr int32 [H_q, N_b+1], col_idx int32 [H_q, cap],
    dir_mask uint8 [H_q, 2, N_b] or None).  c_struct is the route score: C_struct, or D_JS
    from crisp_jsd when params.route_mode is ROUTE_BY_JSD."""
    _inputs(q, k)
    sh = shape_of(q, k, block)
    nb = n_blocks(q.shape[1], block)
    dev = q.device
    _tensor(c_struct, "c_struct", torch.float32, (q.shape[0],), dev)
    _tensor(p_v, "p_v", torch.float32, (q.shape[0], nb), dev)
    _tensor(p_s, "p_s", torch.float32, (q.shape[0], nb), dev)
    cap = max(crisp_col_capacity(sh), 1)
    route = torch.empty(q.shape[0], dtype=torch.int8, device=dev)
    row_ptr = torch.empty(q.shape[0], nb + 1, dtype=torch.int32, device=dev)
    col_idx = torch.empty(q.shape[0], cap, dtype=torch.int32, device=dev)
    dmask = torch.empty(q.shape[0], 2, nb, dtype=torch.uint8, device=dev) if want_mask else None
    ws = workspace(sh, dev) if ws is None else _ws(ws, dev)
    _check(lib.crisp_route_select(ctypes.byref(sh), ctypes.byref(params), _ptr(q), _ptr(k), _ptr(c_struct),
                                  _ptr(p_v), _ptr(p_s), _ptr(route), _ptr(row_ptr), _ptr(col_idx), cap,
                                  _ptr(dmask), _ptr(ws), ws.numel(), _stream(dev)), "crisp_route_select")
    return route, row_ptr, col_idx, dmask


def crisp_sparse_attn(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, row_ptr: torch.Tensor,
                      col_idx: torch.Tensor, block: int = 128, softmax_scale: float = 0.0,
                      out: Optional[torch.Tensor] = None, balance: bool = True,
                      ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Stage 4 over caller-given CSR lists -> o bf16 [H_q, n, d].  balance=False passes no
    workspace (fixed row order)."""
    _inputs(q, k, v)
    sh = shape_of(q, k, block)
    _tensor(row_ptr, "row_ptr", torch.int32, (q.shape[0], n_blocks(q.shape[1], block) + 1), q.device)
    _tensor(col_idx, "col_idx", torch.int32, (q.shape[0], None), q.device)
    o = torch.empty_like(q) if out is None else _tensor_out(out, q)
    if balance and ws is not None:
        _ws(ws, q.device)
    if balance and ws is None:
        ws = torch.empty(max(crisp_sparse_workspace_size(sh), 256), dtype=torch.uint8, device=q.device)
    if not balance:
        ws = None
    _check(lib.crisp_sparse_attn(ctypes.byref(sh), softmax_scale, _ptr(q), _ptr(k), _ptr(v), _ptr(row_ptr),
                                 _ptr(col_idx), col_idx.shape[1], _ptr(o), _ptr(ws), 0 if ws is None else ws.numel(),
                                 _stream(q.device)), "crisp_sparse_attn")
    return o


def crisp_sparse_attn_noalloc(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, row_ptr: torch.Tensor,
                              col_idx: torch.Tensor, block: int = 128, softmax_scale: float = 0.0,
                              out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Stage 4 over caller-given CSR lists with the library's own static schedule area (the
    C entry point allocates nothing; calls that overlap on one GPU race) -> o bf16 [H_q, n, d]."""
    _inputs(q, k, v)
    sh = shape_of(q, k, block)
    _tensor(row_ptr, "row_ptr", torch.int32, (q.shape[0], n_blocks(q.shape[1], block) + 1), q.device)
    _tensor(col_idx, "col_idx", torch.int32, (q.shape[0], None), q.device)
    o = torch.empty_like(q) if out is None else _tensor_out(out, q)
    _check(lib.crisp_sparse_attn_noalloc(ctypes.byref(sh), softmax_scale, _ptr(q), _ptr(k), _ptr(v), _ptr(row_ptr),
                                         _ptr(col_idx), col_idx.shape[1], _ptr(o), _stream(q.device)),
           "crisp_sparse_attn_noalloc")
    return o


def crisp_dense_attn(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, block: int = 128,
                     softmax_scale: float = 0.0, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Dense causal baseline with the same kernel -> o bf16 [H_q, n, d]."""
    _inputs(q, k, v)
    sh = shape_of(q, k, block)
    o = torch.empty_like(q) if out is None else _tensor_out(out, q)
    _check(lib.crisp_dense_attn(ctypes.byref(sh), softmax_scale, _ptr(q), _ptr(k), _ptr(v), _ptr(o),
                                _stream(q.device)), "crisp_dense_attn")
    return o


def crisp_prefill_attn(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, params: CrispParams, block: int = 128,
                       return_lists: bool = False, ws: Optional[torch.Tensor] = None,
                       out: Optional[torch.Tensor] = None):
    """All stages (Alg. 1) -> o, or (o, route, row_ptr, col_idx) with return_lists."""
    _inputs(q, k, v)
    sh = shape_of(q, k, block)
    dev = q.device
    o = torch.empty_like(q) if out is None else _tensor_out(out, q)
    if ws is not None:
        _ws(ws, dev)
    if return_lists:
        nb = n_blocks(q.shape[1], block)
        cap = max(crisp_col_capacity(sh), 1)
        route = torch.empty(q.shape[0], dtype=torch.int8, device=dev)
        row_ptr = torch.empty(q.shape[0], nb + 1, dtype=torch.int32, device=dev)
        col_idx = torch.empty(q.shape[0], cap, dtype=torch.int32, device=dev)
        ws = workspace(sh, dev) if ws is None else ws
    else:
        route = row_ptr = col_idx = None
        ws = workspace(sh, dev, prefill=True) if ws is None else ws
    _check(lib.crisp_prefill_attn(ctypes.byref(sh), ctypes.byref(params), _ptr(q), _ptr(k), _ptr(v), _ptr(o),
                                  _ptr(route), _ptr(row_ptr), _ptr(col_idx), _ptr(ws), ws.numel(), _stream(dev)),
                    "crisp_prefill_attn")
    return (o, route, row_ptr, col_idx) if return_lists else o
