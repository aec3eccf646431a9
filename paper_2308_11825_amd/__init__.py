"""Python binding of libagcn (the MI355X Accel-GCN aggregation SpMM).

Argument marshalling only: every step of the path runs in the library's HIP
kernels. PyTorch supplies device memory and the current stream. The
low-level functions carry the C names of ``include/agcn.h``; ``Plan`` wraps
them for torch tensors.

The library must have been built (``python -m paper_2308_11825_amd.build``);
there is no fallback of any kind: if ``libagcn.so`` is missing, importing the
functions that need it raises.
"""
from __future__ import annotations

import ctypes
import os

__all__ = [
    "LIB_PATH", "AgcnError", "load_library", "agcn_default_params", "agcn_plan_create",
    "agcn_spmm_workspace_size", "agcn_spmm", "agcn_spmm_timed", "agcn_plan_info",
    "agcn_plan_export", "agcn_plan_destroy", "agcn_status_string", "agcn_last_error",
    "agcn_release_cached_memory", "agcn_spmm_ex", "agcn_linear", "agcn_gcn_workspace_size",
    "agcn_gcn_layer", "agcn_spmm_noalloc", "AGCN_NOALLOC_MAX_WORKSPACE", "Plan", "linear",
    "PlanParams", "PlanStats", "EXPORTED_SYMBOLS",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libagcn.so")

EXPORTED_SYMBOLS = [
    "agcn_default_params", "agcn_plan_create", "agcn_spmm_workspace_size", "agcn_spmm",
    "agcn_spmm_timed", "agcn_plan_info", "agcn_plan_export", "agcn_plan_destroy",
    "agcn_status_string", "agcn_last_error", "agcn_release_cached_memory", "agcn_spmm_ex",
    "agcn_linear", "agcn_gcn_workspace_size", "agcn_gcn_layer", "agcn_spmm_noalloc",
]

AGCN_OK = 0
AGCN_ERR_INVALID_ARGUMENT = 1
AGCN_ERR_INVALID_INPUT = 2
AGCN_ERR_UNSUPPORTED = 3
AGCN_ERR_OUT_OF_MEMORY = 4
AGCN_ERR_HIP = 5

AGCN_PLAN_WARP_LEVEL = 0x1
AGCN_PLAN_COLUMN_LOOP = 0x2

AGCN_NOALLOC_MAX_WORKSPACE = 64 << 20

AGCN_EPILOGUE_NONE = 0
AGCN_EPILOGUE_RELU = 1
_EPILOGUES = {None: AGCN_EPILOGUE_NONE, "none": AGCN_EPILOGUE_NONE, "relu": AGCN_EPILOGUE_RELU}


class PlanParams(ctypes.Structure):
    _fields_ = [("max_block_waves", ctypes.c_int32), ("max_wave_nzs", ctypes.c_int32),
                ("hub_chunk_nnz", ctypes.c_int32), ("flags", ctypes.c_uint32)]


class PlanStats(ctypes.Structure):
    _fields_ = [("n_rows", ctypes.c_int32), ("n_cols", ctypes.c_int32), ("nnz", ctypes.c_int64),
                ("n_entries", ctypes.c_int64), ("hub_first_entry", ctypes.c_int64),
                ("n_hub_chunks", ctypes.c_int64), ("n_hub_rows", ctypes.c_int32),
                ("hub_first_row", ctypes.c_int32), ("deg_bound", ctypes.c_int32),
                ("hub_chunk_nnz", ctypes.c_int32), ("max_deg", ctypes.c_int32),
                ("max_block_waves", ctypes.c_int32), ("max_wave_nzs", ctypes.c_int32),
                ("flags", ctypes.c_uint32), ("device_bytes", ctypes.c_size_t),
                ("hub_windows", ctypes.c_int32)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


class AgcnError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{_STATUS.get(status, status)}: {message}")
        self.status = status


_STATUS = {0: "AGCN_OK", 1: "AGCN_ERR_INVALID_ARGUMENT", 2: "AGCN_ERR_INVALID_INPUT",
           3: "AGCN_ERR_UNSUPPORTED", 4: "AGCN_ERR_OUT_OF_MEMORY", 5: "AGCN_ERR_HIP"}

_lib = None
_vp = ctypes.c_void_p


def _hip_runtimes_loaded():
    try:
        with open("/proc/self/maps") as f:
            maps = f.read()
    except OSError:
        return []
    import re
    return sorted(set(re.findall(r"(/\S*libamdhip64\.so[.0-9]*)", maps)))


def load_library(path: str | None = None):
    """Load libagcn.so (raises if it has not been built).

    PyTorch ships its own HIP runtime with the same SONAME as ROCm's. Loading
    torch first makes libagcn bind to that runtime, so torch's streams and
    allocations are valid in the library; two runtimes in one process would
    not share them, so that case raises.
    """
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise ImportError(f"{p} is missing: build it with `python -m paper_2308_11825_amd.build`")
    try:
        import torch  # noqa: F401  (binds the HIP runtime first)
    except ImportError:
        pass
    lib = ctypes.CDLL(p)
    runtimes = _hip_runtimes_loaded()
    if len(runtimes) > 1:
        raise ImportError(f"two HIP runtimes loaded in one process: {runtimes}; import torch "
                          "before loading libagcn")
    lib.agcn_default_params.argtypes = [ctypes.POINTER(PlanParams)]
    lib.agcn_default_params.restype = None
    lib.agcn_plan_create.argtypes = [ctypes.POINTER(_vp), ctypes.c_int32, ctypes.c_int32,
                                     ctypes.c_int64, _vp, _vp, _vp, ctypes.POINTER(PlanParams), _vp]
    lib.agcn_plan_create.restype = ctypes.c_int
    lib.agcn_spmm_workspace_size.argtypes = [_vp, ctypes.c_int32, ctypes.POINTER(ctypes.c_size_t)]
    lib.agcn_spmm_workspace_size.restype = ctypes.c_int
    lib.agcn_spmm.argtypes = [_vp, ctypes.c_int32, _vp, ctypes.c_int64, _vp, ctypes.c_int64, _vp,
                              _vp]
    lib.agcn_spmm.restype = ctypes.c_int
    lib.agcn_spmm_timed.argtypes = [_vp, ctypes.c_int32, _vp, ctypes.c_int64, _vp, ctypes.c_int64,
                                    _vp, _vp, _vp, _vp, _vp]
    lib.agcn_spmm_timed.restype = ctypes.c_int
    lib.agcn_spmm_ex.argtypes = [_vp, ctypes.c_int32, _vp, ctypes.c_int64, _vp, ctypes.c_int64,
                                 _vp, _vp, ctypes.c_int32]
    lib.agcn_spmm_ex.restype = ctypes.c_int
    lib.agcn_spmm_noalloc.argtypes = [_vp, ctypes.c_int32, _vp, ctypes.c_int64, _vp,
                                      ctypes.c_int64, _vp, ctypes.c_int32]
    lib.agcn_spmm_noalloc.restype = ctypes.c_int
    lib.agcn_linear.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, _vp,
                                ctypes.c_int64, _vp, ctypes.c_int64, _vp, ctypes.c_int64, _vp]
    lib.agcn_linear.restype = ctypes.c_int
    lib.agcn_gcn_workspace_size.argtypes = [_vp, ctypes.c_int32, ctypes.POINTER(ctypes.c_size_t)]
    lib.agcn_gcn_workspace_size.restype = ctypes.c_int
    lib.agcn_gcn_layer.argtypes = [_vp, ctypes.c_int32, ctypes.c_int32, _vp, ctypes.c_int64, _vp,
                                   ctypes.c_int64, _vp, ctypes.c_int64, _vp, _vp, ctypes.c_int32]
    lib.agcn_gcn_layer.restype = ctypes.c_int
    lib.agcn_plan_info.argtypes = [_vp, ctypes.POINTER(PlanStats)]
    lib.agcn_plan_info.restype = ctypes.c_int
    lib.agcn_plan_export.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp]
    lib.agcn_plan_export.restype = ctypes.c_int
    lib.agcn_plan_destroy.argtypes = [_vp]
    lib.agcn_plan_destroy.restype = None
    lib.agcn_release_cached_memory.argtypes = []
    lib.agcn_release_cached_memory.restype = None
    lib.agcn_status_string.argtypes = [ctypes.c_int]
    lib.agcn_status_string.restype = ctypes.c_char_p
    lib.agcn_last_error.argtypes = []
    lib.agcn_last_error.restype = ctypes.c_char_p
    if path is None:
        _lib = lib
    return lib


def _check(rc):
    if rc != AGCN_OK:
        raise AgcnError(rc, agcn_last_error())


# ---- same-name wrappers of the C ABI (integers are raw device/host addresses) ----

def agcn_default_params() -> PlanParams:
    p = PlanParams()
    load_library().agcn_default_params(ctypes.byref(p))
    return p


def agcn_plan_create(n_rows, n_cols, nnz, d_rowptr, d_colidx, d_vals, params=None, stream=0):
    """Returns the plan handle (int). Raises AgcnError on failure."""
    h = _vp()
    prm = ctypes.byref(params) if params is not None else None
    _check(load_library().agcn_plan_create(ctypes.byref(h), n_rows, n_cols, nnz, d_rowptr, d_colidx,
                                           d_vals, prm, stream))
    return h.value


def agcn_spmm_workspace_size(plan, F) -> int:
    n = ctypes.c_size_t()
    _check(load_library().agcn_spmm_workspace_size(plan, F, ctypes.byref(n)))
    return n.value


def agcn_spmm(plan, F, d_X, ldx, d_Y, ldy, d_ws=None, stream=0):
    _check(load_library().agcn_spmm(plan, F, d_X, ldx, d_Y, ldy, d_ws, stream))


def agcn_spmm_timed(plan, F, d_X, ldx, d_Y, ldy, d_ws, stream, ev_begin, ev_mid, ev_end):
    _check(load_library().agcn_spmm_timed(plan, F, d_X, ldx, d_Y, ldy, d_ws, stream, ev_begin,
                                          ev_mid, ev_end))


def agcn_spmm_ex(plan, F, d_X, ldx, d_Y, ldy, d_ws, stream, epilogue):
    _check(load_library().agcn_spmm_ex(plan, F, d_X, ldx, d_Y, ldy, d_ws, stream, epilogue))


def agcn_spmm_noalloc(plan, F, d_X, ldx, d_Y, ldy, stream, epilogue=AGCN_EPILOGUE_NONE):
    _check(load_library().agcn_spmm_noalloc(plan, F, d_X, ldx, d_Y, ldy, stream, epilogue))


def agcn_linear(n, fin, fout, d_X, ldx, d_W, ldw, d_H, ldh, stream=0):
    _check(load_library().agcn_linear(n, fin, fout, d_X, ldx, d_W, ldw, d_H, ldh, stream))


def agcn_gcn_workspace_size(plan, fout) -> int:
    n = ctypes.c_size_t()
    _check(load_library().agcn_gcn_workspace_size(plan, fout, ctypes.byref(n)))
    return n.value


def agcn_gcn_layer(plan, fin, fout, d_X, ldx, d_W, ldw, d_Y, ldy, d_ws, stream, epilogue):
    _check(load_library().agcn_gcn_layer(plan, fin, fout, d_X, ldx, d_W, ldw, d_Y, ldy, d_ws,
                                         stream, epilogue))


def agcn_plan_info(plan) -> PlanStats:
    s = PlanStats()
    _check(load_library().agcn_plan_info(plan, ctypes.byref(s)))
    return s


def agcn_plan_export(plan, h_perm=None, h_rowptr_s=None, h_colidx_s=None, h_vals_s=None,
                     h_meta=None):
    _check(load_library().agcn_plan_export(plan, h_perm, h_rowptr_s, h_colidx_s, h_vals_s, h_meta))


def agcn_plan_destroy(plan):
    load_library().agcn_plan_destroy(plan)


def agcn_release_cached_memory():
    load_library().agcn_release_cached_memory()


def agcn_status_string(status) -> str:
    return load_library().agcn_status_string(status).decode()


def agcn_last_error() -> str:
    return load_library().agcn_last_error().decode()


# ---- torch-facing wrapper ----

def _stream_handle(device):
    import torch
    return torch.cuda.current_stream(device).cuda_stream


def _unit_col_stride(t):
    return t.shape[1] <= 1 or t.shape[0] == 0 or t.stride(1) == 1


def _row_stride(t):
    """Row stride in elements; any value >= F is valid for 0 or 1 rows."""
    return t.stride(0) if t.shape[0] > 1 else max(t.shape[1], t.stride(0))


class Plan:
    """A degree-sorted, block-partitioned CSR matrix on one GPU.

    ``Plan(rowptr, colidx, vals, n_cols=None, max_block_waves=..., max_wave_nzs=...,
    hub_chunk_nnz=0)`` with int32 / int32 / float32 CUDA tensors; ``plan.spmm(X)``
    returns ``A @ X`` for a float32 CUDA tensor X of shape (n_cols, F).
    """

    def __init__(self, rowptr, colidx, vals, n_cols=None, max_block_waves=None,
                 max_wave_nzs=None, hub_chunk_nnz=None, flags=0, stream=None):
        import torch
        for name, t, dt in (("rowptr", rowptr, torch.int32), ("colidx", colidx, torch.int32),
                            ("vals", vals, torch.float32)):
            if not isinstance(t, torch.Tensor) or t.device.type != "cuda" or t.dtype != dt:
                raise TypeError(f"{name} must be a CUDA tensor of dtype {dt}")
            if t.dim() != 1 or not t.is_contiguous():
                raise ValueError(f"{name} must be 1-D and contiguous")
        self.device = rowptr.device
        self.n_rows = rowptr.numel() - 1
        self.n_cols = self.n_rows if n_cols is None else int(n_cols)
        self.nnz = colidx.numel()
        if vals.numel() != self.nnz:
            raise ValueError("colidx and vals differ in length")
        prm = agcn_default_params()
        if max_block_waves is not None:
            prm.max_block_waves = max_block_waves
        if max_wave_nzs is not None:
            prm.max_wave_nzs = max_wave_nzs
        if hub_chunk_nnz is not None:
            prm.hub_chunk_nnz = hub_chunk_nnz
        prm.flags = flags
        self.params = prm
        self._handle = None
        with torch.cuda.device(self.device):
            st = stream.cuda_stream if stream is not None else _stream_handle(self.device)
            self._handle = agcn_plan_create(self.n_rows, self.n_cols, self.nnz, rowptr.data_ptr(),
                                            colidx.data_ptr() if self.nnz else None,
                                            vals.data_ptr() if self.nnz else None, prm, st)
            # The plan's last kernel may still read the inputs: on another
            # stream, torch's allocator must not reuse their memory before it.
            if stream is not None:
                for t in (rowptr, colidx, vals):
                    t.record_stream(stream)
        self.stats = agcn_plan_info(self._handle)
        self._ws = {}

    @property
    def handle(self):
        if self._handle is None:
            raise RuntimeError("plan destroyed")
        return self._handle

    def workspace_bytes(self, F: int) -> int:
        return agcn_spmm_workspace_size(self.handle, F)

    def workspace(self, F: int, stream=None):
        """A cached device workspace for feature width F on `stream` (None if
        not needed). One per stream, so executes on different streams never
        share hub-row partials."""
        import torch
        nb = self.workspace_bytes(F)
        if nb == 0:
            return None
        key = (F, stream.cuda_stream if stream is not None else _stream_handle(self.device))
        ws = self._ws.get(key)
        if ws is None:
            # allocated on the stream that uses it, so torch's allocator orders
            # any later reuse of the memory after that stream's work
            with torch.cuda.stream(stream if stream is not None else torch.cuda.current_stream(self.device)):
                ws = torch.empty((nb + 3) // 4, dtype=torch.float32, device=self.device)
            self._ws[key] = ws
        return ws

    def spmm(self, X, out=None, ws=None, stream=None, act=None):
        """A @ X, with act ("relu") applied where Y is written."""
        import torch
        if not isinstance(X, torch.Tensor) or X.device != self.device or X.dtype != torch.float32:
            raise TypeError("X must be a float32 tensor on the plan's device")
        if X.dim() != 2 or X.shape[0] != self.n_cols or not _unit_col_stride(X):
            raise ValueError("X must be (n_cols, F) with unit column stride")
        F = X.shape[1]
        if F < 1:
            raise ValueError("F must be >= 1")
        if out is None:
            out = torch.empty((self.n_rows, F), dtype=torch.float32, device=self.device)
        if (tuple(out.shape) != (self.n_rows, F) or not _unit_col_stride(out)
                or out.dtype != torch.float32 or out.device != self.device):
            raise ValueError("out must be a float32 (n_rows, F) tensor with unit column stride")
        if ws is None:
            ws = self.workspace(F, stream)
        st = stream.cuda_stream if stream is not None else _stream_handle(self.device)
        with torch.cuda.device(self.device):
            agcn_spmm_ex(self.handle, F, X.data_ptr(), _row_stride(X), out.data_ptr(),
                         _row_stride(out), ws.data_ptr() if ws is not None else None, st,
                         _EPILOGUES[act])
        return out

    def gcn_layer(self, X, W, act="relu", out=None, ws=None, stream=None):
        """One GCNConv forward: act(A @ (X @ W)), X (n_cols, fin), W (fin, fout)."""
        import torch
        for name, t in (("X", X), ("W", W)):
            if (not isinstance(t, torch.Tensor) or t.device != self.device
                    or t.dtype != torch.float32 or t.dim() != 2 or not _unit_col_stride(t)):
                raise TypeError(f"{name} must be a 2-D float32 tensor on the plan's device with "
                                "unit column stride")
        fin, fout = W.shape
        if X.shape != (self.n_cols, fin):
            raise ValueError("X must be (n_cols, fin) with fin = W.shape[0]")
        if out is None:
            out = torch.empty((self.n_rows, fout), dtype=torch.float32, device=self.device)
        if (tuple(out.shape) != (self.n_rows, fout) or not _unit_col_stride(out)
                or out.dtype != torch.float32 or out.device != self.device):
            raise ValueError("out must be a float32 (n_rows, fout) tensor with unit column stride")
        if ws is None:
            nb = agcn_gcn_workspace_size(self.handle, fout)
            with torch.cuda.stream(stream if stream is not None else torch.cuda.current_stream(self.device)):
                ws = torch.empty((nb + 3) // 4, dtype=torch.float32, device=self.device)
        st = stream.cuda_stream if stream is not None else _stream_handle(self.device)
        with torch.cuda.device(self.device):
            agcn_gcn_layer(self.handle, fin, fout, X.data_ptr(), _row_stride(X), W.data_ptr(),
                           _row_stride(W), out.data_ptr(), _row_stride(out), ws.data_ptr(), st,
                           _EPILOGUES[act])
        return out

    def export(self):
        """Host copies: dict(perm, rowptr_s, colidx_s, vals_s, meta (n_entries x 4))."""
        import numpy as np
        s = self.stats
        perm = np.empty(s.n_rows, np.int32)
        rowptr_s = np.empty(s.n_rows + 1, np.int32)
        colidx_s = np.empty(s.nnz, np.int32)
        vals_s = np.empty(s.nnz, np.float32)
        meta = np.empty((s.n_entries, 4), np.int32)
        import torch
        with torch.cuda.device(self.device):
            agcn_plan_export(self.handle, perm.ctypes.data, rowptr_s.ctypes.data,
                             colidx_s.ctypes.data, vals_s.ctypes.data, meta.ctypes.data)
        return dict(perm=perm, rowptr_s=rowptr_s, colidx_s=colidx_s, vals_s=vals_s, meta=meta)

    def destroy(self):
        if self._handle is not None:
            agcn_plan_destroy(self._handle)
            self._handle = None
        self._ws = {}

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


def linear(X, W, out=None, stream=None):
    """X @ W on the matrix cores: X (n, fin), W (fin, fout), float32 CUDA tensors."""
    import torch
    for name, t in (("X", X), ("W", W)):
        if (not isinstance(t, torch.Tensor) or t.device.type != "cuda" or t.dtype != torch.float32
                or t.dim() != 2 or not _unit_col_stride(t)):
            raise TypeError(f"{name} must be a 2-D float32 CUDA tensor with unit column stride")
    n, fin = X.shape
    if W.shape[0] != fin or W.device != X.device:
        raise ValueError("W must be (fin, fout) on X's device")
    fout = W.shape[1]
    if out is None:
        out = torch.empty((n, fout), dtype=torch.float32, device=X.device)
    if tuple(out.shape) != (n, fout) or not _unit_col_stride(out) or out.dtype != torch.float32:
        raise ValueError("out must be a float32 (n, fout) tensor with unit column stride")
    st = stream.cuda_stream if stream is not None else _stream_handle(X.device)
    with torch.cuda.device(X.device):
        agcn_linear(n, fin, fout, X.data_ptr(), _row_stride(X), W.data_ptr(), _row_stride(W),
                    out.data_ptr(), _row_stride(out), st)
    return out
