"""Python binding of libflexprefill (FlexPrefill sparse prefill attention for MI355X).

Argument marshalling only: tensors are passed as raw device pointers to the C ABI in
include/flexprefill.h, and every step of the method runs in the library's HIP kernels.
PyTorch supplies device memory (outputs and workspaces are allocated with torch) and the
current stream.  If the library has not been built, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
# the in-tree build; FLEXPREFILL_LIB names another build of the same library (e.g. one with
# the host code instrumented by AddressSanitizer)
LIB_PATH = os.environ.get("FLEXPREFILL_LIB") or os.path.join(_PKG, "libflexprefill.so")

FP_OK, FP_ERR_INVALID_ARG, FP_ERR_UNSUPPORTED, FP_ERR_WORKSPACE, FP_ERR_HIP = range(5)
PATTERN_QUERY_AWARE, PATTERN_VERTICAL_SLASH, PATTERN_DENSE = 0, 1, 2
MAX_BATCH = 64
MAX_MIN_BUDGET = 64


class FlexPrefillError(RuntimeError):
    def __init__(self, status: int, what: str, detail: str = ""):
        self.status = status
        super().__init__(f"{what}: status {status} {detail}".strip())


class FpShape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("cu_seqlens", ctypes.POINTER(ctypes.c_int32)),
                ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("block", ctypes.c_int32)]


class FpParams(ctypes.Structure):
    _fields_ = [("gamma", ctypes.c_float), ("tau", ctypes.c_float),
                ("min_budget_blocks", ctypes.c_int32), ("softmax_scale", ctypes.c_float),
                ("force_pattern", ctypes.c_int32), ("max_budget_blocks", ctypes.c_int32),
                ("qa_mode", ctypes.c_int32), ("vs_granularity", ctypes.c_int32)]


class FpIndices(ctypes.Structure):
    _fields_ = [("kb_idx", ctypes.c_void_p), ("kb_cnt", ctypes.c_void_p),
                ("pattern", ctypes.c_void_p), ("js", ctypes.c_void_p), ("units", ctypes.c_void_p),
                ("softmax_scale", ctypes.c_float)]


_lib_handle = None


def lib() -> ctypes.CDLL:
    """Load libflexprefill.so (raises if it has not been built)."""
    global _lib_handle
    if _lib_handle is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2502_20766_amd._build`")
        h = ctypes.CDLL(LIB_PATH)
        S, P, X = ctypes.POINTER(FpShape), ctypes.POINTER(FpParams), ctypes.POINTER(FpIndices)
        sz = ctypes.POINTER(ctypes.c_size_t)
        vp = ctypes.c_void_p
        h.fp_indices_size.argtypes = [S, sz, sz]
        h.fp_select_workspace_size.argtypes = [S, P, sz]
        h.fp_attn_workspace_size.argtypes = [S, sz]
        h.fp_validate.argtypes = [S, P, ctypes.c_size_t]
        h.fp_select.argtypes = [S, vp, vp, P, X, vp, ctypes.c_size_t, vp]
        h.fp_sparse_attn.argtypes = [S, vp, vp, vp, X, vp, vp, ctypes.c_size_t, vp]
        h.fp_sparse_attn_noalloc.argtypes = [S, vp, vp, vp, X, vp, vp]
        h.fp_status_string.argtypes = [ctypes.c_int]
        h.fp_status_string.restype = ctypes.c_char_p
        h.fp_last_error.argtypes = []
        h.fp_last_error.restype = ctypes.c_char_p
        for name in ("fp_indices_size", "fp_select_workspace_size", "fp_attn_workspace_size",
                     "fp_validate", "fp_select", "fp_sparse_attn", "fp_sparse_attn_noalloc"):
            getattr(h, name).restype = ctypes.c_int
        _lib_handle = h
    return _lib_handle


def _check(status: int, what: str):
    if status != FP_OK:
        h = lib()
        detail = h.fp_status_string(status).decode()
        if status == FP_ERR_HIP:
            detail += " (" + h.fp_last_error().decode() + ")"
        raise FlexPrefillError(status, what, detail)


class Shape:
    """fp_shape plus the host copy of cu_seqlens it points to."""

    def __init__(self, cu_seqlens, num_q_heads, num_kv_heads, head_dim, block=128):
        self.cu = np.ascontiguousarray(np.asarray(cu_seqlens, dtype=np.int32))
        self.c = FpShape(len(self.cu) - 1,
                         self.cu.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                         int(num_q_heads), int(num_kv_heads), int(head_dim), int(block))
        self.block = int(block)

    @property
    def seqlens(self):
        return np.diff(self.cu)

    def nb(self):
        return -(-self.seqlens // self.block)


def params(gamma, tau, min_budget=8, softmax_scale=0.0, force_pattern=-1, max_budget=0,
           qa_mode=0, vs_granularity=0) -> FpParams:
    return FpParams(float(gamma), float(tau), int(min_budget), float(softmax_scale),
                    int(force_pattern), int(max_budget), int(qa_mode), int(vs_granularity))


def indices_size(shape: Shape):
    a, b = ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib().fp_indices_size(ctypes.byref(shape.c), ctypes.byref(a), ctypes.byref(b)),
           "fp_indices_size")
    return a.value, b.value


def select_workspace_size(shape: Shape, p: FpParams) -> int:
    out = ctypes.c_size_t()
    _check(lib().fp_select_workspace_size(ctypes.byref(shape.c), ctypes.byref(p),
                                          ctypes.byref(out)), "fp_select_workspace_size")
    return out.value


def attn_workspace_size(shape: Shape) -> int:
    out = ctypes.c_size_t()
    _check(lib().fp_attn_workspace_size(ctypes.byref(shape.c), ctypes.byref(out)),
           "fp_attn_workspace_size")
    return out.value


def validate(shape: Shape, p: FpParams | None, ws_bytes: int) -> int:
    return lib().fp_validate(ctypes.byref(shape.c), ctypes.byref(p) if p is not None else None,
                             int(ws_bytes))


@dataclass
class Indices:
    """Device outputs of select(): torch tensors on the GPU, plus the softmax scale the
    lists were selected with (host float; 0 = 1/sqrt(d)), which sparse_attn attends with."""
    shape: Shape
    kb_idx: object      # int32 [Hq * TRI]
    kb_cnt: object      # int32 [Hq * NB]
    pattern: object     # uint8 [B * Hq]
    js: object          # float32 [B * Hq]
    units: object       # int32 [B * Hq * 2]
    softmax_scale: float = 0.0

    def c(self) -> FpIndices:
        return FpIndices(self.kb_idx.data_ptr(), self.kb_cnt.data_ptr(), self.pattern.data_ptr(),
                         self.js.data_ptr(), self.units.data_ptr(), float(self.softmax_scale))


def _stream_ptr(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _check_tensor(x, name, ndim, dtype=None):
    import torch
    dtype = torch.bfloat16 if dtype is None else dtype
    if not (x.is_cuda and x.dtype == dtype and x.dim() == ndim and x.is_contiguous()):
        raise ValueError(f"{name} must be a contiguous {dtype} CUDA tensor of {ndim} dims")


def check_shapes(shape: Shape, q=None, k=None, v=None, o=None, index_lens=None):
    """Host-only check of one call's buffer shapes against the problem `shape`, before any
    launch: the C ABI sees raw device pointers and cannot check buffer sizes itself.
    q, k, v, o: shape tuples (or None); index_lens: element counts (kb_idx, kb_cnt,
    pattern, js, units) of the index buffers (or None).  Requires q and o = (T, Hq, d),
    k and v = (T, Hkv, d) with T = cu_seqlens[-1], and index buffers at least as long as
    the problem needs.  Raises ValueError naming the first mismatch."""
    T = int(shape.cu[-1])
    hq, hkv, d = shape.c.num_q_heads, shape.c.num_kv_heads, shape.c.head_dim
    want = {"q": (T, hq, d), "k": (T, hkv, d), "v": (T, hkv, d), "o": (T, hq, d)}
    for name, got in (("q", q), ("k", k), ("v", v), ("o", o)):
        if got is not None and tuple(int(x) for x in got) != want[name]:
            raise ValueError(f"{name} has shape {tuple(got)}; the problem (T={T}, Hq={hq}, "
                             f"Hkv={hkv}, d={d}) needs {want[name]}")
    if index_lens is not None:
        n_idx, n_cnt = indices_size(shape)
        b = shape.c.batch
        need = (max(n_idx, 1), max(n_cnt, 1), b * hq, b * hq, b * hq * 2)
        for name, got, n in zip(("kb_idx", "kb_cnt", "pattern", "js", "units"), index_lens, need):
            if got is not None and int(got) < n:
                raise ValueError(f"{name} holds {got} elements; the problem needs {n}")


def empty_indices(shape: Shape, device):
    import torch
    n_idx, n_cnt = indices_size(shape)
    b, hq = shape.c.batch, shape.c.num_q_heads
    return Indices(shape,
                   torch.empty(max(n_idx, 1), dtype=torch.int32, device=device),
                   torch.empty(max(n_cnt, 1), dtype=torch.int32, device=device),
                   torch.empty(b * hq, dtype=torch.uint8, device=device),
                   torch.empty(b * hq, dtype=torch.float32, device=device),
                   torch.empty(b * hq * 2, dtype=torch.int32, device=device))


def select(q, k, cu_seqlens, gamma, tau, min_budget=8, block=128, softmax_scale=0.0,
           force_pattern=-1, out: Indices | None = None, workspace=None, stream=None,
           max_budget=0, qa_mode=0, vs_granularity=0) -> Indices:
    """Pattern search + index selection (Algorithms 2-4) for a packed layer.

    q: [T, Hq, d] bf16 CUDA, k: [T, Hkv, d] bf16 CUDA, cu_seqlens: host ints [B+1]."""
    import torch
    _check_tensor(q, "q", 3)
    _check_tensor(k, "k", 3)
    shape = Shape(cu_seqlens, q.shape[1], k.shape[1], q.shape[2], block)
    check_shapes(shape, q=q.shape, k=k.shape)
    p = params(gamma, tau, min_budget, softmax_scale, force_pattern, max_budget, qa_mode,
               vs_granularity)
    ws_bytes = select_workspace_size(shape, p)
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=q.device)
    if out is None:
        out = empty_indices(shape, q.device)
    _check_indices(out, shape)
    oc = out.c()
    _check(lib().fp_select(ctypes.byref(shape.c), ctypes.c_void_p(q.data_ptr()),
                           ctypes.c_void_p(k.data_ptr()), ctypes.byref(p), ctypes.byref(oc),
                           ctypes.c_void_p(workspace.data_ptr()), workspace.numel(),
                           _stream_ptr(stream)), "fp_select")
    out.shape = shape
    out.softmax_scale = float(oc.softmax_scale)
    return out


def _check_indices(ind: Indices, shape: Shape):
    import torch
    for name, x, dt in (("kb_idx", ind.kb_idx, torch.int32), ("kb_cnt", ind.kb_cnt, torch.int32),
                        ("pattern", ind.pattern, torch.uint8), ("js", ind.js, torch.float32),
                        ("units", ind.units, torch.int32)):
        _check_tensor(x, name, 1, dt)
    check_shapes(shape, index_lens=(ind.kb_idx.numel(), ind.kb_cnt.numel(), ind.pattern.numel(),
                                    ind.js.numel(), ind.units.numel()))


def sparse_attn(q, k, v, indices: Indices, out=None, workspace=None, stream=None):
    """O = A(Q, K, V, S) over the key-block lists in `indices`, with the softmax scale the
    lists were selected with (indices.softmax_scale)."""
    import torch
    for name, x in (("q", q), ("k", k), ("v", v)):
        _check_tensor(x, name, 3)
    shape = indices.shape
    if out is None:
        out = torch.empty_like(q)
    _check_tensor(out, "out", 3)
    check_shapes(shape, q=q.shape, k=k.shape, v=v.shape, o=out.shape)
    _check_indices(indices, shape)
    ws_bytes = attn_workspace_size(shape)
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=q.device)
    ic = indices.c()
    _check(lib().fp_sparse_attn(ctypes.byref(shape.c), ctypes.c_void_p(q.data_ptr()),
                                ctypes.c_void_p(k.data_ptr()), ctypes.c_void_p(v.data_ptr()),
                                ctypes.byref(ic), ctypes.c_void_p(out.data_ptr()),
                                ctypes.c_void_p(workspace.data_ptr()), workspace.numel(),
                                _stream_ptr(stream)), "fp_sparse_attn")
    return out


NOALLOC_SCRATCH_BYTES = 64 << 20     # FP_NOALLOC_SCRATCH_BYTES


def sparse_attn_noalloc(q, k, v, indices: Indices, out, stream=None):
    """sparse_attn through fp_sparse_attn_noalloc: no workspace argument, the library's fixed
    device scratch array instead (problems up to NOALLOC_SCRATCH_BYTES of workspace).
    `out` is required: this call allocates nothing."""
    for name, x in (("q", q), ("k", k), ("v", v), ("out", out)):
        _check_tensor(x, name, 3)
    shape = indices.shape
    check_shapes(shape, q=q.shape, k=k.shape, v=v.shape, o=out.shape)
    _check_indices(indices, shape)
    ic = indices.c()
    _check(lib().fp_sparse_attn_noalloc(ctypes.byref(shape.c), ctypes.c_void_p(q.data_ptr()),
                                        ctypes.c_void_p(k.data_ptr()),
                                        ctypes.c_void_p(v.data_ptr()), ctypes.byref(ic),
                                        ctypes.c_void_p(out.data_ptr()), _stream_ptr(stream)),
           "fp_sparse_attn_noalloc")
    return out


def indices_from_masks(shape: Shape, masks, device, softmax_scale=0.0):
    """Pack host block masks {(s, h): bool [nb, nb]} into the kb_idx / kb_cnt layout
    (ascending key blocks per row), to be attended with `softmax_scale` (0 = 1/sqrt(d)).
    Host-side data marshalling for callers that bring their own index sets."""
    import torch
    n_idx, n_cnt = indices_size(shape)
    hq = shape.c.num_q_heads
    nbs = shape.nb()
    tri = np.concatenate([[0], np.cumsum(nbs * (nbs + 1) // 2)])
    nb_off = np.concatenate([[0], np.cumsum(nbs)])
    TRI, NB = int(tri[-1]), int(nb_off[-1])
    kb_idx = np.zeros(max(n_idx, 1), dtype=np.int32)
    kb_cnt = np.zeros(max(n_cnt, 1), dtype=np.int32)
    for (s, h), m in masks.items():
        nb = int(nbs[s])
        for I in range(nb):
            js = np.nonzero(m[I, :I + 1])[0].astype(np.int32)
            base = h * TRI + int(tri[s]) + I * (I + 1) // 2
            kb_idx[base:base + js.size] = js
            kb_cnt[h * NB + int(nb_off[s]) + I] = js.size
    b = shape.c.batch
    return Indices(shape, torch.from_numpy(kb_idx).to(device), torch.from_numpy(kb_cnt).to(device),
                   torch.zeros(b * hq, dtype=torch.uint8, device=device),
                   torch.zeros(b * hq, dtype=torch.float32, device=device),
                   torch.zeros(b * hq * 2, dtype=torch.int32, device=device),
                   float(softmax_scale))


def masks_from_indices(indices: Indices):
    """Unpack device kb_idx / kb_cnt into host bool masks {(s, h): [nb, nb]}."""
    shape = indices.shape
    hq = shape.c.num_q_heads
    nbs = shape.nb()
    tri = np.concatenate([[0], np.cumsum(nbs * (nbs + 1) // 2)])
    nb_off = np.concatenate([[0], np.cumsum(nbs)])
    TRI, NB = int(tri[-1]), int(nb_off[-1])
    kb_idx = indices.kb_idx.cpu().numpy()
    kb_cnt = indices.kb_cnt.cpu().numpy()
    out = {}
    for s in range(len(nbs)):
        nb = int(nbs[s])
        for h in range(hq):
            m = np.zeros((nb, nb), dtype=bool)
            for I in range(nb):
                c = int(kb_cnt[h * NB + int(nb_off[s]) + I])
                base = h * TRI + int(tri[s]) + I * (I + 1) // 2
                m[I, kb_idx[base:base + c]] = True
            out[(s, h)] = m
    return out
