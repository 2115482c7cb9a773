"""Thin Python binding of liblosa.so (include/losa.h).

Argument marshalling only: torch tensors in, device pointers and sizes out,
the current HIP stream passed through.  Every step of the computation runs in
the library's HIP kernels; if the library is missing this module raises on
import instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import math
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# the in-tree build; LOSA_LIBRARY names another build of the same sources
# (the host-sanitizer check uses it)
LIB_PATH = os.environ.get("LOSA_LIBRARY") or os.path.join(_HERE, "liblosa.so")

LOSA_DTYPE_F32 = 0
LOSA_DTYPE_BF16 = 1
STATUS = {0: "LOSA_OK", 1: "LOSA_ERR_NULL_POINTER", 2: "LOSA_ERR_INVALID_SHAPE",
          3: "LOSA_ERR_INVALID_TAU", 4: "LOSA_ERR_ALIGNMENT", 5: "LOSA_ERR_UNSUPPORTED",
          6: "LOSA_ERR_CAPACITY", 7: "LOSA_ERR_HIP"}

EXPORTED = ("losa_calibrate_mass", "losa_select_blocks", "losa_select_blocks_topk",
            "losa_block_recall", "losa_sparse_attn_fwd", "losa_sparse_attn_fwd_noalloc",
            "losa_construct", "losa_workspace_bytes", "losa_status_string", "losa_last_error",
            "losa_version")

# bytes of library-held scratch behind losa_sparse_attn_fwd_noalloc (per GPU)
NOALLOC_SCRATCH_BYTES = 128 << 20


class LosaError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)}: {detail}")


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2608_12032_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    P, I, F, Z, L = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t, ctypes.c_int64
    lib.losa_calibrate_mass.argtypes = [P, P, I, I, I, I, I, I, I, F, P, P, P, Z, P]
    lib.losa_calibrate_mass.restype = I
    lib.losa_select_blocks.argtypes = [P, I, I, I, I, I, F, P, P, L, P, Z, P]
    lib.losa_select_blocks.restype = I
    lib.losa_select_blocks_topk.argtypes = [P, I, I, I, I, I, I, P, P, L, P, Z, P]
    lib.losa_select_blocks_topk.restype = I
    lib.losa_block_recall.argtypes = [P, I, I, I, I, I, P, P, L, P, P, P, Z, P]
    lib.losa_block_recall.restype = I
    lib.losa_sparse_attn_fwd.argtypes = [P, P, P, I, I, I, I, I, I, I, F, P, P, L, P, P, P, Z, P]
    lib.losa_sparse_attn_fwd.restype = I
    lib.losa_sparse_attn_fwd_noalloc.argtypes = [P, P, P, I, I, I, I, I, I, I, F, P, P, L, P, P,
                                                 P]
    lib.losa_sparse_attn_fwd_noalloc.restype = I
    lib.losa_construct.argtypes = [P, P, P, I, I, I, I, I, I, I, F, P, P, P, P, Z, P]
    lib.losa_construct.restype = I
    lib.losa_workspace_bytes.argtypes = [I, I, I, I, I, I, I, I]
    lib.losa_workspace_bytes.restype = Z
    lib.losa_status_string.argtypes = [I]
    lib.losa_status_string.restype = ctypes.c_char_p
    lib.losa_last_error.argtypes = []
    lib.losa_last_error.restype = ctypes.c_char_p
    lib.losa_version.argtypes = []
    lib.losa_version.restype = I
    return lib


lib = _load()


def _check(st: int, where: str):
    if st != 0:
        raise LosaError(st, where, lib.losa_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return LOSA_DTYPE_BF16
    if t.dtype == torch.float32:
        return LOSA_DTYPE_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _arg(t, name, device, dtype=None, shape=None, numel=None, nbytes=None):
    """Check a tensor argument before its pointer reaches the library, which
    sees raw device pointers and cannot tell a host tensor, a wrong element
    type or a short buffer from a valid one."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda or t.device != device:
        raise ValueError(f"{name} must live on {device} (got {t.device})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)} (got {tuple(t.shape)})")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} holds {t.numel()} elements, needs {numel}")
    if nbytes is not None and t.numel() * t.element_size() < nbytes:
        raise ValueError(f"{name} holds {t.numel() * t.element_size()} bytes, needs {nbytes}")
    return t


def _qkv(q, others, N: int, block_q: int, block_k: int):
    """Shape of Q ([B, H, N_pad, d] on a GPU, N_pad = padded_len(N, ...)), and
    K / V alike."""
    if not isinstance(q, torch.Tensor) or q.dim() != 4:
        raise ValueError("q must be a [B, H, N_pad, d] tensor")
    _arg(q, "q", q.device)
    B, H, Np, d = q.shape
    if N < 1 or Np != padded_len(N, block_q, block_k):
        raise ValueError(f"q has N_pad = {Np}; N = {N} with blocks {block_q} x {block_k} "
                         f"needs {padded_len(max(N, 1), block_q, block_k)}")
    for name, t in others.items():
        _arg(t, name, q.device, dtype=q.dtype, shape=q.shape)
    return B, H, Np, d


def _mass_shape(mass, N: int, block_q: int, block_k: int):
    if not isinstance(mass, torch.Tensor) or mass.dim() != 4:
        raise ValueError("mass must be a [B, H, n_q, n_k] tensor")
    Np = padded_len(N, block_q, block_k)
    B, H = mass.shape[:2]
    _arg(mass, "mass", mass.device, dtype=torch.float32, shape=(B, H, Np // block_q,
                                                                  Np // block_k))
    return B, H, Np // block_q, Np // block_k


def padded_len(N: int, block_q: int, block_k: int) -> int:
    L = max(block_q, block_k)
    return -(-N // L) * L


def workspace_bytes(which: int, dtype_code: int, B, H, N, d, block_q, block_k) -> int:
    return int(lib.losa_workspace_bytes(which, dtype_code, B, H, N, d, block_q, block_k))


def losa_calibrate_mass(q, k, N: int, block_q: int, block_k: int | None = None,
                        scale: float | None = None, want_lse: bool = True, mass=None, lse=None,
                        workspace=None, two_sweep: bool = False):
    """Exact block masses of a dense step -> (mass [B,H,n_q,n_k] fp32, lse or None).

    bf16 takes one sweep over the keys plus a reduction of per-(query, key
    block) statistics held in ``workspace`` (allocated at the suggested size
    when not given); ``two_sweep=True`` passes no workspace and takes two
    sweeps instead."""
    block_k = block_k or block_q
    B, H, Np, d = _qkv(q, {"k": k}, N, block_q, block_k)
    dev = q.device
    n_q, n_k = Np // block_q, Np // block_k
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    if mass is None:
        mass = torch.empty((B, H, n_q, n_k), dtype=torch.float32, device=dev)
    _arg(mass, "mass", dev, dtype=torch.float32, shape=(B, H, n_q, n_k))
    if want_lse and lse is None:
        lse = torch.empty((B, H, Np), dtype=torch.float32, device=dev)
    if not want_lse:
        lse = None
    if lse is not None:
        _arg(lse, "lse", dev, dtype=torch.float32, shape=(B, H, Np))
    dcode = _dtype_code(q)
    if two_sweep or dcode != LOSA_DTYPE_BF16:
        workspace = None
    elif workspace is None:
        need = workspace_bytes(0, dcode, B, H, N, d, block_q, block_k)
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    if workspace is not None:
        _arg(workspace, "workspace", dev)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib.losa_calibrate_mass(_ptr(q), _ptr(k), dcode, B, H, N, d, block_q, block_k,
                                 scale, _ptr(mass), _ptr(lse), _ptr(workspace), ws_bytes,
                                 _stream(dev))
    _check(st, "losa_calibrate_mass")
    return mass, lse


def _csr_out(row_ptr, col_idx, workspace, rows, n_k, dev, need):
    if row_ptr is None:
        row_ptr = torch.empty(rows + 1, dtype=torch.int32, device=dev)
    if col_idx is None:
        col_idx = torch.empty(rows * n_k, dtype=torch.int32, device=dev)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
    _arg(row_ptr, "row_ptr", dev, dtype=torch.int32, numel=rows + 1)
    _arg(col_idx, "col_idx", dev, dtype=torch.int32)
    _arg(workspace, "workspace", dev, nbytes=need)
    return row_ptr, col_idx, workspace


def losa_select_blocks(mass, N: int, block_q: int, block_k: int | None, tau: float,
                       row_ptr=None, col_idx=None, workspace=None):
    """Shortest-prefix selection -> (row_ptr int32 [rows+1], col_idx int32 buffer).

    col_idx has the worst-case capacity B*H*n_q*n_k; its first row_ptr[-1]
    entries are valid (read row_ptr[-1] after a sync, or use ``nnz``).
    """
    block_k = block_k or block_q
    B, H, n_q, n_k = _mass_shape(mass, N, block_q, block_k)
    rows = B * H * n_q
    dev = mass.device
    need = workspace_bytes(1, LOSA_DTYPE_F32, B, H, N, 1, block_q, block_k)
    row_ptr, col_idx, workspace = _csr_out(row_ptr, col_idx, workspace, rows, n_k, dev, need)
    st = lib.losa_select_blocks(_ptr(mass), B, H, N, block_q, block_k, float(tau),
                                _ptr(row_ptr), _ptr(col_idx), col_idx.numel(), _ptr(workspace),
                                workspace.numel() * workspace.element_size(), _stream(dev))
    _check(st, "losa_select_blocks")
    return row_ptr, col_idx


def losa_select_blocks_topk(mass, N: int, block_q: int, block_k: int | None, k: int,
                            row_ptr=None, col_idx=None, workspace=None):
    """Fixed-ratio top-k selection (k blocks per row) -> (row_ptr, col_idx buffer)."""
    block_k = block_k or block_q
    B, H, n_q, n_k = _mass_shape(mass, N, block_q, block_k)
    rows = B * H * n_q
    dev = mass.device
    need = workspace_bytes(1, LOSA_DTYPE_F32, B, H, N, 1, block_q, block_k)
    row_ptr, col_idx, workspace = _csr_out(row_ptr, col_idx, workspace, rows, n_k, dev, need)
    st = lib.losa_select_blocks_topk(_ptr(mass), B, H, N, block_q, block_k, int(k),
                                     _ptr(row_ptr), _ptr(col_idx), col_idx.numel(),
                                     _ptr(workspace), workspace.numel() * workspace.element_size(),
                                     _stream(dev))
    _check(st, "losa_select_blocks_topk")
    return row_ptr, col_idx


def losa_block_recall(mass, N: int, block_q: int, block_k: int | None, row_ptr, col_idx,
                      want_rows: bool = True, want_heads: bool = True, workspace=None):
    """Recall of a frozen support on these masses -> (recall_rows or None, recall_heads or None)."""
    block_k = block_k or block_q
    B, H, n_q, n_k = _mass_shape(mass, N, block_q, block_k)
    dev = mass.device
    _arg(row_ptr, "row_ptr", dev, dtype=torch.int32, numel=B * H * n_q + 1)
    _arg(col_idx, "col_idx", dev, dtype=torch.int32)
    rec_rows = torch.empty(B * H * n_q, dtype=torch.float32, device=dev) if want_rows else None
    rec_heads = torch.empty((B, H), dtype=torch.float32, device=dev) if want_heads else None
    need = workspace_bytes(3, LOSA_DTYPE_F32, B, H, N, 1, block_q, block_k)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
    _arg(workspace, "workspace", dev, nbytes=need)
    st = lib.losa_block_recall(_ptr(mass), B, H, N, block_q, block_k, _ptr(row_ptr),
                               _ptr(col_idx), col_idx.numel(), _ptr(rec_rows), _ptr(rec_heads),
                               _ptr(workspace), workspace.numel() * workspace.element_size(),
                               _stream(dev))
    _check(st, "losa_block_recall")
    return rec_rows, rec_heads


def nnz(row_ptr) -> int:
    return int(row_ptr[-1].item())


def losa_sparse_attn_fwd(q, k, v, N: int, block_q: int, block_k: int | None, row_ptr, col_idx,
                         scale: float | None = None, want_lse: bool = False, out=None,
                         lse=None, workspace=None):
    """Frozen-support block-sparse attention -> o (and lse if requested)."""
    block_k = block_k or block_q
    B, H, Np, d = _qkv(q, {"k": k, "v": v}, N, block_q, block_k)
    dev = q.device
    _arg(row_ptr, "row_ptr", dev, dtype=torch.int32, numel=B * H * (Np // block_q) + 1)
    _arg(col_idx, "col_idx", dev, dtype=torch.int32)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    dcode = _dtype_code(q)
    o = torch.empty_like(q) if out is None else out
    _arg(o, "out", dev, dtype=q.dtype, shape=q.shape)
    if want_lse and lse is None:
        lse = torch.empty((B, H, Np), dtype=torch.float32, device=dev)
    if want_lse:
        _arg(lse, "lse", dev, dtype=torch.float32, shape=(B, H, Np))
    need = workspace_bytes(2, dcode, B, H, N, d, block_q, block_k)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    if workspace is not None:
        _arg(workspace, "workspace", dev, nbytes=need)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib.losa_sparse_attn_fwd(_ptr(q), _ptr(k), _ptr(v), dcode, B, H, N, d, block_q, block_k,
                                  scale, _ptr(row_ptr), _ptr(col_idx), col_idx.numel(), _ptr(o),
                                  _ptr(lse if want_lse else None), _ptr(workspace), ws_bytes,
                                  _stream(dev))
    _check(st, "losa_sparse_attn_fwd")
    return (o, lse) if want_lse else o


def losa_sparse_attn_fwd_noalloc(q, k, v, N: int, block_q: int, block_k: int | None, row_ptr,
                                 col_idx, scale: float | None = None, want_lse: bool = False,
                                 out=None, lse=None):
    """losa_sparse_attn_fwd without a workspace: the library's own scratch
    (NOALLOC_SCRATCH_BYTES per GPU) holds it.  Allocates only the outputs
    that are not given; pass ``out`` (and ``lse``) to allocate nothing."""
    block_k = block_k or block_q
    B, H, Np, d = _qkv(q, {"k": k, "v": v}, N, block_q, block_k)
    dev = q.device
    _arg(row_ptr, "row_ptr", dev, dtype=torch.int32, numel=B * H * (Np // block_q) + 1)
    _arg(col_idx, "col_idx", dev, dtype=torch.int32)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    o = torch.empty_like(q) if out is None else out
    _arg(o, "out", dev, dtype=q.dtype, shape=q.shape)
    if want_lse and lse is None:
        lse = torch.empty((B, H, Np), dtype=torch.float32, device=dev)
    if want_lse:
        _arg(lse, "lse", dev, dtype=torch.float32, shape=(B, H, Np))
    if torch.cuda.current_device() != dev.index:
        raise ValueError(f"the tensors live on {dev}; make it the current device")
    st = lib.losa_sparse_attn_fwd_noalloc(_ptr(q), _ptr(k), _ptr(v), _dtype_code(q), B, H, N, d,
                                          block_q, block_k, scale, _ptr(row_ptr), _ptr(col_idx),
                                          col_idx.numel(), _ptr(o),
                                          _ptr(lse if want_lse else None), _stream(dev))
    _check(st, "losa_sparse_attn_fwd_noalloc")
    return (o, lse) if want_lse else o


def losa_construct(q, k, v, N: int, block_q: int, block_k: int | None = None,
                   scale: float | None = None, want_lse: bool = False, out=None, mass=None,
                   lse=None, workspace=None):
    """Construction step: dense attention output and exact block masses of the
    same step -> (o, mass) or (o, mass, lse)."""
    block_k = block_k or block_q
    B, H, Np, d = _qkv(q, {"k": k, "v": v}, N, block_q, block_k)
    dev = q.device
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    dcode = _dtype_code(q)
    o = torch.empty_like(q) if out is None else out
    _arg(o, "out", dev, dtype=q.dtype, shape=q.shape)
    if mass is None:
        mass = torch.empty((B, H, Np // block_q, Np // block_k), dtype=torch.float32, device=dev)
    _arg(mass, "mass", dev, dtype=torch.float32, shape=(B, H, Np // block_q, Np // block_k))
    if want_lse and lse is None:
        lse = torch.empty((B, H, Np), dtype=torch.float32, device=dev)
    if not want_lse:
        lse = None
    if lse is not None:
        _arg(lse, "lse", dev, dtype=torch.float32, shape=(B, H, Np))
    need = workspace_bytes(4, dcode, B, H, N, d, block_q, block_k)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    if workspace is not None:
        _arg(workspace, "workspace", dev)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib.losa_construct(_ptr(q), _ptr(k), _ptr(v), dcode, B, H, N, d, block_q, block_k, scale,
                            _ptr(o), _ptr(mass), _ptr(lse), _ptr(workspace), ws_bytes,
                            _stream(dev))
    _check(st, "losa_construct")
    return (o, mass, lse) if want_lse else (o, mass)


# shorter aliases
calibrate_mass = losa_calibrate_mass
select_blocks = losa_select_blocks
select_blocks_topk = losa_select_blocks_topk
block_recall = losa_block_recall
sparse_attn_fwd = losa_sparse_attn_fwd
sparse_attn_fwd_noalloc = losa_sparse_attn_fwd_noalloc
construct = losa_construct
