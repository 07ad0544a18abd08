"""Python binding of libwise (include/wise.h): argument marshalling only.

Each function takes torch tensors (device memory owned by the caller), passes
their data pointers and the current HIP stream to the C entry point of the
same name, and raises WiseError on a non-OK status.  All arithmetic runs in
the library's HIP kernels; there is no fallback path — if libwise.so is
missing or cannot be loaded, `load()` raises.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libwise.so")

WISE_FORCE_SINK = 1
WISE_FORCE_DIAG = 2
WISE_DEFAULT_FLAGS = WISE_FORCE_SINK | WISE_FORCE_DIAG
NOALLOC_SCRATCH_BYTES = 4 << 20    # WISE_NOALLOC_SCRATCH_BYTES

STATUS_NAMES = {0: "WISE_OK", 1: "WISE_ERR_NULL", 2: "WISE_ERR_SHAPE", 3: "WISE_ERR_UNSUPPORTED",
                4: "WISE_ERR_RANGE", 5: "WISE_ERR_WORKSPACE", 6: "WISE_ERR_HIP"}

# Every symbol include/wise.h declares.
EXPORTS = ("wise_dense_attn_accum", "wise_select_support", "wise_select_support_noalloc",
           "wise_sparse_attn", "wise_sparse_attn_grouped", "wise_sparse_group_rows",
           "wise_select_step", "wise_support_from_masks", "wise_mask_union", "wise_mask_overlap",
           "wise_support_mass", "wise_mass_workspace_bytes", "wise_mass_workspace_min_bytes",
           "wise_mask_words",
           "wise_select_workspace_bytes",
           "wise_support_capacity", "wise_status_string", "wise_abi_version")


class WiseError(RuntimeError):
    def __init__(self, status: int, fn: str):
        self.status = status
        msg = _lib().wise_status_string(status).decode() if _LIB is not None else str(status)
        super().__init__(f"{fn}: {msg}")


class wise_shape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("heads", ctypes.c_int32),
                ("seq_len", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("block", ctypes.c_int32), ("scale", ctypes.c_float),
                ("kv_heads", ctypes.c_int32)]

    def __repr__(self):
        return (f"wise_shape(batch={self.batch}, heads={self.heads}, seq_len={self.seq_len}, "
                f"head_dim={self.head_dim}, block={self.block}, scale={self.scale}, "
                f"kv_heads={self.kv_heads})")


def make_shape(batch: int, heads: int, seq_len: int, head_dim: int, block: int,
               scale: float = 0.0, kv_heads: int = 0) -> wise_shape:
    """kv_heads = 0: one key-value head per query head."""
    return wise_shape(batch, heads, seq_len, head_dim, block, scale, kv_heads)


_LIB: Optional[ctypes.CDLL] = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libwise.so (once).  Raises if it is missing: there is no fallback."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(path):
        raise RuntimeError(f"libwise.so not built at {path}: run "
                           "`python -m paper_2609_27373_amd.build` (or __graft_entry__.build())")
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    S = ctypes.POINTER(wise_shape)
    lib.wise_dense_attn_accum.argtypes = [S, P, P, P, P, P, P, P, ctypes.c_size_t, P]
    lib.wise_dense_attn_accum.restype = ctypes.c_int
    lib.wise_select_support.argtypes = [S, P, ctypes.c_float, ctypes.c_uint32, P, P, P, P,
                                        ctypes.c_size_t, P]
    lib.wise_select_support.restype = ctypes.c_int
    lib.wise_select_support_noalloc.argtypes = [S, P, ctypes.c_float, ctypes.c_uint32, P, P, P, P]
    lib.wise_select_support_noalloc.restype = ctypes.c_int
    lib.wise_sparse_attn.argtypes = [S, P, P, P, P, P, P, P, P, P]
    lib.wise_sparse_attn.restype = ctypes.c_int
    lib.wise_sparse_attn_grouped.argtypes = [S, P, P, P, P, P, P, P, P]
    lib.wise_sparse_attn_grouped.restype = ctypes.c_int
    lib.wise_sparse_group_rows.argtypes = [S]
    lib.wise_sparse_group_rows.restype = ctypes.c_int32
    lib.wise_select_step.argtypes = [S, P, ctypes.c_float, P, P]
    lib.wise_select_step.restype = ctypes.c_int
    lib.wise_support_from_masks.argtypes = [S, P, ctypes.c_int32, ctypes.c_uint32, P, P, P, P,
                                            ctypes.c_size_t, P]
    lib.wise_support_from_masks.restype = ctypes.c_int
    lib.wise_mask_union.argtypes = [S, P, ctypes.c_int32, P, P]
    lib.wise_mask_union.restype = ctypes.c_int
    lib.wise_mask_overlap.argtypes = [S, P, P, P, P]
    lib.wise_mask_overlap.restype = ctypes.c_int
    lib.wise_support_mass.argtypes = [S, P, P, P, P, P, P]
    lib.wise_support_mass.restype = ctypes.c_int
    lib.wise_mass_workspace_bytes.argtypes = [S]
    lib.wise_mass_workspace_bytes.restype = ctypes.c_size_t
    lib.wise_mass_workspace_min_bytes.argtypes = [S]
    lib.wise_mass_workspace_min_bytes.restype = ctypes.c_size_t
    lib.wise_mask_words.argtypes = [S]
    lib.wise_mask_words.restype = ctypes.c_int32
    lib.wise_select_workspace_bytes.argtypes = [S]
    lib.wise_select_workspace_bytes.restype = ctypes.c_size_t
    lib.wise_support_capacity.argtypes = [S]
    lib.wise_support_capacity.restype = ctypes.c_int64
    lib.wise_status_string.argtypes = [ctypes.c_int]
    lib.wise_status_string.restype = ctypes.c_char_p
    lib.wise_abi_version.argtypes = []
    lib.wise_abi_version.restype = ctypes.c_int32
    _LIB = lib
    return lib


def _lib() -> ctypes.CDLL:
    return _LIB if _LIB is not None else load()


def _ptr(t: Optional[torch.Tensor], dtype=None, name="tensor", numel=None):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} holds {t.numel()} elements, needs {numel}")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _check(status: int, fn: str):
    if status != 0:
        raise WiseError(status, fn)


def _sizes(s: wise_shape):
    bh = s.batch * s.heads
    nb = s.seq_len // s.block if s.block > 0 else 0
    return bh * s.seq_len * s.head_dim, bh * s.seq_len, bh * nb * nb, bh * nb


def _kv_numel(s: wise_shape) -> int:
    return s.batch * (s.kv_heads or s.heads) * s.seq_len * s.head_dim


def wise_dense_attn_accum(s: wise_shape, q, k, v, o, lse=None, acc=None, workspace=None,
                          stream=None) -> None:
    """`workspace` (any dtype) is required with `acc`: mass_workspace()
    allocates one; wise_mass_workspace_bytes(s) bytes run one launch, any
    size down to wise_mass_workspace_min_bytes(s) runs the heads in turn."""
    nqkv, nlse, nacc, _ = _sizes(s)
    nkv = _kv_numel(s)
    bf = torch.bfloat16
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(_lib().wise_dense_attn_accum(
        ctypes.byref(s), _ptr(q, bf, "q", nqkv), _ptr(k, bf, "k", nkv), _ptr(v, bf, "v", nkv),
        _ptr(o, bf, "o", nqkv), _ptr(lse, torch.float32, "lse", nlse),
        _ptr(acc, torch.float32, "acc", nacc), _ptr(workspace, None, "workspace"),
        ctypes.c_size_t(ws_bytes), _stream(stream)), "wise_dense_attn_accum")


def mass_workspace(s: wise_shape, device="cuda", max_bytes=None) -> torch.Tensor:
    """A device buffer of wise_mass_workspace_bytes(s) bytes, or of at most
    max_bytes (not below wise_mass_workspace_min_bytes(s))."""
    n = wise_mass_workspace_bytes(s)
    if max_bytes is not None:
        n = max(min(n, int(max_bytes)), wise_mass_workspace_min_bytes(s))
    return torch.empty(max(n, 1), dtype=torch.uint8, device=device)


def _capacity(s: wise_shape) -> int:
    """Entries col_idx must hold for a selection to write (0 for an invalid
    shape, which the library then rejects)."""
    return max(wise_support_capacity(s), 0)


def wise_select_support(s: wise_shape, acc, tau: float, flags: int, row_ptr, col_idx,
                        row_order=None, workspace=None, stream=None) -> None:
    _, _, nacc, rows = _sizes(s)
    i32 = torch.int32
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(_lib().wise_select_support(
        ctypes.byref(s), _ptr(acc, torch.float32, "acc", nacc), ctypes.c_float(tau),
        ctypes.c_uint32(flags), _ptr(row_ptr, i32, "row_ptr", rows + 1),
        _ptr(col_idx, i32, "col_idx", _capacity(s)), _ptr(row_order, i32, "row_order", rows),
        _ptr(workspace, None, "workspace"), ctypes.c_size_t(ws_bytes), _stream(stream)),
        "wise_select_support")


def wise_select_support_noalloc(s: wise_shape, acc, tau: float, flags: int, row_ptr, col_idx,
                                row_order=None, stream=None) -> None:
    """wise_select_support on the library's own per-device scratch (no workspace)."""
    _, _, nacc, rows = _sizes(s)
    i32 = torch.int32
    _check(_lib().wise_select_support_noalloc(
        ctypes.byref(s), _ptr(acc, torch.float32, "acc", nacc), ctypes.c_float(tau),
        ctypes.c_uint32(flags), _ptr(row_ptr, i32, "row_ptr", rows + 1),
        _ptr(col_idx, i32, "col_idx", _capacity(s)), _ptr(row_order, i32, "row_order", rows),
        _stream(stream)), "wise_select_support_noalloc")


def wise_sparse_attn(s: wise_shape, q, k, v, row_ptr, col_idx, row_order, o, lse=None,
                     stream=None) -> None:
    nqkv, nlse, _, rows = _sizes(s)
    nkv = _kv_numel(s)
    bf, i32 = torch.bfloat16, torch.int32
    _check(_lib().wise_sparse_attn(
        ctypes.byref(s), _ptr(q, bf, "q", nqkv), _ptr(k, bf, "k", nkv), _ptr(v, bf, "v", nkv),
        _ptr(row_ptr, i32, "row_ptr", rows + 1), _ptr(col_idx, i32, "col_idx"),
        _ptr(row_order, i32, "row_order", rows), _ptr(o, bf, "o", nqkv),
        _ptr(lse, torch.float32, "lse", nlse), _stream(stream)), "wise_sparse_attn")


def wise_sparse_attn_grouped(s: wise_shape, q, k, v, row_ptr, col_idx, o, lse=None,
                             stream=None) -> None:
    nqkv, nlse, _, rows = _sizes(s)
    nkv = _kv_numel(s)
    bf, i32 = torch.bfloat16, torch.int32
    _check(_lib().wise_sparse_attn_grouped(
        ctypes.byref(s), _ptr(q, bf, "q", nqkv), _ptr(k, bf, "k", nkv), _ptr(v, bf, "v", nkv),
        _ptr(row_ptr, i32, "row_ptr", rows + 1), _ptr(col_idx, i32, "col_idx"),
        _ptr(o, bf, "o", nqkv), _ptr(lse, torch.float32, "lse", nlse), _stream(stream)),
        "wise_sparse_attn_grouped")


def wise_sparse_group_rows(s: wise_shape) -> int:
    return int(_lib().wise_sparse_group_rows(ctypes.byref(s)))


def _mask_elems(s: wise_shape, n: int = 1) -> int:
    return n * _sizes(s)[3] * max(wise_mask_words(s), 0)


def wise_select_step(s: wise_shape, r, tau: float, mask, stream=None) -> None:
    _, _, nacc, _ = _sizes(s)
    _check(_lib().wise_select_step(
        ctypes.byref(s), _ptr(r, torch.float32, "r", nacc), ctypes.c_float(tau),
        _ptr(mask, torch.int64, "mask", _mask_elems(s)), _stream(stream)), "wise_select_step")


def wise_support_from_masks(s: wise_shape, masks, n_masks: int, flags: int, row_ptr, col_idx,
                            row_order=None, workspace=None, stream=None) -> None:
    _, _, _, rows = _sizes(s)
    i32 = torch.int32
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(_lib().wise_support_from_masks(
        ctypes.byref(s), _ptr(masks, torch.int64, "masks", _mask_elems(s, max(n_masks, 0))),
        ctypes.c_int32(n_masks), ctypes.c_uint32(flags), _ptr(row_ptr, i32, "row_ptr", rows + 1),
        _ptr(col_idx, i32, "col_idx", _capacity(s)), _ptr(row_order, i32, "row_order", rows),
        _ptr(workspace, None, "workspace"), ctypes.c_size_t(ws_bytes), _stream(stream)),
        "wise_support_from_masks")


def wise_mask_union(s: wise_shape, masks, n_masks: int, out, stream=None) -> None:
    _check(_lib().wise_mask_union(
        ctypes.byref(s), _ptr(masks, torch.int64, "masks", _mask_elems(s, max(n_masks, 0))),
        ctypes.c_int32(n_masks), _ptr(out, torch.int64, "out", _mask_elems(s)), _stream(stream)),
        "wise_mask_union")


def wise_mask_overlap(s: wise_shape, a, b, counts, stream=None) -> None:
    n = _mask_elems(s)
    _check(_lib().wise_mask_overlap(
        ctypes.byref(s), _ptr(a, torch.int64, "a", n), _ptr(b, torch.int64, "b", n),
        _ptr(counts, torch.int64, "counts", 2), _stream(stream)), "wise_mask_overlap")


def wise_support_mass(s: wise_shape, r, row_ptr, col_idx, row_mass, totals=None,
                      stream=None) -> None:
    _, _, nacc, rows = _sizes(s)
    i32, f64 = torch.int32, torch.float64
    _check(_lib().wise_support_mass(
        ctypes.byref(s), _ptr(r, torch.float32, "r", nacc), _ptr(row_ptr, i32, "row_ptr", rows + 1),
        _ptr(col_idx, i32, "col_idx"), _ptr(row_mass, f64, "row_mass", 2 * rows),
        _ptr(totals, f64, "totals", 2), _stream(stream)), "wise_support_mass")


def wise_mass_workspace_bytes(s: wise_shape) -> int:
    return int(_lib().wise_mass_workspace_bytes(ctypes.byref(s)))


def wise_mass_workspace_min_bytes(s: wise_shape) -> int:
    return int(_lib().wise_mass_workspace_min_bytes(ctypes.byref(s)))


def wise_mask_words(s: wise_shape) -> int:
    return int(_lib().wise_mask_words(ctypes.byref(s)))


def wise_select_workspace_bytes(s: wise_shape) -> int:
    return int(_lib().wise_select_workspace_bytes(ctypes.byref(s)))


def wise_support_capacity(s: wise_shape) -> int:
    return int(_lib().wise_support_capacity(ctypes.byref(s)))


def wise_status_string(status: int) -> str:
    return _lib().wise_status_string(status).decode()


def wise_abi_version() -> int:
    return int(_lib().wise_abi_version())


class Schedule:
    """Device buffers of one support schedule (CSR + row order + workspace),
    sized by the library's own size queries."""

    def __init__(self, s: wise_shape, device="cuda"):
        _, _, _, rows = _sizes(s)
        cap = wise_support_capacity(s)
        if cap < 0:
            raise WiseError(2, "wise_support_capacity")
        self.shape = s
        self.row_ptr = torch.empty(rows + 1, dtype=torch.int32, device=device)
        self.col_idx = torch.empty(max(cap, 1), dtype=torch.int32, device=device)
        self.row_order = torch.empty(rows, dtype=torch.int32, device=device)
        self.workspace = torch.empty(wise_select_workspace_bytes(s), dtype=torch.uint8,
                                     device=device)

    def select(self, acc, tau: float, flags: int = WISE_DEFAULT_FLAGS, stream=None):
        wise_select_support(self.shape, acc, tau, flags, self.row_ptr, self.col_idx,
                            self.row_order, self.workspace, stream)
        return self

    def from_masks(self, masks, n_masks: int, flags: int = WISE_DEFAULT_FLAGS, stream=None):
        """The union of n_masks per-step supports (back to back in `masks`)."""
        wise_support_from_masks(self.shape, masks, n_masks, flags, self.row_ptr, self.col_idx,
                                self.row_order, self.workspace, stream)
        return self

    def nnz(self) -> int:
        return int(self.row_ptr[-1].item())
