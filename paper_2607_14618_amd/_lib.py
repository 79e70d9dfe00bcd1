"""ctypes binding of libpolyq.so: argument marshalling only.

Every step of the computation runs in the library's HIP kernels; torch supplies
device memory and the current HIP stream.  There is no fallback: if the library
is missing or a call fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
import threading
from typing import Dict, Optional, Sequence, Tuple

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libpolyq.so")

MAX_BLOCKS = 5
QUANTUM = 32
GROUP = 128
TILE_ROWS = 64
MAX_M_GEMV = 16
MAX_BATCH = 8

STATUS = {0: "POLYQ_OK", 1: "POLYQ_ERR_ARG", 2: "POLYQ_ERR_BITS", 3: "POLYQ_ERR_QUANTUM",
          4: "POLYQ_ERR_SHAPE", 5: "POLYQ_ERR_CAPACITY", 6: "POLYQ_ERR_UNSUPPORTED",
          7: "POLYQ_ERR_DEVICE"}

# every symbol include/polyq.h declares
EXPORTS = ("polyq_plan", "polyq_pack", "polyq_pack_rows", "polyq_unpack", "polyq_permute", "polyq_gemv_workspace_bytes",
           "polyq_gemv", "polyq_gemv_batch_workspace_bytes", "polyq_gemv_batch_workspace_zero_bytes",
           "polyq_gemv_batch",
           "polyq_gemm_workspace_bytes", "polyq_gemm", "polyq_gemm_batch_workspace_bytes",
           "polyq_gemm_batch", "polyq_read_probe", "polyq_gemv_batch_noalloc", "polyq_channel_error",
           "polyq_waterfill", "polyq_quanta_match", "polyq_cluster", "polyq_bit_scaling", "polyq_status_str")


class Block(ctypes.Structure):
    _fields_ = [("bits", ctypes.c_int32), ("len", ctypes.c_int32)]


class Layout(ctypes.Structure):
    _fields_ = [
        ("n", ctypes.c_int32), ("k", ctypes.c_int32), ("nblocks", ctypes.c_int32),
        ("n_groups", ctypes.c_int32), ("n_tiles", ctypes.c_int32), ("n_chunks", ctypes.c_int32),
        ("block", Block * MAX_BLOCKS),
        ("k_begin", ctypes.c_int32 * MAX_BLOCKS),
        ("group_begin", ctypes.c_int32 * MAX_BLOCKS),
        ("block_offset", ctypes.c_int64 * MAX_BLOCKS),
        ("tile_bytes", ctypes.c_int64 * MAX_BLOCKS),
        ("record_bytes", ctypes.c_int64 * MAX_BLOCKS),
        ("packed_bytes", ctypes.c_int64),
        ("code_bits", ctypes.c_int64),
        ("weight_bytes", ctypes.c_int64),
    ]

    @property
    def blocks(self):
        return [(self.block[i].bits, self.block[i].len) for i in range(self.nblocks)]

    def __repr__(self):
        return (f"Layout(n={self.n}, k={self.k}, blocks={self.blocks}, n_groups={self.n_groups}, "
                f"packed_bytes={self.packed_bytes}, weight_bytes={self.weight_bytes})")


class GemvItem(ctypes.Structure):
    _fields_ = [("layout", ctypes.POINTER(Layout)), ("packed", ctypes.c_void_p),
                ("perm", ctypes.c_void_p), ("x", ctypes.c_void_p), ("y", ctypes.c_void_p),
                ("xscale", ctypes.c_void_p)]


def _item6(item):
    """(layout, packed, perm, x, y[, xscale]) -> the six fields (xscale None if absent)."""
    if len(item) == 5:
        return (*item, None)
    return tuple(item)


def _check_xscale(xscale, layout) -> None:
    if xscale is not None and (xscale.dtype != torch.float16 or xscale.numel() != layout.k
                               or not xscale.is_contiguous()):
        raise ValueError("xscale must be a contiguous fp16 [k] tensor")


class PolyQError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)}: {_status_str(status)}")


_lib = None
_lock = threading.Lock()


def lib() -> ctypes.CDLL:
    """Load libpolyq.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise ImportError(f"{LIB_PATH} is missing: run __graft_entry__.build() "
                                  "(or python -m paper_2607_14618_amd.build) first")
            L = ctypes.CDLL(LIB_PATH)
            vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
            lp = ctypes.POINTER(Layout)
            L.polyq_plan.argtypes = [i32, i32, ctypes.POINTER(Block), i32, lp]
            L.polyq_pack.argtypes = [lp, vp, vp, vp, vp, vp]
            L.polyq_pack_rows.argtypes = [lp, vp, vp, vp, vp, vp, vp]
            L.polyq_unpack.argtypes = [lp, vp, vp, vp, vp, vp]
            L.polyq_permute.argtypes = [vp, vp, vp, i32, i32, vp]
            L.polyq_gemv_workspace_bytes.argtypes = [lp, i32]
            L.polyq_gemv_workspace_bytes.restype = sz
            L.polyq_gemv.argtypes = [lp, vp, vp, vp, i32, vp, vp, sz, vp]
            ip = ctypes.POINTER(GemvItem)
            L.polyq_gemv_batch_workspace_bytes.argtypes = [ip, i32, i32]
            L.polyq_gemv_batch_workspace_bytes.restype = sz
            L.polyq_gemv_batch_workspace_zero_bytes.argtypes = [ip, i32, i32]
            L.polyq_gemv_batch_workspace_zero_bytes.restype = sz
            L.polyq_gemv_batch.argtypes = [ip, i32, i32, vp, sz, vp]
            L.polyq_gemm_workspace_bytes.argtypes = [lp, i32, ctypes.c_int]
            L.polyq_gemm_workspace_bytes.restype = sz
            L.polyq_gemm.argtypes = [lp, vp, vp, vp, i32, vp, vp, sz, vp]
            L.polyq_gemm_batch_workspace_bytes.argtypes = [ip, i32, i32]
            L.polyq_gemm_batch_workspace_bytes.restype = sz
            L.polyq_gemm_batch.argtypes = [ip, i32, i32, vp, sz, vp]
            L.polyq_read_probe.argtypes = [vp, ctypes.c_int64, i32, vp, vp]
            L.polyq_gemv_batch_noalloc.argtypes = [ip, i32, i32, vp]
            L.polyq_channel_error.argtypes = [vp, i32, i32, vp, vp, vp]
            L.polyq_waterfill.argtypes = [vp, i32, ctypes.c_double, vp]
            L.polyq_quanta_match.argtypes = [vp, i32, i32, ctypes.c_double, vp, vp]
            L.polyq_cluster.argtypes = [vp, i32, vp, ctypes.POINTER(Block), ctypes.POINTER(i32)]
            L.polyq_bit_scaling.argtypes = [vp, i32, i32, vp, vp, vp, vp, i32, vp, vp]
            L.polyq_status_str.argtypes = [ctypes.c_int]
            L.polyq_status_str.restype = ctypes.c_char_p
            for name in ("polyq_plan", "polyq_pack", "polyq_pack_rows", "polyq_unpack", "polyq_permute",
                         "polyq_gemv", "polyq_gemv_batch", "polyq_gemm", "polyq_gemm_batch",
                         "polyq_read_probe", "polyq_gemv_batch_noalloc", "polyq_channel_error",
                         "polyq_waterfill", "polyq_quanta_match", "polyq_cluster", "polyq_bit_scaling"):
                getattr(L, name).restype = ctypes.c_int
            _lib = L
    return _lib


def _status_str(status: int) -> str:
    try:
        return lib().polyq_status_str(status).decode()
    except Exception:  # library not loadable
        return "?"


def _check(status: int, where: str) -> None:
    if status != 0:
        raise PolyQError(status, where)


# --------------------------------------------------------------------------- helpers
def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(dev: torch.device) -> int:
    return torch.cuda.current_stream(dev).cuda_stream


def _need_cuda(*ts: Optional[torch.Tensor]) -> torch.device:
    dev = None
    for t in ts:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError("polyq device calls take GPU tensors")
        if not t.is_contiguous():
            raise ValueError("polyq device calls take contiguous tensors")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError("all tensors must be on the same device")
    return dev


def _as_u16(t: torch.Tensor) -> torch.Tensor:
    if t.element_size() != 2:
        raise ValueError(f"expected a 2-byte dtype, got {t.dtype}")
    return t


def _aligned_empty(nbytes: int, dev, align: int = 256) -> torch.Tensor:
    buf = torch.empty(nbytes + align, dtype=torch.uint8, device=dev)
    off = (-buf.data_ptr()) % align
    return buf[off:off + nbytes]


# --------------------------------------------------------------------------- API
def plan(n: int, k: int, blocks: Sequence[Tuple[int, int]]) -> Layout:
    """Validate a block list and return the packed layout (host only)."""
    blocks = [(int(b), int(l)) for b, l in blocks]
    arr = (Block * max(1, len(blocks)))(*[Block(b, l) for b, l in blocks])
    out = Layout()
    _check(lib().polyq_plan(int(n), int(k), arr, len(blocks), ctypes.byref(out)), "polyq_plan")
    return out


def pack(layout: Layout, codes: torch.Tensor, scales: torch.Tensor, zeros: torch.Tensor
         ) -> torch.Tensor:
    """Packed buffer (uint8, 256-byte aligned) on the codes' device."""
    dev = _need_cuda(codes, scales, zeros)
    _as_u16(codes), _as_u16(scales), _as_u16(zeros)
    if tuple(codes.shape) != (layout.n, layout.k):
        raise ValueError(f"codes shape {tuple(codes.shape)} != ({layout.n}, {layout.k})")
    if tuple(scales.shape) != (layout.n, layout.n_groups) or scales.shape != zeros.shape:
        raise ValueError("scales/zeros must be [n][n_groups]")
    packed = _aligned_empty(layout.packed_bytes, dev)
    _check(lib().polyq_pack(ctypes.byref(layout), _ptr(codes), _ptr(scales) if layout.n_groups else None,
                            _ptr(zeros) if layout.n_groups else None, _ptr(packed), _stream(dev)),
           "polyq_pack")
    return packed


def pack_rows(layout: Layout, codes: torch.Tensor, scales: torch.Tensor, zeros: torch.Tensor,
              row_perm: torch.Tensor) -> torch.Tensor:
    """Packed buffer whose row r is source row row_perm[r] (Eq. 10: the layer then
    emits y'[:, r] = y[:, row_perm[r]], a consumer's clustered input when
    row_perm is that consumer's permutation)."""
    dev = _need_cuda(codes, scales, zeros, row_perm)
    _as_u16(codes), _as_u16(scales), _as_u16(zeros)
    if tuple(codes.shape) != (layout.n, layout.k):
        raise ValueError(f"codes shape {tuple(codes.shape)} != ({layout.n}, {layout.k})")
    if tuple(scales.shape) != (layout.n, layout.n_groups) or scales.shape != zeros.shape:
        raise ValueError("scales/zeros must be [n][n_groups]")
    if row_perm.dtype != torch.int32 or tuple(row_perm.shape) != (layout.n,) or not row_perm.is_contiguous():
        raise ValueError(f"row_perm must be contiguous int32 [{layout.n}]")
    packed = _aligned_empty(layout.packed_bytes, dev)
    _check(lib().polyq_pack_rows(ctypes.byref(layout), _ptr(codes), _ptr(scales) if layout.n_groups else None,
                                 _ptr(zeros) if layout.n_groups else None, _ptr(row_perm), _ptr(packed),
                                 _stream(dev)),
           "polyq_pack_rows")
    return packed


def unpack(layout: Layout, packed: torch.Tensor):
    """(codes int16 [n][k], scales fp16 [n][G], zeros fp16 [n][G]) from a packed buffer."""
    dev = _need_cuda(packed)
    codes = torch.empty((layout.n, layout.k), dtype=torch.int16, device=dev)
    scales = torch.empty((layout.n, layout.n_groups), dtype=torch.float16, device=dev)
    zeros = torch.empty((layout.n, layout.n_groups), dtype=torch.float16, device=dev)
    g = layout.n_groups > 0
    _check(lib().polyq_unpack(ctypes.byref(layout), _ptr(packed), _ptr(codes),
                              _ptr(scales) if g else None, _ptr(zeros) if g else None, _stream(dev)),
           "polyq_unpack")
    return codes, scales, zeros


def permute(perm: torch.Tensor, x: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """x_out[i][k'] = x[i][perm[k']] for 2-byte x (fp16 / bf16)."""
    x2 = x if x.dim() == 2 else x.reshape(1, -1)
    dev = _need_cuda(perm, x2)
    _as_u16(x2)
    if perm.dtype != torch.int32 or perm.numel() != x2.shape[1]:
        raise ValueError("perm must be int32 [k]")
    out = torch.empty_like(x2) if out is None else out
    _check(lib().polyq_permute(_ptr(perm), _ptr(x2), _ptr(out), x2.shape[0], x2.shape[1],
                               _stream(dev)), "polyq_permute")
    return out if x.dim() == 2 else out.reshape(x.shape)


_ws: Dict[Tuple[str, int, int], list] = {}


def _workspace(kind: str, nbytes: int, dev: torch.device, zero_bytes: int = 0) -> Optional[torch.Tensor]:
    """A cached 256-byte aligned workspace per (kind, device, stream) whose first
    zero_bytes bytes are zero (the GEMV's split-K state; the bytes after it are
    the call's scratch, which the call leaves non-zero).  The cache remembers
    how long a prefix is known to be zero and clears only the difference."""
    if nbytes == 0:
        return None
    key = (kind, dev.index if dev.index is not None else torch.cuda.current_device(), _stream(dev))
    ent = _ws.get(key)
    if ent is None or ent[0].numel() < nbytes:
        size = max(nbytes, 2 * (ent[0].numel() if ent is not None else 0))
        raw = torch.zeros(size + 256, dtype=torch.uint8, device=dev)
        off = (-raw.data_ptr()) % 256
        ent = [raw[off:off + size], size]   # buffer, known-zero prefix
        _ws[key] = ent
    buf, clean = ent
    if zero_bytes > clean:
        buf[clean:zero_bytes].zero_()
        clean = zero_bytes
    # after the call [0, zero_bytes) is zero again; scratch after it is not
    ent[1] = zero_bytes if nbytes > zero_bytes else clean
    return buf


def gemv_workspace_bytes(layout: Layout, m: int) -> int:
    return int(lib().polyq_gemv_workspace_bytes(ctypes.byref(layout), int(m)))


def gemm_workspace_bytes(layout: Layout, m: int, perm_given: bool) -> int:
    return int(lib().polyq_gemm_workspace_bytes(ctypes.byref(layout), int(m), int(bool(perm_given))))


def gemv(layout: Layout, packed: torch.Tensor, perm: Optional[torch.Tensor], x: torch.Tensor,
         y: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """y fp32 [m][n] = x (fp16 [m][k]) times the packed layer; perm None = x pre-permuted."""
    x2 = x if x.dim() == 2 else x.reshape(1, -1)
    dev = _need_cuda(packed, perm, x2, y, workspace)
    if x2.dtype != torch.float16 or x2.shape[1] != layout.k:
        raise ValueError("x must be fp16 [m][k]")
    m = x2.shape[0]
    if perm is not None and (perm.dtype != torch.int32 or perm.numel() != layout.k):
        raise ValueError("perm must be int32 [k]")
    if y is None:
        y = torch.empty((m, layout.n), dtype=torch.float32, device=dev)
    if 1 <= m <= MAX_M_GEMV:
        one = (GemvItem * 1)(GemvItem(ctypes.pointer(layout), _ptr(packed), _ptr(perm), _ptr(x2), _ptr(y)))
        need = int(lib().polyq_gemv_batch_workspace_bytes(one, 1, m))
        zero = int(lib().polyq_gemv_batch_workspace_zero_bytes(one, 1, m))
    else:
        need = zero = 0
    ws = workspace if workspace is not None else _workspace("gemv", need, dev, zero)
    _check(lib().polyq_gemv(ctypes.byref(layout), _ptr(packed), _ptr(perm), _ptr(x2), m, _ptr(y),
                            _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(),
                            _stream(dev)), "polyq_gemv")
    return y


def gemv_batch(items: Sequence[Tuple[Layout, torch.Tensor, Optional[torch.Tensor], torch.Tensor,
                                     Optional[torch.Tensor]]],
               workspace: Optional[torch.Tensor] = None):
    """One launch of several GEMVs: items are (layout, packed, perm, x, y or None)
    with the same token count m.  Returns the list of outputs."""
    if not 1 <= len(items) <= MAX_BATCH:
        raise ValueError(f"1..{MAX_BATCH} items per batch")
    arr = (GemvItem * len(items))()
    keep, ys, m, dev = [], [], None, None
    for i, item in enumerate(items):
        layout, packed, perm, x, y, xscale = _item6(item)
        _check_xscale(xscale, layout)
        x2 = x if x.dim() == 2 else x.reshape(1, -1)
        d = _need_cuda(packed, perm, xscale, x2, y, workspace)
        dev = d if dev is None else dev
        if d != dev:
            raise ValueError("all tensors must be on the same device")
        if x2.dtype != torch.float16 or x2.shape[1] != layout.k:
            raise ValueError("x must be fp16 [m][k]")
        if m is None:
            m = x2.shape[0]
        elif x2.shape[0] != m:
            raise ValueError("every item of a batch has the same m")
        if perm is not None and (perm.dtype != torch.int32 or perm.numel() != layout.k):
            raise ValueError("perm must be int32 [k]")
        if y is None:
            y = torch.empty((m, layout.n), dtype=torch.float32, device=dev)
        arr[i] = GemvItem(ctypes.pointer(layout), _ptr(packed), _ptr(perm), _ptr(x2), _ptr(y), _ptr(xscale))
        keep.append(x2)
        ys.append(y)
    if 1 <= m <= MAX_M_GEMV:
        need = int(lib().polyq_gemv_batch_workspace_bytes(arr, len(items), m))
        zero = int(lib().polyq_gemv_batch_workspace_zero_bytes(arr, len(items), m))
    else:
        need = zero = 0
    ws = workspace if workspace is not None else _workspace("gemv", need, dev, zero)
    _check(lib().polyq_gemv_batch(arr, len(items), m, _ptr(ws),
                                  0 if ws is None else ws.numel() * ws.element_size(), _stream(dev)),
           "polyq_gemv_batch")
    return ys


def gemm(layout: Layout, packed: torch.Tensor, perm: Optional[torch.Tensor], x: torch.Tensor,
         y: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """y fp32 [m][n] = x (bf16 [m][k]) times the packed layer (prefill)."""
    x2 = x if x.dim() == 2 else x.reshape(1, -1)
    dev = _need_cuda(packed, perm, x2, y, workspace)
    if x2.dtype != torch.bfloat16 or x2.shape[1] != layout.k:
        raise ValueError("x must be bf16 [m][k]")
    m = x2.shape[0]
    if y is None:
        y = torch.empty((m, layout.n), dtype=torch.float32, device=dev)
    need = gemm_workspace_bytes(layout, m, perm is not None)
    ws = workspace if workspace is not None else _workspace("gemm", need, dev)
    _check(lib().polyq_gemm(ctypes.byref(layout), _ptr(packed), _ptr(perm), _ptr(x2), m, _ptr(y),
                            _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(),
                            _stream(dev)), "polyq_gemm")
    return y


def gemm_batch(items: Sequence[Tuple[Layout, torch.Tensor, Optional[torch.Tensor], torch.Tensor,
                                     Optional[torch.Tensor]]],
               workspace: Optional[torch.Tensor] = None):
    """One launch of several prefill GEMMs: items are (layout, packed, perm, x,
    y or None) with bf16 x and the same token count m.  Returns the outputs."""
    if not 1 <= len(items) <= MAX_BATCH:
        raise ValueError(f"1..{MAX_BATCH} items per batch")
    arr = (GemvItem * len(items))()
    keep, ys, m, dev = [], [], None, None
    for i, item in enumerate(items):
        layout, packed, perm, x, y, xscale = _item6(item)
        _check_xscale(xscale, layout)
        x2 = x if x.dim() == 2 else x.reshape(1, -1)
        d = _need_cuda(packed, perm, xscale, x2, y, workspace)
        dev = d if dev is None else dev
        if d != dev:
            raise ValueError("all tensors must be on the same device")
        if x2.dtype != torch.bfloat16 or x2.shape[1] != layout.k:
            raise ValueError("x must be bf16 [m][k]")
        if m is None:
            m = x2.shape[0]
        elif x2.shape[0] != m:
            raise ValueError("every item of a batch has the same m")
        if perm is not None and (perm.dtype != torch.int32 or perm.numel() != layout.k):
            raise ValueError("perm must be int32 [k]")
        if y is None:
            y = torch.empty((m, layout.n), dtype=torch.float32, device=dev)
        arr[i] = GemvItem(ctypes.pointer(layout), _ptr(packed), _ptr(perm), _ptr(x2), _ptr(y), _ptr(xscale))
        keep.append(x2)
        ys.append(y)
    need = int(lib().polyq_gemm_batch_workspace_bytes(arr, len(items), m))
    ws = workspace if workspace is not None else _workspace("gemm", need, dev)
    _check(lib().polyq_gemm_batch(arr, len(items), m, _ptr(ws),
                                  0 if ws is None else ws.numel() * ws.element_size(), _stream(dev)),
           "polyq_gemm_batch")
    return ys


class PreparedBatch:
    """One polyq_gemv_batch (kind "gemv") or polyq_gemm_batch (kind "gemm")
    launch whose arguments are marshalled once: the item array, the token count,
    the workspace (queried once and allocated once, zero-filled for the GEMV) and
    the output tensors are kept, so ``run()`` is a single library call.  The
    activations are read from the same tensors on every run (write new values
    into them in place).  items: (layout, packed, perm or None, x, y or None)."""

    def __init__(self, kind: str, items, workspace: Optional[torch.Tensor] = None):
        if kind not in ("gemv", "gemm"):
            raise ValueError(kind)
        if not 1 <= len(items) <= MAX_BATCH:
            raise ValueError(f"1..{MAX_BATCH} items per batch")
        want = torch.float16 if kind == "gemv" else torch.bfloat16
        self.kind = kind
        self.arr = (GemvItem * len(items))()
        self.keep, self.ys, self.layouts = [], [], []
        m, dev = None, None
        for i, item in enumerate(items):
            layout, packed, perm, x, y, xscale = _item6(item)
            _check_xscale(xscale, layout)
            x2 = x if x.dim() == 2 else x.reshape(1, -1)
            d = _need_cuda(packed, perm, xscale, x2, y, workspace)
            dev = d if dev is None else dev
            if d != dev:
                raise ValueError("all tensors must be on the same device")
            if x2.dtype != want or x2.shape[1] != layout.k:
                raise ValueError(f"x must be {want} [m][k]")
            if m is None:
                m = x2.shape[0]
            elif x2.shape[0] != m:
                raise ValueError("every item of a batch has the same m")
            if perm is not None and (perm.dtype != torch.int32 or perm.numel() != layout.k):
                raise ValueError("perm must be int32 [k]")
            if y is None:
                y = torch.empty((m, layout.n), dtype=torch.float32, device=dev)
            self.arr[i] = GemvItem(ctypes.pointer(layout), _ptr(packed), _ptr(perm), _ptr(x2), _ptr(y), _ptr(xscale))
            self.keep += [layout, packed, perm, x2, xscale]
            self.ys.append(y)
        self.m, self.count, self.dev = m, len(items), dev
        L = lib()
        if kind == "gemv":
            need = int(L.polyq_gemv_batch_workspace_bytes(self.arr, self.count, m)) if 1 <= m <= MAX_M_GEMV else 0
        else:
            need = int(L.polyq_gemm_batch_workspace_bytes(self.arr, self.count, m))
        # A workspace of its own (or one shared by prepared launches of the
        # same plan, which all leave the split-K state zero and write their
        # scratch after it): allocated zero-filled.
        if workspace is None and need:
            raw = (torch.zeros if kind == "gemv" else torch.empty)(need + 256, dtype=torch.uint8, device=dev)
            off = (-raw.data_ptr()) % 256
            workspace = raw[off:off + need]
        self.workspace = workspace
        self.ws_ptr = _ptr(workspace)
        self.ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
        self.fn = L.polyq_gemv_batch if kind == "gemv" else L.polyq_gemm_batch
        self.name = "polyq_gemv_batch" if kind == "gemv" else "polyq_gemm_batch"

    def run(self):
        _check(self.fn(self.arr, self.count, self.m, self.ws_ptr, self.ws_bytes, _stream(self.dev)), self.name)
        return self.ys


def read_probe(buf: torch.Tensor, nbytes: int, work_groups: int, sink: torch.Tensor) -> None:
    """Launch the streaming-read probe over the first nbytes of buf (a
    measurement utility: the reference read rate of a launch of that size)."""
    dev = _need_cuda(buf, sink)
    if sink.dtype != torch.int32 or sink.numel() < work_groups:
        raise ValueError("sink must be int32 with at least work_groups entries")
    if nbytes > buf.numel() * buf.element_size():
        raise ValueError("nbytes exceeds the buffer")
    _check(lib().polyq_read_probe(_ptr(buf), int(nbytes), int(work_groups), _ptr(sink), _stream(dev)),
           "polyq_read_probe")


NOALLOC_SCRATCH_BYTES = 16 << 20


def gemv_batch_noalloc(items):
    """polyq_gemv_batch_noalloc: the decode launch of gemv_batch with the
    library's own device scratch array as workspace (no allocation by the
    library; outputs must be given or are allocated here by torch).  items:
    (layout, packed, perm or None, x fp16 [m][k], y or None)."""
    if not 1 <= len(items) <= MAX_BATCH:
        raise ValueError(f"1..{MAX_BATCH} items per batch")
    arr = (GemvItem * len(items))()
    keep, ys, m, dev = [], [], None, None
    for i, item in enumerate(items):
        layout, packed, perm, x, y, xscale = _item6(item)
        _check_xscale(xscale, layout)
        x2 = x if x.dim() == 2 else x.reshape(1, -1)
        d = _need_cuda(packed, perm, xscale, x2, y)
        dev = d if dev is None else dev
        if d != dev:
            raise ValueError("all tensors must be on the same device")
        if x2.dtype != torch.float16 or x2.shape[1] != layout.k:
            raise ValueError("x must be fp16 [m][k]")
        if m is None:
            m = x2.shape[0]
        elif x2.shape[0] != m:
            raise ValueError("every item of a batch has the same m")
        if y is None:
            y = torch.empty((m, layout.n), dtype=torch.float32, device=dev)
        arr[i] = GemvItem(ctypes.pointer(layout), _ptr(packed), _ptr(perm), _ptr(x2), _ptr(y), _ptr(xscale))
        keep.append(x2)
        ys.append(y)
    _check(lib().polyq_gemv_batch_noalloc(arr, len(items), m, _stream(dev)), "polyq_gemv_batch_noalloc")
    return ys


# ---------------------------------------------------------------- bit allocation (host)
BITS = (2, 3, 4, 8, 16)


def _host(a, dtype):
    import numpy as np
    a = np.ascontiguousarray(a.detach().cpu().numpy() if isinstance(a, torch.Tensor) else a, dtype=dtype)
    return a, a.ctypes.data


def channel_error(w, x2, scale=None):
    """Eq. 2 error proxy (polyq_channel_error): w fp32 [n][k], x2 = E[x^2] [k],
    optional per-channel scales [k]; returns fp64 [5][k] (bits 2, 3, 4, 8, 16)."""
    import numpy as np
    wa, wp = _host(w, np.float32)
    n, k = wa.shape
    xa, xp = _host(x2, np.float64)
    sa, sp = (None, None) if scale is None else _host(scale, np.float32)
    err = np.empty((len(BITS), k), dtype=np.float64)
    _check(lib().polyq_channel_error(wp, n, k, xp, sp, err.ctypes.data), "polyq_channel_error")
    return err


def waterfill(err, budget: float):
    """Eq. 3-5 (polyq_waterfill): bits per channel."""
    import numpy as np
    ea, ep = _host(err, np.float64)
    k = ea.shape[1]
    bits = np.empty(k, dtype=np.int32)
    _check(lib().polyq_waterfill(ep, k, float(budget), bits.ctypes.data), "polyq_waterfill")
    return bits


def quanta_match(err, bits, quantum: int, budget: float):
    """Eq. 6 (polyq_quanta_match): snapped bits per channel and the per-bit counts."""
    import numpy as np
    ea, ep = _host(err, np.float64)
    out = np.array(bits, dtype=np.int32, copy=True)
    counts = np.empty(len(BITS), dtype=np.int32)
    _check(lib().polyq_quanta_match(ep, out.size, int(quantum), float(budget), out.ctypes.data,
                                    counts.ctypes.data), "polyq_quanta_match")
    return out, {b: int(c) for b, c in zip(BITS, counts)}


def cluster(bits):
    """Sec. 4.1 (polyq_cluster): perm (clustered position -> original channel) and blocks."""
    import numpy as np
    ba, bp = _host(bits, np.int32)
    perm = np.empty(ba.size, dtype=np.int32)
    blocks = (Block * MAX_BLOCKS)()
    nb = ctypes.c_int32(0)
    _check(lib().polyq_cluster(bp, ba.size, perm.ctypes.data, blocks, ctypes.byref(nb)), "polyq_cluster")
    return perm, [(blocks[i].bits, blocks[i].len) for i in range(nb.value)]


def allocate(w, x2, budget: float, quantum: int = QUANTUM, scale=None):
    """Sec. 3.1-3.3 end to end on the host: (bits, perm, blocks, counts)."""
    err = channel_error(w, x2, scale)
    bits, counts = quanta_match(err, waterfill(err, budget), quantum, budget)
    perm, blocks = cluster(bits)
    return bits, perm, blocks, counts


SCALE_GRID = tuple(i / 10 for i in range(11))


def bit_scaling(w, x2, saliency, bits, grid=SCALE_GRID):
    """Eq. 8 (polyq_bit_scaling): per-channel power-of-two scales s [k] (fp32)
    and the chosen exponent per bit-width {b: alpha_b}."""
    import numpy as np
    wa, wp = _host(w, np.float32)
    n, k = wa.shape
    xa, xp = _host(x2, np.float64)
    ma, mp = _host(saliency, np.float64)
    ba, bp = _host(bits, np.int32)
    ga, gp = _host(np.asarray(grid, dtype=np.float32), np.float32)
    scale = np.empty(k, dtype=np.float32)
    alpha = np.empty(len(BITS), dtype=np.float32)
    _check(lib().polyq_bit_scaling(wp, n, k, xp, mp, bp, gp, ga.size, scale.ctypes.data, alpha.ctypes.data),
           "polyq_bit_scaling")
    return scale, {b: float(a) for b, a in zip(BITS, alpha)}
