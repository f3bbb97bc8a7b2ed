"""Python binding of libvdattn.so: argument marshalling over the C ABI.

Every step of the attention path runs in the library's HIP kernels; this
module only checks shapes, dtypes and devices on the host and passes device
pointers, sizes and the current stream through ``ctypes``.  If the library is
not built, loading fails with an error (there is no other implementation).

Names follow ``include/vdattn.h``.
"""
from __future__ import annotations

import ctypes
import math
import os
import re
from dataclasses import dataclass
from typing import Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
# the in-tree build, or another build of the same sources (VDATTN_LIB: e.g. the
# host code built with sanitizers, oracle/sanitize.py)
LIB_PATH = os.environ.get("VDATTN_LIB") or os.path.join(HERE, "libvdattn.so")
HEADER = os.path.join(ROOT, "include", "vdattn.h")

VD_OK = 0
VD_ABI_VERSION = 4
VD_DTYPE_BF16 = 1
NOALLOC_SCRATCH_BYTES = 128 << 20  # VD_NOALLOC_SCRATCH_BYTES
TILE_KEYS = 64
SPLIT_KEYS = 1024
PAGE_SIZE = 16


class VdError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__("%s failed: %s (%d)" % (what, status_string(status), status))


class _Desc(ctypes.Structure):
    _fields_ = [("abi_version", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("softmax_scale", ctypes.c_float), ("window", ctypes.c_int32)]


class _Batch(ctypes.Structure):
    _fields_ = [("num_seqs", ctypes.c_int32), ("total_q_tokens", ctypes.c_int64),
                ("q", ctypes.c_void_p), ("cu_q_lens", ctypes.c_void_p),
                ("context_lens", ctypes.c_void_p), ("page_table", ctypes.c_void_p),
                ("pt_stride", ctypes.c_int32), ("k_pool", ctypes.c_void_p),
                ("v_pool", ctypes.c_void_p), ("num_pages", ctypes.c_int64),
                ("max_q_len", ctypes.c_int32), ("max_context_len", ctypes.c_int32),
                ("k_new", ctypes.c_void_p), ("v_new", ctypes.c_void_p),
                ("shared_pages", ctypes.c_int32), ("lse", ctypes.c_void_p)]


_lib = None


def load_library(path: str = LIB_PATH):
    """Loads libvdattn.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("libvdattn.so is not built (%s); run __graft_entry__.build() or "
                           "python -m paper_2609_38981_amd.build" % path)
    lib = ctypes.CDLL(path)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    sig = {
        "vd_attn_create": (ctypes.c_int, [ctypes.POINTER(_Desc), ctypes.POINTER(P)]),
        "vd_attn_destroy": (None, [P]),
        "vd_attn_workspace_size": (ctypes.c_int, [P, I32, I32, I32, ctypes.POINTER(SZ)]),
        "vd_attn_forward": (ctypes.c_int, [P, ctypes.POINTER(_Batch), P, P, SZ, P]),
        "vd_attn_forward_noalloc": (ctypes.c_int, [P, ctypes.POINTER(_Batch), P, P]),
        "vd_attn_forward_plan": (ctypes.c_int, [P, ctypes.POINTER(_Batch), P, SZ, P]),
        "vd_attn_forward_splits": (ctypes.c_int, [P, ctypes.POINTER(_Batch), P, P, SZ, P]),
        "vd_attn_forward_chunks": (ctypes.c_int, [P, ctypes.POINTER(_Batch), P, P, SZ, P]),
        "vd_attn_forward_merge": (ctypes.c_int, [P, ctypes.POINTER(_Batch), P, P, SZ, P]),
        "vd_attn_forward_splits_timed": (ctypes.c_int,
                                         [P, ctypes.POINTER(_Batch), P, P, SZ, P, P, P]),
        "vd_attn_forward_chunks_timed": (ctypes.c_int,
                                         [P, ctypes.POINTER(_Batch), P, P, SZ, P, P, P]),
        "vd_pool_bytes": (ctypes.c_int, [P, I64, ctypes.POINTER(SZ)]),
        "vd_attn_validate": (ctypes.c_int, [P, ctypes.POINTER(_Batch), P, P]),
        "vd_kv_write": (ctypes.c_int, [P, P, P, P, I64, P, P, I64, P]),
        "vd_linear": (ctypes.c_int, [P, I64, P, I64, P, I64, I64, I32, I32, P]),
        "vd_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "vd_attn_tiling": (ctypes.c_int, [P, ctypes.POINTER(I32), ctypes.POINTER(I32),
                                          ctypes.POINTER(I32)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def declared_functions(header: str = HEADER):
    """Names of the functions include/vdattn.h declares."""
    text = open(header).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(vd_[a-z_]+)\s*\(", text)))


def status_string(status: int) -> str:
    return load_library().vd_status_string(int(status)).decode()


def _check(status: int, what: str):
    if status != VD_OK:
        raise VdError(status, what)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _need(t: torch.Tensor, name: str, dtype, numel: Optional[int] = None):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a tensor" % name)
    if t.device.type != "cuda":
        raise ValueError("%s must be a device tensor" % name)
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if numel is not None and t.numel() < numel:
        raise ValueError("%s has %d elements, needs %d" % (name, t.numel(), numel))


@dataclass
class Batch:
    """One call's packed inputs (device tensors) and host hints."""
    q: torch.Tensor             # [T, Hq, D] bf16
    cu_q_lens: torch.Tensor     # [B + 1] int32
    context_lens: torch.Tensor  # [B] int32
    page_table: torch.Tensor    # [B, stride] int32
    k_pool: torch.Tensor        # bf16, vd_pool_bytes(num_pages) bytes
    v_pool: torch.Tensor
    num_pages: int
    max_q_len: int
    max_context_len: int
    # optional K/V of the query rows, written into the pool before attention
    k_new: Optional[torch.Tensor] = None  # [T, Hkv, D] bf16, row t = query row t
    v_new: Optional[torch.Tensor] = None  # [T, Hkv, D] bf16
    # host hint: some pages are read by several requests (keeps K/V cached)
    shared_pages: bool = False
    # optional output: [T, Hq] float32 log-sum-exp of each row's visible scaled scores
    lse: Optional[torch.Tensor] = None


class VdAttn:
    """Handle of one fixed attention configuration (immutable)."""

    def __init__(self, num_q_heads: int, num_kv_heads: int, head_dim: int, page_size: int = 16,
                 softmax_scale: float = 0.0, window: int = 0):
        self.lib = load_library()
        d = _Desc(VD_ABI_VERSION, num_q_heads, num_kv_heads, head_dim, page_size, VD_DTYPE_BF16,
                  float(softmax_scale), int(window))
        h = ctypes.c_void_p()
        _check(self.lib.vd_attn_create(ctypes.byref(d), ctypes.byref(h)), "vd_attn_create")
        self._h = h
        self.num_q_heads, self.num_kv_heads, self.head_dim = num_q_heads, num_kv_heads, head_dim
        self.page_size = page_size
        self.window = int(window)
        self.softmax_scale = softmax_scale if softmax_scale > 0 else 1.0 / math.sqrt(head_dim)

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            self.lib.vd_attn_destroy(h)
            self._h = None

    # -- sizes -------------------------------------------------------------
    def workspace_size(self, num_seqs: int, max_q_len: int, max_context_len: int) -> int:
        n = ctypes.c_size_t()
        _check(self.lib.vd_attn_workspace_size(self._h, num_seqs, max_q_len, max_context_len,
                                               ctypes.byref(n)), "vd_attn_workspace_size")
        return n.value

    def pool_bytes(self, num_pages: int) -> int:
        n = ctypes.c_size_t()
        _check(self.lib.vd_pool_bytes(self._h, num_pages, ctypes.byref(n)), "vd_pool_bytes")
        return n.value

    def tiling(self):
        a, b, c = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        _check(self.lib.vd_attn_tiling(self._h, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)),
               "vd_attn_tiling")
        return a.value, b.value, c.value

    # -- allocation helpers (torch owns the memory) ------------------------
    def new_pool(self, num_pages: int, device="cuda") -> torch.Tensor:
        return torch.empty(self.pool_bytes(num_pages) // 2, dtype=torch.bfloat16, device=device)

    def new_workspace(self, num_seqs: int, max_q_len: int, max_context_len: int,
                      device="cuda") -> torch.Tensor:
        n = self.workspace_size(num_seqs, max_q_len, max_context_len)
        return torch.empty(max(n, 1), dtype=torch.uint8, device=device)

    # -- calls ---------------------------------------------------------------
    def _batch(self, b: Batch) -> _Batch:
        B = int(b.context_lens.numel())
        T = int(b.q.shape[0]) if b.q.dim() else 0
        _need(b.q, "q", torch.bfloat16)
        if tuple(b.q.shape[1:]) != (self.num_q_heads, self.head_dim):
            raise ValueError("q must be [T, %d, %d], got %s" % (self.num_q_heads, self.head_dim,
                                                               tuple(b.q.shape)))
        _need(b.cu_q_lens, "cu_q_lens", torch.int32)
        _need(b.context_lens, "context_lens", torch.int32)
        _need(b.page_table, "page_table", torch.int32)
        if b.cu_q_lens.numel() != B + 1:
            raise ValueError("cu_q_lens must have num_seqs + 1 entries")
        if b.page_table.dim() != 2 or b.page_table.shape[0] != B:
            raise ValueError("page_table must be [num_seqs, stride]")
        pool_elems = self.pool_bytes(b.num_pages) // 2
        _need(b.k_pool, "k_pool", torch.bfloat16, pool_elems)
        _need(b.v_pool, "v_pool", torch.bfloat16, pool_elems)
        stride = int(b.page_table.shape[1]) if B else 1
        if (b.k_new is None) != (b.v_new is None):
            raise ValueError("k_new and v_new go together")
        if b.k_new is not None:
            per = self.num_kv_heads * self.head_dim
            _need(b.k_new, "k_new", torch.bfloat16, T * per)
            _need(b.v_new, "v_new", torch.bfloat16, T * per)
        if b.lse is not None:
            _need(b.lse, "lse", torch.float32, T * self.num_q_heads)
        return _Batch(B, T, _ptr(b.q), _ptr(b.cu_q_lens), _ptr(b.context_lens),
                      _ptr(b.page_table), stride, _ptr(b.k_pool), _ptr(b.v_pool),
                      int(b.num_pages), int(b.max_q_len), int(b.max_context_len),
                      _ptr(b.k_new), _ptr(b.v_new), int(bool(b.shared_pages)), _ptr(b.lse))

    def _ws(self, b: Batch, workspace):
        need = self.workspace_size(int(b.context_lens.numel()), b.max_q_len, b.max_context_len)
        if workspace is None:
            workspace = self.new_workspace(int(b.context_lens.numel()), b.max_q_len,
                                           b.max_context_len, b.q.device)
        _need(workspace, "workspace", torch.uint8, need)
        return workspace

    def _out(self, b: Batch, out):
        if out is None:
            out = torch.empty_like(b.q)
        _need(out, "out", torch.bfloat16, b.q.numel())
        if out.shape != b.q.shape:
            raise ValueError("out must have q's shape")
        return out

    def forward(self, b: Batch, out=None, workspace=None, stream=None) -> torch.Tensor:
        cb = self._batch(b)
        out = self._out(b, out)
        ws = self._ws(b, workspace)
        _check(self.lib.vd_attn_forward(self._h, ctypes.byref(cb), _ptr(out), _ptr(ws), ws.numel(),
                                        _stream(stream)), "vd_attn_forward")
        return out

    def forward_noalloc(self, b: Batch, out: torch.Tensor, stream=None) -> torch.Tensor:
        """vd_attn_forward_noalloc: the call with the library's own static
        scratch as its workspace (the C call allocates nothing); ``out`` is
        the caller's."""
        cb = self._batch(b)
        out = self._out(b, out)
        _check(self.lib.vd_attn_forward_noalloc(self._h, ctypes.byref(cb), _ptr(out),
                                                _stream(stream)), "vd_attn_forward_noalloc")
        return out

    def forward_plan(self, b: Batch, workspace, stream=None):
        cb = self._batch(b)
        ws = self._ws(b, workspace)
        _check(self.lib.vd_attn_forward_plan(self._h, ctypes.byref(cb), _ptr(ws), ws.numel(),
                                             _stream(stream)), "vd_attn_forward_plan")

    def forward_splits(self, b: Batch, out, workspace, stream=None):
        cb = self._batch(b)
        out = self._out(b, out)
        ws = self._ws(b, workspace)
        _check(self.lib.vd_attn_forward_splits(self._h, ctypes.byref(cb), _ptr(out), _ptr(ws),
                                               ws.numel(), _stream(stream)),
               "vd_attn_forward_splits")

    def forward_chunks(self, b: Batch, out, workspace, stream=None):
        cb = self._batch(b)
        out = self._out(b, out)
        ws = self._ws(b, workspace)
        _check(self.lib.vd_attn_forward_chunks(self._h, ctypes.byref(cb), _ptr(out), _ptr(ws),
                                               ws.numel(), _stream(stream)),
               "vd_attn_forward_chunks")

    def forward_merge(self, b: Batch, out, workspace, stream=None):
        cb = self._batch(b)
        out = self._out(b, out)
        ws = self._ws(b, workspace)
        _check(self.lib.vd_attn_forward_merge(self._h, ctypes.byref(cb), _ptr(out), _ptr(ws),
                                              ws.numel(), _stream(stream)), "vd_attn_forward_merge")

    def prepare(self, b: Batch, out=None, workspace=None, stream=None) -> "PreparedCall":
        """Marshals one call's arguments once, for callers that launch the same
        call (same tensors, same stream) many times."""
        return PreparedCall(self, b, out, workspace, stream)

    def validate(self, b: Batch, stream=None) -> torch.Tensor:
        """Per-request bit masks of the device-side preconditions each request
        violates (0: none), as int32 [num_seqs] on the device; see vd_attn_validate."""
        cb = self._batch(b)
        status = torch.full((int(b.context_lens.numel()),), -1, dtype=torch.int32, device="cuda")
        _check(self.lib.vd_attn_validate(self._h, ctypes.byref(cb), _ptr(status), _stream(stream)),
               "vd_attn_validate")
        return status

    def kv_write(self, k_new: torch.Tensor, v_new: torch.Tensor, slot_mapping: torch.Tensor,
                 k_pool: torch.Tensor, v_pool: torch.Tensor, num_pages: int, stream=None):
        T = int(slot_mapping.numel())
        per = self.num_kv_heads * self.head_dim
        _need(k_new, "k_new", torch.bfloat16, T * per)
        _need(v_new, "v_new", torch.bfloat16, T * per)
        _need(slot_mapping, "slot_mapping", torch.int64)
        pool_elems = self.pool_bytes(num_pages) // 2
        _need(k_pool, "k_pool", torch.bfloat16, pool_elems)
        _need(v_pool, "v_pool", torch.bfloat16, pool_elems)
        _check(self.lib.vd_kv_write(self._h, _ptr(k_new), _ptr(v_new), _ptr(slot_mapping), T,
                                    _ptr(k_pool), _ptr(v_pool), int(num_pages), _stream(stream)),
               "vd_kv_write")


class PreparedCall:
    """The C arguments of one attention call, checked and marshalled once.

    Holds references to every tensor it points at.  Each method is one C call
    with those arguments; the phases compose exactly like forward()."""

    def __init__(self, attn: VdAttn, b: Batch, out=None, workspace=None, stream=None):
        self.attn, self.batch = attn, b
        self.cb = attn._batch(b)
        self.out = attn._out(b, out)
        self.workspace = attn._ws(b, workspace)
        self.stream = stream
        lib, h = attn.lib, attn._h
        pcb, sp = ctypes.byref(self.cb), _stream(stream)
        o, w, wn = _ptr(self.out), _ptr(self.workspace), self.workspace.numel()
        self._fwd = (lib.vd_attn_forward, (h, pcb, o, w, wn, sp))
        self._plan = (lib.vd_attn_forward_plan, (h, pcb, w, wn, sp))
        self._splits = (lib.vd_attn_forward_splits, (h, pcb, o, w, wn, sp))
        self._chunks = (lib.vd_attn_forward_chunks, (h, pcb, o, w, wn, sp))
        self._merge = (lib.vd_attn_forward_merge, (h, pcb, o, w, wn, sp))
        self._splits_timed = (lib.vd_attn_forward_splits_timed, (h, pcb, o, w, wn, sp))
        self._chunks_timed = (lib.vd_attn_forward_chunks_timed, (h, pcb, o, w, wn, sp))

    @staticmethod
    def _run(fa, what):
        fn, args = fa
        _check(fn(*args), what)

    def forward(self) -> torch.Tensor:
        self._run(self._fwd, "vd_attn_forward")
        return self.out

    def plan(self):
        self._run(self._plan, "vd_attn_forward_plan")

    @staticmethod
    def _timed(fa, events, what):
        """events: a pair of torch.cuda.Event(enable_timing=True); the kernel's
        dispatch records them at its start and end."""
        fn, args = fa
        for e in events:
            if not e.cuda_event:  # torch creates the event at its first record
                e.record()
        _check(fn(*args, events[0].cuda_event, events[1].cuda_event), what)

    def splits(self, events=None):
        if events is None:
            self._run(self._splits, "vd_attn_forward_splits")
        else:
            self._timed(self._splits_timed, events, "vd_attn_forward_splits_timed")

    def chunks(self, events=None):
        if events is None:
            self._run(self._chunks, "vd_attn_forward_chunks")
        else:
            self._timed(self._chunks_timed, events, "vd_attn_forward_chunks_timed")

    def merge(self):
        self._run(self._merge, "vd_attn_forward_merge")


def linear(a: torch.Tensor, b: torch.Tensor, out: Optional[torch.Tensor] = None,
           stream=None) -> torch.Tensor:
    """Batch-invariant linear layer (vd_linear): out = a @ b^T with a [M, K]
    bf16 activations and b [N, K] bf16 weights, out [M, N] bf16; row m of the
    output depends only on row m of a and on b.  Rows may be strided (the
    last dimension contiguous)."""
    lib = load_library()
    for t, name in ((a, "a"), (b, "b")):
        if not isinstance(t, torch.Tensor) or t.device.type != "cuda" or t.dtype != torch.bfloat16:
            raise TypeError("%s must be a bf16 device tensor" % name)
        if t.dim() != 2 or t.stride(1) != 1:
            raise ValueError("%s must be 2-D with contiguous rows" % name)
    M, K = a.shape
    N, Kb = b.shape
    if Kb != K:
        raise ValueError("a is [M, %d] but b is [N, %d]" % (K, Kb))
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device=a.device)
    if out.dtype != torch.bfloat16 or out.dim() != 2 or out.shape != (M, N) or out.stride(1) != 1:
        raise ValueError("out must be bf16 [M, N] with contiguous rows")
    _check(lib.vd_linear(a.data_ptr(), a.stride(0), b.data_ptr(), b.stride(0), out.data_ptr(),
                         out.stride(0), M, N, K, _stream(stream)), "vd_linear")
    return out
