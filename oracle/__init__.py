"""Plain CPU oracle for paged causal attention and for the linear layer --
TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never imports, links or calls it, and the oracle imports
nothing from the product.

The arithmetic lives in ``vd_oracle.c`` (IEEE double, plain loops, ascending
sums), which follows the problem statement of the paper's Appendix A.1 and the
causal contract of Section 5.3: row ``i`` of a request with query length ``s``
and key length ``n`` is logical position ``p = n - s + i`` and attends to the
logical keys ``0..p`` gathered through the request's page table.

Pool layout read by the oracle: ``[num_pages, num_kv_heads, page_size,
head_dim]`` bf16 bit patterns (uint16).  This is the oracle's own plain layout;
the GPU library keeps its pool in a layout of its own.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "vd_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
# another build of the same source, e.g. with sanitizers (oracle/sanitize.py)
_OVERRIDE = os.environ.get("VDO_ORACLE_LIB")
_lock = threading.Lock()
_lib = None

ERRORS = {
    -1: "invalid argument",
    -2: "invalid lengths (need 0 < s <= n, cu_q_lens consistent, pages fit the table)",
    -3: "page id out of range",
    -4: "out of memory / thread start failure",
}


def build(force: bool = True) -> str:
    """Compile the oracle with gcc into ``oracle/liboracle.so``."""
    if not force and os.path.exists(_LIB) and os.path.getmtime(_LIB) >= os.path.getmtime(_SRC):
        return _LIB
    tmp = _LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-std=c11", "-fPIC",
           "-shared", "-pthread", _SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


def bind(path: str):
    """Loads an oracle shared library (the built one, or a test's mutant)."""
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    lib.vdo_paged_attention.restype = ctypes.c_int
    lib.vdo_paged_attention.argtypes = [
        ctypes.c_int, ctypes.c_int64, ctypes.c_int, ctypes.c_int, ctypes.c_int,
        ctypes.c_int, ctypes.c_double, ctypes.c_int, P, P, P, P, ctypes.c_int, P, P,
        ctypes.c_int64, P, P, P, ctypes.c_int]
    lib.vdo_default_threads.restype = ctypes.c_int
    if hasattr(lib, "vdo_dense_attention"):
        lib.vdo_dense_attention.restype = ctypes.c_int
        lib.vdo_dense_attention.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                            ctypes.c_int, ctypes.c_double, ctypes.c_int, P, P, P,
                                            P, P]
    if hasattr(lib, "vdo_linear"):
        lib.vdo_linear.restype = ctypes.c_int
        lib.vdo_linear.argtypes = [ctypes.c_int64, ctypes.c_int, ctypes.c_int, P, ctypes.c_int64,
                                   P, ctypes.c_int64, P, ctypes.c_int]
    return lib


def _load():
    global _lib
    with _lock:
        if _lib is None:
            if _OVERRIDE:
                _lib = bind(_OVERRIDE)
            else:
                build(force=False)
                _lib = bind(_LIB)
    return _lib


def default_threads() -> int:
    return int(_load().vdo_default_threads())


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data_as(ctypes.c_void_p)


def paged_attention(q_bits, cu_q_lens, context_lens, page_table, k_pool_bits, v_pool_bits,
                    *, num_q_heads, num_kv_heads, head_dim, page_size, scale=None,
                    window=0, rows=None, threads=0, lib=None, with_lse=False):
    """Exact (fp64) paged causal attention.

    q_bits:        uint16 [T, Hq, D] bf16 bit patterns, rows packed by request.
    cu_q_lens:     int32 [B+1] query-row offsets (cu[0] = 0, cu[B] = T).
    context_lens:  int32 [B] key lengths n_r (count this call's own tokens).
    page_table:    int32 [B, stride]; the first ceil(n_r / P) entries are used.
    k/v_pool_bits: uint16 [num_pages, Hkv, P, D] bf16 bit patterns.
    scale:         softmax scale (default 1/sqrt(D)).
    window:        0 for the full causal prefix; w > 0 restricts row p to the
                   sliding window of keys p - w < j <= p (Appendix A.5).
    rows:          optional iterable of token indices (or bool mask [T]); only
                   those rows are computed, the rest of the result is NaN.
    threads:       host threads (0 = all online cores).
    lib:           an alternative library from ``bind`` (tests of the pins).
    with_lse:      also return the rows' log-sum-exp of the scaled scores over
                   the visible keys (natural log), float64 [T, Hq].

    Returns float64 [T, Hq, D] (and the log-sum-exp with ``with_lse``).
    """
    lib = _load() if lib is None else lib
    q_bits, qp = _c(q_bits, np.uint16)
    T = q_bits.shape[0]
    assert q_bits.shape == (T, num_q_heads, head_dim), q_bits.shape
    cu, cup = _c(cu_q_lens, np.int32)
    ctx, ctxp = _c(context_lens, np.int32)
    pt, ptp = _c(page_table, np.int32)
    B = ctx.shape[0]
    assert cu.shape == (B + 1,)
    pt = pt.reshape(B, -1) if B else pt.reshape(0, 0)
    stride = pt.shape[1] if B else 0
    kp, kpp = _c(k_pool_bits, np.uint16)
    vp, vpp = _c(v_pool_bits, np.uint16)
    assert kp.shape == vp.shape and kp.ndim == 4
    assert kp.shape[1:] == (num_kv_heads, page_size, head_dim), kp.shape
    if scale is None:
        scale = 1.0 / np.sqrt(head_dim)
    sel = None
    selp = None
    if rows is not None:
        rows_arr = np.asarray(rows)
        if rows_arr.dtype == bool:
            sel = rows_arr.astype(np.uint8)
        else:
            sel = np.zeros(T, np.uint8)
            sel[rows_arr.astype(np.int64)] = 1
        sel, selp = _c(sel, np.uint8)
    out = np.full((T, num_q_heads, head_dim), np.nan, np.float64)
    lse = np.full((T, num_q_heads), np.nan, np.float64) if with_lse else None
    rc = lib.vdo_paged_attention(
        B, T, num_q_heads, num_kv_heads, head_dim, page_size, float(scale), int(window), qp,
        cup, ctxp, ptp, stride, kpp, vpp, kp.shape[0], selp,
        out.ctypes.data_as(ctypes.c_void_p),
        lse.ctypes.data_as(ctypes.c_void_p) if with_lse else None, int(threads))
    if rc != 0:
        raise ValueError("oracle rejected the call: %s (%d)" % (ERRORS.get(rc, "?"), rc))
    return (out, lse) if with_lse else out


def dense_attention(q_bits, k_bits, v_bits, *, num_q_heads, num_kv_heads, head_dim, scale=None,
                    window=0, lib=None, with_lse=False):
    """Exact (fp64) causal attention of one request whose keys and values are
    contiguous (no page table): the dense variant of ``paged_attention``.

    q_bits: uint16 [s, Hq, D]; k_bits, v_bits: uint16 [n, Hkv, D] (bf16 bit
    patterns); row i stands for position n - s + i.  Returns float64
    [s, Hq, D] (and the log-sum-exp [s, Hq] with ``with_lse``)."""
    lib = _load() if lib is None else lib
    q, qp = _c(q_bits, np.uint16)
    k, kp = _c(k_bits, np.uint16)
    v, vp = _c(v_bits, np.uint16)
    s, n = q.shape[0], k.shape[0]
    assert q.shape == (s, num_q_heads, head_dim), q.shape
    assert k.shape == v.shape == (n, num_kv_heads, head_dim), (k.shape, v.shape)
    if scale is None:
        scale = 1.0 / np.sqrt(head_dim)
    out = np.full((s, num_q_heads, head_dim), np.nan, np.float64)
    lse = np.full((s, num_q_heads), np.nan, np.float64) if with_lse else None
    rc = lib.vdo_dense_attention(s, n, num_q_heads, num_kv_heads, head_dim, float(scale),
                                 int(window), qp, kp, vp, out.ctypes.data_as(ctypes.c_void_p),
                                 lse.ctypes.data_as(ctypes.c_void_p) if with_lse else None)
    if rc != 0:
        raise ValueError("oracle rejected the call: %s (%d)" % (ERRORS.get(rc, "?"), rc))
    return (out, lse) if with_lse else out


def linear(a_bits, b_bits, *, k=None, threads=0, lib=None):
    """Exact (fp64) linear layer, c = a . b^T (the matmul contract of the
    paper's Section 5.4, Fig. 3).

    a_bits: uint16 [M, lda] bf16 bit patterns (activations; the first k
            columns are used, k defaults to lda).
    b_bits: uint16 [N, ldb] bf16 bit patterns (weights, one row per output
            column; the first k columns are used).
    Returns float64 [M, N]."""
    lib = _load() if lib is None else lib
    a, ap = _c(a_bits, np.uint16)
    b, bp = _c(b_bits, np.uint16)
    assert a.ndim == 2 and b.ndim == 2
    M, lda = a.shape
    N, ldb = b.shape
    K = lda if k is None else int(k)
    c = np.full((M, N), np.nan, np.float64)
    rc = lib.vdo_linear(M, N, K, ap, lda, bp, ldb, c.ctypes.data_as(ctypes.c_void_p), int(threads))
    if rc != 0:
        raise ValueError("oracle rejected the linear call: %s (%d)" % (ERRORS.get(rc, "?"), rc))
    return c
