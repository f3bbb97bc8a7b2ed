"""CPU checks of the C ABI: the library loads, exports every function the
header declares, and rejects bad host-side arguments before any launch.
Nothing here runs a kernel."""
from __future__ import annotations

import ctypes

import pytest

from paper_2609_38981_amd import vdattn as V


@pytest.fixture(scope="module")
def lib():
    return V.load_library()


def test_exports_every_declared_function(lib):
    names = V.declared_functions()
    assert len(names) >= 11, names
    for name in names:
        assert hasattr(lib, name), name


def _create(lib, **kw):
    d = dict(abi_version=V.VD_ABI_VERSION, num_q_heads=32, num_kv_heads=8, head_dim=128,
             page_size=16, dtype=1, softmax_scale=0.0, window=0)
    d.update(kw)
    desc = V._Desc(**d)
    h = ctypes.c_void_p()
    rc = lib.vd_attn_create(ctypes.byref(desc), ctypes.byref(h))
    return rc, h


def test_create_supported_and_destroy(lib):
    for hq, hkv, d, w in [(32, 8, 128, 0), (64, 8, 128, 0), (4, 2, 64, 0), (8, 8, 64, 0),
                          (32, 8, 128, 4096), (4, 2, 64, 1)]:
        rc, h = _create(lib, num_q_heads=hq, num_kv_heads=hkv, head_dim=d, window=w)
        assert rc == 0 and h.value
        a, b, c = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        assert lib.vd_attn_tiling(h, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)) == 0
        assert (a.value, b.value, c.value) == (64, 1024, 16)
        lib.vd_attn_destroy(h)
    lib.vd_attn_destroy(None)


@pytest.mark.parametrize("kw,code", [
    (dict(head_dim=96), -2), (dict(head_dim=256), -2), (dict(page_size=32), -2),
    (dict(dtype=2), -2), (dict(num_q_heads=12, num_kv_heads=8), -2),
    (dict(num_q_heads=64, num_kv_heads=1), -2), (dict(abi_version=5), -1),
    (dict(num_kv_heads=0), -1), (dict(softmax_scale=float("nan")), -1), (dict(window=-1), -1),
    (dict(abi_version=1), -1), (dict(abi_version=2), -1), (dict(abi_version=3), -1),
])
def test_create_rejects(lib, kw, code):
    rc, h = _create(lib, **kw)
    assert rc == code and not h.value


def test_status_strings(lib):
    for code in (0, -1, -2, -3, -4, 7):
        assert lib.vd_status_string(code)


def test_workspace_and_pool_sizes(lib):
    rc, h = _create(lib)
    n = ctypes.c_size_t()
    assert lib.vd_attn_workspace_size(h, 64, 8, 4096, ctypes.byref(n)) == 0
    # m, z and U (D floats) per (request, KV head, 32 columns, 4 splits of 1024 keys)
    entries = 64 * 8 * 32 * 4
    assert n.value >= entries * (2 + 128) * 4
    # single-token rows of 4 query heads per KV head: 4 columns
    assert lib.vd_attn_workspace_size(h, 64, 1, 4096, ctypes.byref(n)) == 0
    assert 64 * 8 * 4 * 4 * (2 + 128) * 4 <= n.value < 64 * 8 * 8 * 4 * (2 + 128) * 4
    assert lib.vd_attn_workspace_size(h, -1, 1, 1, ctypes.byref(n)) == -1
    assert lib.vd_pool_bytes(h, 10, ctypes.byref(n)) == 0
    assert n.value == 10 * 8 * 16 * 128 * 2
    lib.vd_attn_destroy(h)


def test_forward_rejects_before_launch(lib):
    rc, h = _create(lib)
    fake = 0x1000  # never dereferenced: every case below fails a host check
    b = V._Batch(1, 1, fake, fake, fake, fake, 1, fake, fake, 4, 1, 16, None, None, 0)
    ws = ctypes.c_size_t()
    lib.vd_attn_workspace_size(h, 1, 1, 16, ctypes.byref(ws))
    # missing workspace / too small
    assert lib.vd_attn_forward(h, ctypes.byref(b), fake, None, 0, None) == -3
    assert lib.vd_attn_forward(h, ctypes.byref(b), fake, fake, ws.value - 1, None) == -3
    # null output
    assert lib.vd_attn_forward(h, ctypes.byref(b), None, fake, ws.value, None) == -1
    # null input pointers, bad sizes, inconsistent hints
    for field, val in [("q", None), ("page_table", None), ("pt_stride", 0), ("num_pages", 0),
                       ("max_q_len", 0), ("max_context_len", 0), ("num_seqs", -1)]:
        bb = V._Batch(1, 1, fake, fake, fake, fake, 1, fake, fake, 4, 1, 16, None, None, 0)
        setattr(bb, field, val)
        assert lib.vd_attn_forward(h, ctypes.byref(bb), fake, fake, ws.value, None) == -1, field
    bb = V._Batch(1, 1, fake, fake, fake, fake, 1, fake, fake, 4, 32, 16, None, None, 0)  # max_q > max_ctx
    assert lib.vd_attn_forward(h, ctypes.byref(bb), fake, fake, ws.value, None) == -1
    # an empty batch is a no-op
    e = V._Batch(0, 0, None, None, None, None, 0, None, None, 0, 0, 0, None, None, 0)
    assert lib.vd_attn_forward(h, ctypes.byref(e), None, None, 0, None) == 0
    assert lib.vd_attn_forward(None, ctypes.byref(e), None, None, 0, None) == -1
    # fused new tokens: k_new without v_new, or v_new without k_new
    for kn, vn in [(fake, None), (None, fake)]:
        bb = V._Batch(1, 1, fake, fake, fake, fake, 1, fake, fake, 4, 1, 16, kn, vn, 0)
        for fn in (lib.vd_attn_forward_plan,):
            assert fn(h, ctypes.byref(bb), fake, ws.value, None) == -1
        assert lib.vd_attn_forward(h, ctypes.byref(bb), fake, fake, ws.value, None) == -1
    # kv write
    assert lib.vd_kv_write(h, fake, fake, fake, -1, fake, fake, 4, None) == -1
    assert lib.vd_kv_write(h, None, fake, fake, 3, fake, fake, 4, None) == -1
    assert lib.vd_kv_write(h, fake, fake, fake, 0, fake, fake, 4, None) == 0
    lib.vd_attn_destroy(h)


def test_linear_rejects_before_launch(lib):
    """vd_linear's host checks: every case returns before a kernel is launched."""
    fake = 0x1000  # 16-byte aligned, never dereferenced
    f = lib.vd_linear
    i64, i32 = ctypes.c_int64, ctypes.c_int32
    ok = dict(a=fake, lda=64, b=fake, ldb=64, c=fake, ldc=16, M=4, N=16, K=64)

    def call(**kw):
        d = dict(ok)
        d.update(kw)
        return f(ctypes.c_void_p(d["a"]), i64(d["lda"]), ctypes.c_void_p(d["b"]), i64(d["ldb"]),
                 ctypes.c_void_p(d["c"]), i64(d["ldc"]), i64(d["M"]), i32(d["N"]), i32(d["K"]),
                 None)

    # an empty output is a no-op
    assert call(M=0) == 0 and call(N=0) == 0
    # negative sizes, a missing or too narrow output, misaligned rows or pointers
    for kw in (dict(M=-1), dict(N=-1), dict(K=-1), dict(c=0), dict(ldc=8), dict(c=fake + 1),
               dict(a=0), dict(b=0), dict(lda=32), dict(ldb=32), dict(lda=68), dict(ldb=68),
               dict(a=fake + 8), dict(b=fake + 8)):
        assert call(**kw) == -1, kw
    # K must be a multiple of the 64-wide step
    assert call(K=96, lda=96, ldb=96) == -2


def test_forward_rejects_misaligned_pointers(lib):
    """Every buffer the kernels access with vector loads must be aligned: a
    misaligned one is rejected before any launch (VD_ERR_INVALID_ARG), on every
    entry point that takes the batch."""
    rc, h = _create(lib)
    fake = 0x10000  # 16-byte aligned, never dereferenced
    ws = ctypes.c_size_t()
    lib.vd_attn_workspace_size(h, 1, 1, 16, ctypes.byref(ws))

    def batch(**kw):
        b = V._Batch(1, 1, fake, fake, fake, fake, 1, fake, fake, 4, 1, 16, None, None, 0, None)
        for k, v in kw.items():
            setattr(b, k, v)
        return b

    # bf16 buffers at 16 bytes, int32 / fp32 arrays at 4
    cases = [dict(q=fake + 8), dict(k_pool=fake + 2), dict(v_pool=fake + 4),
             dict(k_new=fake + 8, v_new=fake), dict(k_new=fake, v_new=fake + 2),
             dict(cu_q_lens=fake + 2), dict(context_lens=fake + 1), dict(page_table=fake + 2),
             dict(lse=fake + 2)]
    for kw in cases:
        b = batch(**kw)
        assert lib.vd_attn_forward(h, ctypes.byref(b), fake, fake, ws.value, None) == -1, kw
        assert lib.vd_attn_forward_plan(h, ctypes.byref(b), fake, ws.value, None) == -1, kw
        assert lib.vd_attn_forward_splits(h, ctypes.byref(b), fake, fake, ws.value, None) == -1, kw
        assert lib.vd_attn_forward_chunks(h, ctypes.byref(b), fake, fake, ws.value, None) == -1, kw
        assert lib.vd_attn_forward_merge(h, ctypes.byref(b), fake, fake, ws.value, None) == -1, kw
        st = ctypes.c_void_p(fake)
        assert lib.vd_attn_validate(h, ctypes.byref(b), st, None) == -1, kw
    # the output and the workspace at 16
    b = batch()
    for out, w in [(fake + 8, fake), (fake, fake + 8), (fake + 2, fake + 4)]:
        assert lib.vd_attn_forward(h, ctypes.byref(b), out, w, ws.value, None) == -1, (out, w)
        assert lib.vd_attn_forward_splits(h, ctypes.byref(b), out, w, ws.value, None) == -1
        assert lib.vd_attn_forward_chunks(h, ctypes.byref(b), out, w, ws.value, None) == -1
        assert lib.vd_attn_forward_merge(h, ctypes.byref(b), out, w, ws.value, None) == -1
    assert lib.vd_attn_forward_plan(h, ctypes.byref(b), fake + 8, ws.value, None) == -1
    # the validator's status array at 4
    assert lib.vd_attn_validate(h, ctypes.byref(b), ctypes.c_void_p(fake + 2), None) == -1
    # the KV write: bf16 rows and pools at 16, slot ids at 8
    for args in [(fake + 8, fake, fake, fake, fake), (fake, fake + 2, fake, fake, fake),
                 (fake, fake, fake + 4, fake, fake), (fake, fake, fake, fake + 8, fake),
                 (fake, fake, fake, fake, fake + 2)]:
        kn, vn, sm, kp, vp = args
        assert lib.vd_kv_write(h, kn, vn, sm, 3, kp, vp, 4, None) == -1, args
    lib.vd_attn_destroy(h)


def test_noalloc_host_checks(lib):
    """vd_attn_forward_noalloc: the checks of vd_attn_forward, and a call whose
    workspace would exceed the library's static scratch is refused with
    VD_ERR_WORKSPACE -- all before any device call."""
    rc, h = _create(lib)
    fake = 0x10000
    limit = V.NOALLOC_SCRATCH_BYTES
    n = ctypes.c_size_t()
    # the workloads of the benchmark that fit, and the one that does not
    for B, q, ctx, fits in [(64, 1, 4096, True), (8, 1, 131072, True), (256, 4, 2560, True),
                            (128, 512, 8704, False)]:
        hq = 64 if q == 4 else 32
        rc2, h2 = _create(lib, num_q_heads=hq)
        assert lib.vd_attn_workspace_size(h2, B, q, ctx, ctypes.byref(n)) == 0
        assert (n.value <= limit) == fits, (B, q, ctx, n.value)
        lib.vd_attn_destroy(h2)
    big = V._Batch(128, 128 * 512, fake, fake, fake, fake, 600, fake, fake, 4, 512, 8704, None,
                   None, 0, None)
    assert lib.vd_attn_forward_noalloc(h, ctypes.byref(big), fake, None) == -3
    b = V._Batch(1, 1, fake, fake, fake, fake, 1, fake, fake, 4, 1, 16, None, None, 0, None)
    assert lib.vd_attn_forward_noalloc(h, ctypes.byref(b), None, None) == -1        # no output
    assert lib.vd_attn_forward_noalloc(h, ctypes.byref(b), fake + 8, None) == -1    # misaligned
    b.q = fake + 2
    assert lib.vd_attn_forward_noalloc(h, ctypes.byref(b), fake, None) == -1
    e = V._Batch(0, 0, None, None, None, None, 0, None, None, 0, 0, 0, None, None, 0, None)
    assert lib.vd_attn_forward_noalloc(h, ctypes.byref(e), None, None) == 0        # nothing to do
    assert lib.vd_attn_forward_noalloc(None, ctypes.byref(b), fake, None) == -1
    lib.vd_attn_destroy(h)
