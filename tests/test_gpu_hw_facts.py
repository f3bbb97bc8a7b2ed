"""GPU: the gfx950 instruction facts the kernels' bitwise guarantees rest on,
pinned by running the instructions themselves (tests/probes/vd_probes.hip,
built by __graft_entry__.build()) and checking their results on the host.

* v_mfma_f32_16x16x32_bf16: an output cell depends only on its own row of A,
  column of B and accumulator (not on its slot in the tile or on the other
  rows and columns; a NaN stays in its row), so a row's bits do not depend on
  which rows share its tile; with an all-zero B it returns the accumulator
  bit for bit (every finite value, denormals included, -0 aside); and its
  32-term dot product is not what a chain of fp32 fused multiply-adds gives
  (in either order) nor the exact sum rounded once -- the reason decode
  issues the same matrix instruction as prefill instead of a vector-ALU dot
  product (the paper's Section 5.3 contract: one operation sequence per
  logical position, whatever the query length).
* v_exp_f32: exp2(+-0) = 1, exp2(-inf) = 0 (the identity and masked steps of
  the softmax), and results below the normal range are flushed to +0.
* v_cvt_pk_bf16_f32: round to nearest, ties to even (the P operand's cast).
* v_permlane16_swap_b32 / v_permlane32_swap_b32 (the softmax's exchanges
  between the four lanes of a column): the odd 16-lane rows of the first
  register trade places with the even rows of the second, and the upper half
  of the first with the lower half of the second.
* atomicAdd on a device-memory int32 (a vector atomic at agent scope): the
  values workgroups on all eight dies take from one counter are each handed
  out once, 0 .. N - 1 -- the split launch claims its later slots this way.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import pytest
import torch

from paper_2609_38981_amd import workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu
LIB = os.path.join(os.path.dirname(os.path.abspath(__file__)), "probes", "libvdprobes.so")


@pytest.fixture(scope="module")
def probes():
    U.require_gpu()
    if not os.path.exists(LIB):
        pytest.fail("tests/probes/libvdprobes.so is not built: run __graft_entry__.build()")
    lib = ctypes.CDLL(LIB)
    vp = ctypes.c_void_p
    lib.vdp_mfma_bf16.argtypes = [vp, vp, vp, vp, ctypes.c_int, vp]
    lib.vdp_exp2.argtypes = [vp, vp, ctypes.c_int64, vp]
    lib.vdp_cvt_bf16.argtypes = [vp, vp, ctypes.c_int64, vp]
    lib.vdp_row_swap.argtypes = [vp, vp, vp, vp]
    lib.vdp_claims.argtypes = [vp, vp, ctypes.c_int, ctypes.c_int, vp]
    for f in (lib.vdp_mfma_bf16, lib.vdp_exp2, lib.vdp_cvt_bf16, lib.vdp_row_swap, lib.vdp_claims):
        f.restype = ctypes.c_int
    return lib


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def run_mfma(lib, a_bits, b_bits, c):
    """D of every tile: a_bits [T, 16, 32] and b_bits [T, 32, 16] bf16 bits,
    c [T, 16, 16] float32."""
    t = a_bits.shape[0]
    assert a_bits.shape == (t, 16, 32) and b_bits.shape == (t, 32, 16) and c.shape == (t, 16, 16)
    da = torch.from_numpy(np.ascontiguousarray(a_bits).view(np.int16)).cuda()
    db = torch.from_numpy(np.ascontiguousarray(b_bits).view(np.int16)).cuda()
    dc = torch.from_numpy(np.ascontiguousarray(c, dtype=np.float32)).cuda()
    dd = torch.full((t, 16, 16), float("nan"), dtype=torch.float32, device="cuda")
    assert lib.vdp_mfma_bf16(da.data_ptr(), db.data_ptr(), dc.data_ptr(), dd.data_ptr(), t, _stream()) == 0
    torch.cuda.synchronize()
    return dd.cpu().numpy()


def bits32(x):
    return np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)


def random_tiles(rng, t):
    a = W.normal_bf16(rng, (t, 16, 32))
    b = W.normal_bf16(rng, (t, 32, 16))
    return a, b


def test_mfma_dot_product_models(probes):
    """51,200 dot products of 32 N(0, 1) bf16 pairs, accumulator +0: which
    fp32 model reproduces the instruction's bits.  A bf16 x bf16 product is
    exact in fp32, so a fused multiply-add step is one rounded fp32 add of
    the exact product."""
    rng = W.rng_for(40, 1)
    t = 200
    a, b = random_tiles(rng, t)
    d = run_mfma(probes, a, b, np.zeros((t, 16, 16), np.float32))
    fa = W.bf16_to_f32(a).astype(np.float64)
    fb = W.bf16_to_f32(b).astype(np.float64)
    prod = fa[:, :, None, :] * np.transpose(fb, (0, 2, 1))[:, None, :, :]  # [t, 16, 16, 32], exact
    assert np.array_equal(prod.astype(np.float32).astype(np.float64), prod)
    fwd = np.zeros((t, 16, 16), np.float32)
    for k in range(32):
        fwd = (fwd + prod[..., k].astype(np.float32)).astype(np.float32)
    rev = np.zeros((t, 16, 16), np.float32)
    for k in reversed(range(32)):
        rev = (rev + prod[..., k].astype(np.float32)).astype(np.float32)
    # the exact sum as an integer multiple of 2^-200 (every product here is
    # one: bf16 exponents of N(0, 1) values stay far above 2^-100)
    scaled = prod.reshape(-1, 32) * 2.0**200
    assert np.array_equal(np.floor(scaled), scaled)
    once = np.array([round_f32(sum(int(v) for v in row), 200) for row in scaled],
                    np.float32).reshape(t, 16, 16)
    n = d.size
    got = bits32(d)
    rates = {name: float(np.mean(got == bits32(m))) for name, m in
             (("fma chain k = 0..31", fwd), ("fma chain k = 31..0", rev), ("exact sum, one rounding", once))}
    for name, r in rates.items():
        U.say("  mfma vs %-26s: %6d of %d equal (%.1f%%)" % (name, round(r * n), n, 100 * r))
    # none of the three reproduces the instruction, so a vector-ALU decode
    # could not give the bits that the matrix-core prefill gives
    assert all(r < 1.0 for r in rates.values())
    # but each is an fp32-accuracy dot product: within 32 units of 2^-24 of
    # the sum of the terms' magnitudes
    err = np.abs(d.astype(np.float64) - once.astype(np.float64))
    assert bool(np.all(err <= 32 * 2.0**-24 * np.abs(prod).sum(-1)))


def round_f32(s: int, k: int) -> np.float32:
    """s * 2^-k rounded once to float32, nearest even (normal range)."""
    if s == 0:
        return np.float32(0.0)
    sign = -1.0 if s < 0 else 1.0
    m = abs(s)
    shift = m.bit_length() - 24
    if shift > 0:
        q, rem, half = m >> shift, m & ((1 << shift) - 1), 1 << (shift - 1)
        if rem > half or (rem == half and q & 1):
            q += 1
        m = q
    else:
        shift = 0
    return np.float32(sign * float(m) * 2.0 ** (shift - k))


def test_mfma_cell_depends_only_on_its_row_column_and_accumulator(probes):
    """Permuting a tile's rows of A (with C's rows) and columns of B (with
    C's columns) permutes D's cells and changes no bit; replacing every other
    row and column leaves a cell's bits alone; a NaN in one row of A reaches
    only that row of D."""
    rng = W.rng_for(40, 2)
    t = 200
    a, b = random_tiles(rng, t)
    c = rng.standard_normal((t, 16, 16)).astype(np.float32)
    d = run_mfma(probes, a, b, c)
    pr = np.array([rng.permutation(16) for _ in range(t)])
    pc = np.array([rng.permutation(16) for _ in range(t)])
    ti = np.arange(t)[:, None]
    a2 = a[ti, pr]                                   # rows of A
    b2 = np.transpose(np.transpose(b, (0, 2, 1))[ti, pc], (0, 2, 1))  # columns of B
    c2 = c[ti, pr][ti[:, :, None], np.arange(16)[None, :, None], pc[:, None, :]]
    d2 = run_mfma(probes, a2, b2, c2)
    want = d[ti, pr][ti[:, :, None], np.arange(16)[None, :, None], pc[:, None, :]]
    moved = int(np.sum(bits32(d2) != bits32(want)))
    # every row but 0 and column but 0 replaced
    a3, b3 = random_tiles(rng, t)
    a3[:, 0] = a[:, 0]
    b3[:, :, 0] = b[:, :, 0]
    c3 = rng.standard_normal((t, 16, 16)).astype(np.float32)
    c3[:, 0, 0] = c[:, 0, 0]
    d3 = run_mfma(probes, a3, b3, c3)
    replaced = int(np.sum(bits32(d3[:, 0, 0]) != bits32(d[:, 0, 0])))
    # a NaN in row 5 of A
    a4 = a.copy()
    a4[:, 5, 7] = 0x7FC0
    d4 = run_mfma(probes, a4, b, c)
    rows = np.ones(16, bool)
    rows[5] = False
    leak = int(np.sum(bits32(d4[:, rows]) != bits32(d[:, rows])))
    assert np.isnan(d4[:, 5]).all()
    U.say("  mfma slot independence: %d of %d cells changed by permutation, %d of %d by other "
          "rows and columns; NaN cells outside its row: %d" % (moved, d.size, replaced, t, leak))
    assert moved == 0 and replaced == 0 and leak == 0


def test_mfma_zero_b_returns_the_accumulator(probes):
    """B = +0 or -0 everywhere, A random finite, C every kind of finite fp32
    (random bit patterns, denormals, +-0): D equals C bit for bit, except that
    -0 comes back +0 -- the identity step of a column without a visible key
    (alpha = 1, zero weights)."""
    rng = W.rng_for(40, 3)
    t = 4096
    a = W.normal_bf16(rng, (t, 16, 32))
    u = rng.integers(0, 2**32, size=(t, 16, 16), dtype=np.uint64).astype(np.uint32)
    u = np.where(((u >> 23) & 0xFF) == 0xFF, u & 0x807FFFFF, u)  # finite only
    u[:, :2] = rng.integers(0, 2**23, size=(t, 2, 16), dtype=np.uint64).astype(np.uint32) | \
        (rng.integers(0, 2, size=(t, 2, 16), dtype=np.uint64).astype(np.uint32) << 31)  # denormals
    u[:, 2, :8] = 0x80000000
    u[:, 2, 8:] = 0
    c = u.view(np.float32)
    for zero in (0x0000, 0x8000):
        b = np.full((t, 32, 16), zero, np.uint16)
        d = run_mfma(probes, a, b, c)
        want = np.where(u == 0x80000000, np.uint32(0), u)
        bad = int(np.sum(bits32(d) != want))
        den = int(np.sum(((u & 0x7F800000) == 0) & ((u & 0x7FFFFFFF) != 0)))
        U.say("  mfma with B = %s: %d of %d accumulators changed (%d denormal, %d -0 -> +0)"
              % ("+0" if zero == 0 else "-0", bad, d.size, den, int(np.sum(u == 0x80000000))))
        assert bad == 0


def test_exp2_special_values(probes):
    x = np.array([0.0, -0.0, -np.inf, -130.0, -140.0, -149.0, -200.0, -1.0, -126.0, 0.5],
                 np.float32)
    dx = torch.from_numpy(x).cuda()
    dy = torch.full_like(dx, float("nan"))
    assert probes.vdp_exp2(dx.data_ptr(), dy.data_ptr(), x.size, _stream()) == 0
    torch.cuda.synchronize()
    y = dy.cpu().numpy()
    assert bits32(y[:3]).tolist() == [0x3F800000, 0x3F800000, 0]
    # results below the normal range are flushed to +0
    assert bits32(y[3:7]).tolist() == [0, 0, 0, 0]
    for xi, yi in zip(x[7:], y[7:]):
        assert abs(float(yi) - 2.0 ** float(xi)) <= 2.0 ** float(xi) * 2.0**-22
    U.say("  exp2: +-0 -> 1, -inf -> +0, 2^-130 .. 2^-200 -> +0; exp2(-1) = %r, exp2(-126) = %r, "
          "exp2(0.5) = %r" % (float(y[7]), float(y[8]), float(y[9])))


def rne_bf16_reference(x: np.ndarray) -> np.ndarray:
    """Nearest bf16 to each finite float32, ties to the even mantissa: the two
    bf16 neighbours of x (truncation and one step away from zero) compared
    exactly in float64."""
    u = bits32(x).astype(np.uint64)
    lo = (u & 0xFFFF0000).astype(np.uint32)
    hi = (lo.astype(np.uint64) + 0x10000).astype(np.uint32)
    xv = x.astype(np.float64)
    dlo = np.abs(xv - lo.view(np.float32).astype(np.float64))
    dhi = np.abs(hi.view(np.float32).astype(np.float64) - xv)
    even_lo = ((lo >> 16) & 1) == 0
    pick_lo = (dlo < dhi) | ((dlo == dhi) & even_lo)
    return np.where(pick_lo, lo >> 16, hi >> 16).astype(np.uint16)


def test_cvt_bf16_rounds_to_nearest_even(probes):
    rng = W.rng_for(40, 4)
    n = 1 << 20
    u = rng.integers(0, 2**32, size=n, dtype=np.uint64).astype(np.uint32)
    u = np.where(((u >> 23) & 0xFF) >= 0xFE, u & 0x807FFFFF, u)  # finite, no overflow to inf
    u[: n // 2] = (u[: n // 2] & 0xFFFF0000) | 0x8000           # exact ties
    x = u.view(np.float32)
    dx = torch.from_numpy(x.copy()).cuda()
    dy = torch.zeros(n, dtype=torch.int16, device="cuda")
    assert probes.vdp_cvt_bf16(dx.data_ptr(), dy.data_ptr(), n, _stream()) == 0
    torch.cuda.synchronize()
    got = dy.cpu().numpy().view(np.uint16)
    bad = int(np.sum(got != rne_bf16_reference(x)))
    U.say("  cvt to bf16: %d of %d differ from nearest-even (%d exact ties)" % (bad, n, n // 2))
    assert bad == 0


def test_row_swaps_exchange_rows_between_two_registers(probes):
    a = np.arange(64, dtype=np.float32)
    b = 1000.0 + np.arange(64, dtype=np.float32)
    da, db = torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda()
    out = torch.zeros(256, dtype=torch.float32, device="cuda")
    assert probes.vdp_row_swap(da.data_ptr(), db.data_ptr(), out.data_ptr(), _stream()) == 0
    torch.cuda.synchronize()
    got = out.cpu().numpy().reshape(4, 64)
    r = lambda x, k: x[16 * k: 16 * k + 16]  # noqa: E731  (row k of 16 lanes)
    # 16-lane swap: odd rows of the first register <-> even rows of the second
    want_a16 = np.concatenate([r(a, 0), r(b, 0), r(a, 2), r(b, 2)])
    want_b16 = np.concatenate([r(a, 1), r(b, 1), r(a, 3), r(b, 3)])
    # 32-lane swap: upper half of the first <-> lower half of the second
    want_a32 = np.concatenate([a[:32], b[:32]])
    want_b32 = np.concatenate([a[32:], b[32:]])
    for name, g, w in (("first after 16", got[0], want_a16), ("second after 16", got[1], want_b16),
                       ("first after 32", got[2], want_a32), ("second after 32", got[3], want_b32)):
        U.say("  row swap, %s register: %s" % (name, "as expected" if np.array_equal(g, w) else g))
        assert np.array_equal(g, w)


@pytest.mark.parametrize("wgs,per", [(4096, 4), (20000, 1)])
def test_counter_claims_are_unique_across_dies(probes, wgs, per):
    counter = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    out = torch.full((wgs * per,), -1, dtype=torch.int32, device="cuda")
    for rep in range(3):
        assert probes.vdp_claims(counter.data_ptr(), out.data_ptr(), wgs, per, _stream()) == 0
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        ok = np.array_equal(np.sort(got), np.arange(wgs * per))
        U.say("  %d workgroups x %d claims, run %d: %s; counter ends at %d" % (
            wgs, per, rep, "each value once" if ok else "NOT a permutation", int(counter.item())))
        assert ok
        assert int(counter.item()) == wgs * per
        # a workgroup's own claims increase
        assert (np.diff(got.reshape(wgs, per), axis=1) > 0).all()
