"""GPU tests of the batch-invariant linear layer (vd_linear, the matmul
contract of the paper's Section 5.4, Fig. 3): parity with the fp64 oracle
within a bound derived from the arithmetic, bitwise row invariance across the
number of rows, the row's position and the row stride, and edge cases."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from paper_2609_38981_amd import staging as S
from paper_2609_38981_amd import vdattn as V
from paper_2609_38981_amd import workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    U.require_gpu()


def _draw(seed, M, N, K):
    rng = np.random.default_rng(seed)
    return W.normal_bf16(rng, (M, K)), W.normal_bf16(rng, (N, K))


def _gpu_linear(a_bits, b_bits, lda=None):
    a = S.bf16_tensor(a_bits, "cuda")
    if lda is not None and lda != a.shape[1]:
        # a strided copy: rows of lda values, NaN past K (never read)
        big = torch.full((a.shape[0], lda), float("nan"), dtype=torch.bfloat16, device="cuda")
        big[:, :a.shape[1]] = a
        a = big[:, :a_bits.shape[1]]
    out = V.linear(a, S.bf16_tensor(b_bits, "cuda"))
    torch.cuda.synchronize()
    return S.bits_of(out)


def _abs_bits(x):
    return (np.asarray(x, np.uint16) & np.uint16(0x7FFF)).astype(np.uint16)


def _check_parity(a_bits, b_bits, got_bits, rows=None):
    """|c_gpu - c| <= 2^-8 |c| + (K + 64) 2^-24 sum_k |a_k b_k| + 2^-133.

    The bf16 cast of the fp32 result is within half an ulp, 2^-9 of its
    magnitude (2^-8 of the exact value leaves room for the fp32 error); the
    fp32 chain of K / 32 MFMA steps, each adding 32 exact bf16 x bf16 products
    and the accumulator, is within (K + K / 32) 2^-24 sum |a_k b_k| of the
    exact sum (one rounding per operand added, as for any order of fp32
    additions); the last term covers values below the bf16 normal range."""
    rows = np.arange(a_bits.shape[0]) if rows is None else np.asarray(rows)
    K = a_bits.shape[1]
    ref = oracle.linear(a_bits[rows], b_bits)
    mag = oracle.linear(_abs_bits(a_bits[rows]), _abs_bits(b_bits))
    got = W.bf16_to_f32(got_bits[rows]).astype(np.float64)
    assert np.isfinite(got).all()
    err = np.abs(got - ref)
    bound = 2.0 ** -8 * np.abs(ref) + (K + 64) * 2.0 ** -24 * mag + 2.0 ** -133
    assert (err <= bound).all(), "max excess %g" % float((err - bound).max())
    return float(err.max()), float((err / np.maximum(np.abs(ref), 1e-30)).max())


@pytest.mark.parametrize("M,N,K", [(1, 16, 64), (37, 160, 256), (129, 300, 192),
                                   (300, 128, 512), (5, 1000, 128)])
def test_linear_parity(M, N, K):
    a, b = _draw(M * 131 + N * 7 + K, M, N, K)
    got = _gpu_linear(a, b)
    U.say("linear %dx%dx%d: max abs err %.3g, max rel err %.3g" % (M, N, K, *_check_parity(a, b, got)))


def test_linear_row_invariance():
    """Row x of an M-row call equals row 0 of the one-row call, bit for bit,
    for several M, positions and row strides; a column depends only on its
    own weight row (a subset of the weights gives the same columns)."""
    M, N, K = 300, 272, 320
    a, b = _draw(7, M, N, K)
    full = _gpu_linear(a, b)
    n = 0
    for x in [0, 1, 127, 128, 129, 255, 299]:
        one = _gpu_linear(a[x:x + 1], b)
        assert np.array_equal(one[0], full[x]), x
        n += 1
    for m in [2, 17, 128, 131, 257]:
        part = _gpu_linear(a[M - m:], b)
        assert np.array_equal(part, full[M - m:]), m
    assert np.array_equal(_gpu_linear(a, b, lda=K + 40), full)
    sub = _gpu_linear(a, b[33:33 + 150])
    assert np.array_equal(sub, full[:, 33:33 + 150])
    U.say("linear row invariance: %d single rows, 5 suffixes, a strided copy, a weight subset" % n)


def test_linear_edges():
    a, b = _draw(11, 3, 20, 64)
    # K = 0: the empty sum is +0
    z = V.linear(torch.zeros((3, 0), dtype=torch.bfloat16, device="cuda"),
                 torch.zeros((20, 0), dtype=torch.bfloat16, device="cuda"))
    torch.cuda.synchronize()
    assert (S.bits_of(z) == 0).all()
    # M = 0: nothing to do
    e = V.linear(torch.zeros((0, 64), dtype=torch.bfloat16, device="cuda"), S.bf16_tensor(b, "cuda"))
    assert e.shape == (0, 20)
    # K not a multiple of the K step: rejected (a missing configuration)
    with pytest.raises(V.VdError):
        V.linear(torch.zeros((3, 80), dtype=torch.bfloat16, device="cuda"),
                 torch.zeros((20, 80), dtype=torch.bfloat16, device="cuda"))
    # a row stride that breaks 16-byte alignment: rejected
    big = torch.zeros((3, 68), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(V.VdError):
        V.linear(big[:, 2:66], S.bf16_tensor(b, "cuda"))


def test_linear_full_size_sampled():
    """Llama-3-8B QKV projection at full size (4096 tokens, 4096 -> 6144):
    sampled rows against the oracle, and those rows alone bit-identical."""
    M, N, K = 4096, 6144, 4096
    a, b = _draw(2026, M, N, K)
    full = _gpu_linear(a, b)
    rows = [0, 1, 777, 2048, 4095]
    U.say("linear full size: %s" % (_check_parity(a, b, full, rows=rows),))
    for x in rows[1:]:
        assert np.array_equal(_gpu_linear(a[x:x + 1], b)[0], full[x]), x


@pytest.mark.parametrize("case", range(8))
def test_linear_random_shapes(case):
    """Seeded random shapes (N off every tile multiple among them, K up to
    4096, padded row strides): sampled rows within the bound of the oracle,
    rows bit-identical computed in another M at other positions, columns
    bit-identical computed from a subset of the weight rows."""
    rng = np.random.default_rng(8100 + case)
    M = int(rng.choice([1, 17, 65, 255, 257, 1000]))
    N = int(rng.choice([8, 17, 95, 97, 193, 1000, 4095]))
    K = 64 * int(rng.integers(1, 65))
    lda = K + 8 * int(rng.choice([0, 1, 5]))
    a, b = _draw(8200 + case, M, N, K)
    got = _gpu_linear(a, b, lda=lda)
    rows = rng.choice(M, size=min(4, M), replace=False)
    err, rel = _check_parity(a, b, got, rows=rows)
    sub = np.sort(rng.choice(M, size=min(M, 20), replace=False))
    perm = rng.permutation(len(sub))
    assert np.array_equal(_gpu_linear(np.ascontiguousarray(a[sub][perm]), b), got[sub][perm])
    cols = np.sort(rng.choice(N, size=min(N, 24), replace=False))
    assert np.array_equal(_gpu_linear(a, np.ascontiguousarray(b[cols])), got[:, cols])
    U.say("linear %dx%dx%d (lda %d): max abs err %.3g; %d rows and %d columns bit-identical" % (
        M, N, K, lda, err, len(sub), len(cols)))
