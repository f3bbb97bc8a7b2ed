"""Pins of the CPU oracle against facts that do not come from the oracle.

Each ``pin_*`` function takes an oracle library handle (the built oracle, or a
deliberately broken copy of it) and raises AssertionError when the oracle
disagrees with the fact it is pinned to:

* a library routine: ``torch.nn.functional.scaled_dot_product_attention`` in
  float64 (causal prefill, a chunk at a key offset via an explicit ``tril``
  mask, grouped-query heads via ``enable_gqa``, a sliding window via a banded
  mask), and ``scipy.special.softmax``;
* the log-sum-exp output: scipy's ``logsumexp``; log(count) for a zero query,
  the score of a single key, weights exp(score - lse) summing to one;
* closed forms: a single visible key (n = 1, row 0, or a window of 1) returns
  that key's value exactly; a zero query or identical keys give the plain mean
  of the visible values (the prefix, or the window); one dominant score
  returns (nearly) that key's value;
* the paper's worked example of Fig. 4 (golden fixture);
* invariants the paper requires of the attention result: physical page
  placement, prompt chunking, batch composition and order, and data at
  positions after p (causal masking) or before the window do not change a
  row; a window covering the prefix is full attention.
"""
from __future__ import annotations

import json
import os

import numpy as np
import scipy.special
import torch
import torch.nn.functional as F

import oracle
from paper_2609_38981_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


# ---------------------------------------------------------------------------
# helpers: pack dense per-request data into a paged call for the oracle
# ---------------------------------------------------------------------------
def pack(reqs, hq, hkv, d, P, num_pages=None, rng=None, pages=None, poison=True):
    """reqs: list of dicts with q [s, hq, d], k/v [n, hkv, d] (uint16 bits).

    Places each request's pages at random (or at ``pages[r]``) in a pool of
    plain layout [pages, hkv, P, d] filled with NaN elsewhere."""
    need = [-(-r["k"].shape[0] // P) for r in reqs]
    total = sum(need)
    if num_pages is None:
        num_pages = max(2 * total, 1)
    rng = np.random.default_rng(0) if rng is None else rng
    perm = rng.permutation(num_pages)
    fill = W.BF16_QNAN if poison else np.uint16(0)
    kp = np.full((num_pages, hkv, P, d), fill, np.uint16)
    vp = np.full_like(kp, fill)
    stride = max(need) if need else 1
    pt = np.full((len(reqs), stride), -1, np.int32)
    cur = 0
    for i, r in enumerate(reqs):
        pg = list(pages[i]) if pages is not None else perm[cur:cur + need[i]].tolist()
        cur += need[i]
        pt[i, :len(pg)] = pg
        n = r["k"].shape[0]
        for j in range(n):
            kp[pg[j // P], :, j % P, :] = r["k"][j]
            vp[pg[j // P], :, j % P, :] = r["v"][j]
    cu = np.concatenate([[0], np.cumsum([r["q"].shape[0] for r in reqs])]).astype(np.int32)
    ctx = np.array([r["k"].shape[0] for r in reqs], np.int32)
    q = np.concatenate([r["q"] for r in reqs]) if reqs else np.zeros((0, hq, d), np.uint16)
    return q, cu, ctx, pt, kp, vp


def run(lib, reqs, hq, hkv, d, P, scale=None, window=0, with_lse=False, **kw):
    q, cu, ctx, pt, kp, vp = pack(reqs, hq, hkv, d, P, **kw)
    return oracle.paged_attention(q, cu, ctx, pt, kp, vp, num_q_heads=hq, num_kv_heads=hkv,
                                  head_dim=d, page_size=P, scale=scale, window=window, lib=lib,
                                  with_lse=with_lse)


def rand_req(rng, s, n, hq, hkv, d):
    return dict(q=W.normal_bf16(rng, (s, hq, d)), k=W.normal_bf16(rng, (n, hkv, d)),
                v=W.normal_bf16(rng, (n, hkv, d)))


def f64(bits):
    return W.bf16_to_f32(bits).astype(np.float64)


def sdpa_reference(req, hq, hkv, scale=None, window=0):
    """Library attention for one request, rows at positions n - s .. n - 1;
    with window w > 0 the mask is the band tril(n - s) minus tril(n - s - w)
    (the sliding window of Appendix A.5)."""
    q = torch.from_numpy(f64(req["q"])).permute(1, 0, 2)[None]  # [1, hq, s, d]
    k = torch.from_numpy(f64(req["k"])).permute(1, 0, 2)[None]  # [1, hkv, n, d]
    v = torch.from_numpy(f64(req["v"])).permute(1, 0, 2)[None]
    s, n = q.shape[2], k.shape[2]
    mask = torch.ones(s, n, dtype=torch.bool).tril(diagonal=n - s)
    if window > 0:
        mask &= ~torch.ones(s, n, dtype=torch.bool).tril(diagonal=n - s - window)
    o = F.scaled_dot_product_attention(q, k, v, attn_mask=mask, enable_gqa=(hq != hkv), scale=scale)
    return o[0].permute(1, 0, 2).numpy()  # [s, hq, d]


# ---------------------------------------------------------------------------
# pins
# ---------------------------------------------------------------------------
def pin_sdpa_prefill(lib):
    """Whole-prompt prefill (s = n) equals causal SDPA."""
    rng = np.random.default_rng(11)
    for (n, hq, hkv, d, P) in [(37, 4, 2, 64, 16), (21, 2, 2, 16, 4), (70, 8, 2, 32, 16)]:
        req = rand_req(rng, n, n, hq, hkv, d)
        got = run(lib, [req], hq, hkv, d, P)
        ref = sdpa_reference(req, hq, hkv)
        np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)


def pin_sdpa_chunk_offset(lib):
    """A chunk at a key offset (s < n) equals SDPA with a tril(n - s) mask, in
    a packed batch with scattered pages and GQA."""
    rng = np.random.default_rng(12)
    hq, hkv, d, P = 8, 2, 32, 16
    reqs = [rand_req(rng, s, n, hq, hkv, d) for s, n in [(1, 37), (8, 100), (5, 5), (3, 17)]]
    got = run(lib, reqs, hq, hkv, d, P)
    off = 0
    for r in reqs:
        s = r["q"].shape[0]
        np.testing.assert_allclose(got[off:off + s], sdpa_reference(r, hq, hkv), rtol=0, atol=1e-12)
        off += s


def pin_sdpa_scale(lib):
    """An explicit softmax scale is honoured like SDPA's ``scale``."""
    rng = np.random.default_rng(13)
    hq, hkv, d, P = 4, 4, 16, 8
    req = rand_req(rng, 3, 30, hq, hkv, d)
    got = run(lib, [req], hq, hkv, d, P, scale=0.37)
    np.testing.assert_allclose(got, sdpa_reference(req, hq, hkv, scale=0.37), rtol=0, atol=1e-12)


def pin_scipy_softmax_dense(lib):
    """Dense brute force with scipy's softmax on a tiny request."""
    rng = np.random.default_rng(14)
    hq, hkv, d, P = 2, 1, 8, 2
    s, n = 3, 7
    req = rand_req(rng, s, n, hq, hkv, d)
    got = run(lib, [req], hq, hkv, d, P)
    q, k, v = f64(req["q"]), f64(req["k"]), f64(req["v"])
    for i in range(s):
        p = n - s + i
        for h in range(hq):
            sc = (k[:p + 1, 0, :] @ q[i, h]) / np.sqrt(d)
            w = scipy.special.softmax(sc)
            np.testing.assert_allclose(got[i, h], w @ v[:p + 1, 0, :], rtol=0, atol=1e-12)


def pin_single_key(lib):
    """n = 1, and row 0 of a whole-prompt prefill, return v_0 bit for bit."""
    rng = np.random.default_rng(15)
    hq, hkv, d, P = 4, 2, 16, 16
    r1 = rand_req(rng, 1, 1, hq, hkv, d)
    r2 = rand_req(rng, 5, 5, hq, hkv, d)
    got = run(lib, [r1, r2], hq, hkv, d, P)
    for h in range(hq):
        g = h // (hq // hkv)
        assert np.array_equal(got[0, h], f64(r1["v"])[0, g])
        assert np.array_equal(got[1, h], f64(r2["v"])[0, g])


def pin_zero_query_mean(lib):
    """q = 0 gives uniform weights: the mean of v_0..v_p."""
    rng = np.random.default_rng(16)
    hq, hkv, d, P = 4, 2, 16, 4
    req = rand_req(rng, 4, 23, hq, hkv, d)
    req["q"][:] = 0
    got = run(lib, [req], hq, hkv, d, P)
    v = f64(req["v"])
    for i in range(4):
        p = 19 + i
        for h in range(hq):
            np.testing.assert_allclose(got[i, h], v[:p + 1, h // 2].mean(axis=0), rtol=0, atol=1e-12)


def pin_identical_keys_mean(lib):
    """All keys equal give the mean of the visible values whatever q is."""
    rng = np.random.default_rng(17)
    hq, hkv, d, P = 2, 1, 16, 4
    req = rand_req(rng, 2, 9, hq, hkv, d)
    req["k"][:] = req["k"][0]
    got = run(lib, [req], hq, hkv, d, P)
    v = f64(req["v"])
    for i, p in enumerate([7, 8]):
        for h in range(hq):
            np.testing.assert_allclose(got[i, h], v[:p + 1, 0].mean(axis=0), rtol=0, atol=1e-12)


def pin_dominant_key(lib):
    """A key aligned with q and scaled far above the rest takes all weight."""
    rng = np.random.default_rng(18)
    hq, hkv, d, P = 1, 1, 16, 4
    req = rand_req(rng, 1, 12, hq, hkv, d)
    req["q"][0, 0] = W.bf16_bits(np.full(d, 1.0, np.float32))
    req["k"][5, 0] = W.bf16_bits(np.full(d, 64.0, np.float32))
    got = run(lib, [req], hq, hkv, d, P)
    np.testing.assert_allclose(got[0, 0], f64(req["v"])[5, 0], rtol=0, atol=1e-12)


def pin_fig4_example(lib):
    """Paper Fig. 4: prefill row 3 of a 6-token prompt equals the decode row
    at k_len 4, with different physical pages, bit for bit; changing the
    masked future KV (positions 4, 5) does not change it."""
    with open(os.path.join(GOLDEN, "fig4_position_example.json")) as f:
        ex = json.load(f)
    P, pos = ex["page_size"], ex["position"]
    pre, dec = ex["prefill"], ex["decode"]
    assert pre["k_len"] - pre["q_len"] + pre["row"] == pos
    assert dec["k_len"] - dec["q_len"] + dec["row"] == pos
    rng = np.random.default_rng(19)
    hq, hkv, d = 4, 2, 16
    full = rand_req(rng, pre["q_len"], pre["k_len"], hq, hkv, d)
    dreq = dict(q=full["q"][pos:pos + 1].copy(), k=full["k"][:dec["k_len"]].copy(),
                v=full["v"][:dec["k_len"]].copy())
    kw = dict(num_pages=ex["pool_pages"])
    a = run(lib, [full], hq, hkv, d, P, pages=[pre["pages"]], **kw)
    b = run(lib, [dreq], hq, hkv, d, P, pages=[dec["pages"]], **kw)
    assert np.array_equal(a[pre["row"]], b[dec["row"]])
    # masked future positions do not matter
    alt = {k: v.copy() for k, v in full.items()}
    alt["k"][pos + 1:] = W.normal_bf16(rng, alt["k"][pos + 1:].shape)
    alt["v"][pos + 1:] = W.normal_bf16(rng, alt["v"][pos + 1:].shape)
    c = run(lib, [alt], hq, hkv, d, P, pages=[pre["pages"]], **kw)
    assert np.array_equal(a[pre["row"]], c[pre["row"]])
    # and the rows after p do see them (the example is not vacuous)
    assert not np.array_equal(a[pre["row"] + 1], c[pre["row"] + 1])


def pin_invariances(lib):
    """Page placement, chunking, batch composition and order leave rows
    bit-identical (tiny workload family)."""
    sh = W.TINY
    kw = dict(num_q_heads=sh.num_q_heads, num_kv_heads=sh.num_kv_heads, head_dim=sh.head_dim,
              page_size=sh.page_size, lib=lib)

    def out(call):
        kp, vp = call.std_pool()
        o = oracle.paged_attention(call.q_bits(), call.cu_q_lens, call.context_lens,
                                   call.page_table, kp, vp, **kw)
        res = {}
        for ri, r in enumerate(call.reqs):
            for p in r.positions:
                res[(r.prompt, p)] = o[call.row_of(ri, p)]
        return res

    base = out(W.config1(variant="both"))
    variants = [W.config1(perm_stream=5, variant="both"), W.config1(variant="BA"),
                W.config1(variant="A"), W.config1(variant="B"), W.config1(variant="B44a"),
                W.config1(variant="B44b")]
    for call in variants:
        for key, val in out(call).items():
            assert np.array_equal(val, base[key]), key


def pin_paged_equals_dense(lib):
    """The page-table gather: every request of a paged call (random page
    placement in a NaN-poisoned pool, several requests, GQA, a window) gives
    exactly the bits of the same request over contiguous keys and values (the
    dense variant, written separately with no page table)."""
    rng = np.random.default_rng(41)
    hq, hkv, d, P = 6, 2, 32, 16
    reqs = [rand_req(rng, s, n, hq, hkv, d) for s, n in [(1, 1), (3, 17), (1, 64), (5, 70),
                                                       (16, 33), (2, 130)]]
    for window in (0, 20):
        for scale in (None, 0.3):
            out, lse = run(lib, reqs, hq, hkv, d, P, scale=scale, window=window, with_lse=True,
                           rng=np.random.default_rng(window + 7))
            t = 0
            for r in reqs:
                s = r["q"].shape[0]
                dense, dlse = oracle.dense_attention(r["q"], r["k"], r["v"], num_q_heads=hq,
                                                     num_kv_heads=hkv, head_dim=d, scale=scale,
                                                     window=window, lib=lib, with_lse=True)
                assert np.array_equal(out[t:t + s], dense), (s, window, scale)
                assert np.array_equal(lse[t:t + s], dlse), (s, window, scale)
                t += s


# -- sliding window (Appendix A.5: key j visible to p when p - w < j <= p) ----
def pin_sdpa_window(lib):
    """Chunks at key offsets with a sliding window equal SDPA with a banded
    causal mask (GQA, scattered pages, windows shorter and longer than s)."""
    rng = np.random.default_rng(21)
    hq, hkv, d, P = 8, 2, 32, 16
    for w in (3, 16, 40):
        reqs = [rand_req(rng, s, n, hq, hkv, d) for s, n in [(1, 37), (8, 100), (5, 5), (20, 61)]]
        got = run(lib, reqs, hq, hkv, d, P, window=w)
        off = 0
        for r in reqs:
            s = r["q"].shape[0]
            np.testing.assert_allclose(got[off:off + s], sdpa_reference(r, hq, hkv, window=w),
                                       rtol=0, atol=1e-12)
            off += s


def pin_window_one_key(lib):
    """w = 1 leaves one visible key: every row returns v_p bit for bit."""
    rng = np.random.default_rng(22)
    hq, hkv, d, P = 4, 2, 16, 4
    req = rand_req(rng, 6, 19, hq, hkv, d)
    got = run(lib, [req], hq, hkv, d, P, window=1)
    v = f64(req["v"])
    for i in range(6):
        for h in range(hq):
            assert np.array_equal(got[i, h], v[13 + i, h // 2])


def pin_window_zero_query_mean(lib):
    """q = 0 gives the mean of the window's values v_(p-w+1)..v_p."""
    rng = np.random.default_rng(23)
    hq, hkv, d, P, w = 2, 1, 16, 4, 7
    req = rand_req(rng, 10, 30, hq, hkv, d)
    req["q"][:] = 0
    got = run(lib, [req], hq, hkv, d, P, window=w)
    v = f64(req["v"])
    for i in range(10):
        p = 20 + i
        for h in range(hq):
            np.testing.assert_allclose(got[i, h], v[p - w + 1:p + 1, 0].mean(axis=0), rtol=0,
                                       atol=1e-12)


def pin_window_limits(lib):
    """A window covering the whole prefix is full attention bit for bit, and
    K/V before the window do not change a row (while a row whose window
    includes them does change)."""
    rng = np.random.default_rng(24)
    hq, hkv, d, P = 4, 2, 16, 8
    req = rand_req(rng, 5, 33, hq, hkv, d)
    full = run(lib, [req], hq, hkv, d, P)
    assert np.array_equal(full, run(lib, [req], hq, hkv, d, P, window=33))
    assert np.array_equal(full, run(lib, [req], hq, hkv, d, P, window=1000))
    w = 10
    a = run(lib, [req], hq, hkv, d, P, window=w)
    alt = {k: v.copy() for k, v in req.items()}
    alt["k"][:19] = W.normal_bf16(rng, alt["k"][:19].shape)   # rows p >= 28 see keys >= 19
    alt["v"][:19] = W.normal_bf16(rng, alt["v"][:19].shape)
    b = run(lib, [alt], hq, hkv, d, P, window=w)
    assert np.array_equal(a[0], b[0])  # p = 28: window 19..28
    alt["k"][19] = W.normal_bf16(rng, alt["k"][19].shape)
    c = run(lib, [alt], hq, hkv, d, P, window=w)
    assert not np.array_equal(a[0], c[0])


# -- log-sum-exp of the visible scaled scores (natural log) ---------------------
def pin_lse_scipy(lib):
    """Dense brute force with scipy's logsumexp on tiny requests, with and
    without a window."""
    rng = np.random.default_rng(31)
    hq, hkv, d, P = 2, 1, 8, 2
    s, n = 4, 11
    req = rand_req(rng, s, n, hq, hkv, d)
    for w in (0, 3):
        _, lse = run(lib, [req], hq, hkv, d, P, window=w, with_lse=True)
        q, k = f64(req["q"]), f64(req["k"])
        for i in range(s):
            p = n - s + i
            lo = max(0, p - w + 1) if w else 0
            for h in range(hq):
                sc = (k[lo:p + 1, 0, :] @ q[i, h]) / np.sqrt(d)
                np.testing.assert_allclose(lse[i, h], scipy.special.logsumexp(sc), rtol=0,
                                           atol=1e-12)


def pin_lse_closed_forms(lib):
    """q = 0 gives lse = log(number of visible keys); one visible key gives
    its own score; and the weights exp(score - lse) sum to one."""
    rng = np.random.default_rng(32)
    hq, hkv, d, P = 4, 2, 16, 4
    req = rand_req(rng, 5, 23, hq, hkv, d)
    zq = {k: v.copy() for k, v in req.items()}
    zq["q"][:] = 0
    for w in (0, 7):
        _, lse = run(lib, [zq], hq, hkv, d, P, window=w, with_lse=True)
        for i in range(5):
            p = 18 + i
            cnt = min(p + 1, w) if w else p + 1
            assert np.all(lse[i] == np.log(cnt)), (w, i)
    one = rand_req(rng, 1, 1, hq, hkv, d)
    _, lse = run(lib, [one], hq, hkv, d, P, with_lse=True)
    q, k = f64(one["q"]), f64(one["k"])
    for h in range(hq):
        np.testing.assert_allclose(lse[0, h], (q[0, h] @ k[0, h // 2]) / np.sqrt(d), rtol=0,
                                   atol=1e-12)
    _, lse = run(lib, [req], hq, hkv, d, P, with_lse=True)
    q, k = f64(req["q"]), f64(req["k"])
    for i in range(5):
        p = 18 + i
        for h in range(hq):
            sc = (k[:p + 1, h // 2, :] @ q[i, h]) / np.sqrt(d)
            np.testing.assert_allclose(np.exp(sc - lse[i, h]).sum(), 1.0, rtol=0, atol=1e-12)


# ---------------------------------------------------------------------------
# linear layer (the matmul contract of Section 5.4, Fig. 3): c = a . b^T
# ---------------------------------------------------------------------------
def _bf16_ints(rng, shape, lo=-8, hi=8):
    """bf16 bit patterns of small integers (exact in bf16), and the integers."""
    vals = rng.integers(lo, hi + 1, size=shape)
    return W.bf16_bits(vals.astype(np.float32)), vals.astype(np.int64)


def pin_linear_integer_exact(lib):
    """Small-integer inputs make every product and every partial sum exact in
    fp64, so the oracle equals numpy's int64 matmul a @ b^T; the shapes are
    not square and the operands not symmetric, so a transposed operand, a
    dropped or repeated term or a wrong index fails."""
    rng = np.random.default_rng(31)
    for M, N, K in [(5, 7, 3), (1, 9, 33), (13, 2, 64), (4, 4, 4)]:
        ab, ai = _bf16_ints(rng, (M, K))
        bb, bi = _bf16_ints(rng, (N, K))
        c = oracle.linear(ab, bb, lib=lib)
        assert np.array_equal(c, (ai @ bi.T).astype(np.float64)), (M, N, K)


def pin_linear_one_hot(lib):
    """A one-hot activation row (a single 1 at column k_m) selects one column
    of the weights: c[m, n] = b[n, k_m] bit for bit (random bf16 weights)."""
    rng = np.random.default_rng(32)
    M, N, K = 6, 11, 40
    hot = rng.integers(0, K, size=M)
    a = np.zeros((M, K), np.float32)
    a[np.arange(M), hot] = 1.0
    bb = W.normal_bf16(rng, (N, K))
    c = oracle.linear(W.bf16_bits(a), bb, lib=lib)
    assert np.array_equal(c, f64(bb)[:, hot].T)


def pin_linear_strided(lib):
    """Only the first k columns of a and b are read: with NaN in the columns
    past k (a row stride larger than k) the result equals the contiguous one."""
    rng = np.random.default_rng(33)
    M, N, K = 7, 5, 24
    a = W.normal_bf16(rng, (M, K))
    b = W.normal_bf16(rng, (N, K))
    a_pad = np.full((M, K + 9), W.BF16_QNAN, np.uint16)
    b_pad = np.full((N, K + 3), W.BF16_QNAN, np.uint16)
    a_pad[:, :K] = a
    b_pad[:, :K] = b
    c = oracle.linear(a_pad, b_pad, k=K, lib=lib)
    assert np.array_equal(c, oracle.linear(a, b, lib=lib))


def pin_linear_fsum_bound(lib):
    """Random bf16 inputs: every bf16 x bf16 product is exact in fp64, so the
    ascending fp64 sum lies within K * 2^-53 * sum |a_k b_k| of the exactly
    rounded sum of the same products (math.fsum)."""
    import math

    rng = np.random.default_rng(34)
    M, N, K = 3, 4, 300
    a = W.normal_bf16(rng, (M, K))
    b = W.normal_bf16(rng, (N, K))
    c = oracle.linear(a, b, lib=lib)
    af, bf = f64(a), f64(b)
    for m in range(M):
        for n in range(N):
            prods = [af[m, k] * bf[n, k] for k in range(K)]
            bound = K * 2.0 ** -53 * sum(abs(x) for x in prods)
            assert abs(c[m, n] - math.fsum(prods)) <= bound, (m, n)


ALL_PINS = [pin_paged_equals_dense, pin_sdpa_prefill, pin_sdpa_chunk_offset, pin_sdpa_scale,
            pin_scipy_softmax_dense,
            pin_single_key, pin_zero_query_mean, pin_identical_keys_mean, pin_dominant_key,
            pin_fig4_example, pin_invariances, pin_sdpa_window, pin_window_one_key,
            pin_window_zero_query_mean, pin_window_limits, pin_lse_scipy, pin_lse_closed_forms,
            pin_linear_integer_exact, pin_linear_one_hot, pin_linear_strided,
            pin_linear_fsum_bound]


if __name__ == "__main__":
    # Runs every pin against the oracle library named on the command line and
    # prints the names of the pins that fail (used on deliberately broken
    # copies of the oracle, which may also crash outright).
    import sys

    mlib = oracle.bind(sys.argv[1])
    for pin in ALL_PINS:
        try:
            with np.errstate(all="ignore"):
                pin(mlib)
        except (AssertionError, ValueError):
            print("CAUGHT", pin.__name__, flush=True)
