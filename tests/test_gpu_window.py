"""Sliding-window attention (Appendix A.5: key j is visible to the row at p
when p - w < j <= p): the HIP path against the fp64 oracle on both kernel
paths, the exact one-key case, and the bitwise invariances with a window
(chunking, query length, batch composition, a window covering the prefix)."""
from __future__ import annotations

from dataclasses import replace

import numpy as np
import pytest

from paper_2609_38981_amd import workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    U.require_gpu()


def ws(shape, w):
    return replace(shape, window=w)


def outs(call, **kw):
    return U.by_position(call, U.gpu_run(call, **kw))


# windows below a page, at and around the tile (64) and split (1024) sizes
CASES = {
    "decode8b": lambda w: W.config2(batch=8, lo=100, hi=1800, shape=ws(W.LLAMA8B, w)),
    "mixed8b": lambda w: W.config3(num_prefill=2, chunk=96, max_off=1500, num_decode=6,
                                   dec_lo=50, dec_hi=1800, shape=ws(W.LLAMA8B, w)),
    "verify70b": lambda w: W.config5(num_req=6, prefix=608, suf_lo=20, suf_hi=300,
                                     shape=ws(W.LLAMA70B, w)),
    "chunks_tiny": lambda w: W.place(ws(W.TINY, w), [W.make_prompt(W.TINY, 1300, 9, 0)],
                                     [W.Req(0, 1300, 1300)], W.rng_for(9, 4)),
}
PARAMS = [(c, w) for c in sorted(CASES) for w in (1, 37, 64, 700)] + \
    [("decode8b", 512), ("decode8b", 1024), ("decode8b", 1500), ("mixed8b", 513),
     ("mixed8b", 1025), ("chunks_tiny", 200)]


@pytest.mark.parametrize("case,w", PARAMS, ids=["%s-w%d" % p for p in PARAMS])
def test_window_parity_small(case, w):
    call = CASES[case](w)
    U.say("window parity %s w=%d: B=%d T=%d max_n=%d" % (case, w, call.num_seqs,
                                                        call.total_q_tokens, call.max_context_len))
    out = U.gpu_run(call)
    U.say("  %s" % U.parity(call, out))


@pytest.mark.parametrize("shape", [W.TINY, W.LLAMA8B], ids=["tiny", "8b"])
def test_window_edge_lengths(shape):
    """Ragged tails at page, tile and split edges with a window that starts
    mid-tile and mid-split."""
    lens = [(1, 1), (17, 1), (65, 1), (513, 1), (1025, 1), (65, 9), (513, 8), (600, 120),
            (1100, 1100)]
    sh = ws(shape, 333)
    prompts = [W.make_prompt(sh, n, 8, i, q_window=s) for i, (n, s) in enumerate(lens)]
    call = W.place(sh, prompts, [W.Req(i, n, s) for i, (n, s) in enumerate(lens)],
                   W.rng_for(8, 4))
    U.say("window edge lengths %s T=%d" % (sh, call.total_q_tokens))
    U.say("  %s" % U.parity(call, U.gpu_run(call)))


def test_window_of_one_is_exact():
    """w = 1: every row sees only its own key and returns v_p bit for bit
    (on the chunk path and the split path)."""
    sh = ws(W.LLAMA8B, 1)
    pr = W.make_prompt(sh, 700, 7, 0)
    call = W.place(sh, [pr], [W.Req(0, 700, 700)], W.rng_for(7, 4))
    dec = W.place(sh, [pr], [W.Req(0, 530, 1), W.Req(0, 600, 4)], W.rng_for(7, 5))
    for c in (call, dec):
        out = U.gpu_run(c)
        for ri, r in enumerate(c.reqs):
            for p in r.positions:
                row = out[c.row_of(ri, p)]
                v = pr.v[p]  # [Hkv, D]
                for h in range(sh.num_q_heads):
                    want = v[h // sh.group].copy()
                    want[want == 0x8000] = 0  # the output maps -0 to +0
                    assert np.array_equal(row[h], want), (p, h)


def test_window_covering_the_prefix_is_full_attention():
    """A window longer than every context gives the bits of the handle
    without a window."""
    base = W.config3(num_prefill=2, chunk=96, max_off=900, num_decode=6, dec_lo=50, dec_hi=1200)
    wide = W.config3(num_prefill=2, chunk=96, max_off=900, num_decode=6, dec_lo=50, dec_hi=1200,
                     shape=ws(W.LLAMA8B, 5000))
    U.assert_same_bits(outs(base), outs(wide), min_common=2 * 96 + 6)


@pytest.mark.parametrize("shape", [ws(W.LLAMA8B, 300), ws(W.TINY, 700)], ids=["8b-w300", "tiny-w700"])
def test_window_chunking_and_query_length(shape):
    """One 1100-token prompt with a window: whole prefill, chunks of 512 and
    128, 4-token verify and 1-token decode steps, and a mixed batch give the
    same bits per position."""
    n_total = 1100
    pr = W.make_prompt(shape, n_total, 12, 0)
    rng = W.rng_for(12, 4)

    def run(pieces):
        res = {}
        for n, s in pieces:
            res.update(outs(W.place(shape, [pr], [W.Req(0, n, s)], rng)))
        return res

    whole = run([(n_total, n_total)])
    c512 = run([(min(n_total, e + 512), min(512, n_total - e)) for e in range(0, n_total, 512)])
    c128 = run([(min(n_total, e + 128), min(128, n_total - e)) for e in range(0, n_total, 128)])
    U.assert_same_bits(whole, c512, min_common=n_total)
    U.assert_same_bits(whole, c128, min_common=n_total)
    spots = [1, 63, 64, 65, 299, 300, 301, 511, 512, 513, 700, 1023, 1024, 1025, 1099]
    steps = [(p + 1, 1) for p in spots] + [(p + 1, 4) for p in spots if p >= 3]
    U.assert_same_bits(whole, run(steps), min_common=len(spots))
    reqs = [W.Req(0, n, s) for n, s in [(1100, 600), (513, 1), (700, 4), (65, 65), (1025, 8)]]
    U.assert_same_bits(whole, outs(W.place(shape, [pr], reqs, rng)), min_common=600)


@pytest.mark.parametrize("shape,w,s", [(W.TINY, 300, 12), (W.LLAMA70B, 700, 4)],
                         ids=["tiny-w300", "70b-w700"])
def test_window_wide_items(shape, w, s):
    """With a window: verify rows of 17..32 query-head rows per KV head run as
    wide split items when every request is on the split path, as column
    halves when the call also prefills a 40-token chunk, and as single-token
    steps: the same bits."""
    sh = ws(shape, w)
    assert 16 < s * sh.group <= 32
    prompts = [W.make_prompt(sh, n, 18, i, q_window=s) for i, n in enumerate((650, 1500, 2300))]
    reqs = [W.Req(i, pr.length, s) for i, pr in enumerate(prompts)]
    wide = outs(W.place(sh, prompts, reqs, W.rng_for(18, 4)))
    extra = W.make_prompt(sh, 400, 18, 9, q_window=40)
    mixed = W.place(sh, prompts + [extra], reqs + [W.Req(len(prompts), 400, 40)], W.rng_for(18, 5))
    n = U.assert_same_bits(wide, outs(mixed), min_common=3 * s)
    steps = [W.Req(i, pr.length - j, 1) for i, pr in enumerate(prompts) for j in range(s)]
    n += U.assert_same_bits(wide, outs(W.place(sh, prompts, steps, W.rng_for(18, 6))), min_common=3 * s)
    U.say("  window %d, wide vs column halves vs steps: %d rows bit-identical" % (w, n))


def test_window_batch_and_placement_invariance():
    """A probe request alone and at random slots of batches of 17 and 64,
    with two placements, gives the same bits under a window."""
    kw = dict(lo=200, hi=2600, shape=ws(W.LLAMA8B, 777))
    solo = outs(W.config2(batch=1, probe_slot=0, **kw))
    for batch, slot, perm in [(17, 5, 4), (64, 41, 5)]:
        U.assert_same_bits(solo, outs(W.config2(batch=batch, probe_slot=slot, perm_stream=perm,
                                                **kw)))


def test_window_full_size_sampled():
    """The sliding-window workload at full size (32 requests, contexts 8K to
    32K, window 4096), in the benchmark's launch configuration: sampled rows
    against the oracle."""
    call = W.config2(batch=32, lo=8192, hi=32768, shape=W.LLAMA8B_SWA4K, cfg=6, pool_factor=1.5)
    U.say("full swa8b: T=%d kv(window)=%.1f MB" % (call.total_q_tokens, call.kv_bytes() / 1e6))
    out = U.gpu_run(call, poison=False)
    rows = np.random.default_rng(4).choice(call.total_q_tokens, 12, replace=False)
    U.say("  %s" % U.parity(call, out, rows=rows))
