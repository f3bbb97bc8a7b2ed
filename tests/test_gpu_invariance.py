"""GPU bitwise invariance: the output of a logical (prompt, position, head)
row is bit-identical across batch composition and order, chunking, query
length (decode vs verify vs prefill), page placement and sharing, and
metadata that must not matter (hints, table stride, pool size, workspace
contents, stream, repetition) -- the causal contract of the paper's
Section 5.3 / Appendix A.1."""
from __future__ import annotations

import json
import os

import numpy as np
import pytest
import torch

from paper_2609_38981_amd import vdattn as V
from paper_2609_38981_amd import workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    U.require_gpu()


def outs(call, **kw):
    return U.by_position(call, U.gpu_run(call, **kw))


# -- tiny workload (config 1) ---------------------------------------------------
def test_tiny_variants():
    base = outs(W.config1(variant="both"))
    n = 0
    for v in ["BA", "A", "B", "B44a", "B44b"]:
        n += U.assert_same_bits(base, outs(W.config1(variant=v)))
    n += U.assert_same_bits(base, outs(W.config1(perm_stream=5)), min_common=9)
    U.say("tiny variants: %d rows bit-identical" % n)


def test_fig4_example_on_gpu():
    """Paper Fig. 4: prefill row 3 of q_len = k_len = 6 equals the decode row
    of q_len 1, k_len 4, on different physical pages (page size 16 here)."""
    ex = json.load(open(os.path.join(GOLDEN, "fig4_position_example.json")))
    pre, dec = ex["prefill"], ex["decode"]
    for sh in (W.TINY, W.LLAMA8B):
        pr = W.make_prompt(sh, pre["k_len"], 11, 0)
        a = W.place(sh, [pr], [W.Req(0, pre["k_len"], pre["q_len"])], W.rng_for(11, 4), min_pages=12)
        b = W.place(sh, [pr], [W.Req(0, dec["k_len"], dec["q_len"])], W.rng_for(11, 5), min_pages=12)
        assert a.page_table[0, 0] != b.page_table[0, 0]
        oa, ob = U.gpu_run(a), U.gpu_run(b)
        assert np.array_equal(oa[pre["row"]], ob[dec["row"]])


# -- query length: whole prefill vs chunks vs verify vs decode stepping --------
@pytest.mark.parametrize("shape", [W.LLAMA8B, W.TINY], ids=["8b", "tiny"])
def test_chunking_and_query_length(shape):
    """One prompt of 1100 tokens: whole (s = n), chunks of 512 and 128, 4-token
    verify steps and 1-token decode steps give the same bits per position."""
    n_total = 1100
    pr = W.make_prompt(shape, n_total, 12, 0)
    rng = W.rng_for(12, 4)

    def run(pieces):
        # pieces: list of (n, s) calls, each a separate invocation
        res = {}
        for n, s in pieces:
            call = W.place(shape, [pr], [W.Req(0, n, s)], rng)
            res.update(outs(call))
        return res

    whole = run([(n_total, n_total)])
    assert len(whole) == n_total
    c512 = run([(min(n_total, e + 512), min(512, n_total - e)) for e in range(0, n_total, 512)])
    c128 = run([(min(n_total, e + 128), min(128, n_total - e)) for e in range(0, n_total, 128)])
    U.assert_same_bits(whole, c512, min_common=n_total)
    U.assert_same_bits(whole, c128, min_common=n_total)
    # verify (s = 4) and decode (s = 1) steps around split and tile edges
    spots = [1, 2, 63, 64, 65, 511, 512, 513, 1023, 1024, 1025, 1099]
    steps = [(p + 1, 1) for p in spots] + [(p + 1, 4) for p in spots if p >= 3]
    U.assert_same_bits(whole, run(steps), min_common=len(spots))
    # a batch that mixes all of them in one call
    reqs = [W.Req(0, n, s) for n, s in [(1100, 600), (513, 1), (700, 4), (65, 65), (1025, 8)]]
    call = W.place(shape, [pr], reqs, rng)
    U.assert_same_bits(whole, outs(call), min_common=600)


# -- batch composition and order (config 2 family) -----------------------------
def test_probe_request_batch_invariance():
    """A fixed probe request alone, and at random slots in batches of 17 and
    64, gives the same bits; page placement and order do not matter."""
    kw = dict(lo=200, hi=2600)
    solo = outs(W.config2(batch=1, probe_slot=0, **kw))
    n = 0
    for batch, slot, perm in [(17, 5, 4), (64, 41, 4), (64, 0, 5), (17, 16, 5)]:
        n += U.assert_same_bits(solo, outs(W.config2(batch=batch, probe_slot=slot,
                                                     perm_stream=perm, **kw)))
    U.say("probe invariance: %d comparisons" % n)


def test_metadata_does_not_matter():
    """Oversized hints, a wider page-table stride, a bigger pool, a NaN-filled
    workspace, another stream, a repeat run and a prepared call (whole or
    phase by phase) give the same bits."""
    mk = lambda **kw: W.config2(batch=9, lo=300, hi=1800, **kw)
    base = outs(mk())
    call = mk()
    variants = {
        "hints": dict(hint_extra_q=7, hint_extra_ctx=3000),
        "hints_long": dict(hint_extra_ctx=20000),
        "ws_nan": dict(workspace_fill=-1),
        "stream": dict(stream=torch.cuda.Stream()),
        "repeat": {},
        "prepared_forward": dict(prepared="forward"),
        "prepared_phases": dict(prepared="phases"),
        "prepared_timed": dict(prepared="timed"),
        # ordinary (cached) K/V loads instead of non-temporal ones
        "shared_pages_hint": dict(shared_pages=True),
    }
    for name, kw in variants.items():
        U.assert_same_bits(base, U.by_position(call, U.gpu_run(call, **kw)), min_common=9)
    wide = W.place(call.shape, call.prompts, call.reqs, W.rng_for(2, 4), stride_extra=37,
                   pool_factor=3.0)
    U.assert_same_bits(base, outs(wide), min_common=9)


def test_mixed_batch_orders():
    """Config 3 family: prefill chunks and decodes in one call, rows ordered
    prefill-first or shuffled, and the timed phase launches, give the same
    bits."""
    kw = dict(num_prefill=3, chunk=96, max_off=900, num_decode=10, dec_lo=60, dec_hi=1500)
    a = outs(W.config3(**kw))
    b = outs(W.config3(shuffle=True, perm_stream=5, **kw))
    U.assert_same_bits(a, b, min_common=3 * 96 + 10)
    # the timed split and chunk launches compute the same bits
    c = outs(W.config3(**kw), prepared="timed")
    U.assert_same_bits(a, c, min_common=3 * 96 + 10)


def test_prefix_sharing_and_verify_steps():
    """Config 5 family: shared vs copied prefix pages, and 4-token verify vs
    single-token steps at each of the 4 positions."""
    kw = dict(num_req=8, prefix=512, suf_lo=30, suf_hi=200)
    shared = outs(W.config5(shared=True, **kw))
    copied = outs(W.config5(shared=False, perm_stream=5, **kw))
    U.assert_same_bits(shared, copied, min_common=4 * 4 + 4)
    for step in range(4):
        U.assert_same_bits(shared, outs(W.config5(step=step, **kw)), min_common=8)
    # non-temporal K/V loads although pages are shared
    U.assert_same_bits(shared, outs(W.config5(shared=True, **kw), shared_pages=False),
                       min_common=4 * 4 + 4)


def test_large_batch_plan_launch():
    """More than 256 requests: the plan launch lists the split items and, with
    the query rows' K/V handed over, writes them.  A probe request gives the
    same bits there as alone or among 17 requests, where the split workgroups
    find their items and write the new tokens themselves."""
    kw = dict(lo=20, hi=600)
    solo = outs(W.config2(batch=1, probe_slot=0, **kw))
    big = W.config2(batch=300, probe_slot=211, perm_stream=5, **kw)
    U.assert_same_bits(solo, outs(big))
    out_append = U.gpu_run(big, append=True)
    U.assert_same_bits(solo, U.by_position(big, out_append))
    U.assert_same_bits(outs(big), U.by_position(big, out_append), min_common=300)
    U.assert_same_bits(solo, outs(W.config2(batch=17, probe_slot=3, **kw), append=True))
    U.say("  300 requests, appended: %s" % U.parity(big, out_append, rows=[0, 150, 211, 299]))
    # prefill rows too: the plan launch's chunk list (263 requests) against the
    # chunk workgroups' own planning (13 requests)
    kw3 = dict(num_prefill=3, chunk=96, max_off=900, dec_lo=20, dec_hi=400)
    small = outs(W.config3(num_decode=10, **kw3))
    large = W.config3(num_decode=260, **kw3)
    U.assert_same_bits(small, outs(large), min_common=3 * 96 + 10)
    U.assert_same_bits(small, outs(large, append=True), min_common=3 * 96 + 10)
    U.assert_same_bits(small, outs(W.config3(num_decode=10, **kw3), append=True),
                       min_common=3 * 96 + 10)


def test_large_batch_column_halves():
    """More than 256 requests with 32 query-head rows per KV head (70B verify,
    s = 4): the plan launch lists one wide item per split (both 16-row
    blocks).  Rows equal those of a few of the requests run alone (the split
    workgroups' own planning), and those without the shared-prefix pass."""
    big = W.config5(num_req=300, prefix=V.SPLIT_KEYS, suf_lo=20, suf_hi=300)
    a = outs(big)
    U.assert_same_bits(a, outs(big.subcall([0, 1, 150, 298, 299])), min_common=4 * 3 + 2)
    U.assert_same_bits(a, outs(big, shared_pages=False), min_common=big.total_q_tokens)
    U.say("  300 verify requests: %s" % U.parity(big, U.gpu_run(big), rows=[0, 3, 601, 749]))


def test_wide_items_vs_column_halves():
    """70B verify (s = 4: 32 query-head rows per KV head) runs as wide split
    items, one per split over both 16-row blocks, when every request is on
    the split path, and as two column-half items per split when the call also
    carries a prefill chunk (40 G rows: the chunk path).  The verify rows are
    the same bits either way, below and above 256 requests (in-wave planning
    and the plan launch), with and without the shared-prefix pass; suffixes
    up to 1500 keys give rows of up to three splits."""
    for num_req in (12, 300):
        base = W.config5(num_req=num_req, prefix=V.SPLIT_KEYS + 304, suf_lo=20, suf_hi=1500)
        sh = base.shape
        wide = outs(base)
        extra = W.make_prompt(sh, 700, 16, 0, q_window=40)
        mixed = W.place(sh, base.prompts + [extra], base.reqs + [W.Req(len(base.prompts), 700, 40)],
                        W.rng_for(16, 4), shared_prefix_pages=(V.SPLIT_KEYS + 304) // sh.page_size)
        assert mixed.max_q_len * sh.group > 32 and base.max_q_len * sh.group == 32
        n = U.assert_same_bits(wide, outs(mixed), min_common=base.total_q_tokens)
        n += U.assert_same_bits(wide, outs(mixed, shared_pages=False), min_common=base.total_q_tokens)
        n += U.assert_same_bits(wide, outs(base, shared_pages=False), min_common=base.total_q_tokens)
        U.say("  %d verify requests, wide vs column halves: %d rows bit-identical" % (num_req, n))


def test_wide_items_head_dim_64():
    """Head dim 64, 2 query heads per KV head: 12-token verify rows (24
    query-head rows per KV head, wide split items) against the same rows in a
    call that also prefills a 40-token chunk (16-row column halves), and
    against single-token steps at each position."""
    sh = W.TINY
    prompts = [W.make_prompt(sh, n, 17, i, q_window=12) for i, n in enumerate((700, 1500, 2100, 90))]
    reqs = [W.Req(i, pr.length, 12) for i, pr in enumerate(prompts)]
    wide = outs(W.place(sh, prompts, reqs, W.rng_for(17, 4)))
    extra = W.make_prompt(sh, 300, 17, 9, q_window=40)
    mixed = W.place(sh, prompts + [extra], reqs + [W.Req(len(prompts), 300, 40)], W.rng_for(17, 5))
    n = U.assert_same_bits(wide, outs(mixed), min_common=48)
    steps = [W.Req(i, pr.length - j, 1) for i, pr in enumerate(prompts) for j in range(12)]
    n += U.assert_same_bits(wide, outs(W.place(sh, prompts, steps, W.rng_for(17, 6))), min_common=48)
    U.say("  head dim 64, wide vs column halves vs steps: %d rows bit-identical" % n)


def test_chunk_order_above_64_requests():
    """70 prefill chunks (more than 64 on the chunk path: the in-wave planner
    keeps request order) against 9 of them alone (listed longest first), and
    in reverse order."""
    kw = dict(chunk=96, max_off=1500, num_decode=3, dec_lo=20, dec_hi=400)
    big = W.config3(num_prefill=70, **kw)
    a = outs(big)
    sub = [0, 1, 5, 17, 33, 40, 64, 69, 71]
    n = U.assert_same_bits(a, outs(big.subcall(sub)), min_common=8 * 96 + 1)
    rev = W.place(big.shape, big.prompts, big.reqs[::-1], W.rng_for(3, 9))
    n += U.assert_same_bits(a, outs(rev), min_common=big.total_q_tokens)
    U.say("  70 chunk-path requests vs 9 alone and reversed: %d rows bit-identical" % n)


def test_long_context_batch_and_placement():
    """Config 4 family (scaled down): batch 1 vs batch 4, two placements."""
    kw = dict(lo=6000, hi=12000)
    b4 = outs(W.config4(batch=4, **kw))
    for i in range(4):
        U.assert_same_bits(b4, outs(W.config4(batch=4, only=i, perm_stream=5, **kw)))


def test_full_size_long_decode_batch_one_vs_eight():
    """Long-context decode at full size: requests alone (another placement)
    and in the batch of 8 give the same bits."""
    b8 = outs(W.config4())
    for i in (2, 6):
        U.assert_same_bits(b8, outs(W.config4(only=i, perm_stream=5)))


def test_full_size_decode_probe_batch_1_17_64():
    """Llama-3-8B decode at full size: the probe request alone, in 17 and in
    64 requests (contexts 512..4096)."""
    solo = outs(W.config2(batch=1, probe_slot=0))
    for batch, slot in [(17, 9), (64, 33)]:
        U.assert_same_bits(solo, outs(W.config2(batch=batch, probe_slot=slot, perm_stream=5)))
