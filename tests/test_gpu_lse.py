"""GPU log-sum-exp output (the row's ln sum exp(scale * q.k) over its visible
keys, from the final online-softmax state): parity with the oracle's, bit
invariance across execution variations, and no effect on the attention
output.  Every output path is covered: rows written by the split kernel
(one split), the short and the long merge, and the chunk kernel."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2609_38981_amd import workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

# Max abs error allowed against the fp64 oracle's log-sum-exp.  Budget (in
# natural-log units): the fp32 dot products behind the running maximum M
# (128 bf16 products accumulated in fp32: below 2e-4 for these N(0,1) inputs),
# the fp32 normaliser Z (tile trees, up to ~2,000 sequential tile updates and
# 256 split folds: relative error below 2e-4, the same in its log), and
# v_log_f32 / v_exp_f32 (a few ulp).  1e-3 keeps a 2x margin.
LSE_TOL = 1e-3


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    U.require_gpu()


CASES = {
    "tiny": lambda: W.config1(),                                       # single-split rows
    "decode_small": lambda: W.config2(batch=8, lo=100, hi=1500),       # short merge
    "mixed_small": lambda: W.config3(num_prefill=2, chunk=40, max_off=700, num_decode=6,
                                     dec_lo=50, dec_hi=1200),          # chunk kernel
    "long_mid": lambda: W.config4(batch=2, lo=9000, hi=40000),         # long merge
    "verify_small": lambda: W.config5(num_req=6, prefix=256, suf_lo=20, suf_hi=80),
    "window": lambda: W.config2(batch=6, lo=300, hi=2600, shape=W.Shape(32, 8, 128, window=700),
                                cfg=6),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_lse_parity_and_output_unchanged(name):
    call = CASES[name]()
    U.say("lse %s: B=%d T=%d max_n=%d" % (name, call.num_seqs, call.total_q_tokens,
                                         call.max_context_len))
    out, lse = U.gpu_run(call, with_lse=True)
    assert np.array_equal(out, U.gpu_run(call)), "asking for the log-sum-exp changed the output"
    assert np.isfinite(lse).all()
    rows = np.arange(call.total_q_tokens)
    if call.total_q_tokens > 400:
        rows = np.unique(np.linspace(0, call.total_q_tokens - 1, 200).astype(int))
    sub_reqs = sorted({call.request_of_row(int(t)) for t in rows})
    sub = call.subcall(sub_reqs)
    ref_rows, got_rows = [], []
    for t in rows:
        ri = call.request_of_row(int(t))
        p = call.reqs[ri].n - call.reqs[ri].s + (int(t) - int(call.cu_q_lens[ri]))
        ref_rows.append(sub.row_of(sub_reqs.index(ri), p))
        got_rows.append(int(t))
    _, ref = U.oracle_run(sub, rows=ref_rows, with_lse=True)
    err = np.abs(lse[got_rows].astype(np.float64) - ref[ref_rows])
    U.say("  lse max abs err %.3g over %d rows" % (err.max(), len(rows)))
    assert err.max() <= LSE_TOL, err.max()


def _lse_by_position(call, lse):
    res = {}
    for ri, r in enumerate(call.reqs):
        tag = call.prompts[r.prompt].tag
        for p in r.positions:
            res[(tag, p)] = lse[call.row_of(ri, p)]
    return res


def test_lse_bit_invariance():
    """The log-sum-exp of a logical row is bit-identical alone and batched,
    chunked or stepped, and under another page placement."""
    def lse_of(call, **kw):
        return _lse_by_position(call, U.gpu_run(call, with_lse=True, **kw)[1])

    base = lse_of(W.config1(variant="both"))
    for v in ["BA", "A", "B", "B44a", "B44b"]:
        U.assert_same_bits(base, lse_of(W.config1(variant=v)))
    kw = dict(lo=200, hi=2600)
    solo = lse_of(W.config2(batch=1, probe_slot=0, **kw))
    for batch, slot, perm in [(17, 5, 4), (64, 41, 5)]:
        U.assert_same_bits(solo, lse_of(W.config2(batch=batch, probe_slot=slot,
                                                  perm_stream=perm, **kw)))
    # a 700-token prompt whole (chunk kernel) vs 4-token verify and 1-token steps
    pr = W.make_prompt(W.LLAMA8B, 700, 13, 0)
    rng = W.rng_for(13, 4)
    whole = lse_of(W.place(W.LLAMA8B, [pr], [W.Req(0, 700, 700)], rng))
    for n, s in [(4, 4), (513, 1), (516, 4), (700, 1)]:
        U.assert_same_bits(whole, lse_of(W.place(W.LLAMA8B, [pr], [W.Req(0, n, s)], rng)))
    # appended tokens written by the split items
    U.assert_same_bits(solo, lse_of(W.config2(batch=17, probe_slot=5, **kw), append=True))
