"""GPU tests of the shared-prefix pass (calls with the shared_pages hint): the
plan launch finds adjacent requests whose page tables start with the same
pages, and the shared-prefix kernel computes their shared splits once
for all their rows, storing the partial states the rows' own split items would
have stored; the merge folds them with the rest.  Its output must be
bit-identical to the same call without the pass (every split read by
the request's own split items) and to a call with copied prefix pages, and
within tolerance of the oracle."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2609_38981_amd import vdattn as V
from paper_2609_38981_amd import workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    U.require_gpu()


def _groups_call(shape: W.Shape, shared: bool, cfg: int = 21) -> W.Call:
    """Ten requests in groups of different depths (S = the split size).

    * 0..3 on a 2S-token prefix X (2 splits): verify, decode, a 120-row
      prefill chunk (chunk path: in the group's range, not a member), decode;
    * 4: an unrelated decode (ends the group);
    * 5, 6: two requests reading one (4S - 48)-token prompt Y, at n = 3S + 300
      and n = 4S - 48 (verify): they share 3 splits;
    * 7..9 on X again, apart from 0..3: decode at n = 2S + 400, decode at
      n = 2S - 24 reading the same prompt as 7 (its row lies inside X's second
      split), and a verify: they share 1 split.
    ``shared``: the prompts on X share X's physical pages (else they hold
    copies)."""
    S = V.SPLIT_KEYS
    X = W.make_prompt(shape, 2 * S, cfg, 90_000, q_window=0)
    Y = W.make_prompt(shape, 4 * S - 48, cfg, 90_001, q_window=S)
    prompts = []

    def on_x(n, qw):
        prompts.append(W.make_prompt(shape, n, cfg, len(prompts), q_window=qw, prefix=X,
                                     prefix_len=2 * S))
        return len(prompts) - 1

    a0, a1 = on_x(2 * S + 100, 4), on_x(2 * S + 300, 1)
    a2, a3 = on_x(2 * S + 200, 120), on_x(2 * S + 50, 1)
    prompts.append(W.make_prompt(shape, 2 * S - 124, cfg, len(prompts), q_window=1))
    z = len(prompts) - 1
    prompts.append(Y)
    y = len(prompts) - 1
    a7, a9 = on_x(2 * S + 400, 430), on_x(2 * S + 60, 4)
    reqs = [W.Req(a0, 2 * S + 100, 4), W.Req(a1, 2 * S + 300, 1), W.Req(a2, 2 * S + 200, 120),
            W.Req(a3, 2 * S + 50, 1), W.Req(z, 2 * S - 124, 1), W.Req(y, 3 * S + 300, 1),
            W.Req(y, 4 * S - 48, 4), W.Req(a7, 2 * S + 400, 1), W.Req(a7, 2 * S - 24, 1),
            W.Req(a9, 2 * S + 60, 4)]
    return W.place(shape, prompts, reqs, W.rng_for(cfg, 4 if shared else 5),
                   shared_prefix_pages=(2 * S) // shape.page_size if shared else 0)


@pytest.mark.parametrize("shape", [W.LLAMA70B, W.Shape(16, 4, 64)], ids=["70b", "g4_d64"])
def test_prefix_groups(shape):
    shared = _groups_call(shape, True)
    copied = _groups_call(shape, False)
    U.say("prefix groups %s: B=%d T=%d" % (shape, shared.num_seqs, shared.total_q_tokens))
    a_bits = U.gpu_run(shared, shared_pages=True)
    a = U.by_position(shared, a_bits)
    rows = shared.total_q_tokens
    # the same call without the pass, and with copied prefix pages
    U.assert_same_bits(a, U.by_position(shared, U.gpu_run(shared, shared_pages=False)),
                       min_common=rows)
    U.assert_same_bits(a, U.by_position(copied, U.gpu_run(copied, shared_pages=True)),
                       min_common=rows)
    # the phases run one by one, and their timed form
    for how in ("phases", "timed"):
        U.assert_same_bits(a, U.by_position(shared, U.gpu_run(shared, shared_pages=True,
                                                              prepared=how)), min_common=rows)
    U.say("  %s" % U.parity(shared, a_bits))


def test_prefix_many_requests():
    """300 requests on a prefix of one split (the plan launch lists the split
    items), and 1030 requests (more than the pass examines: it is off)."""
    kw = dict(prefix=V.SPLIT_KEYS, suf_lo=20, suf_hi=120, shape=W.LLAMA8B)
    big = W.config5(num_req=300, **kw)
    a_bits = U.gpu_run(big, shared_pages=True)
    a = U.by_position(big, a_bits)
    U.assert_same_bits(a, U.by_position(big, U.gpu_run(big, shared_pages=False)),
                       min_common=big.total_q_tokens)
    # a request alone (no sharing) gives the same bits
    solo = W.config5(num_req=300, **kw).subcall([211])
    U.assert_same_bits(a, U.by_position(solo, U.gpu_run(solo)), min_common=solo.total_q_tokens)
    U.say("  300 requests: %s" % U.parity(big, a_bits, rows=[0, 1, 150, 299, big.total_q_tokens - 1]))
    huge = W.config5(num_req=1030, prefix=512, suf_lo=10, suf_hi=40, shape=W.LLAMA8B)
    h = U.by_position(huge, U.gpu_run(huge, shared_pages=True))
    U.assert_same_bits(h, U.by_position(huge, U.gpu_run(huge, shared_pages=False)),
                       min_common=huge.total_q_tokens)


def test_prefix_with_new_tokens():
    """The call's new tokens handed over (k_new / v_new): written by the split
    items (at most 256 requests) or by the plan launch (more), with the pass
    on; the same bits as without it and as with the tokens already in the
    pool."""
    for num_req in (12, 300):
        call = W.config5(num_req=num_req, prefix=V.SPLIT_KEYS, suf_lo=30, suf_hi=200,
                         shape=W.LLAMA8B)
        base = U.by_position(call, U.gpu_run(call, shared_pages=False))
        for sp in (True, False):
            U.assert_same_bits(base, U.by_position(call, U.gpu_run(call, append=True, shared_pages=sp)),
                               min_common=call.total_q_tokens)


def test_prefix_lse():
    call = _groups_call(W.LLAMA70B, True, cfg=22)
    out, lse = U.gpu_run(call, shared_pages=True, with_lse=True)
    out0, lse0 = U.gpu_run(call, shared_pages=False, with_lse=True)
    assert np.array_equal(out, out0)
    assert np.array_equal(lse.view(np.uint32), lse0.view(np.uint32))
    _, ref = U.oracle_run(call, with_lse=True)
    err = float(np.abs(lse.astype(np.float64) - ref).max())
    U.say("  prefix lse: max abs err %.3g" % err)
    assert err <= 1e-3


def test_prefix_deep():
    """A 36-split shared prefix: the pass covers its first 32 splits, the split
    items the rest, and the long merge (more than 16 splits) folds them all."""
    call = W.config5(num_req=4, prefix=36 * V.SPLIT_KEYS, suf_lo=100, suf_hi=600,
                     shape=W.LLAMA70B)
    a_bits = U.gpu_run(call, shared_pages=True)
    a = U.by_position(call, a_bits)
    U.assert_same_bits(a, U.by_position(call, U.gpu_run(call, shared_pages=False)),
                       min_common=call.total_q_tokens)
    U.say("  deep prefix: %s" % U.parity(call, a_bits))


def test_prefix_full_size_verify():
    """The 70B prefix-shared verify batch at full size (256 requests on a
    2048-token prefix, s = 4 / 1), in the launch configuration the benchmark
    times: every row bit-identical with and without the pass."""
    call = W.config5()
    with_pass = U.by_position(call, U.gpu_run(call, poison=False, shared_pages=True))
    without = U.by_position(call, U.gpu_run(call, poison=False, shared_pages=False))
    U.say("  full cfg5: %d rows compared" % U.assert_same_bits(with_pass, without,
                                                              min_common=call.total_q_tokens))
