"""GPU: seeded random batches across the shapes and call options the library
takes -- head dim 64 and 128, 1 to 12 query heads per KV head (3, 7 and 12
among them: groups need not be powers of two), sliding windows, a shared
prefix with and without the shared_pages hint, new tokens handed over in
k_new / v_new, batch sizes on both sides of the in-wave planners' limits (64
and 256 requests) -- with query lengths mixing decode (s = 1), verify (s up
to 16) and prefill chunks (up to 600).  In every case the rows of a few
requests run alone are bit-identical to their rows in the batch (the causal
contract of the paper's Section 5.3 / Appendix A.1), and sampled rows match
the oracle within the parity tolerance.  New tokens are kept off the shared
prefix pages: a call may not read one request's new-token slot as another
request's key (Section 4.1: new tokens go to private slots)."""
from __future__ import annotations

import numpy as np
import pytest

from paper_2609_38981_amd import workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

# (id, shape, requests, shared prefix, hint, append)
CASES = [
    ("d64-g2-64req-append", W.Shape(4, 2, 64), 64, False, None, True),
    ("d64-g1-65req", W.Shape(8, 8, 64), 65, False, None, False),
    ("d128-g8-17req-prefix-hint-append", W.Shape(16, 2, 128), 17, True, True, True),
    ("d128-g8-256req-prefix-hint", W.Shape(64, 8, 128), 256, True, True, False),
    ("d128-g4-257req-window-append", W.Shape(32, 8, 128, window=1500), 257, False, None, True),
    ("d64-g2-300req-window", W.Shape(4, 2, 64, window=300), 300, False, None, False),
    ("d128-g4-3req-long", W.Shape(32, 8, 128), 3, False, None, False),
    ("d128-g8-255req-prefix-append", W.Shape(64, 8, 128), 255, True, False, True),
    ("d64-g2-256req-prefix-hint-append", W.Shape(4, 2, 64), 256, True, True, True),
    # groups that are not powers of two
    ("d64-g3-63req", W.Shape(6, 2, 64), 63, False, None, False),
    ("d128-g7-100req-append", W.Shape(28, 4, 128), 100, False, None, True),
    ("d128-g12-64req-prefix-hint", W.Shape(24, 2, 128), 64, True, True, False),
    ("d64-g7-257req-window-append", W.Shape(21, 3, 64, window=2500), 257, False, None, True),
]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    U.require_gpu()


def random_call(case_index: int, shape: W.Shape, num_req: int, prefix: bool):
    """Lengths and query lengths drawn from the case's seed.  With ``prefix``
    about 80% of the requests read a common prefix of 1 to 3 splits plus up to
    19 pages (a 1024-key split boundary need not end it) from the same
    physical pages, and their new tokens lie past it."""
    rng = W.rng_for(61, case_index)
    maxlen = 20000 if num_req <= 3 else (6000 if num_req <= 65 else 2500)
    p0 = int(rng.integers(1, 4)) * 1024 + 16 * int(rng.integers(0, 20)) if prefix else 0
    pre = W.make_prompt(shape, p0, 61, 10**6 + case_index) if prefix else None
    prompts, reqs = [], []
    for r in range(num_req):
        on_prefix = prefix and rng.random() < 0.8
        n = p0 + int(rng.integers(1, 700)) if on_prefix else int(rng.integers(1, maxlen))
        u = rng.random()
        s = 1 if u < 0.6 else (int(rng.integers(2, 17)) if u < 0.8 else int(rng.integers(17, 600)))
        shares = prefix and n > p0
        s = max(1, min(s, n - p0 if shares else n))
        if shares:
            prompts.append(W.make_prompt(shape, n, 61, 1000 * case_index + r, q_window=s,
                                         prefix=pre, prefix_len=p0))
        else:
            prompts.append(W.make_prompt(shape, n, 61, 1000 * case_index + r, q_window=s))
        reqs.append(W.Req(r, n, s))
    return W.place(shape, prompts, reqs, rng, shared_prefix_pages=p0 // shape.page_size)


@pytest.mark.parametrize("case", range(len(CASES)), ids=[c[0] for c in CASES])
def test_random_batch(case):
    name, shape, num_req, prefix, hint, append = CASES[case]
    call = random_call(case, shape, num_req, prefix)
    G = shape.group
    U.say("%s: %d requests (%d on the chunk path), %d query rows, longest context %d" % (
        name, num_req, sum(r.s * G > 32 for r in call.reqs), call.total_q_tokens,
        call.max_context_len))
    out = U.gpu_run(call, append=append, shared_pages=hint)
    rows = U.by_position(call, out)
    U.assert_written(rows)
    rng = np.random.default_rng(case)
    # alone: a chunk-path request, a split-path request with several rows and
    # a random one (when the batch has them)
    chunk = [i for i, r in enumerate(call.reqs) if r.s * G > 32]
    multi = [i for i, r in enumerate(call.reqs) if 1 < r.s and r.s * G <= 32]
    picks = {int(rng.choice(num_req))}
    for group in (chunk, multi):
        if group:
            picks.add(int(rng.choice(group)))
    alone = 0
    for ri in sorted(picks):
        sub = call.subcall([ri])
        alone += U.assert_same_bits(rows, U.by_position(sub, U.gpu_run(sub)))
    sel = rng.choice(call.total_q_tokens, size=min(6, call.total_q_tokens), replace=False)
    st = U.parity(call, out, rows=sel)
    U.say("  %d rows alone == batched; oracle max abs error %.2e over %d rows" % (
        alone, st["max_abs"], st["rows"]))
