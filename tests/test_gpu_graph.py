"""GPU: a call captured in a HIP graph (torch.cuda.CUDAGraph) and replayed gives
the eager call's bits on every replay, with the program's own eager work and
synchronizations between the replays: an eager call of the same batch on the
same workspace, and the workspace overwritten with 0xFF bytes.

* A long-context decode batch with more split items than the split launch has
  workgroups: the graph holds the one-wavefront launch that zeroes the slot
  counter (a kernel, not a memset), so each replay claims from zero whatever
  the previous call or the overwrite left there.
* The 8B decode batch (every item in the launch's first round).
* The allocation-free entry point (for callers that capture graphs and cannot
  allocate), whose workspace is the library's static scratch.
The bits of a row depend only on its request (Section 5.3), so every replay
must equal the eager run exactly."""
from __future__ import annotations

import pytest
import torch

from paper_2609_38981_amd import staging as S
from paper_2609_38981_amd import workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

CALLS = {
    # 6 requests x 8 KV heads x 88-108 splits: about 4,900 split items
    "long-decode-d64-claims": (lambda: W.config4(batch=6, lo=90000, hi=110000,
                                                 shape=W.Shape(16, 8, 64)), False),
    "decode8b": (lambda: W.config2(), False),
    "decode8b-noalloc": (lambda: W.config2(), True),
}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    U.require_gpu()


@pytest.mark.parametrize("name", list(CALLS))
def test_graph_replays_equal_eager(name):
    make, noalloc = CALLS[name]
    call = make()
    attn = U.handle(call.shape)
    dc = S.to_device(attn, call, poison=True)
    b = dc.batch
    ws = attn.new_workspace(call.num_seqs, b.max_q_len, b.max_context_len)
    out = torch.empty_like(b.q)

    def run(dst):
        if noalloc:
            attn.forward_noalloc(b, dst)
        else:
            attn.forward(b, out=dst, workspace=ws)

    # eager reference (it also does the library's one-time set-up per device)
    out.view(torch.int16).fill_(U.FILL)
    run(out)
    torch.cuda.synchronize()
    rows = U.by_position(call, S.bits_of(out))
    U.assert_written(rows)

    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            run(out)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    other = torch.empty_like(b.q)
    n = 0
    for rep in range(4):
        # the program's own work between replays: an eager call of the same
        # batch on the same workspace, or the workspace overwritten
        if rep % 2 == 0:
            other.view(torch.int16).fill_(U.FILL)
            run(other)
            torch.cuda.synchronize()
            n += U.assert_same_bits(rows, U.by_position(call, S.bits_of(other)))
        else:
            ws.view(torch.int8).fill_(-1)
            torch.cuda.synchronize()
        out.view(torch.int16).fill_(U.FILL)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        n += U.assert_same_bits(rows, U.by_position(call, S.bits_of(out)),
                                min_common=call.total_q_tokens)
    U.say("%s: %d requests, 4 replays and 2 eager calls, %d rows bit-identical to the eager run" % (
        name, call.num_seqs, n))
    del g
