"""GPU tests of the opt-in validator of a batch's device-side data
(vd_attn_validate) and of what vd_attn_forward does with the requests it
flags: requests with invalid lengths are skipped (their rows keep the NaN the
output was filled with), a page id outside the pool reads as zeros, and the
other requests' rows are bit-identical to those of the clean batch."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from paper_2609_38981_amd import staging as S
from paper_2609_38981_amd import workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    U.require_gpu()


def expected_status(cu, ctx, pt, num_pages, T, max_q, max_ctx):
    """The status codes the boundary documents, from the host copies."""
    out = []
    stride = pt.shape[1]
    for r in range(len(ctx)):
        q0, q1, n = int(cu[r]), int(cu[r + 1]), int(ctx[r])
        s, st = q1 - q0, 0
        if s < 1 or s > n:
            st |= 1
        if s > max_q or n > max_ctx:
            st |= 2
        npages = -(-n // 16) if n > 0 else 0
        if npages > stride:
            st |= 4
        if q0 < 0 or q1 > T:
            st |= 8
        ids = pt[r, :min(npages, stride)]
        if ((ids < 0) | (ids >= num_pages)).any():
            st |= 16
        out.append(st)
    return np.array(out, np.int32)


def _forward_bits(attn, b, shared_pages):
    b.shared_pages = shared_pages
    B = int(b.context_lens.numel())
    ws = attn.new_workspace(B, b.max_q_len, b.max_context_len)
    out = torch.empty_like(b.q)
    out.view(torch.int16).fill_(0x7FC0)
    attn.forward(b, out=out, workspace=ws)
    torch.cuda.synchronize()
    return S.bits_of(out)


@pytest.mark.parametrize("batch", [8, 300])
def test_validate_flags_and_forward_skips(batch):
    call = W.config2(batch=batch, lo=100, hi=1500, cfg=8)
    attn = U.handle(call.shape)
    clean = U.gpu_run(call)
    dc = S.to_device(attn, call, hint_extra_ctx=200)
    b = dc.batch
    B, T = call.num_seqs, call.total_q_tokens
    assert (attn.validate(b).cpu().numpy() == 0).all()
    stride = b.page_table.shape[1]
    # planted violations of the device-side preconditions
    b.context_lens[2] = 0                         # s = 1 > n = 0
    b.context_lens[3] = b.max_context_len + 100   # over the hint (and past the stride)
    b.page_table[4, 0] = b.num_pages + 5          # a page id outside the pool
    b.context_lens[5] = 16 * stride + 1           # more pages than the table stride
    b.cu_q_lens[B] = T + 3                        # the last request's rows reach past T
    torch.cuda.synchronize()
    want = expected_status(b.cu_q_lens.cpu().numpy(), b.context_lens.cpu().numpy(),
                           b.page_table.cpu().numpy(), b.num_pages, T, b.max_q_len,
                           b.max_context_len)
    got = attn.validate(b).cpu().numpy()
    U.say("  B=%d status %s" % (B, {r: int(got[r]) for r in range(B) if got[r]}))
    assert np.array_equal(got, want)
    assert got[2] & 1 and got[3] & 2 and got[4] == 16 and got[5] & 4 and got[B - 1] & 8
    cu = call.cu_q_lens
    skipped = [2, 3, 5, B - 1]
    for shared in (False, True):
        bits = _forward_bits(attn, b, shared)
        for r in range(B):
            rows = slice(int(cu[r]), int(cu[r + 1]))
            if r in skipped:
                assert (bits[rows].view(np.int16) == 0x7FC0).all(), (r, shared)
            elif r == 4:
                assert np.isfinite(W.bf16_to_f32(bits[rows])).all()
            else:
                assert np.array_equal(bits[rows], clean[rows]), (r, shared)
