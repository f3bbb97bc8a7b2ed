"""Helpers of the GPU tests: run a synthetic call through the HIP library and
through the CPU oracle, and compare rows by logical (prompt, position)."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
from paper_2609_38981_amd import staging as S
from paper_2609_38981_amd import workloads as W
from paper_2609_38981_amd.vdattn import VdAttn

# Max abs error allowed against the fp64 oracle for bf16 outputs with fp32
# accumulation.  Budget: the bf16 cast of the weights before P.V (relative
# 2^-9 per weight) and the bf16 output rounding (half an ulp, 2^-9 relative,
# <= 7.8e-3 for |o| < 4) dominate; exp2 and fp32 sums add < 1e-4.
TOL = 2e-2


def say(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def require_gpu():
    if not torch.cuda.is_available():
        raise RuntimeError("GPU tests need a visible MI355X")


_handles = {}


def handle(shape: W.Shape) -> VdAttn:
    if shape not in _handles:
        _handles[shape] = S.handle_for(shape)
    return _handles[shape]


def gpu_run(call: W.Call, poison: bool = True, stream=None, workspace_fill=None,
            prepared=None, with_lse: bool = False, **kw):
    """Output bits (uint16 [T, Hq, D]) of one vd_attn_forward call (or, with
    prepared = "forward" / "phases" / "timed", of a prepared call run whole, phase
    by phase, or phase by phase with the kernels' dispatches recording events).
    With ``with_lse``: (output bits, log-sum-exp float32 [T, Hq])."""
    attn = handle(call.shape)
    dc = S.to_device(attn, call, poison=poison, lse=with_lse, **kw)
    ws = attn.new_workspace(call.num_seqs, dc.batch.max_q_len, dc.batch.max_context_len)
    if workspace_fill is not None:
        ws.view(torch.int8).fill_(workspace_fill)
    out = torch.empty_like(dc.batch.q)
    out.view(torch.int16).fill_(0x7FC0)
    if prepared is not None:
        pc = attn.prepare(dc.batch, out, ws)
        if prepared == "forward":
            pc.forward()
        elif prepared == "timed":
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
            pc.plan()
            pc.splits(events=ev[:2])
            pc.chunks(events=ev[2:])
            pc.merge()
            torch.cuda.synchronize()
            for a, b in (ev[:2], ev[2:]):
                assert a.elapsed_time(b) >= 0.0
        else:
            pc.plan()
            pc.splits()
            pc.chunks()
            pc.merge()
    elif stream is None:
        attn.forward(dc.batch, out=out, workspace=ws)
    else:
        with torch.cuda.stream(stream):
            attn.forward(dc.batch, out=out, workspace=ws, stream=stream)
        stream.synchronize()
    torch.cuda.synchronize()
    if with_lse:
        return S.bits_of(out), dc.batch.lse.cpu().numpy()
    return S.bits_of(out)


def oracle_run(call: W.Call, rows=None, with_lse: bool = False):
    sh = call.shape
    kp, vp = call.std_pool()
    return oracle.paged_attention(call.q_bits(), call.cu_q_lens, call.context_lens,
                                  call.page_table, kp, vp, num_q_heads=sh.num_q_heads,
                                  num_kv_heads=sh.num_kv_heads, head_dim=sh.head_dim,
                                  page_size=sh.page_size, window=sh.window, rows=rows,
                                  with_lse=with_lse)


def by_position(call: W.Call, out: np.ndarray):
    """{(prompt identity, position): output row [Hq, D]} for every row."""
    res = {}
    for ri, r in enumerate(call.reqs):
        tag = call.prompts[r.prompt].tag
        for p in r.positions:
            res[(tag, p)] = out[call.row_of(ri, p)]
    return res


def parity(call: W.Call, gpu_bits: np.ndarray, rows=None) -> dict:
    """Compares GPU rows with the oracle; returns error statistics.

    With ``rows``, the oracle runs on a compact copy of just the requests
    holding those rows (their logical data and lengths are unchanged)."""
    got = W.bf16_to_f32(gpu_bits).astype(np.float64)
    if rows is None:
        sel = np.arange(call.total_q_tokens)
        ref = oracle_run(call)[sel]
    else:
        sel = np.asarray(rows)
        reqs = sorted({call.request_of_row(int(t)) for t in sel})
        sub = call.subcall(reqs)
        sub_rows = []
        for t in sel:
            ri = call.request_of_row(int(t))
            p = call.reqs[ri].n - call.reqs[ri].s + (int(t) - int(call.cu_q_lens[ri]))
            sub_rows.append(sub.row_of(reqs.index(ri), p))
        ref = oracle_run(sub, sub_rows)[sub_rows]
    diff = np.abs(got[sel] - ref)
    assert np.isfinite(got[sel]).all(), "non-finite GPU output"
    # the error in units of the bf16 spacing at the reference value (8 significant
    # bits: 2^(e - 7) for |ref| in [2^e, 2^(e+1)), down to the smallest normal)
    e = np.floor(np.log2(np.maximum(np.abs(ref), 2.0 ** -126)))
    ulps = diff / np.exp2(e - 7)
    st = dict(max_abs=float(diff.max()) if diff.size else 0.0,
              mean_abs=float(diff.mean()) if diff.size else 0.0,
              max_bf16_ulp=float(ulps.max()) if ulps.size else 0.0, rows=int(len(sel)))
    assert st["max_abs"] <= TOL, st
    return st


def assert_same_bits(a: dict, b: dict, min_common: int = 1):
    common = sorted(set(a) & set(b))
    assert len(common) >= min_common, (len(common), min_common)
    bad = [k for k in common if not np.array_equal(a[k], b[k])]
    assert not bad, "bitwise mismatch at %d of %d (prompt, position) rows, e.g. %s" % (
        len(bad), len(common), bad[:3])
    return len(common)
