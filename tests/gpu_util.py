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
# ... and relative to the largest reference magnitude of each (row, head):
# o_d = sum_j w_j v_jd has spread ||w||_2 over d, and the weight cast adds a
# random error of about 2^-9 ||w||_2 / sqrt(3) to each o_d, the output
# rounding half an ulp of o_d.  An emulation of that arithmetic in numpy
# (bf16 weights, fp32 sums, bf16 output) on 10^5 rows of 2 .. 131072 N(0, 1)
# keys gave at most 0.58% of the row's largest |o_d|; 2^-6 (1.56%) leaves
# 2.7x headroom.  Unlike the absolute bound it stays tight at long contexts,
# where |o_d| ~ 1.6 / sqrt(n) (about 5e-3 at 100K keys) and an all-zero or
# scrambled row would pass 2e-2.
REL_TOL = 2.0 ** -6


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
    # per (row, head): the error against the largest magnitude of the row
    row_max = np.abs(ref).max(axis=-1, keepdims=True)
    rel = diff / np.maximum(row_max, 1e-30)
    # the error in units of the bf16 spacing at the reference value (8 significant
    # bits: 2^(e - 7) for |ref| in [2^e, 2^(e+1)), down to the smallest normal)
    e = np.floor(np.log2(np.maximum(np.abs(ref), 2.0 ** -126)))
    ulps = diff / np.exp2(e - 7)
    st = dict(max_abs=float(diff.max()) if diff.size else 0.0,
              mean_abs=float(diff.mean()) if diff.size else 0.0,
              max_bf16_ulp=float(ulps.max()) if ulps.size else 0.0,
              max_rel_row=float(rel.max()) if rel.size else 0.0, rows=int(len(sel)))
    assert st["max_abs"] <= TOL, st
    assert (diff <= REL_TOL * row_max + 1e-7).all(), st
    return st


# gpu_run fills the output with this bf16 quiet NaN before the call
FILL = 0x7FC0


def assert_written(rows: dict, keys=None):
    """Every compared row was written: no bf16 NaN or infinity (exponent all
    ones), which includes the 0x7FC0 fill of rows the library left unwritten."""
    keys = rows.keys() if keys is None else keys

    def bad_row(x):
        x = np.asarray(x)
        if x.dtype == np.uint16:  # bf16 bit patterns
            return ((x & 0x7F80) == 0x7F80).any()
        return not np.isfinite(x).all()  # e.g. float32 log-sum-exp values

    bad = [k for k in keys if bad_row(rows[k])]
    assert not bad, "unwritten or non-finite output at %d rows, e.g. %s" % (len(bad), bad[:3])


def assert_same_bits(a: dict, b: dict, min_common: int = 1):
    common = sorted(set(a) & set(b))
    assert len(common) >= min_common, (len(common), min_common)
    # two variants that both leave a row unwritten would compare equal
    assert_written(a, common)
    assert_written(b, common)
    bad = [k for k in common if not np.array_equal(a[k], b[k])]
    assert not bad, "bitwise mismatch at %d of %d (prompt, position) rows, e.g. %s" % (
        len(bad), len(common), bad[:3])
    return len(common)


class Session:
    """Device pools holding a fixed placement of prompts, against which calls
    with any requests over those prompts run without restaging the pools.

    ``base`` places the prompts: the page-table row of its longest request on
    each prompt gives that prompt's pages for every later call.  With
    ``prefill`` every slot of the base call is written once (vd_kv_write);
    without it the pools start as bf16 NaN and only calls that hand their new
    tokens over (``append``) fill them, in call order, as an engine's chunked
    prefill would."""

    def __init__(self, base: W.Call, prefill: bool = True):
        self.base = base
        self.attn = handle(base.shape)
        self.k_pool = self.attn.new_pool(base.num_pages)
        self.v_pool = self.attn.new_pool(base.num_pages)
        self.k_pool.view(torch.int16).fill_(FILL)
        self.v_pool.view(torch.int16).fill_(FILL)
        if prefill:
            S.fill_pool(self.attn, base, self.k_pool, self.v_pool)
        self.rows = {}
        for ri, r in enumerate(base.reqs):
            if r.prompt not in self.rows or r.n > base.reqs[self.rows[r.prompt]].n:
                self.rows[r.prompt] = ri
        torch.cuda.synchronize()

    def call(self, reqs) -> W.Call:
        """A call of (prompt, n, s) requests on the session's pages."""
        rq = [W.Req(p, n, s) for p, n, s in reqs]
        pt = np.stack([self.base.page_table[self.rows[p]] for p, _, _ in reqs])
        return W.Call(self.base.shape, self.base.prompts, rq, pt, self.base.num_pages,
                      self.base.page_owner)

    def run(self, reqs, append: bool = False, hint_ctx: int = 0, shared_pages: bool = False):
        """Output bits (uint16 [T, Hq, D]) of one call of (prompt, n, s)
        requests, and the call.  ``hint_ctx``: a max_context_len hint above the
        true maximum (0: the true maximum)."""
        call = self.call(reqs)
        dev = "cuda"
        extra = {}
        if append:
            kn, vn = call.query_kv()
            extra = dict(k_new=S.bf16_tensor(kn, dev), v_new=S.bf16_tensor(vn, dev))
        batch = S.Batch(
            q=S.bf16_tensor(call.q_bits(), dev),
            cu_q_lens=torch.from_numpy(call.cu_q_lens).to(dev),
            context_lens=torch.from_numpy(call.context_lens).to(dev),
            page_table=torch.from_numpy(np.ascontiguousarray(call.page_table)).to(dev),
            k_pool=self.k_pool, v_pool=self.v_pool, num_pages=call.num_pages,
            max_q_len=call.max_q_len, max_context_len=max(call.max_context_len, hint_ctx),
            shared_pages=shared_pages, **extra)
        ws = self.attn.new_workspace(call.num_seqs, batch.max_q_len, batch.max_context_len)
        out = torch.empty_like(batch.q)
        out.view(torch.int16).fill_(FILL)
        self.attn.forward(batch, out=out, workspace=ws)
        torch.cuda.synchronize()
        return S.bits_of(out), call


def request_spans(call: W.Call):
    """(prompt tag, first position, first packed row, rows) of every request."""
    cu = call.cu_q_lens
    return [(call.prompts[r.prompt].tag, r.n - r.s, int(cu[i]), r.s) for i, r in enumerate(call.reqs)]


def assert_rows_equal(ref_call: W.Call, ref_out: np.ndarray, call: W.Call, out: np.ndarray,
                      min_rows: int = 1) -> int:
    """Every row of ``call`` whose (prompt, position) ``ref_call`` also holds
    equals that row of ``ref_out`` bit for bit (both written); returns how many
    rows were compared.  Compares whole runs of rows at once."""
    spans = {}
    for tag, p0, row0, s in request_spans(ref_call):
        spans.setdefault(tag, []).append((p0, row0, s))
    n = 0
    for tag, p0, row0, s in request_spans(call):
        for q0, qrow0, qs in spans.get(tag, []):
            lo, hi = max(p0, q0), min(p0 + s, q0 + qs)
            if lo >= hi:
                continue
            a = out[row0 + lo - p0:row0 + hi - p0]
            b = ref_out[qrow0 + lo - q0:qrow0 + hi - q0]
            for x, what in ((a, "variant"), (b, "reference")):
                assert not ((x & 0x7F80) == 0x7F80).any(), \
                    "unwritten or non-finite %s rows at positions %d..%d of %s" % (what, lo, hi, tag)
            if not np.array_equal(a, b):
                bad = [lo + i for i in range(hi - lo) if not np.array_equal(a[i], b[i])]
                raise AssertionError("bitwise mismatch at %d of %d rows of %s, positions %s"
                                     % (len(bad), hi - lo, tag, bad[:5]))
            n += hi - lo
    assert n >= min_rows, (n, min_rows)
    return n
