"""GPU parity: the HIP path against the fp64 CPU oracle (max abs error within
TOL on bf16 outputs), the KV write bit for bit against the documented pool
layout, and exact closed forms."""
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


# -- a0: the KV write ---------------------------------------------------------
@pytest.mark.parametrize("shape", [W.TINY, W.LLAMA8B], ids=["d64", "d128"])
def test_kv_write_layout(shape):
    U.say("kv_write layout %s" % (shape,))
    attn = U.handle(shape)
    rng = np.random.default_rng(5)
    num_pages, T = 37, 300
    slots = rng.choice(num_pages * 16, size=T, replace=False).astype(np.int64)
    slots[7] = -1  # skipped
    slots[9] = num_pages * 16 + 3  # out of range: skipped
    k = W.normal_bf16(rng, (T, shape.num_kv_heads, shape.head_dim))
    v = W.normal_bf16(rng, (T, shape.num_kv_heads, shape.head_dim))
    kp, vp = attn.new_pool(num_pages), attn.new_pool(num_pages)
    kp.view(torch.int16).fill_(0x1234)
    vp.view(torch.int16).fill_(0x1234)
    attn.kv_write(S.bf16_tensor(k, "cuda"), S.bf16_tensor(v, "cuda"),
                  torch.from_numpy(slots).cuda(), kp, vp, num_pages)
    torch.cuda.synchronize()
    D, H = shape.head_dim, shape.num_kv_heads
    kb = S.bits_of(kp).reshape(num_pages, H, 16 * D)
    vb = S.bits_of(vp).reshape(num_pages, H, 16 * D)
    # decode the layout stated in include/vdattn.h
    d = np.arange(D)
    for t in range(T):
        sl = slots[t]
        if sl < 0 or sl >= num_pages * 16:
            continue
        page, s = sl // 16, sl % 16
        kidx = ((d // 8) * 16 + s) * 8 + d % 8
        vidx = ((d // 16) * 4 + s // 4) * 64 + (d % 16) * 4 + s % 4
        assert np.array_equal(kb[page][:, kidx], k[t]), t
        assert np.array_equal(vb[page][:, vidx], v[t]), t
    written = set(int(x) for x in slots if 0 <= x < num_pages * 16)
    untouched = [sl for sl in range(num_pages * 16) if sl not in written][:50]
    for sl in untouched:
        page, s = sl // 16, sl % 16
        assert (kb[page][:, ((d // 8) * 16 + s) * 8 + d % 8] == 0x1234).all()


# -- parity against the oracle, sizes the oracle finishes in seconds ----------
SMALL = {
    "cfg1_tiny": lambda: W.config1(),
    "cfg1_tiny_permB": lambda: W.config1(perm_stream=5),
    "cfg2_decode_small": lambda: W.config2(batch=8, lo=100, hi=1500),
    "cfg3_mixed_small": lambda: W.config3(num_prefill=2, chunk=40, max_off=700, num_decode=6,
                                          dec_lo=50, dec_hi=1200),
    "cfg4_long_small": lambda: W.config4(batch=2, lo=3000, hi=5000),
    # more than 16 splits per request: the long merge
    "cfg4_long_mid": lambda: W.config4(batch=3, lo=9000, hi=40000),
    "cfg5_verify_small": lambda: W.config5(num_req=6, prefix=256, suf_lo=20, suf_hi=80),
    "d64_prefill_chunks": lambda: W.place(W.TINY, [W.make_prompt(W.TINY, 700, 9, 0)],
                                          [W.Req(0, 700, 700)], W.rng_for(9, 4)),
    # 32 query heads per KV head: a one-row decode has 32 query-head rows, two
    # split items per split (column halves)
    "g32_decode": lambda: W.config2(batch=6, lo=100, hi=2500, shape=W.Shape(32, 1, 128), cfg=7),
    "g32_d64_mixed": lambda: W.config3(num_prefill=1, chunk=20, max_off=900, num_decode=5,
                                       dec_lo=50, dec_hi=2200, shape=W.Shape(64, 2, 64), cfg=7),
}


@pytest.mark.parametrize("name", sorted(SMALL))
def test_parity_small(name):
    call = SMALL[name]()
    U.say("parity %s: B=%d T=%d max_n=%d" % (name, call.num_seqs, call.total_q_tokens,
                                             call.max_context_len))
    out = U.gpu_run(call)
    st = U.parity(call, out)
    U.say("  %s" % st)


EDGE_LENGTHS = [(1, 1), (2, 1), (16, 1), (17, 1), (63, 1), (64, 1), (65, 1), (511, 1), (512, 1),
                (513, 1), (1023, 1), (1024, 1), (1025, 1), (2047, 1), (2048, 1), (2049, 1),
                (16, 16), (65, 9), (513, 8), (1025, 8), (600, 120), (1100, 1100)]


@pytest.mark.parametrize("shape", [W.TINY, W.LLAMA8B, W.LLAMA70B], ids=["tiny", "8b", "70b"])
def test_parity_edge_lengths(shape):
    """Ragged tails around page (16), tile (64) and split (1024) boundaries, on
    both the split path (few query rows) and the chunk path (many)."""
    prompts = [W.make_prompt(shape, n, 8, i, q_window=s) for i, (n, s) in enumerate(EDGE_LENGTHS)]
    reqs = [W.Req(i, n, s) for i, (n, s) in enumerate(EDGE_LENGTHS)]
    call = W.place(shape, prompts, reqs, W.rng_for(8, 4))
    U.say("edge lengths %s T=%d" % (shape, call.total_q_tokens))
    out = U.gpu_run(call)
    U.say("  %s" % U.parity(call, out))


def test_single_key_is_exact():
    """n = 1 (and row p = 0 of a whole prefill) returns v_0 bit for bit: one
    visible key gives weight exp2(0) = 1, z = 1, 1/z = 1."""
    sh = W.LLAMA8B
    prompts = [W.make_prompt(sh, 1, 7, 0), W.make_prompt(sh, 40, 7, 1)]
    call = W.place(sh, prompts, [W.Req(0, 1, 1), W.Req(1, 40, 40)], W.rng_for(7, 4))
    out = U.gpu_run(call)
    for ri, pid in [(0, 0), (1, 1)]:
        row = out[call.row_of(ri, 0)]
        v0 = prompts[pid].v[0]  # [Hkv, D]
        for h in range(sh.num_q_heads):
            assert np.array_equal(row[h], v0[h // sh.group]), (ri, h)


def test_parity_full_size_decode_sampled():
    """Llama-3-8B decode at full size (64 requests, contexts 512..4096): 16
    sampled rows against the oracle, in the launch configuration the
    benchmark times."""
    call = W.config2()
    U.say("full cfg2: T=%d kv=%.1f MB" % (call.total_q_tokens, call.kv_bytes() / 1e6))
    out = U.gpu_run(call, poison=False)
    rows = np.random.default_rng(3).choice(call.total_q_tokens, 16, replace=False)
    U.say("  %s" % U.parity(call, out, rows=rows))


def _sample_rows(call, per_req=2, max_reqs=6, seed=0):
    """First and last query row of up to ``max_reqs`` requests, plus random rows."""
    rng = np.random.default_rng(seed)
    reqs = sorted(rng.choice(call.num_seqs, min(max_reqs, call.num_seqs), replace=False))
    rows = set()
    for ri in reqs:
        lo, hi = int(call.cu_q_lens[ri]), int(call.cu_q_lens[ri + 1])
        rows.update({lo, hi - 1})
        rows.update(int(x) for x in rng.integers(lo, hi, size=per_req))
    return sorted(rows)


def test_parity_full_size_mixed_sampled():
    """Mixed 8B batch at full size: 8 prefill chunks of 512 at offsets up to
    8192 plus 120 decodes, in the benchmark's launch configuration."""
    call = W.config3()
    U.say("full cfg3: T=%d kv=%.2f GB" % (call.total_q_tokens, call.kv_bytes() / 1e9))
    out = U.gpu_run(call, poison=False)
    rows = _sample_rows(call, per_req=3, max_reqs=10)
    rows += [int(call.cu_q_lens[i]) for i in range(8)]  # first row of every chunk
    U.say("  %s" % U.parity(call, out, rows=sorted(set(rows))))


def test_parity_full_size_long_decode():
    """Long-context decode at full size (8 requests, contexts 32K..128K): every
    row against the oracle (up to 121 splits per row: the long merge folds
    them in chunks of 64).  The batch has more split items than the split
    launch has workgroups, so the later items go to whichever workgroups ask
    first: a second run (another assignment) and the first and last requests
    alone (a few hundred items, no claims) give the same bits."""
    call = W.config4()
    U.say("full cfg4: kv=%.2f GB max_n=%d" % (call.kv_bytes() / 1e9, call.max_context_len))
    out = U.gpu_run(call, poison=False)
    U.say("  %s" % U.parity(call, out))
    rows = U.by_position(call, out)
    again = U.gpu_run(call, poison=True)
    n = U.assert_same_bits(rows, U.by_position(call, again), min_common=len(call.reqs))
    for i in (0, len(call.reqs) - 1):
        sub = call.subcall([i])
        n += U.assert_same_bits(rows, U.by_position(sub, U.gpu_run(sub)))
    U.say("  %d rows bit-identical across runs and alone" % n)


def test_claimed_items_with_empty_slots_in_the_last_die_range():
    """3 KV heads: 4,461 split items, not a multiple of the 8 dies, so the
    last die's range ends with 3 slots that hold no item; a workgroup that
    claims one of them claims again.  Sampled rows against the oracle, a
    second run and requests alone bit for bit."""
    rng = W.rng_for(8, 0)
    sh = W.Shape(12, 3, 128)
    prompts, reqs = [], []
    for r in range(13):
        n = int(rng.integers(110000, 125001))
        prompts.append(W.make_prompt(sh, n, 8, r, q_window=1))
        reqs.append(W.Req(r, n, 1))
    call = W.place(sh, prompts, reqs, rng)
    items = sum((r.n - 1) // 1024 + 1 for r in reqs) * sh.num_kv_heads
    assert items > 4096 and items % 8 != 0, items
    U.say("3 KV heads: %d requests, %d split items" % (len(reqs), items))
    out = U.gpu_run(call)
    U.say("  %s" % U.parity(call, out, rows=[0, 6, 12]))
    rows = U.by_position(call, out)
    n = U.assert_same_bits(rows, U.by_position(call, U.gpu_run(call)), min_common=len(reqs))
    for i in (0, 12):
        sub = call.subcall([i])
        n += U.assert_same_bits(rows, U.by_position(sub, U.gpu_run(sub)))
    U.say("  %d rows bit-identical across runs and alone" % n)


def test_parity_full_size_verify_sampled():
    """70B prefix-shared verify at full size (256 requests on a shared
    2048-token prefix, s = 4 / 1)."""
    call = W.config5()
    U.say("full cfg5: T=%d kv(logical)=%.2f GB" % (call.total_q_tokens, call.kv_bytes() / 1e9))
    out = U.gpu_run(call, poison=False)
    U.say("  %s" % U.parity(call, out, rows=_sample_rows(call, per_req=2, max_reqs=8)))


@pytest.mark.parametrize("name", ["cfg1_tiny", "cfg3_mixed_small", "cfg5_verify_small"])
def test_append_then_attend(name):
    """The call's own tokens handed to vd_attn_forward (written by the split
    items themselves, or by the plan launch when the call has prefill rows)
    instead of written beforehand with vd_kv_write: the same bits, and within
    tolerance of the oracle."""
    call = SMALL[name]()
    a = U.gpu_run(call, append=True)
    b = U.gpu_run(call)
    assert np.array_equal(a, b)
    U.say("  append %s: %s" % (name, U.parity(call, a)))


APPEND_LENS = [(300, 100), (97, 40), (1500, 1), (700, 4), (64, 64), (1100, 33), (17, 17)]


@pytest.mark.parametrize("shape", [W.TINY, W.LLAMA8B, W.LLAMA70B, W.Shape(8, 8, 64)],
                         ids=["g2_d64", "g4_d128", "g8_d128", "g1_d64"])
def test_append_writes_the_pool_like_kv_write(shape):
    """A call handed its new tokens (k_new / v_new) leaves the pools bit for
    bit as vd_kv_write of every token would: runs of new positions that start
    and end inside pages, rows on the split path (written by the split items)
    and on the chunk path (written by the split launch's append workgroups, or
    by the plan launch when a split-path request may hold more than 16 rows);
    the slots of other positions keep their NaN fill.  The outputs equal those
    of the call whose tokens were written beforehand."""
    prompts = [W.make_prompt(shape, n, 16, i, q_window=s) for i, (n, s) in enumerate(APPEND_LENS)]
    call = W.place(shape, prompts, [W.Req(i, n, s) for i, (n, s) in enumerate(APPEND_LENS)],
                   W.rng_for(16, 4))
    attn = U.handle(shape)
    outs, pools = [], []
    for append in (True, False):
        dc = S.to_device(attn, call, poison=True, append=append)
        out = torch.empty_like(dc.batch.q)
        out.view(torch.int16).fill_(U.FILL)
        ws = attn.new_workspace(call.num_seqs, dc.batch.max_q_len, dc.batch.max_context_len)
        attn.forward(dc.batch, out=out, workspace=ws)
        torch.cuda.synchronize()
        outs.append(S.bits_of(out))
        pools.append((S.bits_of(dc.batch.k_pool), S.bits_of(dc.batch.v_pool)))
    assert np.array_equal(pools[0][0], pools[1][0]), "K pool differs from vd_kv_write's"
    assert np.array_equal(pools[0][1], pools[1][1]), "V pool differs from vd_kv_write's"
    U.assert_same_bits(U.by_position(call, outs[0]), U.by_position(call, outs[1]),
                       min_common=call.total_q_tokens)
    U.say("  append %s: %s" % (shape, U.parity(call, outs[0])))
