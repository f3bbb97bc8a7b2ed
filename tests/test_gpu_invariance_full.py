"""Bitwise invariance at the workloads' real sizes -- the causal contract of
Section 5.3 / Appendix A.1 (a row's bits depend only on its position, its
query and the keys and values it sees), where the kernels' ways of folding
splits meet:

* the mixed 8B batch's 8 chunk prompts (up to about 8,700 tokens) prefilled
  whole, in 512-, 128- and 64-token chunks (all chunks batched in one call),
  in 512- and 128-token chunks one call per chunk step handing its new tokens
  over, against each other and against their 512 rows in the mixed batch;
* single-token decode and 4-token verify steps of those prompts at split
  edges 1023 .. 8192 (those below their lengths), where the split path's
  merge kernel (4, 8 or 16 splits, or the long merge under a larger
  max_context_len hint) meets the chunk kernel's in-register fold of a whole
  prefill;
* an 18,500-token prompt: decode and verify rows in splits 16 .. 18 (the
  long merge) and rows of 3 .. 16 splits against the whole prefill;
* the 70B prefix-shared verify batch at full size: copied prefix pages, and
  every 4-token verify as four single-token calls, with the shared-prefix pass;
* a 100,000-key context where one key dominates the scores: every row that
  sees it returns that key's value bit for bit, whichever split and tile holds
  it (a dropped, duplicated or misplaced tile would not).
"""
from __future__ import annotations

import numpy as np
import pytest

from paper_2609_38981_amd import workloads as W
from tests import gpu_util as U

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    U.require_gpu()


# -- the mixed 8B batch's chunk prompts --------------------------------------
def cfg3_with_full_prompts():
    """The mixed 8B batch (8 chunks of 512 at offsets U[0, 8192] plus 120
    decodes), its 8 chunk prompts drawn with a query at every position (their
    keys and values are those of the batch's own draw, and so is the
    placement)."""
    call = W.config3()
    sh = call.shape
    prompts = list(call.prompts)
    for i in range(8):
        prompts[i] = W.make_prompt(sh, call.reqs[i].n, 3, i)
        assert np.array_equal(prompts[i].k, call.prompts[i].k)
        assert np.array_equal(prompts[i].v, call.prompts[i].v)
    return W.place(sh, prompts, call.reqs, W.rng_for(3, 4))


@pytest.fixture(scope="module")
def cfg3():
    mixed = cfg3_with_full_prompts()
    lens = [mixed.reqs[i].n for i in range(8)]
    # the 8 prompts alone, each prefilled whole (s = n): the reference rows
    base = W.place(mixed.shape, mixed.prompts[:8], [W.Req(i, n, n) for i, n in enumerate(lens)],
                   W.rng_for(3, 5))
    U.say("cfg3 prompts: lengths %s, %d rows whole" % (lens, sum(lens)))
    whole = U.gpu_run(base, poison=False)
    return mixed, base, whole, lens


def chunk_reqs(lens, size, step=None):
    """(prompt, n, s) requests of chunked prefill: chunk j of prompt i holds
    positions [j size, min((j + 1) size, n_i)); all chunks, or only step j's."""
    return [(i, min(e + size, n), min(size, n - e)) for i, n in enumerate(lens)
            for e in range(0, n, size) if step is None or e == step * size]


def test_cfg3_prompts_whole_vs_chunks(cfg3):
    mixed, base, whole, lens = cfg3
    total = sum(lens)
    # the whole prefills against the oracle on sampled rows
    rows = sorted({int(x) for x in np.random.default_rng(4).choice(total, 12, replace=False)})
    U.say("  whole vs oracle: %s" % U.parity(base, whole, rows=rows))
    sess = U.Session(base)
    for size in (512, 128, 64):
        # every chunk of every prompt in one call (64: more than the 256
        # requests whose workgroups plan their own items, so the plan launch
        # lists them)
        out, call = sess.run(chunk_reqs(lens, size))
        n = U.assert_rows_equal(base, whole, call, out, min_rows=total)
        U.say("  %d-token chunks, one call of %d requests: %d rows bit-identical"
              % (size, call.num_seqs, n))
    for size in (512, 128):
        # an engine's chunked prefill: one call per chunk step, the pools empty
        # at first, each call handing over its new tokens
        sess = U.Session(base, prefill=False)
        n, j = 0, 0
        while True:
            reqs = chunk_reqs(lens, size, step=j)
            if not reqs:
                break
            out, call = sess.run(reqs, append=True)
            n += U.assert_rows_equal(base, whole, call, out, min_rows=sum(s for _, _, s in reqs))
            j += 1
        assert n == total
        U.say("  %d-token chunks, %d calls appending their tokens: %d rows bit-identical"
              % (size, j, n))


def test_cfg3_mixed_batch_rows_vs_whole(cfg3):
    """The mixed batch itself (chunks and decodes in one call, with and
    without its new tokens handed over): every chunk's 512 rows equal those
    of the whole prefills."""
    mixed, base, whole, lens = cfg3
    for append in (False, True):
        out = U.gpu_run(mixed, poison=False, append=append)
        n = U.assert_rows_equal(base, whole, mixed, out, min_rows=8 * 512)
        U.say("  mixed batch (append=%s): %d chunk rows bit-identical" % (append, n))


SPLIT_EDGES = (1023, 1024, 1025, 2047, 4095, 4096, 8191, 8192)


def test_cfg3_prompts_steps_at_split_edges(cfg3):
    """Decode (s = 1) and verify (s = 4) calls whose last position is a split
    edge (or the prompt's last position), alone -- so that the merge kernel
    is sized for 1-4, 5-8 or 9-16 splits -- and with a 20,000-key
    max_context_len hint, which sends rows of 3 or more splits to the long
    merge; then all of them batched.  The whole prefills fold the same splits
    in registers."""
    mixed, base, whole, lens = cfg3
    sess = U.Session(base)
    pos = {i: sorted({p for p in SPLIT_EDGES if p < n} | {n - 1}) for i, n in enumerate(lens)}
    n = calls = 0
    for i, ps in pos.items():
        for p in ps:
            for s in (1, 4):
                for hint in (0, 20000):
                    out, call = sess.run([(i, p + 1, s)], hint_ctx=hint)
                    n += U.assert_rows_equal(base, whole, call, out, min_rows=s)
                    calls += 1
    dec = [(i, p + 1, 1) for i, ps in pos.items() for p in ps]
    ver = [(i, p + 1, 4) for i, ps in pos.items() for p in ps]
    for reqs in (dec, ver, dec + ver):
        for hint in (0, 20000):
            out, call = sess.run(reqs, hint_ctx=hint)
            n += U.assert_rows_equal(base, whole, call, out, min_rows=len(reqs))
            calls += 1
    U.say("  %d calls, %d rows bit-identical to the whole prefills" % (calls, n))


def test_long_prompt_long_merge_vs_register_fold():
    """An 18,500-token prompt (19 splits, a ragged last tile): rows in splits
    16, 17 and 18 as decode and verify steps (the long merge: more than 16
    splits) against the whole prefill (the chunk kernel's in-register fold);
    rows of 3, 8, 9 and 16 splits alone (the merge sized for 4, 8 or 16
    splits) and with a hint that sends them to the long merge."""
    sh = W.LLAMA8B
    n = 18500
    pr = W.make_prompt(sh, n, 14, 0)
    base = W.place(sh, [pr], [W.Req(0, n, n)], W.rng_for(14, 4))
    whole = U.gpu_run(base, poison=False)
    U.say("  18,500-token prefill vs oracle: %s"
          % U.parity(base, whole, rows=[0, 1023, 16384, 17500, n - 1]))
    sess = U.Session(base)
    ps = [3000, 8191, 8192, 9000, 16383, 16384, 16385, 17407, 17408, 18431, 18432, n - 1]
    cnt = 0
    for p in ps:
        for s in (1, 4):
            for hint in (0, 20000):
                out, call = sess.run([(0, p + 1, s)], hint_ctx=hint)
                cnt += U.assert_rows_equal(base, whole, call, out, min_rows=s)
    reqs = [(0, p + 1, s) for p in ps for s in (1, 4)]
    out, call = sess.run(reqs)
    cnt += U.assert_rows_equal(base, whole, call, out, min_rows=5 * len(ps))
    U.say("  %d rows bit-identical" % cnt)


# -- the 70B prefix-shared verify batch at full size --------------------------
def test_cfg5_full_size_copied_pages_and_single_token_steps():
    """256 requests on a shared 2048-token prefix (the shared-prefix pass
    reads it once): the same requests with the prefix copied into private
    pages, with and without the shared_pages hint, and each 4-token verify
    replaced by four single-token calls (positions n - 4 .. n - 1) with the
    prefix shared."""
    base = W.config5()
    sh = base.shape
    assert base.shares_pages()
    ref = U.gpu_run(base, poison=False)
    copied = W.place(sh, base.prompts, base.reqs, W.rng_for(5, 5))
    assert not copied.shares_pages()
    n = 0
    for hint in (False, True):
        out = U.gpu_run(copied, poison=False, shared_pages=hint)
        n += U.assert_rows_equal(base, ref, copied, out, min_rows=base.total_q_tokens)
    for step in range(4):
        reqs = [W.Req(r.prompt, r.n - 3 + step, 1) if r.s == 4 else r for r in base.reqs]
        c = W.place(sh, base.prompts, reqs, W.rng_for(5, 6 + step), shared_prefix_pages=2048 // 16)
        assert c.shares_pages()
        n += U.assert_rows_equal(base, ref, c, U.gpu_run(c, poison=False), min_rows=256)
    U.say("  full-size verify: %d rows bit-identical" % n)


# -- every key counts at 100K ---------------------------------------------------
N_LONG = 100_000
# the dominant key: first, middle and last key of splits 0, 50 and the last
# split (97: keys 99,328 .. 99,999), and the ragged last tile (99,968 ..)
DOMINANT = (0, 511, 1023, 50 * 1024, 50 * 1024 + 512, 51 * 1024 - 1, 97 * 1024,
            97 * 1024 + 300, N_LONG - 32, N_LONG - 1)


def dominant_key_call():
    """Prompt 0: N(0, 1) keys and values at 100,000 positions.  Prompt 1 + r:
    the same, except that every query head of KV head g asks one vector u_g
    (all rows) and key DOMINANT[r] is 4 u_g, so its scaled score (about 45)
    exceeds every other (about N(0, 1)) by more than 35: its weight is 1 and the
    sum of all others is below 2^-40, far under half an ulp of fp32.  The
    prompts share their pages but the one holding their dominant key."""
    sh = W.LLAMA8B
    G, P = sh.group, sh.page_size
    base = W.make_prompt(sh, N_LONG, 15, 0, q_window=64)
    prompts = [base]
    for r, j in enumerate(DOMINANT):
        u = W.normal_bf16(W.rng_for(15, 1, 100 + r), (sh.num_kv_heads, sh.head_dim))
        q = np.repeat(u[:, None, :], G, axis=1).reshape(sh.num_q_heads, sh.head_dim)
        k = base.k.copy()
        k[j] = W.bf16_bits(4.0 * W.bf16_to_f32(u))
        prompts.append(W.Prompt(N_LONG, k, base.v, N_LONG - 64,
                                np.ascontiguousarray(np.broadcast_to(q, (64,) + q.shape)),
                                tag=(15, 1 + r)))
    npg = -(-N_LONG // P)
    num_pages = npg + len(DOMINANT) + 37
    perm = W.rng_for(15, 4).permutation(num_pages)
    pt = np.tile(perm[:npg], (len(prompts), 1)).astype(np.int32)
    owner = {int(pg): (0, b) for b, pg in enumerate(perm[:npg])}
    for r, j in enumerate(DOMINANT):
        pg = int(perm[npg + r])
        pt[1 + r, j // P] = pg
        owner[pg] = (1 + r, j // P)
    reqs = [W.Req(i, N_LONG, 1) for i in range(len(prompts))]
    return W.Call(sh, prompts, reqs, pt, num_pages, owner)


def test_dominant_key_at_100k():
    base = dominant_key_call()
    sh = base.shape
    sess = U.Session(base)
    R = len(DOMINANT)
    dec = [(1 + r, N_LONG, 1) for r in range(R)]
    # chunk-path rows too (40 rows x 4 query heads per KV head = 160 columns)
    chunk = [(1 + r, N_LONG, 40) for r in (1, 4, 8, 9)]
    checked = 0
    for reqs, hint, shared in [([(0, N_LONG, 1)] + dec, 0, False), (dec, 0, True),
                               (dec + chunk, 0, False), (dec, 131072, False)]:
        out, call = sess.run(reqs, hint_ctx=hint, shared_pages=shared)
        for ri, (pid, n, s) in enumerate(reqs):
            if pid == 0:
                continue
            j = DOMINANT[pid - 1]
            want = np.repeat(base.prompts[pid].v[j][:, None, :], sh.group, axis=1).reshape(
                sh.num_q_heads, sh.head_dim)
            for p in range(max(n - s, j), n):
                got = out[call.row_of(ri, p)]
                bad = np.flatnonzero((got != want).any(axis=1))
                assert not len(bad), ("dominant key %d, row %d, heads %s: %s vs %s"
                                      % (j, p, bad[:4], got[bad[0]][:4], want[bad[0]][:4]))
                checked += 1
        if reqs[0][0] == 0:
            # the control request (no dominant key) against the oracle
            U.say("  control row at 100K keys vs oracle: %s" % U.parity(call, out, rows=[0]))
    U.say("  %d rows equal their dominant key's value bit for bit" % checked)
