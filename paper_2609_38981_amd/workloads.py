"""Seeded synthetic inputs for paged causal attention.

This module only *generates and places data*: request lengths, bf16 query /
key / value values drawn from N(0, 1), page placements in a pool, and the
packed per-call metadata (``cu_q_lens``, ``context_lens``, page table).  It
holds none of the attention arithmetic, so both the CPU oracle side and the
GPU side of the tests (and the benchmark) can draw their inputs from it.

Seeding: every draw uses ``numpy.random.Generator(PCG64(SeedSequence([1000 *
cfg + stream, *extra])))`` with streams
    0: lengths and offsets, 1: Q, 2: K, 3: V, 4: page placement A,
    5: page placement B, 6: the probe request, 7: companion requests.

Values: iid N(0, 1) float32 (torch's CPU generator, seeded from the stream
above) rounded to bf16 with round-to-nearest-even.
Pools: pages are a random permutation of the pool; each request takes
consecutive entries of it, so its pages are scattered.  Unused pages and
slots at positions >= n hold a poison value (bf16 quiet NaN) unless told
otherwise.

Shapes of the five workload families (head_dim D, page size 16 throughout):
    tiny      Hq 4  / Hkv 2, D 64
    llama8b   Hq 32 / Hkv 8, D 128
    llama70b  Hq 64 / Hkv 8, D 128
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

BF16_QNAN = np.uint16(0x7FC0)


# ---------------------------------------------------------------------------
# bf16 encoding helpers (data encoding only)
# ---------------------------------------------------------------------------
def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even.

    NaN inputs map to the canonical quiet NaN.  (For every non-NaN input the
    sum below stays below 2**32, so uint32 arithmetic is exact.)  Works in
    cache-sized chunks."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.reshape(-1).view(np.uint32)
    out = np.empty(u.shape, np.uint16)
    step = 1 << 18
    tmp = np.empty(step, np.uint32)
    for lo in range(0, u.size, step):
        hi = min(lo + step, u.size)
        t = tmp[:hi - lo]
        np.right_shift(u[lo:hi], 16, out=t)
        np.bitwise_and(t, 1, out=t)
        t += np.uint32(0x7FFF)
        t += u[lo:hi]
        np.right_shift(t, 16, out=t)
        out[lo:hi] = t
    nan = np.isnan(x.reshape(-1))
    if nan.any():
        out[nan] = BF16_QNAN
    return out.reshape(x.shape)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float32 (exact)."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def rng_for(cfg: int, stream: int, *extra: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([1000 * cfg + stream, *extra])))


def normal_bf16(rng: np.random.Generator, shape) -> np.ndarray:
    """iid N(0, 1) values rounded to bf16 (nearest even), as uint16 bits.

    The values come from torch's CPU generator (deterministic for a given
    seed whatever the thread count, and several times faster than numpy's
    for the gigabyte-sized pools), seeded from ``rng``."""
    import torch

    g = torch.Generator().manual_seed(int(rng.integers(0, 2**63 - 1)))
    n = int(np.prod(shape)) if len(shape) else 1
    x = torch.randn(n, generator=g, dtype=torch.float32).to(torch.bfloat16)
    return x.view(torch.int16).numpy().view(np.uint16).reshape(shape)


# ---------------------------------------------------------------------------
# Shapes
# ---------------------------------------------------------------------------
@dataclass(frozen=True)
class Shape:
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int = 16
    window: int = 0  # sliding-window attention span in keys; 0 = full causal prefix

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads


TINY = Shape(4, 2, 64)
LLAMA8B = Shape(32, 8, 128)
LLAMA70B = Shape(64, 8, 128)
# Llama-3-8B head geometry with a 4096-key sliding window (Appendix A.5)
LLAMA8B_SWA4K = Shape(32, 8, 128, window=4096)


# ---------------------------------------------------------------------------
# Prompts: the logical per-position data of one synthetic sequence
# ---------------------------------------------------------------------------
@dataclass
class Prompt:
    """Logical K/V for positions [0, length) and queries for [q_lo, length).

    k, v: uint16 [length, Hkv, D];  q: uint16 [length - q_lo, Hq, D].
    """
    length: int
    k: np.ndarray
    v: np.ndarray
    q_lo: int
    q: np.ndarray
    prefix_key: Optional[int] = None  # identity of a shared prefix, if any
    prefix_len: int = 0
    tag: Tuple[int, ...] = ()          # identity of the draw: (cfg, pid)

    def q_rows(self, lo: int, hi: int) -> np.ndarray:
        assert self.q_lo <= lo <= hi <= self.length, (self.q_lo, lo, hi, self.length)
        return self.q[lo - self.q_lo:hi - self.q_lo]


def make_prompt(shape: Shape, length: int, cfg: int, pid: int, q_window: Optional[int] = None,
                prefix: Optional[Prompt] = None, prefix_len: int = 0) -> Prompt:
    """Draws one prompt.  With ``prefix``, positions [0, prefix_len) copy that
    prompt's K/V (a shared, page-aligned prefix); the rest is fresh."""
    hkv, hq, d = shape.num_kv_heads, shape.num_q_heads, shape.head_dim
    q_window = length if q_window is None else min(q_window, length)
    q_lo = length - q_window
    own = length - prefix_len
    k = np.empty((length, hkv, d), np.uint16)
    v = np.empty((length, hkv, d), np.uint16)
    if prefix_len:
        assert prefix is not None and prefix.length >= prefix_len
        k[:prefix_len] = prefix.k[:prefix_len]
        v[:prefix_len] = prefix.v[:prefix_len]
    k[prefix_len:] = normal_bf16(rng_for(cfg, 2, pid), (own, hkv, d))
    v[prefix_len:] = normal_bf16(rng_for(cfg, 3, pid), (own, hkv, d))
    q = normal_bf16(rng_for(cfg, 1, pid), (q_window, hq, d))
    key = id(prefix) if prefix_len else None
    return Prompt(length, k, v, q_lo, q, key, prefix_len, (cfg, pid))


# ---------------------------------------------------------------------------
# A call: requests packed into one invocation with a page placement
# ---------------------------------------------------------------------------
@dataclass
class Req:
    prompt: int  # index into Call.prompts
    n: int       # key length (counts this call's own query tokens)
    s: int       # query length

    @property
    def positions(self) -> range:
        return range(self.n - self.s, self.n)


@dataclass
class Call:
    shape: Shape
    prompts: List[Prompt]
    reqs: List[Req]
    page_table: np.ndarray          # int32 [B, stride]
    num_pages: int
    # physical page -> (prompt, logical page) it holds (for writing the pool)
    page_owner: Dict[int, Tuple[int, int]] = field(default_factory=dict)

    # -- packed metadata ----------------------------------------------------
    @property
    def num_seqs(self) -> int:
        return len(self.reqs)

    @property
    def cu_q_lens(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum([r.s for r in self.reqs])]).astype(np.int32)

    @property
    def context_lens(self) -> np.ndarray:
        return np.array([r.n for r in self.reqs], np.int32)

    @property
    def total_q_tokens(self) -> int:
        return int(sum(r.s for r in self.reqs))

    @property
    def max_q_len(self) -> int:
        return max((r.s for r in self.reqs), default=0)

    @property
    def max_context_len(self) -> int:
        return max((r.n for r in self.reqs), default=0)

    def q_bits(self) -> np.ndarray:
        sh = self.shape
        if not self.reqs:
            return np.zeros((0, sh.num_q_heads, sh.head_dim), np.uint16)
        return np.concatenate([self.prompts[r.prompt].q_rows(r.n - r.s, r.n) for r in self.reqs])

    def row_of(self, req_index: int, position: int) -> int:
        """Packed token index of (request, logical position)."""
        r = self.reqs[req_index]
        assert r.n - r.s <= position < r.n
        return int(self.cu_q_lens[req_index]) + position - (r.n - r.s)

    def subcall(self, req_indices: Sequence[int]) -> "Call":
        """The same requests' logical data in a compact pool: only the pages
        of the selected requests, renumbered in table order."""
        P = self.shape.page_size
        remap: Dict[int, int] = {}
        owner: Dict[int, Tuple[int, int]] = {}
        pt = np.full((len(req_indices), max(self.page_table.shape[1], 1)), -1, np.int32)
        for k, i in enumerate(req_indices):
            r = self.reqs[i]
            for b in range(-(-r.n // P)):
                pg = int(self.page_table[i, b])
                if pg not in remap:
                    remap[pg] = len(remap)
                    # a page shared by several prompts holds the same data for
                    # each of them: take it from this request's prompt
                    owner[remap[pg]] = (r.prompt, b)
                pt[k, b] = remap[pg]
        return Call(self.shape, self.prompts, [self.reqs[i] for i in req_indices], pt,
                    max(len(remap), 1), owner)

    def request_of_row(self, row: int) -> int:
        cu = self.cu_q_lens
        return int(np.searchsorted(cu, row, side="right") - 1)

    # -- pool contents ------------------------------------------------------
    def first_key(self, ri: int) -> int:
        """First key any row of request ri can see: 0, or with a sliding
        window of w keys the window start of its first row, max(0, n - s - w + 1)."""
        r, w = self.reqs[ri], self.shape.window
        return max(0, r.n - r.s - w + 1) if w > 0 else 0

    def kv_bytes(self) -> int:
        """Algorithmic K+V bytes: every request reads each key its rows can see
        (keys first_key .. n - 1) once."""
        sh = self.shape
        keys = sum(r.n - self.first_key(ri) for ri, r in enumerate(self.reqs))
        return int(keys) * sh.num_kv_heads * sh.head_dim * 2 * 2

    def unique_kv_bytes(self, req_indices=None) -> int:
        """K+V bytes of the distinct cache slots the given requests (default:
        all) read (the keys their rows can see): a slot of a page shared by
        several requests counts once."""
        sh = self.shape
        P = sh.page_size
        idx = range(len(self.reqs)) if req_indices is None else req_indices
        used = {}  # page -> bit mask of its slots read
        for ri in idx:
            n, lo = int(self.context_lens[ri]), self.first_key(ri)
            for lp in range(lo // P, -(-n // P)):
                page = int(self.page_table[ri, lp])
                a, b = max(0, lo - lp * P), min(P, n - lp * P)
                used[page] = used.get(page, 0) | (((1 << (b - a)) - 1) << a)
        slots = sum(bin(m).count("1") for m in used.values())
        return int(slots) * sh.num_kv_heads * sh.head_dim * 2 * 2

    def new_tokens(self) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
        """This call's own tokens (positions n - s .. n - 1 of every request):
        (k_rows, v_rows [N, Hkv, D] uint16, slot ids int64 [N])."""
        P = self.shape.page_size
        ks, vs, slots, seen = [], [], [], set()
        for ri, r in enumerate(self.reqs):
            pr = self.prompts[r.prompt]
            for p in r.positions:
                sl = int(self.page_table[ri, p // P]) * P + p % P
                if sl in seen:
                    continue
                seen.add(sl)
                ks.append(pr.k[p])
                vs.append(pr.v[p])
                slots.append(sl)
        sh = self.shape
        if not ks:
            e = np.zeros((0, sh.num_kv_heads, sh.head_dim), np.uint16)
            return e, e.copy(), np.zeros(0, np.int64)
        return np.stack(ks), np.stack(vs), np.array(slots, np.int64)

    def query_kv(self) -> Tuple[np.ndarray, np.ndarray]:
        """K and V of the query rows, row t = query row t (position n - s + i
        of its request): (k_rows, v_rows [T, Hkv, D] uint16)."""
        sh = self.shape
        if not self.reqs:
            e = np.zeros((0, sh.num_kv_heads, sh.head_dim), np.uint16)
            return e, e.copy()
        k = np.concatenate([self.prompts[r.prompt].k[r.n - r.s:r.n] for r in self.reqs])
        v = np.concatenate([self.prompts[r.prompt].v[r.n - r.s:r.n] for r in self.reqs])
        return k, v

    def shares_pages(self) -> bool:
        """Whether some page is read by more than one request of the call."""
        P = self.shape.page_size
        seen = set()
        for ri in range(len(self.reqs)):
            n, lo = int(self.context_lens[ri]), self.first_key(ri)
            pages = {int(self.page_table[ri, lp]) for lp in range(lo // P, -(-n // P))}
            if pages & seen:
                return True
            seen |= pages
        return False

    def write_list(self, exclude_new: bool = False) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
        """Every valid physical slot once: (k_rows, v_rows [W, Hkv, D] uint16,
        slot ids int64 [W] with slot = page * P + offset).  With
        ``exclude_new``, the slots of this call's own tokens are left out."""
        P = self.shape.page_size
        ks, vs, slots = [], [], []
        for page, (pid, lp) in sorted(self.page_owner.items()):
            pr = self.prompts[pid]
            lo = lp * P
            hi = min(lo + P, self.filled_len(pid))
            if hi <= lo:
                continue
            ks.append(pr.k[lo:hi])
            vs.append(pr.v[lo:hi])
            slots.append(page * P + np.arange(hi - lo, dtype=np.int64))
        sh = self.shape
        if not ks:
            e = np.zeros((0, sh.num_kv_heads, sh.head_dim), np.uint16)
            return e, e.copy(), np.zeros(0, np.int64)
        k, v, sl = np.concatenate(ks), np.concatenate(vs), np.concatenate(slots)
        if exclude_new:
            keep = ~np.isin(sl, self.new_tokens()[2])
            k, v, sl = k[keep], v[keep], sl[keep]
        return k, v, sl

    def filled_len(self, pid: int) -> int:
        """Positions of prompt ``pid`` present in the pool: the longest n of
        any request of this call that reads it."""
        return max(r.n for r in self.reqs if r.prompt == pid)

    def std_pool(self, poison: bool = True, prompts=None) -> Tuple[np.ndarray, np.ndarray]:
        """Pool in the plain layout [num_pages, Hkv, P, D] (uint16).  With
        ``prompts`` (a set of prompt indices) only their pages are filled."""
        sh = self.shape
        P = sh.page_size
        shape = (self.num_pages, sh.num_kv_heads, P, sh.head_dim)
        fill = BF16_QNAN if poison else np.uint16(0)
        kp = np.full(shape, fill, np.uint16)
        vp = np.full(shape, fill, np.uint16)
        by_prompt: Dict[int, List[Tuple[int, int]]] = {}
        for page, (pid, lp) in self.page_owner.items():
            if prompts is None or pid in prompts:
                by_prompt.setdefault(pid, []).append((lp, page))
        for pid, lst in by_prompt.items():
            lst.sort()
            pr = self.prompts[pid]
            n = self.filled_len(pid)
            lps = np.array([lp for lp, _ in lst])
            pages = np.array([pg for _, pg in lst])
            full = lps < n // P  # pages with all P slots filled
            if full.any():
                idx = lps[full][:, None] * P + np.arange(P)  # [pages, P] positions
                kp[pages[full]] = pr.k[idx].transpose(0, 2, 1, 3)
                vp[pages[full]] = pr.v[idx].transpose(0, 2, 1, 3)
            for lp, page in zip(lps[~full], pages[~full]):
                lo, hi = lp * P, min(lp * P + P, n)
                if hi > lo:
                    kp[page, :, :hi - lo, :] = pr.k[lo:hi].transpose(1, 0, 2)
                    vp[page, :, :hi - lo, :] = pr.v[lo:hi].transpose(1, 0, 2)
        return kp, vp


def place(shape: Shape, prompts: List[Prompt], reqs: List[Req], rng: np.random.Generator,
          pool_factor: float = 1.5, min_pages: int = 0, stride_extra: int = 0,
          shared_prefix_pages: int = 0) -> Call:
    """Places every request's pages in a randomly permuted pool.

    Each distinct prompt gets its own pages (requests reading the same prompt
    in one call share them: a prompt's page b is one physical page).  With
    ``shared_prefix_pages`` > 0, logical pages [0, shared_prefix_pages) of all
    prompts built on one common prefix map to the same physical pages."""
    P = shape.page_size
    need: Dict[int, int] = {}
    for r in reqs:
        need[r.prompt] = max(need.get(r.prompt, 0), -(-r.n // P))
    # pages required
    shared_groups: Dict[int, List[int]] = {}
    if shared_prefix_pages:
        for pid in sorted(need):
            pr = prompts[pid]
            if pr.prefix_key is not None and pr.prefix_len >= shared_prefix_pages * P:
                shared_groups.setdefault(pr.prefix_key, []).append(pid)
    total = 0
    for pid, npg in need.items():
        total += npg
    if shared_prefix_pages:
        total -= sum((len(g) - 1) * shared_prefix_pages for g in shared_groups.values())
    num_pages = max(int(np.ceil(total * pool_factor)), total, min_pages, 1)
    perm = rng.permutation(num_pages).astype(np.int64)
    cursor = 0
    table: Dict[int, List[int]] = {}
    owner: Dict[int, Tuple[int, int]] = {}
    if shared_prefix_pages:
        for grp in shared_groups.values():
            pages = perm[cursor:cursor + shared_prefix_pages].tolist()
            cursor += shared_prefix_pages
            for pid in grp:
                table[pid] = list(pages)
            for b, pg in enumerate(pages):
                owner[pg] = (grp[0], b)
    for pid in sorted(need):
        start = len(table.get(pid, []))
        pages = perm[cursor:cursor + need[pid] - start].tolist()
        cursor += need[pid] - start
        table[pid] = table.get(pid, []) + pages
        for b, pg in enumerate(pages, start=start):
            owner[pg] = (pid, b)
    stride = max((need[p] for p in need), default=0) + stride_extra
    stride = max(stride, 1)
    pt = np.full((len(reqs), stride), -1, np.int32)
    for i, r in enumerate(reqs):
        pg = table[r.prompt]
        pt[i, :len(pg)] = pg
    return Call(shape, prompts, reqs, pt, num_pages, owner)


# ---------------------------------------------------------------------------
# The five workload families
# ---------------------------------------------------------------------------
def config1(perm_stream: int = 4, variant: str = "both") -> Call:
    """Tiny: request A (context 37, decodes 1 token) and request B (context
    100, prefills an 8-token chunk), Hq 4 / Hkv 2, D 64, P 16, 32-page pool.

    variant: "both" (A and B co-batched), "A" (A alone), "B" (B alone),
    "B44a" / "B44b" (B's chunk as 4 + 4: n = 96, s = 4 then n = 100, s = 4),
    "BA" (order swapped)."""
    sh = TINY
    pa = make_prompt(sh, 37, 1, 0)
    pb = make_prompt(sh, 100, 1, 1)
    prompts = [pa, pb]
    reqs = {
        "both": [Req(0, 37, 1), Req(1, 100, 8)],
        "BA": [Req(1, 100, 8), Req(0, 37, 1)],
        "A": [Req(0, 37, 1)],
        "B": [Req(1, 100, 8)],
        "B44a": [Req(1, 96, 4)],
        "B44b": [Req(1, 100, 4)],
    }[variant]
    return place(sh, prompts, reqs, rng_for(1, perm_stream), min_pages=32, pool_factor=1.0)


def _uniform_int(rng, lo, hi, size):
    return rng.integers(lo, hi + 1, size=size)


def config2(batch: int = 64, lo: int = 512, hi: int = 4096, perm_stream: int = 4,
            probe_slot: Optional[int] = None, shape: Shape = LLAMA8B, cfg: int = 2,
            pool_factor: float = 1.5) -> Call:
    """Llama-3-8B-shaped decode: ``batch`` requests with contexts uniform in
    [lo, hi], one query token each.  With ``probe_slot``, the fixed probe
    request (stream 6) takes that slot and companions fill the rest."""
    lens = _uniform_int(rng_for(cfg, 0), lo, hi, batch)
    prompts, reqs = [], []
    probe_len = int(_uniform_int(rng_for(cfg, 6), lo, hi, 1)[0])
    for i in range(batch):
        if probe_slot is not None and i == probe_slot:
            prompts.append(make_prompt(shape, probe_len, cfg, 10_000, q_window=1))
            reqs.append(Req(len(prompts) - 1, probe_len, 1))
        else:
            n = int(lens[i])
            prompts.append(make_prompt(shape, n, cfg, i, q_window=1))
            reqs.append(Req(len(prompts) - 1, n, 1))
    return place(shape, prompts, reqs, rng_for(cfg, perm_stream), pool_factor=pool_factor)


def config3(num_prefill: int = 8, chunk: int = 512, max_off: int = 8192, num_decode: int = 120,
            dec_lo: int = 256, dec_hi: int = 8192, shuffle: bool = False,
            perm_stream: int = 4, shape: Shape = LLAMA8B, cfg: int = 3) -> Call:
    """Mixed chunked-prefill batch: ``num_prefill`` chunks of ``chunk`` tokens
    at prefix offsets uniform in [0, max_off] plus ``num_decode`` single-token
    decodes with contexts uniform in [dec_lo, dec_hi]."""
    r0 = rng_for(cfg, 0)
    offs = _uniform_int(r0, 0, max_off, num_prefill)
    dlens = _uniform_int(r0, dec_lo, dec_hi, num_decode)
    prompts, reqs = [], []
    for i in range(num_prefill):
        n = int(offs[i]) + chunk
        prompts.append(make_prompt(shape, n, cfg, i, q_window=chunk))
        reqs.append(Req(i, n, chunk))
    for j in range(num_decode):
        n = int(dlens[j])
        prompts.append(make_prompt(shape, n, cfg, 1000 + j, q_window=1))
        reqs.append(Req(num_prefill + j, n, 1))
    if shuffle:
        order = rng_for(cfg, 7).permutation(len(reqs))
        reqs = [reqs[k] for k in order]
    return place(shape, prompts, reqs, rng_for(cfg, perm_stream))


def config4(batch: int = 8, lo: int = 32768, hi: int = 131072, perm_stream: int = 4,
            only: Optional[int] = None, shape: Shape = LLAMA8B, cfg: int = 4) -> Call:
    """Long-context decode: ``batch`` requests with contexts uniform in
    [lo, hi].  ``only`` keeps a single request (the batch-1 variant)."""
    lens = _uniform_int(rng_for(cfg, 0), lo, hi, batch)
    prompts = [make_prompt(shape, int(n), cfg, i, q_window=1) for i, n in enumerate(lens)]
    reqs = [Req(i, int(n), 1) for i, n in enumerate(lens)]
    if only is not None:
        reqs = [reqs[only]]
    return place(shape, prompts, reqs, rng_for(cfg, perm_stream))


def config5(num_req: int = 256, prefix: int = 2048, suf_lo: int = 64, suf_hi: int = 512,
            shared: bool = True, step: Optional[int] = None, perm_stream: int = 4,
            shape: Shape = LLAMA70B, cfg: int = 5) -> Call:
    """Prefix-shared verify: ``num_req`` requests on a common ``prefix``-token
    prefix (shared pages when ``shared``) plus unique suffixes uniform in
    [suf_lo, suf_hi]; even requests verify 4 tokens, odd ones decode 1.

    ``step`` in 0..3 turns every 4-token verify into the single-token call at
    position n - 4 + step (the query-length-1 stepping variant)."""
    P = shape.page_size
    assert prefix % P == 0
    sufs = _uniform_int(rng_for(cfg, 0), suf_lo, suf_hi, num_req)
    base = make_prompt(shape, prefix, cfg, 99_999, q_window=0)
    prompts, reqs = [], []
    for i in range(num_req):
        n = prefix + int(sufs[i])
        prompts.append(make_prompt(shape, n, cfg, i, q_window=4, prefix=base, prefix_len=prefix))
        s = 4 if i % 2 == 0 else 1
        if step is not None and s == 4:
            reqs.append(Req(i, n - 3 + step, 1))
        else:
            reqs.append(Req(i, n, s))
    return place(shape, prompts, reqs, rng_for(cfg, perm_stream),
                 shared_prefix_pages=(prefix // P) if shared else 0)


def chunked(call_prompts: List[Prompt], shape: Shape, pid_lens: Sequence[Tuple[int, int, int]],
            rng: np.random.Generator) -> Call:
    """A call of (prompt, n, s) triples over existing prompts."""
    reqs = [Req(p, n, s) for p, n, s in pid_lens]
    return place(shape, call_prompts, reqs, rng)
