"""Batch metadata for the five synthetic mixes and the scheduler replay.

A *row* is what one scheduling iteration hands to the attention step for one
request: ``(req_id, chunk_start, chunk_len, ctx_len)``.  ``chunk_start`` is the
number of tokens of that request already in the KV cache, ``chunk_len`` the
number of new tokens processed in this iteration (1 for a decode row), and
``ctx_len = chunk_start + chunk_len`` the number of keys the row's last query
sees.  Decode rows are admitted before prefill chunks and prefill chunks get
the residual token budget (Sec. 3.1.1 and 3.1.3 of the paper); one chunk per
request per round (Sec. 3.1.3, Algorithm 1 returns one chunk size).

Lognormal draws use sigma = 1 (natural log); the paper does not state the
spread of these synthetic mixes.
"""

from __future__ import annotations

import math
from collections import deque
from dataclasses import dataclass, field

import numpy as np

CONFIG_NAMES = {
    1: "tiny-gqa2-d64-b16",
    2: "llama3-8b-budget512",
    3: "llama3-8b-prefill-heavy-budget2048",
    4: "llama3-8b-decode-dominated",
    5: "llama-70b-replay-20it-budget4096",
}


@dataclass
class Batch:
    """One scheduling iteration's batch plus the pool it reads.

    rows          int32 [n_rows, 4]  (req_id, chunk_start, chunk_len, ctx_len), q-row order
    block_tables  int32 [R, max_blocks_per_req]; entries past a request's
                  allocation point at ``poison_block`` (never read by a correct kernel)
    num_blocks    physical blocks in each of the K and V pools
    """

    name: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    block_size: int
    rows: np.ndarray
    block_tables: np.ndarray
    num_blocks: int
    poison_block: int
    sm_scale: float = 0.0
    referenced: np.ndarray = field(default=None, repr=False)  # bool [num_blocks]

    def __post_init__(self):
        if not self.sm_scale:
            self.sm_scale = float(np.float32(1.0 / math.sqrt(self.head_dim)))
        self.rows = np.ascontiguousarray(self.rows, dtype=np.int32).reshape(-1, 4)
        self.block_tables = np.ascontiguousarray(self.block_tables, dtype=np.int32)

    @property
    def n_rows(self) -> int:
        return int(self.rows.shape[0])

    @property
    def num_tokens(self) -> int:
        return int(self.rows[:, 2].sum()) if self.n_rows else 0

    @property
    def max_blocks_per_req(self) -> int:
        return int(self.block_tables.shape[1])

    @property
    def num_reqs_in_table(self) -> int:
        return int(self.block_tables.shape[0])

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    def tok_offsets(self) -> np.ndarray:
        off = np.zeros(self.n_rows + 1, dtype=np.int64)
        np.cumsum(self.rows[:, 2], out=off[1:])
        return off

    def describe(self) -> dict:
        r = self.rows
        dec = r[r[:, 2] == 1]
        pf = r[r[:, 2] > 1]
        return {
            "rows": self.n_rows,
            "tokens": self.num_tokens,
            "decode_rows": int(dec.shape[0]),
            "prefill_rows": int(pf.shape[0]),
            "sum_decode_ctx": int(dec[:, 3].sum()) if dec.size else 0,
            "max_ctx": int(r[:, 3].max()) if r.size else 0,
            "heads": (self.num_q_heads, self.num_kv_heads),
            "head_dim": self.head_dim,
            "block_size": self.block_size,
            "num_blocks": self.num_blocks,
        }


def _lognormal_int(rng, median, n, lo, hi):
    x = rng.lognormal(mean=math.log(median), sigma=1.0, size=n)
    return np.clip(np.round(x), lo, hi).astype(np.int64)


def make_batch(name, hq, hkv, d, bsz, starts_lens, rng, n_spare=2, shuffle_req_ids=True,
               mbr=None, pool=None) -> Batch:
    """Builds a batch whose block tables deal a random permutation of the pool.

    starts_lens: list of (chunk_start, chunk_len) in row order.
    The pool holds exactly the blocks the rows need plus ``n_spare`` spare
    blocks, unless ``pool`` fixes its size (then the rows' blocks are a random
    draw without replacement from it); spare block ``poison_block`` backs
    every unused table entry.
    """
    starts_lens = [(int(s), int(c)) for s, c in starts_lens]
    n = len(starts_lens)
    nblk = [-(-(s + c) // bsz) for s, c in starts_lens]
    used = int(sum(nblk))
    if pool is None:
        pool = used + max(1, n_spare)
        perm = rng.permutation(pool).astype(np.int64)
    else:
        if pool < used + 1:
            raise ValueError(f"pool of {pool} blocks cannot hold {used} blocks and a spare")
        perm = rng.permutation(pool)[: used + 1].astype(np.int64)
    poison = int(perm[used])  # first spare block in permutation order
    mbr = int(mbr if mbr is not None else max([1] + nblk))
    req_ids = rng.permutation(n) if shuffle_req_ids else np.arange(n)
    bt = np.full((max(n, 1), mbr), poison, dtype=np.int32)
    rows = np.zeros((n, 4), dtype=np.int32)
    k = 0
    for i, (s, c) in enumerate(starts_lens):
        rid = int(req_ids[i])
        bt[rid, : nblk[i]] = perm[k: k + nblk[i]]
        k += nblk[i]
        rows[i] = (rid, s, c, s + c)
    referenced = np.zeros(pool, dtype=bool)
    referenced[perm[:used]] = True
    return Batch(name, hq, hkv, d, bsz, rows, bt, pool, poison, referenced=referenced)


def subset(batch: Batch, keep, suffix: str) -> Batch:
    """The rows of ``batch`` selected by the boolean mask ``keep``, over the same
    pool and block tables (their tokens are renumbered in row order)."""
    keep = np.asarray(keep, dtype=bool)
    return Batch(f"{batch.name}-{suffix}", batch.num_q_heads, batch.num_kv_heads,
                 batch.head_dim, batch.block_size, batch.rows[keep].copy(),
                 batch.block_tables, batch.num_blocks, batch.poison_block, batch.sm_scale,
                 referenced=batch.referenced)


def tiny_batch(seed: int = 1) -> Batch:
    """4 q heads, 2 kv heads, head_dim 64, block 16: a 64-token chunk at ctx 0,
    a 48-token chunk after 128 cached tokens, decode rows with ctx 200 and 37."""
    rng = np.random.default_rng(seed)
    return make_batch(CONFIG_NAMES[1], 4, 2, 64, 16,
                      [(0, 64), (128, 48), (199, 1), (36, 1)], rng)


def _config2(rng):
    prior = rng.integers(0, 4097, size=2)
    dctx = _lognormal_int(rng, 1024, 128, 16, 8192)
    sl = [(int(c) - 1, 1) for c in dctx] + [(int(p), 192) for p in prior]
    return make_batch(CONFIG_NAMES[2], 32, 8, 128, 16, sl, rng)


def _config3(rng):
    dctx = _lognormal_int(rng, 2048, 128, 16, 32768)
    sl = [(int(c) - 1, 1) for c in dctx] + [(p, 480) for p in (0, 8192, 16384, 31744)]
    return make_batch(CONFIG_NAMES[3], 32, 8, 128, 16, sl, rng)


def _config4(rng):
    is_long = rng.random(256) < 0.3
    short = _lognormal_int(rng, 512, 256, 16, 8192)
    long_ = rng.integers(8192, 32769, size=256)
    dctx = np.where(is_long, long_, short)
    sl = [(int(c) - 1, 1) for c in dctx] + [(0, 256)]
    return make_batch(CONFIG_NAMES[4], 32, 8, 128, 16, sl, rng)


def make_config(n: int) -> Batch:
    """Metadata of synthetic mix ``n`` (1..4) from ``numpy.random.default_rng(n)``.
    Mix 5 is a multi-iteration replay: use :func:`replay_schedule`."""
    if n == 1:
        return tiny_batch(1)
    rng = np.random.default_rng(n)
    if n == 2:
        return _config2(rng)
    if n == 3:
        return _config3(rng)
    if n == 4:
        return _config4(rng)
    raise ValueError("mix 5 is a replay; call replay_schedule()")


@dataclass
class ReplayRequest:
    prompt: int
    output: int
    arrival: int
    done: int = 0          # prompt tokens already prefilled
    generated: int = 0     # output tokens produced (first one comes from the prefill)
    finished: bool = False
    blocks: list = field(default_factory=list)

    @property
    def remaining(self) -> int:
        return self.prompt - self.done

    @property
    def in_decode(self) -> bool:
        return (not self.finished) and self.done == self.prompt and self.generated >= 1


def replay_schedule(n_req=64, iters=20, budget=4096, c_max=4, s_max=64, l_min=32,
                    hq=64, hkv=8, d=128, bsz=32, alpha=1.0, beta=-1.0 / 256.0,
                    seed=5, pool_seed=105):
    """Open-loop replay of an Aging + active-prefill-control schedule.

    Per iteration: every request in decode emits one row first (decode-first
    admission, Sec. 3.1.3); arrived requests still in prefill are ranked by the
    time-invariant aging key K_i = -alpha*a_i + beta*r_i (Eq. 4, max first, ties
    to the lower id); the activity cap C_t (Eq. 12) and the minimum-progress /
    warm-start rule (Eq. 13-14) gate each candidate; the proposed chunk is the
    static fill h_i = min(r_i, B_max - U_t) (Eq. 6-7); the remaining work is
    updated by Eq. 2.  Blocks come from a seeded shuffled free list when a
    request's context crosses a block boundary and return to it on finish.

    Returns ``(batches, info)``: one :class:`Batch` per iteration (all sharing
    one pool) and a dict with the request draws.
    """
    rng = np.random.default_rng(seed)
    prompts = _lognormal_int(rng, 1500, n_req, 16, 32768)
    outputs = _lognormal_int(rng, 200, n_req, 1, 4096)
    reqs = [ReplayRequest(int(p), int(o), i // 4) for i, (p, o) in enumerate(zip(prompts, outputs))]
    need = [-(-(r.prompt + r.output) // bsz) for r in reqs]
    pool_used = int(sum(need))
    poison = pool_used  # one extra block, never handed out, backs unused table entries
    pool = pool_used + 1
    free = deque(int(b) for b in np.random.default_rng(pool_seed).permutation(pool_used))
    mbr = int(max(need))
    batches = []
    for it in range(iters):
        rows = []
        used = 0
        decodes = [i for i, r in enumerate(reqs) if r.in_decode]
        for i in decodes:
            r = reqs[i]
            pos = r.prompt + r.generated - 1
            rows.append((i, pos, 1))
            used += 1
        cands = [i for i, r in enumerate(reqs)
                 if (not r.finished) and r.arrival <= it and r.remaining > 0]
        cands.sort(key=lambda i: (-(-alpha * reqs[i].arrival + beta * reqs[i].remaining), i))
        n_pf = 0
        for i in cands:
            r = reqs[i]
            cap = min(c_max, s_max - len(decodes), (budget - used) // l_min)
            h = min(r.remaining, budget - used)
            if h <= 0:
                continue
            c_star = h
            m = min(r.remaining, l_min)
            if n_pf < cap and c_star >= m:
                c = c_star
            elif c_star < m and n_pf == 0:
                c = min(h, m)
            else:
                c = 0
            if c <= 0:
                continue
            rows.append((i, r.done, c))
            used += c
            n_pf += 1
        # blocks for every row's new positions
        for i, s, c in rows:
            r = reqs[i]
            while len(r.blocks) * bsz < s + c:
                r.blocks.append(free.popleft())
        bt = np.full((n_req, mbr), poison, dtype=np.int32)
        for i, r in enumerate(reqs):
            if r.blocks:
                bt[i, : len(r.blocks)] = r.blocks
        arr = np.array([(i, s, c, s + c) for i, s, c in rows], dtype=np.int32).reshape(-1, 4)
        referenced = np.zeros(pool, dtype=bool)
        for r in reqs:
            referenced[r.blocks] = True
        batches.append(Batch(f"{CONFIG_NAMES[5]}:it{it}", hq, hkv, d, bsz, arr, bt, pool,
                             poison, referenced=referenced))
        # state update (Eq. 2 for prefill chunks; one token per decode row)
        for i, s, c in rows:
            r = reqs[i]
            if c == 1 and r.in_decode and s == r.prompt + r.generated - 1:
                r.generated += 1
            else:
                r.done += c
                if r.done == r.prompt:
                    r.generated = 1
            if r.done == r.prompt and r.generated >= r.output:
                r.finished = True
                free.extend(r.blocks)
                r.blocks = []
    info = {"prompts": prompts, "outputs": outputs, "pool": pool, "poison_block": poison}
    return batches, info
