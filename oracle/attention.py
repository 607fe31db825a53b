"""Plain fp64 definitions of the decode-attention sweep, its shards and their merge.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``): only tests, ``smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may use this module.

Paper: Q-First, arXiv:2608.15473.
  §2 (decode protocol): the device attends over the j-1 cached positions with the query alone and
      returns o_<j and lse_<j; scores are s = q.k / sqrt(d).
  §5 (the cache may be split anywhere): Z(S) = sum exp(s_i), W(S) = sum exp(s_i) v_i,
      O(S) = W/Z; a shard returns (O, log Z); the merge is
      O(A u B) = lerp(O(B), O(A), sigmoid(log Z(A) - log Z(B))),
      log Z(A u B) = logaddexp(log Z(A), log Z(B));
      an empty shard has log Z = -inf and a vector that is never read.
  §2 (overflow paragraph): sigmoid written as 1 / (1 + exp(-x)).
  Appendix E (numerical caveats): logaddexp must be the stabilised form.

All arithmetic is float64 on exact copies of the bf16 inputs (bf16 -> float64 is exact).  Sums use
numpy's own reductions; nothing is blocked, fused or reordered beyond what the definitions state.

Parity status: every function here is pinned by ``tests/test_oracle_pins.py`` (closed forms,
invariants, brute force, library special cases, the paper's split experiment).  The paper's
worked example of a 400-position shard whose scores spread over 30 nats (Appendix A) is NOT reproduced by any
reading of it and is therefore not used as a pin (parity unpinned for that example only).
"""

from __future__ import annotations

import numpy as np

NEG_INF = -np.inf


# --------------------------------------------------------------------------------------------
# work map
# --------------------------------------------------------------------------------------------
def shard_ranges(n: int, n_shards: int, page_size: int) -> list[tuple[int, int]]:
    """Position ranges [lo, hi) of the ``n_shards`` shards of a request with ``n`` cached positions.

    By §5 any partition of the positions merges to the same result, so the split is free.  The
    library fixes one, restated here from its description: the request's positions fill
    ceil(n / P) pages; every shard takes the next ceil(pages / S) pages (the last shards may get
    fewer pages, or none); the positions of the last page are clipped to n.
    """
    if n_shards < 1:
        raise ValueError("n_shards must be >= 1")
    pages = -(-n // page_size)
    per_shard = -(-pages // n_shards) if pages else 0
    ranges = []
    for s in range(n_shards):
        first = min(s * per_shard, pages)
        last = min((s + 1) * per_shard, pages)
        ranges.append((min(first * page_size, n), min(last * page_size, n)))
    return ranges


def gather_rows(cache, table_row, head: int, n: int, page_size: int) -> np.ndarray:
    """Rows 0..n-1 of one KV head of one request, as float64 [n, D].

    Logical position i lives in physical page ``table_row[i // P]`` at slot ``i % P`` (the paged
    layout the paper takes from PagedAttention, §4).  ``cache`` is [num_pages, Hkv, P, D].
    """
    idx = np.arange(n)
    pages = np.asarray(table_row)[idx // page_size]
    return np.asarray(cache[pages, head, idx % page_size, :], dtype=np.float64)


# --------------------------------------------------------------------------------------------
# the sweep over one set of positions
# --------------------------------------------------------------------------------------------
def attend(q, K, V, scale: float) -> tuple[np.ndarray, float]:
    """(O, log Z) of one query over the positions whose keys/values are the rows of K, V.

    §5 definitions with the §2 score s_i = scale * q . k_i:  Z = sum_i exp(s_i),
    O = sum_i exp(s_i) v_i / Z, returned as (O, ln Z).  An empty set gives (0, -inf) (§5: the
    empty shard).  float64 overflows exp() only above s = 709, so the unshifted sum is used
    unless the largest score passes 700; then exp(max s) is factored out of Z and W alike, which
    is the same quantity.  NaN in any input reaches O and ln Z.
    """
    q = np.asarray(q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    if K.shape[0] == 0:
        return np.zeros(V.shape[1]), NEG_INF
    s = float(scale) * (K @ q)
    top = np.max(s)
    if top > 700.0:
        return attend_shifted(q, K, V, scale)
    with np.errstate(invalid="ignore", over="ignore"):
        e = np.exp(s)
        Z = np.sum(e)
        O = (e @ V) / Z
        return O, float(np.log(Z))


def attend_shifted(q, K, V, scale: float) -> tuple[np.ndarray, float]:
    """The same (O, ln Z) as :func:`attend`, always with exp(max s) factored out of Z and W."""
    q = np.asarray(q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    if K.shape[0] == 0:
        return np.zeros(V.shape[1]), NEG_INF
    s = float(scale) * (K @ q)
    with np.errstate(invalid="ignore", over="ignore"):
        m = np.max(s)
        e = np.exp(s - m)
        Zs = np.sum(e)
        O = (e @ V) / Zs
        return O, float(m + np.log(Zs))


# --------------------------------------------------------------------------------------------
# the whole decode step: per-shard partials and the unsplit result
# --------------------------------------------------------------------------------------------
def _table_row(block_table, b: int, max_pages: int):
    if block_table is None:  # identity: request b owns pages b*max_pages .. b*max_pages+max_pages-1
        return np.arange(b * max_pages, (b + 1) * max_pages)
    return np.asarray(block_table)[b]


def _selected(pairs, B, Hq):
    if pairs is None:
        return [(b, h) for b in range(B) for h in range(Hq)]
    return list(pairs)


def decode_split(q, k_cache, v_cache, block_table, ctx_lens, n_shards, scale: float,
                 max_shards: int, page_size: int = 16, max_pages: int | None = None,
                 pairs=None):
    """Per-shard partials (O_s, ln Z_s) for every request and query head.

    Returns ``part_out`` float64 [B, max_shards, Hq, D] and ``part_lse`` float64
    [B, max_shards, Hq].  Shard s of request b covers ``shard_ranges(n_b, S_b, P)[s]``; query head
    h reads KV head h // (Hq / Hkv) (grouped-query attention, heads of a group contiguous).  Empty
    shards and slots s >= S_b hold (0, -inf).  ``pairs`` restricts the work to a list of (b, h);
    the other entries are NaN.
    """
    q = np.asarray(q)
    B, Hq, D = q.shape
    Hkv = k_cache.shape[1]
    G = Hq // Hkv
    if max_pages is None:
        max_pages = (np.asarray(block_table).shape[1] if block_table is not None
                     else k_cache.shape[0] // B)
    part_out = np.full((B, max_shards, Hq, D), np.nan)
    part_lse = np.full((B, max_shards, Hq), np.nan)
    todo = _selected(pairs, B, Hq)
    cached = {}
    for b, h in todo:
        n = int(ctx_lens[b])
        S = int(n_shards[b])
        g = h // G
        if (b, g) not in cached:
            row = _table_row(block_table, b, max_pages)
            cached.clear()
            cached[(b, g)] = (gather_rows(k_cache, row, g, n, page_size),
                              gather_rows(v_cache, row, g, n, page_size))
        K, V = cached[(b, g)]
        part_out[b, :, h, :] = 0.0
        part_lse[b, :, h] = NEG_INF
        for s, (lo, hi) in enumerate(shard_ranges(n, S, page_size)):
            O, lse = attend(q[b, h], K[lo:hi], V[lo:hi], scale)
            part_out[b, s, h] = O
            part_lse[b, s, h] = lse
    return part_out, part_lse


def decode_unsplit(q, k_cache, v_cache, block_table, ctx_lens, scale: float,
                   page_size: int = 16, max_pages: int | None = None, pairs=None):
    """(out, lse) of one sweep over each request's whole cache: float64 [B, Hq, D] and [B, Hq].

    This is the result every split must reproduce (§5).  n_b = 0 gives (0, -inf).  ``pairs``
    restricts the work as in :func:`decode_split`.
    """
    q = np.asarray(q)
    B, Hq, D = q.shape
    Hkv = k_cache.shape[1]
    G = Hq // Hkv
    if max_pages is None:
        max_pages = (np.asarray(block_table).shape[1] if block_table is not None
                     else k_cache.shape[0] // B)
    out = np.full((B, Hq, D), np.nan)
    lse = np.full((B, Hq), np.nan)
    cached = {}
    for b, h in _selected(pairs, B, Hq):
        n = int(ctx_lens[b])
        g = h // G
        if (b, g) not in cached:
            row = _table_row(block_table, b, max_pages)
            cached.clear()
            cached[(b, g)] = (gather_rows(k_cache, row, g, n, page_size),
                              gather_rows(v_cache, row, g, n, page_size))
        K, V = cached[(b, g)]
        out[b, h], lse[b, h] = attend(q[b, h], K, V, scale)
    return out, lse


# --------------------------------------------------------------------------------------------
# the merge
# --------------------------------------------------------------------------------------------
def _sigmoid(x: float) -> float:
    """sigma(x) = 1 / (1 + exp(-x)), the form §2 recommends; exp(-x) may overflow to inf -> 0."""
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-x))


def merge_pair(O_a, lse_a, O_b, lse_b):
    """(O, ln Z) of A u B from the two shards' pairs, §5.

    O(A u B) = lerp(O(B), O(A), sigma(ln Z_A - ln Z_B)) with lerp(x, y, t) = (1 - t) x + t y, and
    ln Z(A u B) = logaddexp(ln Z_A, ln Z_B).  An empty side (ln Z = -inf) is the identity and its
    vector is not read (§5, last paragraph), so garbage there cannot leak into the result.
    """
    if lse_a == NEG_INF:
        return np.array(O_b, dtype=np.float64), lse_b
    if lse_b == NEG_INF:
        return np.array(O_a, dtype=np.float64), lse_a
    t = _sigmoid(lse_a - lse_b)
    O = (1.0 - t) * np.asarray(O_b, dtype=np.float64) + t * np.asarray(O_a, dtype=np.float64)
    return O, float(np.logaddexp(lse_a, lse_b))


def fold_combine(part_out, part_lse, order=None, rng=None):
    """Merge every shard slot of every (request, head) by folding :func:`merge_pair`.

    part_out [B, S, Hq, D], part_lse [B, S, Hq] -> (out [B, Hq, D], lse [B, Hq]).  The slots are
    folded in ``order`` (a permutation of range(S)), or in a random order drawn from ``rng`` per
    (request, head), or in index order; §5 says the order cannot matter.  All slots empty gives
    (0, -inf).
    """
    part_out = np.asarray(part_out, dtype=np.float64)
    part_lse = np.asarray(part_lse, dtype=np.float64)
    B, S, Hq, D = part_out.shape
    out = np.zeros((B, Hq, D))
    lse = np.full((B, Hq), NEG_INF)
    for b in range(B):
        for h in range(Hq):
            if order is not None:
                seq = list(order)
            elif rng is not None:
                seq = list(rng.permutation(S))
            else:
                seq = list(range(S))
            acc_O, acc_lse = np.zeros(D), NEG_INF
            for s in seq:
                acc_O, acc_lse = merge_pair(part_out[b, s, h], part_lse[b, s, h], acc_O, acc_lse)
            out[b, h], lse[b, h] = acc_O, acc_lse
    return out, lse


def combine_max_shifted(part_out, part_lse):
    """The N-way form of the same merge: with m = max_s ln Z_s over non-empty slots,
    out = sum_s exp(ln Z_s - m) O_s / sum_s exp(ln Z_s - m) and ln Z = m + ln(sum_s exp(ln Z_s - m)).

    Empty slots are selected out, never multiplied (§5).  This is the algebra of the pairwise fold
    written for S slots at once (§5 cites the online-softmax recurrence); it must equal
    :func:`fold_combine`.
    """
    part_out = np.asarray(part_out, dtype=np.float64)
    part_lse = np.asarray(part_lse, dtype=np.float64)
    B, S, Hq, D = part_out.shape
    out = np.zeros((B, Hq, D))
    lse = np.full((B, Hq), NEG_INF)
    for b in range(B):
        for h in range(Hq):
            l = part_lse[b, :, h]
            live = l != NEG_INF
            if not live.any():
                continue
            m = np.max(l[live])
            w = np.exp(l[live] - m)
            out[b, h] = (w @ part_out[b, live, h, :]) / np.sum(w)
            lse[b, h] = m + np.log(np.sum(w))
    return out, lse


# --------------------------------------------------------------------------------------------
# the current token (§2 protocol table and combine, Appendix A fold) and the cache append
# --------------------------------------------------------------------------------------------
def fold_current(O_prev, lse_prev, q, k_cur, v_cur, scale: float):
    """Fold the current token into the cache's (o_<j, lse_<j) for every request and query head.

    §2 and Appendix A: s_jj = scale * q_j . k_j, out = lerp(v_j, o_<j, sigma(lse_<j - s_jj)),
    lse = logaddexp(lse_<j, s_jj).  The cached history acts as one pseudo-token of score lse_<j
    and value o_<j, so this is a two-way softmax.  An empty cache (lse_<j = -inf) gives
    (v_j, s_jj) and its o_<j is not read.

    O_prev [B, Hq, D], lse_prev [B, Hq], q [B, Hq, D], k_cur / v_cur [B, Hkv, D] (query head h
    uses KV head h // (Hq / Hkv)).  Returns float64 (out [B, Hq, D], lse [B, Hq]).
    """
    O_prev = np.asarray(O_prev, dtype=np.float64)
    lse_prev = np.asarray(lse_prev, dtype=np.float64)
    q = np.asarray(q, dtype=np.float64)
    k_cur = np.asarray(k_cur, dtype=np.float64)
    v_cur = np.asarray(v_cur, dtype=np.float64)
    B, Hq, D = q.shape
    G = Hq // k_cur.shape[1]
    out = np.zeros((B, Hq, D))
    lse = np.zeros((B, Hq))
    for b in range(B):
        for h in range(Hq):
            g = h // G
            s_jj = float(scale) * float(q[b, h] @ k_cur[b, g])
            if lse_prev[b, h] == NEG_INF:
                out[b, h], lse[b, h] = v_cur[b, g], s_jj
                continue
            t = _sigmoid(lse_prev[b, h] - s_jj)
            out[b, h] = (1.0 - t) * v_cur[b, g] + t * O_prev[b, h]
            lse[b, h] = float(np.logaddexp(lse_prev[b, h], s_jj))
    return out, lse


def append_kv(k_cache, v_cache, block_table, ctx_lens, k_new, v_new, page_size: int = 16,
              max_pages: int | None = None):
    """The cache write of §2 (k_j and v_j appended, a write nothing waits on): returns copies of
    the caches with request b's new key/value stored at its position n_b = ctx_lens[b], i.e.
    physical page block_table[b, n_b // P], slot n_b % P, for every KV head."""
    k = np.array(k_cache, copy=True)
    v = np.array(v_cache, copy=True)
    B = len(ctx_lens)
    if max_pages is None:
        max_pages = (np.asarray(block_table).shape[1] if block_table is not None
                     else k.shape[0] // B)
    for b in range(B):
        n = int(ctx_lens[b])
        page = int(_table_row(block_table, b, max_pages)[n // page_size])
        if not 0 <= page < k.shape[0]:
            raise ValueError(f"request {b}: no page allocated for position {n}")
        k[page, :, n % page_size, :] = k_new[b]
        v[page, :, n % page_size, :] = v_new[b]
    return k, v
