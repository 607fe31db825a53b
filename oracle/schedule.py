"""The layer-wise decode schedule, layer by layer (test infrastructure only).

TEST INFRASTRUCTURE ONLY: only tests may use this module.

Q-First, arXiv:2608.15473, Appendix D (the wiring as a schedule, worked).  Requests arrive with
an attention (sweep) time `a` that is the same at every layer; each layer's feed-forward is a pool
that serves one departure at a time, a departure takes `ffn_time` and carries every request
waiting at that moment, and the pool leaves only with at least `min_batch` waiting.
Communication is free.

Q-First wiring (Appendix D, the recurrence for the ready time e of each layer):
    e_1 = arrival + a,   e_l = max(e_{l-1} + a, ffn_{l-1}),   finish = ffn_L,
where ffn_l is the time the request's feed-forward of layer l returns.  At e_l the request
joins pool l (its residual exists) and the sweep of layer l+1 starts (its query exists).
Composed wiring (same appendix): the feed-forward of layer l reads layer l's attention output,
so the request joins pool l when sweep l ends, and sweep l+1 starts when that feed-forward
returns.

Under either wiring the times at which requests join pool l depend only on what happened at
layer l-1, so the schedule is computed one layer at a time: first every request's join time for
layer l, then the departures of pool l from those join times alone.

The pool (one server, batch service): with the server free from F and the oldest request that has
not left yet joining at j_k, the next departure is at the first instant t >= F at which either
min_batch requests have joined and not left, or the oldest has waited max_wait (t >= j_k +
max_wait; Appendix D's hazard paragraph: the rule needs a maximum wait, or the last request can be
stranded).  Every request that has joined by t (join time <= t) rides; the server is busy until
t + ffn_time.  A request that never departs is stranded (finish None), and so are its later
layers.
"""

from __future__ import annotations

import math


def pool_departures(joins, min_batch, ffn_time, max_wait):
    """One feed-forward pool.  `joins`: list of (join time, request).  Returns a list of
    (departure time, members) in time order; requests that never leave are in no departure."""
    order = sorted(joins, key=lambda jr: jr[0])
    times = [t for t, _ in order]
    n = len(order)
    out = []
    k = 0                       # first request that has not left
    free = -math.inf            # the server is free from this time on
    while k < n:
        # earliest t >= free with min_batch requests joined and not yet left
        t_batch = max(free, times[k + min_batch - 1]) if k + min_batch - 1 < n else math.inf
        # earliest t >= free at which the oldest has waited max_wait
        t_wait = max(free, times[k] + max_wait)
        t = min(t_batch, t_wait)
        if t == math.inf:
            break               # the rest are stranded
        end = k
        while end < n and times[end] <= t:
            end += 1
        out.append((t, tuple(sorted(r for _, r in order[k:end]))))
        k = end
        free = t + ffn_time
    return out


def simulate(arrival, attn_time, n_layers, wiring="qfirst", ffn_time=1.0, min_batch=2,
             max_wait=math.inf):
    """Returns dict(finish, sweep, depart, returned, batches): finish[r] (None if stranded);
    sweep[r][l] = (start, end) or None; depart / returned [r][l] or None; batches = list of
    (layer, time, members) in layer order, then time order."""
    R, L = len(arrival), n_layers
    sweep = [[None] * L for _ in range(R)]
    depart = [[None] * L for _ in range(R)]
    ret = [[None] * L for _ in range(R)]
    finish = [None] * R
    batches = []

    start = list(arrival)        # start of this layer's sweep (None: never)
    for l in range(L):
        joins = []
        for r in range(R):
            if start[r] is None:
                continue
            s = start[r]
            end = s + attn_time[r]
            sweep[r][l] = (s, end)
            if wiring == "qfirst":
                # e_l: the sweep is done and, past layer 1, the previous feed-forward has returned
                if l == 0:
                    joins.append((end, r))
                elif ret[r][l - 1] is not None:
                    joins.append((max(end, ret[r][l - 1]), r))
            else:
                joins.append((end, r))
        for t, members in pool_departures(joins, min_batch, ffn_time, max_wait):
            batches.append((l, t, members))
            for r in members:
                depart[r][l] = t
                ret[r][l] = t + ffn_time
        nxt = [None] * R
        for t_join, r in joins:
            if wiring == "qfirst":
                nxt[r] = t_join                  # the sweep of layer l+1 starts at e_l
            elif ret[r][l] is not None:
                nxt[r] = ret[r][l]               # composed: after this layer's feed-forward
        start = nxt
    for r in range(R):
        if ret[r][L - 1] is not None:
            finish[r] = ret[r][L - 1]
    return dict(finish=finish, sweep=sweep, depart=depart, returned=ret, batches=batches)
