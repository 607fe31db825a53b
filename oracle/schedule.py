"""Plain discrete-event simulation of the layer-wise decode schedule (test infrastructure only).

TEST INFRASTRUCTURE ONLY: only tests may use this module.

Q-First, arXiv:2608.15473, Appendix D (the wiring as a schedule, worked): requests with an
arrival time and an attention (sweep) time per layer; the feed-forward of each layer is a pool
that serves one departure at a time, each departure taking `ffn_time`, and departs only with at
least `min_batch` requests waiting (all waiting requests ride).  Communication is free.

  Q-First wiring: e_1 = arrival + a;  e_l = max(e_{l-1} + a, ffn_{l-1});  finish = ffn_L.
      At e_l the request joins feed-forward pool l and, if l < L, its sweep of layer l+1 starts.
  Composed wiring: the feed-forward of layer l reads layer l's attention output, so it joins pool
      l when sweep l ends, and sweep l+1 starts when that feed-forward returns.

A request whose last feed-forward never departs is stranded (finish = None); Appendix D notes an
implementation needs a maximum wait, modelled by ``max_wait``: a pool whose oldest waiting
request has waited that long departs with whatever is waiting.

Simultaneous events: at each time every completion is applied (and anything it makes ready at
that same time) before any pool decides whether to depart.
"""

from __future__ import annotations

import math


def simulate(arrival, attn_time, n_layers, wiring="qfirst", ffn_time=1.0, min_batch=2,
             max_wait=math.inf):
    R = len(arrival)
    L = n_layers
    sweep = [[None] * L for _ in range(R)]
    depart = [[None] * L for _ in range(R)]
    ret = [[None] * L for _ in range(R)]
    finish = [None] * R
    swept = [[False] * L for _ in range(R)]
    joined = [[False] * L for _ in range(R)]
    waiting = [[] for _ in range(L)]          # (enqueue time, request), FIFO
    free_at = [-math.inf] * L
    events = {}                               # time -> list of (kind, data)
    batches = []                              # (layer, time, members)

    def at(t, kind, data):
        events.setdefault(t, []).append((kind, data))

    def start_sweep(r, l, t):
        sweep[r][l] = (t, t + attn_time[r])
        at(t + attn_time[r], "swept", (r, l))

    def join(r, l, t):
        if not joined[r][l]:
            joined[r][l] = True
            waiting[l].append((t, r))

    def ready(r, l, t):                       # Q-First: layer l's output exists at t?
        if swept[r][l] and (l == 0 or ret[r][l - 1] is not None) and not joined[r][l]:
            join(r, l, t)
            if l + 1 < L:
                start_sweep(r, l + 1, t)

    for r in range(R):
        start_sweep(r, 0, arrival[r])

    while events:
        t = min(events)
        while t in events:                    # completions at t, to a fixed point
            for kind, data in events.pop(t):
                if kind == "swept":
                    r, l = data
                    swept[r][l] = True
                    if wiring == "qfirst":
                        ready(r, l, t)
                    else:
                        join(r, l, t)
                elif kind == "returned":
                    l, members = data
                    for r in members:
                        ret[r][l] = t
                        if l + 1 == L:
                            finish[r] = t
                        elif wiring == "qfirst":
                            ready(r, l + 1, t)
                        else:
                            start_sweep(r, l + 1, t)
        for l in range(L):                    # departures at t
            if not waiting[l] or free_at[l] > t:
                continue
            if len(waiting[l]) >= min_batch or t - waiting[l][0][0] >= max_wait:
                members = tuple(r for _, r in waiting[l])
                waiting[l] = []
                free_at[l] = t + ffn_time
                for r in members:
                    depart[r][l] = t
                batches.append((l, t, members))
                at(t + ffn_time, "returned", (l, members))
        for l in range(L):                    # wake-ups: a busy pool, or a pending time-out
            if waiting[l]:
                if free_at[l] > t:
                    events.setdefault(free_at[l], [])
                elif math.isfinite(max_wait):
                    events.setdefault(max(waiting[l][0][0] + max_wait, t), [])
    return dict(finish=finish, sweep=sweep, depart=depart, returned=ret, batches=batches)
