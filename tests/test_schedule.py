"""The layer-wise decode schedule (Appendix D).

The oracle computes the schedule one layer at a time from the appendix's recurrence; the native
simulator in libqfattn is a discrete-event loop.  The oracle is pinned to the worked example the
paper prints and to closed forms; the two are then compared on random instances, integer and
fractional (every native call runs in a child process under a time limit, so a simulator that does
not terminate fails instead of hanging the suite)."""

import json
import math
import os
import random

import pytest

from oracle import schedule as oracle_schedule

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_schedule.json")


def _instance():
    g = json.load(open(GOLDEN))
    reqs = g["instance"]["requests"]
    return g, [r["arrival"] for r in reqs], [r["attn"] for r in reqs], [r["name"] for r in reqs]


def _last_finish(res):
    return max(f for f in res["finish"] if f is not None)


def test_oracle_reproduces_the_worked_example():
    g, arr, att, names = _instance()
    inst = g["instance"]
    res = {w: oracle_schedule.simulate(arr, att, inst["layers"], w, inst["ffn_time"],
                                       inst["min_batch"]) for w in ("qfirst", "composed")}
    for w in ("qfirst", "composed"):
        assert _last_finish(res[w]) == g["last_finish"][w]
        assert [names[i] for i, f in enumerate(res[w]["finish"]) if f is None] == \
            g["stranded"]["requests"]
    r1 = names.index(g["slowest_sweeps_qfirst"]["request"])
    assert [list(s) for s in res["qfirst"]["sweep"][r1]] == g["slowest_sweeps_qfirst"]["intervals"]
    # the same batches in the same order per layer, only shifted in time
    for l in range(inst["layers"]):
        q = [set(m) for (ll, t, m) in res["qfirst"]["batches"] if ll == l]
        c = [set(m) for (ll, t, m) in res["composed"]["batches"] if ll == l]
        assert q == c


def test_oracle_recurrence_holds():
    """e_l = max(e_{l-1} + a, ffn_{l-1}) under Q-First: sweep l+1 starts when layer l is ready."""
    _, arr, att, _ = _instance()
    res = oracle_schedule.simulate(arr, att, 3, "qfirst")
    for r in range(len(arr)):
        for l in range(2):
            if res["sweep"][r][l + 1] is None:
                continue
            e_l = res["sweep"][r][l + 1][0]
            prev_ret = res["returned"][r][l - 1] if l > 0 else -math.inf
            assert e_l == max(res["sweep"][r][l][1], prev_ret)


def test_max_wait_releases_the_stranded_request():
    _, arr, att, _ = _instance()
    res = oracle_schedule.simulate(arr, att, 3, "qfirst", max_wait=2.0)
    assert all(f is not None for f in res["finish"])
    assert res["finish"][0] == 12 + 2 + 1      # R1 waits 2, then rides alone for 1


@pytest.mark.parametrize("arr,a,ffn,L", [(0.0, 4.0, 1.0, 3), (1.5, 0.7, 2.25, 5), (2.0, 0.0, 0.5, 2),
                                         (0.25, 3.0, 3.0, 4)])
def test_oracle_lone_request_closed_forms(arr, a, ffn, L):
    """One request alone.  With min_batch 1 every pool departs the moment the request joins, so the
    recurrence gives e_l = arr + a + (l-1) max(a, ffn) under Q-First (finish e_L + ffn) and
    arr + L (a + ffn) composed; with min_batch 2 it is stranded at layer 1 unless a maximum wait w
    releases it, each pool then leaving w after the join: e_l = arr + a + (l-1) max(a, w + ffn)."""
    q = oracle_schedule.simulate([arr], [a], L, "qfirst", ffn, 1)
    assert q["finish"][0] == pytest.approx(arr + a + (L - 1) * max(a, ffn) + ffn, abs=1e-12)
    c = oracle_schedule.simulate([arr], [a], L, "composed", ffn, 1)
    assert c["finish"][0] == pytest.approx(arr + L * (a + ffn), abs=1e-12)
    s = oracle_schedule.simulate([arr], [a], L, "qfirst", ffn, 2)
    assert s["finish"] == [None] and s["returned"][0] == [None] * L
    # stranded in pool 1; its query for layer 2 exists at e_1, so sweep 2 still runs, sweep 3 not
    assert s["sweep"][0][0] == (arr, arr + a)
    assert s["sweep"][0][1] == (arr + a, arr + a + a)
    assert all(x is None for x in s["sweep"][0][2:])
    for w in (0.0, 0.1, 1.75):
        r = oracle_schedule.simulate([arr], [a], L, "qfirst", ffn, 2, w)
        assert r["finish"][0] == pytest.approx(arr + a + (L - 1) * max(a, w + ffn) + w + ffn,
                                               abs=1e-12)
        c = oracle_schedule.simulate([arr], [a], L, "composed", ffn, 2, w)
        assert c["finish"][0] == pytest.approx(arr + L * (a + w + ffn), abs=1e-12)


def test_oracle_pool_rule():
    """One pool by hand: joins at 0, 0.5, 3 and 3.2, batches of 2, service 1, no time-out: the
    first two leave at 0.5 (the second join), the next two at 3.2; with max_wait 0.25 the first
    leaves alone at 0.25, the second at 1.25 (server busy until then, it has waited 0.75), the
    third at 3.2 with the fourth; a request that joins exactly at a departure rides it."""
    pd = oracle_schedule.pool_departures
    joins = [(0.0, 0), (0.5, 1), (3.0, 2), (3.2, 3)]
    assert pd(joins, 2, 1.0, math.inf) == [(0.5, (0, 1)), (3.2, (2, 3))]
    assert pd(joins, 2, 1.0, 0.25) == [(0.25, (0,)), (1.25, (1,)), (3.2, (2, 3))]
    assert pd([(0.0, 0), (1.0, 1), (1.0, 2)], 3, 1.0, 1.0) == [(1.0, (0, 1, 2))]
    assert pd([(0.0, 0)], 2, 1.0, math.inf) == []


def test_oracle_fractional_time_out_terminates():
    """0.7 + 0.1 is not exactly 0.8 in binary floating point; the lone request still leaves once it
    has waited max_wait (at 0.7 + 0.1) and finishes one feed-forward later."""
    res = oracle_schedule.simulate([0.0], [0.7], 1, "qfirst", 1.0, 2, 0.1)
    assert res["depart"][0][0] == 0.7 + 0.1
    assert res["finish"][0] == pytest.approx(1.8, abs=1e-12)


# ------------------------------------------------------------------------------------------------
# the native simulator in libqfattn (host code, no GPU needed)
# ------------------------------------------------------------------------------------------------
qf = pytest.importorskip("paper_2608_15473_amd")
needs_lib = pytest.mark.skipif(not os.path.exists(qf.LIB_PATH), reason="libqfattn.so not built")


def _as_lists(native, R, L):
    nan = lambda x: None if math.isnan(x) else float(x)
    return dict(finish=[nan(x) for x in native["finish"]],
                sweep=[[None if math.isnan(native["sweep_start"][r, l]) else
                        (float(native["sweep_start"][r, l]), float(native["sweep_end"][r, l]))
                        for l in range(L)] for r in range(R)],
                depart=[[nan(native["ffn_depart"][r, l]) for l in range(L)] for r in range(R)],
                returned=[[nan(native["ffn_return"][r, l]) for l in range(L)] for r in range(R)])


@needs_lib
def test_native_reproduces_the_worked_example():
    g, arr, att, names = _instance()
    for w in ("qfirst", "composed"):
        res = qf.schedule_simulate(arr, att, 3, w, 1.0, 2)
        fin = res["finish"]
        assert max(f for f in fin if not math.isnan(f)) == g["last_finish"][w]
        assert [names[i] for i, f in enumerate(fin) if math.isnan(f)] == g["stranded"]["requests"]
    res = qf.schedule_simulate(arr, att, 3, "qfirst")
    r1 = names.index("R1")
    got = [[res["sweep_start"][r1, l], res["sweep_end"][r1, l]] for l in range(3)]
    assert got == g["slowest_sweeps_qfirst"]["intervals"]


def _instance_for(seed, fractional):
    rng = random.Random(seed)
    R = rng.randint(1, 30)
    L = rng.randint(1, 5)
    if fractional:
        arr = [round(rng.uniform(0, 10), rng.choice([1, 2, 17])) for _ in range(R)]
        att = [round(rng.uniform(0, 6), rng.choice([1, 2, 17])) for _ in range(R)]
        ffn = round(rng.uniform(0.05, 3.0), rng.choice([1, 2, 17]))
        mw = rng.choice([math.inf, 0.0, round(rng.uniform(0, 3), 1), rng.uniform(0, 3)])
    else:
        arr = [float(rng.randint(0, 10)) for _ in range(R)]
        att = [float(rng.randint(0, 6)) for _ in range(R)]
        ffn = rng.choice([1.0, 2.0, 3.0])
        mw = rng.choice([math.inf, 0.0, 1.0, 3.0])
    ffn = max(ffn, 0.05)
    return arr, att, L, ffn, rng.randint(1, 4), mw


def _fuzz_native(first_seed, count, fractional):
    """Runs in a child process: native against the oracle on `count` instances; returns the first
    mismatch or None."""
    import paper_2608_15473_amd as lib
    for seed in range(first_seed, first_seed + count):
        arr, att, L, ffn, mb, mw = _instance_for(seed, fractional)
        for w in ("qfirst", "composed"):
            ref = oracle_schedule.simulate(arr, att, L, w, ffn, mb, mw)
            nat = _as_lists(lib.schedule_simulate(arr, att, L, w, ffn, mb, mw), len(arr), L)
            for key in ("finish", "sweep", "depart", "returned"):
                if nat[key] != ref[key]:
                    return (seed, fractional, w, key, nat[key], ref[key])
    return None


def _in_child(fn, *args, timeout=120):
    import multiprocessing as mp
    ctx = mp.get_context("spawn")
    with ctx.Pool(1) as pool:
        res = pool.apply_async(fn, args)
        return res.get(timeout=timeout)     # raises multiprocessing.TimeoutError on a hang


@needs_lib
@pytest.mark.parametrize("fractional", [False, True])
def test_native_equals_oracle_on_random_instances(fractional):
    """6,000 integer and 6,000 fractional instances (arrival, attention, feed-forward and wait times
    with 1, 2 or 17 decimals, or none rounded), both wirings: every time of every request equal."""
    assert _in_child(_fuzz_native, 0, 6000, fractional, timeout=240) is None


@needs_lib
def test_native_fractional_time_out_terminates():
    res = _in_child(_native_lone, timeout=60)
    assert res[0] == 0.7 + 0.1 and abs(res[1] - 1.8) < 1e-12


def _native_lone():
    import paper_2608_15473_amd as lib
    r = lib.schedule_simulate([0.0], [0.7], 1, "qfirst", 1.0, 2, 0.1)
    return float(r["ffn_depart"][0, 0]), float(r["finish"][0])


@needs_lib
def test_native_rejects_bad_arguments():
    with pytest.raises(qf.QFError):
        qf.schedule_simulate([0.0], [1.0], 0)
    with pytest.raises(qf.QFError):
        qf.schedule_simulate([0.0], [-1.0], 2)
    with pytest.raises(qf.QFError):
        qf.schedule_simulate([0.0], [1.0], 2, ffn_time=0.0)
    with pytest.raises(qf.QFError):
        qf.schedule_simulate([0.0], [1.0], 2, max_wait=float("nan"))
    with pytest.raises(qf.QFError):
        qf.schedule_simulate([float("inf")], [1.0], 2)
