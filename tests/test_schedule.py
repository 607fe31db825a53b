"""The layer-wise decode schedule (Appendix D): the fp64-free integer simulation in the oracle and
the native one in libqfattn, pinned to the worked example the paper prints and to each other."""

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


@needs_lib
@pytest.mark.parametrize("seed", range(40))
def test_native_equals_oracle_on_random_instances(seed):
    rng = random.Random(seed)
    R = rng.randint(1, 30)
    L = rng.randint(1, 5)
    arr = [rng.randint(0, 10) for _ in range(R)]
    att = [rng.randint(0, 6) for _ in range(R)]
    ffn = rng.choice([1.0, 2.0, 3.0])
    mb = rng.randint(1, 4)
    mw = rng.choice([math.inf, 0.0, 1.0, 3.0])
    for w in ("qfirst", "composed"):
        ref = oracle_schedule.simulate(arr, att, L, w, ffn, mb, mw)
        nat = _as_lists(qf.schedule_simulate(arr, att, L, w, ffn, mb, mw), R, L)
        for key in ("finish", "sweep", "depart", "returned"):
            assert nat[key] == ref[key], (seed, w, key)


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
