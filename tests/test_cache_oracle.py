"""Pins of the expert-cache oracle (Section 3.4, Eq. 3) against hand-worked
fixtures, a textbook LRU and invariants of the single-policy cases."""
import collections
import json
import os

import numpy as np
import pytest

from oracle import cache_oracle as CO

HERE = os.path.dirname(os.path.abspath(__file__))
FIX = json.load(open(os.path.join(HERE, "golden", "cache_worked_example.json")))


def _cfg(c, weights):
    return CO.CacheConfig(c["n_layers"], c["n_experts"], c["hi_capacity"], c["lo_capacity"],
                          *weights, bits_hi=c["bits_hi"], bits_lo=c["bits_lo"])


def _ev(e):
    return None if e is None else tuple(e)


@pytest.mark.parametrize("policy", ["lfu", "lhu"])
def test_lfu_vs_lhu_worked_example(policy):
    f = FIX["lfu_vs_lhu"]
    exp = f[policy]
    o, out = CO.replay(_cfg(f["config"], exp["weights"]), [tuple(t) for t in f["trace"]])
    assert [int(h) for h, _ in out] == exp["hits"]
    assert [e for _, e in out] == [_ev(e) for e in exp["evicted"]]
    assert o.penalty == pytest.approx(exp["penalty"], abs=0)


def test_fld_worked_example():
    f = FIX["fld"]
    _, out = CO.replay(_cfg(f["config"], f["weights"]), [tuple(t) for t in f["trace"]])
    assert [e for _, e in out] == [_ev(e) for e in f["evicted"]]


def test_mask_worked_example():
    f = FIX["mask"]
    cfg = _cfg(f["config"], f["weights"])
    _, out = CO.replay(cfg, [tuple(t) for t in f["trace"]])
    assert [e for _, e in out] == [_ev(e) for e in f["evicted_unmasked"]]
    o = CO.CacheOracle(cfg)
    o.begin_token()
    o.access(0, 0, True)
    o.access(3, 0, True)
    o.set_mask(*f["mask"], True)
    assert o.access(1, 1, True)[1] == _ev(f["evicted_masked"][-1])


def test_pure_lru_is_textbook_lru():
    """w_lru = 1, one use per token (distinct R_t): the victim is the least
    recently used resident, as in an ordered-dict LRU."""
    rng = np.random.default_rng(11)
    cfg = CO.CacheConfig(3, 5, 4, 0, 1.0, 0.0, 0.0, 0.0)
    trace = [(i + 1, int(rng.integers(3)), int(rng.integers(5)), 1) for i in range(400)]
    _, out = CO.replay(cfg, trace)
    lru = collections.OrderedDict()
    for (tok, l, e, _), (hit, ev) in zip(trace, out):
        t = (l, e)
        want_hit = t in lru
        want_ev = None
        if want_hit:
            lru.move_to_end(t)
        else:
            if len(lru) >= 4:
                want_ev, _ = lru.popitem(last=False)
            lru[t] = True
        assert (hit, ev) == (want_hit, want_ev)


def test_pure_lfu_and_fld_invariants():
    """w_lfu = 1: no resident that stays was used less often than the victim;
    w_fld = 1: no resident that stays is farther ahead of the incoming layer."""
    rng = np.random.default_rng(12)
    L, E = 6, 4
    for w, key in (((0, 1, 0, 0), "lfu"), ((0, 0, 0, 1), "fld")):
        o = CO.CacheOracle(CO.CacheConfig(L, E, 5, 0, *w))
        for tok in range(1, 300):
            o.begin_token()
            for _ in range(3):
                l, e = int(rng.integers(L)), int(rng.integers(E))
                before = set(o.resident[0])
                F_before = dict(o.F)
                F_before[(l, e)] = F_before.get((l, e), 0) + 1
                hit, ev = o.access(l, e, True)
                if ev is None:
                    continue
                for t in before - {ev}:
                    if key == "lfu":
                        assert F_before.get(t, 0) >= F_before.get(ev, 0)
                    else:
                        dist = lambda u: (u[0] - l + L) % L
                        assert dist(t) <= dist(ev)


def test_eq3_closed_form_and_reset():
    o = CO.CacheOracle(CO.CacheConfig(8, 4, 2, 2, 0.1, 0.2, 0.3, 0.4))
    for _ in range(5):
        o.begin_token()
    o.access(2, 1, True)      # R = 5, F = 1, H = 1
    o.begin_token()
    o.access(2, 1, False)     # R = 6, F = 2, H = 1
    o.begin_token()           # T = 7
    # relative to layer 5: distance (2 - 5 + 8) % 8 = 5
    want = 0.1 * 6 / 7 + 0.2 * 2 / 7 + 0.3 * 1 / 7 + 0.4 * (1 - 5 / 8)
    assert o.priority((2, 1), 5) == pytest.approx(want, rel=1e-15)
    o.begin_sequence()
    assert o.T == 0 and o.priority((2, 1), 5) == pytest.approx(0.4 * (1 - 5 / 8), rel=1e-15)
    # contents survive the reset
    assert o.contains(2, 1, True) and o.contains(2, 1, False)


def test_penalty_ratio():
    """A high-precision miss costs C, an int4 miss C * 4 / 16, an int2 miss
    (replacing an int8 expert) C * 2 / 8."""
    for bh, bl, ratio in ((16, 4, 0.25), (8, 2, 0.25), (16, 2, 0.125)):
        o = CO.CacheOracle(CO.CacheConfig(1, 4, 4, 4, 1, 0, 0, 0, bits_hi=bh, bits_lo=bl,
                                          miss_cost=2.0))
        o.begin_token()
        o.access(0, 0, True)
        o.access(0, 1, False)
        assert o.penalty == pytest.approx(2.0 + 2.0 * ratio, abs=0)
        assert (o.hi_misses, o.lo_misses, o.hits) == (1, 1, 0)
