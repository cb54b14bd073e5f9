"""The library's expert cache manager (host code, Section 3.4) against the
oracle: identical hits, evictions and penalties on seeded traces; argument
checks; tags for the layer.  Runs without a GPU."""
import ctypes

import numpy as np
import pytest

import paper_2411_01433_amd as P
from paper_2411_01433_amd import binding as B
from oracle import cache_oracle as CO
from synth import traces as TR

CONFIGS = [
    # (L, E, hi_cap, lo_cap, weights, bits_hi, bits_lo)
    (32, 8, 40, 20, (0.25, 0.25, 0.25, 0.25), 16, 4),
    (32, 8, 64, 64, (1.0, 0.0, 0.0, 0.0), 16, 4),
    (32, 8, 64, 16, (0.0, 1.0, 0.0, 0.0), 16, 4),
    (32, 8, 64, 16, (0.0, 0.0, 1.0, 0.0), 16, 4),
    (32, 8, 64, 16, (0.0, 0.0, 0.0, 1.0), 16, 4),
    (32, 16, 100, 30, (0.4, 0.1, 0.3, 0.2), 8, 2),
    (4, 64, 10, 0, (0.2, 0.3, 0.4, 0.1), 16, 2),
]


def _oracle_replay(cfg, tr):
    tokens, layers, experts, highs, news = tr
    o = CO.CacheOracle(cfg)
    hits, ev = [], []
    last = None
    for i in range(len(tokens)):
        if news[i]:
            o.begin_sequence()
            last = None
        if tokens[i] != last:
            o.begin_token()
            last = tokens[i]
        h, e = o.access(int(layers[i]), int(experts[i]), bool(highs[i]))
        hits.append(int(h))
        ev.append(-1 if e is None else e[0] * cfg.n_experts + e[1])
    return o, np.array(hits), np.array(ev)


@pytest.mark.parametrize("ci", range(len(CONFIGS)))
def test_replay_matches_oracle(ci):
    L, E, hc, lc, w, bh, bl = CONFIGS[ci]
    tr = TR.expert_trace(100 + ci, n_seqs=3, seq_len=40, n_layers=L, n_experts=E)
    cfg = CO.CacheConfig(L, E, hc, lc, *w, bits_hi=bh, bits_lo=bl, miss_cost=1.5)
    o, hits, ev = _oracle_replay(cfg, tr)
    c = P.MoeCache(L, E, hc, lc, *w, bits_hi=bh, bits_lo=bl, miss_cost=1.5)
    g_hits, g_ev = c.replay(*tr)
    np.testing.assert_array_equal(g_hits, hits)
    np.testing.assert_array_equal(g_ev, ev)
    pen, hm, lm, nh = c.stats()
    assert pen == o.penalty and (hm, lm, nh) == (o.hi_misses, o.lo_misses, o.hits)
    for layer in range(L):
        for e in range(E):
            assert c.contains(layer, e, True) == o.contains(layer, e, True)
            assert c.contains(layer, e, False) == o.contains(layer, e, False)
    c.destroy()


def test_step_api_with_masks_matches_oracle():
    """Access one use at a time; the predictor masks a few experts of the
    next layers at every token (Section 3.3) and clears them after."""
    L, E = 16, 8
    cfg = CO.CacheConfig(L, E, 24, 12, 0.3, 0.2, 0.3, 0.2)
    o = CO.CacheOracle(cfg)
    c = P.MoeCache(L, E, 24, 12, 0.3, 0.2, 0.3, 0.2)
    rng = np.random.default_rng(5)
    tr = TR.expert_trace(6, n_seqs=2, seq_len=30, n_layers=L, n_experts=E)
    last = None
    for i in range(len(tr[0])):
        tok, layer, expert, high, new = (int(a[i]) for a in tr)
        if new:
            o.begin_sequence()
            c.begin_sequence()
            last = None
        if tok != last:
            o.begin_token()
            c.begin_token()
            o.clear_masks()
            c.clear_masks()
            for _ in range(3):
                ml, me = int(rng.integers(L)), int(rng.integers(E))
                o.set_mask(ml, me, True)
                c.set_mask(ml, me, True)
            last = tok
        assert c.access(layer, expert, bool(high)) == o.access(layer, expert, bool(high))
    assert c.stats()[0] == o.penalty
    c.destroy()


def test_all_masked_still_evicts():
    c = P.MoeCache(2, 4, 2, 0, 0.0, 0.0, 0.0, 1.0)
    c.begin_token()
    c.access(0, 0, True)
    c.access(1, 0, True)
    c.set_mask(0, 0, True)
    c.set_mask(1, 0, True)
    hit, ev = c.access(0, 1, True)
    assert not hit and ev == (1, 0)  # lowest FLD priority relative to layer 0


def test_layer_tags():
    c = P.MoeCache(2, 4, 3, 2, 1.0, 0.0, 0.0, 0.0, bits_lo=4)
    c.begin_token()
    c.access(1, 2, True)
    c.access(1, 3, False)
    assert c.layer_tags(1).tolist() == [B.TAG_MISS_INT4] * 2 + [B.TAG_FP16, B.TAG_MISS_INT4]
    # an int8 model (Section 4.1): int8 high copies, int2 low copies
    c2 = P.MoeCache(1, 2, 1, 1, 1.0, 0.0, 0.0, 0.0, bits_hi=8, bits_lo=2)
    c2.begin_token()
    c2.access(0, 1, True)
    assert c2.layer_tags(0).tolist() == [B.TAG_MISS_INT8_INT2, B.TAG_INT8]
    c4 = P.MoeCache(1, 2, 1, 1, 1.0, 0.0, 0.0, 0.0, bits_hi=16, bits_lo=2)
    c4.begin_token()
    c4.access(0, 0, True)
    assert c4.layer_tags(0).tolist() == [B.TAG_FP16, B.TAG_MISS_INT2]
    for hi, lo in ((8, 3), (8, 4), (12, 2)):
        c3 = P.MoeCache(1, 2, 1, 1, 1.0, 0.0, 0.0, 0.0, bits_hi=hi, bits_lo=lo)
        with pytest.raises(B.MoeError):
            c3.layer_tags(0)
        c3.destroy()
    for h in (c, c2, c4):
        h.destroy()


@pytest.mark.parametrize("bad", [
    dict(n_layers=0), dict(n_experts=0), dict(hi_capacity=-1), dict(lo_capacity=-2),
    dict(w_lru=0.5), dict(w_lru=-0.5, w_lfu=1.5), dict(w_fld=float("nan")),
    dict(bits_lo=17), dict(bits_lo=0), dict(miss_cost=-1.0), dict(n_layers=5000, n_experts=5000),
])
def test_create_rejects_bad_desc(bad):
    d = dict(n_layers=2, n_experts=4, hi_capacity=2, lo_capacity=2, w_lru=0.25, w_lfu=0.25,
             w_lhu=0.25, w_fld=0.25, bits_hi=16, bits_lo=4, miss_cost=1.0)
    d.update(bad)
    out = ctypes.c_void_p(123)
    st = B.lib().moe_cache_create(ctypes.byref(B.CacheDesc(**d)), ctypes.byref(out))
    assert st == B.MOE_EINVAL and out.value is None
    assert B.lib().moe_last_error()


def test_bad_indices_and_handles():
    L = B.lib()
    c = P.MoeCache(2, 4, 2, 2, 0.25, 0.25, 0.25, 0.25)
    for layer, e in ((-1, 0), (2, 0), (0, 4), (0, -1)):
        with pytest.raises(B.MoeError):
            c.access(layer, e, True)
    with pytest.raises(B.MoeError):
        c.replay([1, 2], [0, 2], [0, 0], [1, 1])
    assert c.stats() == (0.0, 0, 0, 0)  # the failed replay applied nothing
    c.destroy()
    bogus = ctypes.c_void_p(0xdead0)
    assert L.moe_cache_begin_token(bogus) == B.MOE_ESTATE
    assert L.moe_cache_destroy(bogus) == B.MOE_ESTATE
    assert L.moe_cache_destroy(None) == B.MOE_EINVAL
