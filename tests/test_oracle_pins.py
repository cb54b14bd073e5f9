"""Pins of the CPU oracle against things other than itself.

Each test checks one oracle function against what the paper or mathematics
fixes: brute force on tiny inputs, closed forms, library routines,
invariants and hand-worked fixtures under tests/golden/.  A plausible slip
(a dropped term, a wrong sign or index, a transposed operand) in any oracle
function fails at least one test here.
"""
import itertools
import json
import os

import numpy as np
import pytest
import scipy.special

from oracle import moe_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _fp16(rng, shape, std):
    return (rng.standard_normal(shape) * std).astype(np.float16)


def _experts(rng, E, d, f, tags):
    return [O.Expert(_fp16(rng, (f, d), 0.05), _fp16(rng, (f, d), 0.05),
                     _fp16(rng, (d, f), 0.05), int(tags[e])) for e in range(E)]


# ---------------------------------------------------------------- gating
def test_router_logits_vs_loops(rng):
    x = _fp16(rng, (3, 20), 1.0)
    wg = _fp16(rng, (5, 20), 0.1)
    np.testing.assert_allclose(O.router_logits(x, wg),
                               O.brute_router_logits(x, wg), rtol=1e-13,
                               atol=1e-13)
    # shape / orientation: [T, E]
    assert O.router_logits(x, wg).shape == (3, 5)


def test_topk_vs_exhaustive(rng):
    for trial in range(200):
        E = int(rng.integers(2, 9))
        K = int(rng.integers(1, E + 1))
        l = rng.standard_normal(E)
        if trial % 3 == 0:  # force exact ties
            l = np.round(l * 2) / 2
        got = O.topk(l, K)
        assert set(got.tolist()) == O.brute_topk_set(l, K)
        # slot 0 holds the largest, descending order
        assert all(l[got[i]] >= l[got[i + 1]] for i in range(K - 1))
        assert len(set(got.tolist())) == K


def test_topk_tie_goes_to_lower_index():
    l = np.array([1.0, 3.0, 3.0, 0.0, 3.0])
    assert O.topk(l, 2).tolist() == [1, 2]
    assert O.topk(l, 3).tolist() == [1, 2, 4]


def test_gate_weights_closed_forms(rng):
    for _ in range(50):
        E = int(rng.integers(2, 17))
        l = rng.standard_normal(E) * 3
        for K in (1, 2, E):
            sel = O.topk(l, K)
            w = O.gate_weights(l[sel])
            assert abs(w.sum() - 1.0) < 1e-14
            assert np.all(w > 0)
            # equals the full softmax renormalised over the selected set
            full = scipy.special.softmax(l)
            ref = full[sel] / full[sel].sum()
            np.testing.assert_allclose(w, ref, rtol=1e-12)
            if K == 1:
                assert w[0] == 1.0
            if K == E:  # dense soft MoE: library softmax over all experts
                np.testing.assert_allclose(w, full[sel], rtol=1e-12)
            # descending because the logits are
            assert np.all(np.diff(w) <= 0)


# ------------------------------------------------------------- Eq. 2 rule
def test_eq2_worked_examples():
    d = json.load(open(os.path.join(GOLDEN, "eq2_worked_examples.json")))
    for c in d["cases"]:
        w = np.array(c["w"])
        s = O.unimportance_scores(w)
        np.testing.assert_allclose(s, c["scores"], atol=1e-12)
        tags = np.full(len(w), O.TAG_MISS_INT4)
        sel = np.arange(len(w))
        prec = O.token_precisions(w, sel, tags, c["t1"], c["t2"])
        assert prec.tolist() == c["prec"], c["why"]


def test_eq2_closed_form_top2(rng):
    """At K = 2 the second expert's score is the first gate, 1 - g2; the rule
    'int4 when g < 0.3, else fp16' is T1 = 0.7 with skip disabled."""
    for _ in range(500):
        l = rng.standard_normal(2) * 2
        sel = O.topk(l, 2)
        w = O.gate_weights(l[sel])
        s = O.unimportance_scores(w)
        assert s[0] == 0.0
        assert abs(s[1] - w[0]) < 1e-15
        assert abs(s[1] - (1 - w[1])) < 1e-12
        tags = np.array([O.TAG_MISS_INT4, O.TAG_MISS_INT4])
        prec = O.token_precisions(w, np.array([0, 1]), tags, 0.7, 1.0)
        assert prec[0] == O.PREC_HIGH
        if abs(w[1] - 0.3) > 1e-9:
            assert prec[1] == (O.PREC_LOW if w[1] < 0.3 else O.PREC_HIGH)


def test_eq2_invariants(rng):
    for _ in range(300):
        K = int(rng.integers(1, 7))
        w = rng.dirichlet(np.ones(K))
        s = O.unimportance_scores(w)
        order = O.importance_rank(w)
        assert s[order[0]] == 0.0                  # top expert scores 0
        ss = s[order]
        assert np.all(np.diff(ss) >= -1e-15)       # scores grow with rank
        for i in range(1, K):                      # s_i = sum of gates above
            assert abs(ss[i] - w[order[:i]].sum()) < 1e-12
        assert np.all(s <= 1.0 + 1e-12)
        tags = np.full(K, O.TAG_MISS_INT2)
        sel = np.arange(K)
        # T1 >= 1 -> all high ; top expert always high whatever T1, T2
        assert np.all(O.token_precisions(w, sel, tags, 1.0, 1.0) == O.PREC_HIGH)
        p = O.token_precisions(w, sel, tags, 0.0, 0.0)
        assert p[order[0]] == O.PREC_HIGH
        # resident tags ignore the rule
        tags2 = np.array([O.TAG_FP16, O.TAG_INT4, O.TAG_INT2] * 3)[:K]
        p2 = O.token_precisions(w, sel, tags2, 0.0, 0.0)
        for j in range(K):
            assert p2[j] == (O.PREC_HIGH if tags2[j] == O.TAG_FP16 else O.PREC_LOW)
    # top-2 with T1 < 0.5: the second expert's score (>= 0.5) always exceeds T1
    for _ in range(100):
        w = np.sort(rng.dirichlet(np.ones(2)))[::-1]
        p = O.token_precisions(w, np.arange(2), np.full(2, O.TAG_MISS_INT4),
                               0.49, 1.0)
        assert p.tolist() == [O.PREC_HIGH, O.PREC_LOW]


# ------------------------------------------------------------ quantiser
def test_quant_worked_examples():
    d = json.load(open(os.path.join(GOLDEN, "quant_worked_examples.json")))
    for c in d["cases"]:
        b = c["bits"]
        w = (np.array(c["w_over_2m6"]) * 2.0 ** -6).astype(np.float16)
        assert np.all(w.astype(np.float64) == np.array(c["w_over_2m6"]) * 2.0 ** -6)
        q, s = O.quantize(w[None, :], b)
        assert float(s[0, 0]) == c["scale"]
        assert q[0].tolist() == c["q"], c["why"]
        packed = O.pack_codes(q, b)
        assert " ".join("%02x" % v for v in packed[0]) == c["packed_hex"]
        assert O.unpack_codes(packed, b)[0].tolist() == c["q"]


@pytest.mark.parametrize("bits", [4, 2, 8])
def test_quant_brute_nearest(rng, bits):
    w = _fp16(rng, (6, 64), 0.02)
    w[0, :32] = 0                                   # zero group
    w[1, 5] = np.float16(0.0)
    q, s = O.quantize(w, bits)
    sf = s.astype(np.float64)
    for r in range(w.shape[0]):
        for c in range(w.shape[1]):
            g = c // 32
            exp = O.brute_nearest_code(float(w[r, c]), float(sf[r, g]), bits)
            assert q[r, c] == exp, (r, c, float(w[r, c]), float(sf[r, g]))


@pytest.mark.parametrize("bits", [4, 2, 8])
def test_quant_bounds_and_extremes(rng, bits):
    qmax = 2 ** (bits - 1) - 1
    w = _fp16(rng, (64, 256), 0.02)
    q, s = O.quantize(w, bits)
    assert q.min() >= -(2 ** (bits - 1)) and q.max() <= qmax
    # the scale is fp16 of absmax / qmax, absmax taken per 32-group of a row
    m = np.abs(w.astype(np.float64)).reshape(64, 8, 32).max(axis=2)
    assert np.array_equal(s, (m / qmax).astype(np.float16))
    wh = O.dequantize(q, s)
    sf = np.repeat(s.astype(np.float64), 32, axis=1)
    err = np.abs(w.astype(np.float64) - wh)
    # |w - w_hat| <= s/2 unless the clamp engaged (then <= m - qmax*s)
    mf = np.repeat(m, 32, axis=1)
    bound = np.maximum(sf / 2, mf - qmax * sf) + 1e-18
    assert np.all(err <= bound)
    # +-absmax maps to +-qmax exactly
    for r in range(64):
        for g in range(8):
            grp = w[r, g * 32:(g + 1) * 32].astype(np.float64)
            j = int(np.argmax(np.abs(grp)))
            assert abs(q[r, g * 32 + j]) == qmax
            assert np.sign(q[r, g * 32 + j]) == np.sign(grp[j])


@pytest.mark.parametrize("bits", [4, 2, 8])
def test_quant_idempotent(rng, bits):
    w = _fp16(rng, (16, 128), 0.02)
    q, s = O.quantize(w, bits)
    wh = O.dequantize(q, s)          # float64, exact q * s
    q2, s2 = O.quantize(wh, bits)
    assert np.array_equal(q2, q)
    assert np.array_equal(s2, s)


def test_quant_subnormal_group():
    """A group whose absmax/7 is below the smallest normal fp16 gets a
    subnormal scale; codes still come from the nearest-level rule."""
    tiny = np.float16(2.0 ** -20)
    w = np.zeros((1, 32), dtype=np.float16)
    w[0, :6] = np.array([7, -7, 3, 1, 2, -5]) * tiny
    q, s = O.quantize(w, 4)
    assert float(s[0, 0]) == float(np.float16(7 * 2.0 ** -20 / 7))
    assert float(s[0, 0]) < 2.0 ** -14
    for c in range(32):
        assert q[0, c] == O.brute_nearest_code(float(w[0, c]), float(s[0, 0]), 4)


def test_pack_roundtrip_and_layout(rng):
    for bits in (4, 2, 8):
        q = rng.integers(-(2 ** (bits - 1)), 2 ** (bits - 1), size=(5, 64))
        p = O.pack_codes(q, bits)
        assert p.shape == (5, 64 * bits // 8) and p.dtype == np.uint8
        assert np.array_equal(O.unpack_codes(p, bits), q)
        # element j lives at bit bits*(j % per) of byte j // per
        per = 8 // bits
        for j in range(64):
            u = (p[:, j // per] >> (bits * (j % per))) & ((1 << bits) - 1)
            assert np.array_equal(u.astype(np.int64) - 2 ** (bits - 1), q[:, j])


# ---------------------------------------------------------- expert + layer
def test_silu_against_library():
    import torch
    a = np.linspace(-20, 20, 1001)
    np.testing.assert_allclose(
        O.silu(a), torch.nn.functional.silu(torch.tensor(a)).numpy(),
        rtol=1e-13, atol=1e-300)
    assert O.silu(np.array([0.0]))[0] == 0.0


def test_expert_vs_loops(rng):
    d, f = 12, 20            # non-square so a transposed operand fails
    x = _fp16(rng, (1, d), 1.0)
    w1, w3, w2 = _fp16(rng, (f, d), 0.3), _fp16(rng, (f, d), 0.3), _fp16(rng, (d, f), 0.3)
    got = O.swiglu_expert(x.astype(np.float64), w1.astype(np.float64),
                          w3.astype(np.float64), w2.astype(np.float64))[0]
    np.testing.assert_allclose(got, O.brute_expert(x[0], w1, w3, w2),
                               rtol=1e-12, atol=1e-14)


def _dense_reference(x16, wg16, W1, W3, W2, k):
    """Dense masked MoE: every expert on every token, then a gate matrix with
    zeros outside the top-k (library argsort + full softmax renormalised)."""
    x = x16.astype(np.float64)
    l = x @ wg16.astype(np.float64).T
    T, E = l.shape
    G = np.zeros((T, E))
    for t in range(T):
        order = np.lexsort((np.arange(E), -l[t]))[:k]
        p = scipy.special.softmax(l[t])
        G[t, order] = p[order] / p[order].sum()
    a = np.einsum("td,efd->tef", x, W1)
    b = np.einsum("td,efd->tef", x, W3)
    h = a * scipy.special.expit(a) * b
    out = np.einsum("tef,edf->ted", h, W2)
    return np.einsum("te,ted->td", G, out)


def test_layer_all_fp16_equals_dense(rng):
    E, d, f, T, K = 6, 24, 40, 5, 2
    x = _fp16(rng, (T, d), 1.0)
    wg = _fp16(rng, (E, d), 0.3)
    ex = _experts(rng, E, d, f, [O.TAG_FP16] * E)
    y, r = O.layer_forward(x, wg, ex, K, 0.6, 0.9)
    W1 = np.stack([e.w1 for e in ex]).astype(np.float64)
    W3 = np.stack([e.w3 for e in ex]).astype(np.float64)
    W2 = np.stack([e.w2 for e in ex]).astype(np.float64)
    np.testing.assert_allclose(y, _dense_reference(x, wg, W1, W3, W2, K),
                               rtol=1e-11, atol=1e-12)
    assert np.all(r.prec == O.PREC_HIGH)
    np.testing.assert_allclose(r.w.sum(axis=1), 1.0, atol=1e-14)


def test_layer_k_equals_e_is_soft_moe(rng):
    E, d, f, T = 4, 16, 24, 3
    x = _fp16(rng, (T, d), 1.0)
    wg = _fp16(rng, (E, d), 0.3)
    ex = _experts(rng, E, d, f, [O.TAG_FP16] * E)
    y, _ = O.layer_forward(x, wg, ex, E, 1.0, 1.0)
    l = x.astype(np.float64) @ wg.astype(np.float64).T
    G = scipy.special.softmax(l, axis=1)
    ref = np.zeros_like(y)
    for e in range(E):
        ref += G[:, e:e + 1] * np.stack([
            O.brute_expert(x[t], ex[e].w1, ex[e].w3, ex[e].w2) for t in range(T)])
    np.testing.assert_allclose(y, ref, rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("tag,bits,prec", [(O.TAG_INT4, 4, O.PREC_LOW), (O.TAG_INT2, 2, O.PREC_LOW),
                                           (O.TAG_INT8, 8, O.PREC_HIGH)])
def test_layer_all_quantised_equals_dense_dequant(rng, tag, bits, prec):
    """Every expert held as one quantised copy (int4 / int2 low copies, or
    the int8 high copy of an int8 model) equals the dense layer over weights
    dequantised by the brute-force nearest-level rule."""
    E, d, f, T, K = 4, 64, 96, 4, 2
    x = _fp16(rng, (T, d), 1.0)
    wg = _fp16(rng, (E, d), 0.3)
    ex = _experts(rng, E, d, f, [tag] * E)
    y, r = O.layer_forward(x, wg, ex, K, 1.0, 1.0)
    assert np.all(r.prec == prec)

    def dq(w):  # dequantise by the brute-force nearest-level rule
        w64 = w.astype(np.float64)
        out = np.zeros_like(w64)
        qmax = 2 ** (bits - 1) - 1
        for rr in range(w.shape[0]):
            for g in range(w.shape[1] // 32):
                seg = w64[rr, g * 32:(g + 1) * 32]
                s = float(np.float16(np.abs(seg).max() / qmax))
                out[rr, g * 32:(g + 1) * 32] = [
                    O.brute_nearest_code(v, s, bits) * s for v in seg]
        return out
    W1 = np.stack([dq(e.w1) for e in ex])
    W3 = np.stack([dq(e.w3) for e in ex])
    W2 = np.stack([dq(e.w2) for e in ex])
    np.testing.assert_allclose(y, _dense_reference(x, wg, W1, W3, W2, K),
                               rtol=1e-11, atol=1e-12)


def test_layer_skip_and_mixed(rng):
    """T1 = T2 = 0 with miss tags: only the top expert contributes, with its
    (unrenormalised) gate weight."""
    E, d, f, T, K = 4, 32, 32, 3, 2
    x = _fp16(rng, (T, d), 1.0)
    wg = _fp16(rng, (E, d), 0.3)
    ex = _experts(rng, E, d, f, [O.TAG_MISS_INT4] * E)
    y, r = O.layer_forward(x, wg, ex, K, 0.0, 0.0)
    for t in range(T):
        assert r.prec[t].tolist() == [O.PREC_HIGH, O.PREC_SKIP]
        e0 = int(r.idx[t, 0])
        ref = r.w[t, 0] * O.brute_expert(x[t], ex[e0].w1, ex[e0].w3, ex[e0].w2)
        np.testing.assert_allclose(y[t], ref, rtol=1e-11, atol=1e-13)
    # T1 = 0, T2 = 1: second expert runs from its int4 copy
    y2, r2 = O.layer_forward(x, wg, ex, K, 0.0, 1.0)
    for t in range(T):
        assert r2.prec[t].tolist() == [O.PREC_HIGH, O.PREC_LOW]
        e1 = int(r2.idx[t, 1])
        lo = [O.make_low_copy(m, 4).dense() for m in (ex[e1].w1, ex[e1].w3, ex[e1].w2)]
        delta = r2.w[t, 1] * O.brute_expert(x[t], *lo)
        np.testing.assert_allclose(y2[t] - y[t], delta, rtol=1e-9, atol=1e-12)


def test_layer_int8_model_rule(rng):
    """int8 model (Section 4.1: int2 copies replace int8 experts) with the
    thresholds quoted for Mixtral in Section 3.2 (T1 = 0.6, T2 = 0.9).  At
    top-2 the second slot's Eq. 2 score is the first gate w0, so it runs from
    the int8 copy when w0 <= 0.6, from the int2 copy when 0.6 < w0 <= 0.9 and
    is skipped above; the first slot always runs from the int8 copy.  Each
    token's output is rebuilt by brute force from nearest-level codes."""
    E, d, f, T, K = 4, 32, 64, 24, 2
    x = _fp16(rng, (T, d), 1.0)
    wg = _fp16(rng, (E, d), 0.6)
    tags = [O.TAG_INT8, O.TAG_MISS_INT8_INT2, O.TAG_MISS_INT8_INT2, O.TAG_INT8]
    ex = _experts(rng, E, d, f, tags)
    y, r = O.layer_forward(x, wg, ex, K, 0.6, 0.9)

    def dq(w, bits):
        w64 = w.astype(np.float64)
        qmax = 2 ** (bits - 1) - 1
        out = np.zeros_like(w64)
        for rr in range(w.shape[0]):
            for g in range(w.shape[1] // 32):
                seg = w64[rr, g * 32:(g + 1) * 32]
                s = float(np.float16(np.abs(seg).max() / qmax))
                out[rr, g * 32:(g + 1) * 32] = [O.brute_nearest_code(v, s, bits) * s for v in seg]
        return out
    seen = set()
    for t in range(T):
        ref = np.zeros(d)
        for j in range(K):
            e = int(r.idx[t, j])
            if j == 0 or tags[e] == O.TAG_INT8:
                exp_p = O.PREC_HIGH
            else:
                w0 = r.w[t, 0]
                exp_p = O.PREC_HIGH if w0 <= 0.6 else (O.PREC_LOW if w0 <= 0.9 else O.PREC_SKIP)
            assert r.prec[t, j] == exp_p
            if tags[e] == O.TAG_MISS_INT8_INT2 and j == 1:
                seen.add(exp_p)
            if exp_p == O.PREC_SKIP:
                continue
            bits = 8 if exp_p == O.PREC_HIGH else 2
            mats = [dq(m, bits) for m in (ex[e].w1, ex[e].w3, ex[e].w2)]
            ref += r.w[t, j] * O.brute_expert(x[t], *mats)
        np.testing.assert_allclose(y[t], ref, rtol=1e-10, atol=1e-12)
    assert seen == {O.PREC_HIGH, O.PREC_LOW, O.PREC_SKIP}, seen


def test_layer_linear_in_expert_output(rng):
    """Doubling every W2 doubles y (Eq. 1 is linear in each E(x))."""
    E, d, f, T, K = 4, 16, 16, 3, 2
    x = _fp16(rng, (T, d), 1.0)
    wg = _fp16(rng, (E, d), 0.3)
    ex = _experts(rng, E, d, f, [O.TAG_FP16] * E)
    y, _ = O.layer_forward(x, wg, ex, K, 1.0, 1.0)
    ex2 = [O.Expert(e.w1, e.w3, (e.w2 * np.float16(2)).astype(np.float16), e.tag)
           for e in ex]
    y2, _ = O.layer_forward(x, wg, ex2, K, 1.0, 1.0)
    np.testing.assert_allclose(y2, 2 * y, rtol=1e-13, atol=1e-15)


# ------------------------------------------------------------ stack glue
def test_rmsnorm_closed_form(rng):
    h = rng.standard_normal((4, 64)) * 7
    n = O.rmsnorm(h, eps=0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(n * n, axis=1)), 1.0, rtol=1e-13)
    np.testing.assert_allclose(n / h, (n / h)[:, :1] * np.ones_like(h), rtol=1e-12)
    c = np.full((1, 8), 3.0)                      # constant row -> all ones
    np.testing.assert_allclose(O.rmsnorm(c, eps=0.0), 1.0, rtol=1e-15)
    h2, x2 = O.residual_step(h, np.ones_like(h))
    np.testing.assert_allclose(h2, h + 1.0)
    assert x2.dtype == np.float16


# ------------------------------------------ Stacking Computer (Section 3.3)
def test_predictor_worked_example():
    d = json.load(open(os.path.join(GOLDEN, "predictor_worked_example.json")))
    x = np.array(d["x"], dtype=np.float16)
    gates = [np.array(g, dtype=np.float16) for g in d["gates"]]
    pr = O.predict_next_layers(x, gates, d["cached"], d["k"])
    np.testing.assert_array_equal(pr.logits, np.array(d["logits"]))
    assert pr.idx.tolist() == d["idx"]
    np.testing.assert_allclose(pr.w, np.array(d["w"]), rtol=0, atol=1e-15)
    assert (pr.first_miss, pr.preload) == (d["first_miss"], d["preload"])


def test_predictor_one_layer_is_that_layers_router(rng):
    x = _fp16(rng, (5, 48), 1.0)
    wg = _fp16(rng, (8, 48), 0.3)
    pr = O.predict_next_layers(x, [wg], [0], 2)
    r = O.route(x, wg, [O.TAG_FP16] * 8, 2, 1.0, 1.0)
    np.testing.assert_array_equal(pr.idx[:, 0], r.idx)
    np.testing.assert_allclose(pr.w[:, 0], r.w, rtol=0, atol=0)


def test_predictor_walk_brute_force(rng):
    """Sets and the walk written out with Python sets on exhaustive top-k."""
    T, d, E, K, p = 3, 16, 6, 2, 4
    for trial in range(40):
        x = _fp16(rng, (T, d), 1.0)
        gates = [_fp16(rng, (E, d), 0.5) for _ in range(p)]
        cached = [int(v) for v in rng.integers(0, 1 << E, size=p)]
        if trial % 4 == 0:
            cached = [(1 << E) - 1] * p
        pr = O.predict_next_layers(x, gates, cached, K)
        exp_first, exp_pre = 0, 0
        for j in range(p):
            need = set()
            for t in range(T):
                row = [sum(float(x[t, c]) * float(gates[j][e, c]) for c in range(d))
                       for e in range(E)]
                sel = O.brute_topk_set(row, K)
                assert set(pr.idx[t, j].tolist()) == sel
                need |= sel
            missing = {e for e in need if not (cached[j] >> e) & 1}
            if missing:
                exp_first, exp_pre = j + 1, sum(1 << e for e in missing)
                break
        assert (pr.first_miss, pr.preload) == (exp_first, exp_pre)


def test_predictor_walk_extremes(rng):
    x = _fp16(rng, (4, 32), 1.0)
    gates = [_fp16(rng, (8, 32), 0.5) for _ in range(3)]
    full = O.predict_next_layers(x, gates, [0xFF] * 3, 2)
    assert (full.first_miss, full.preload) == (0, 0)
    none = O.predict_next_layers(x, gates, [0] * 3, 2)
    union = 0
    for e in none.idx[:, 0].ravel():
        union |= 1 << int(e)
    assert (none.first_miss, none.preload) == (1, union)
    assert np.allclose(none.w.sum(axis=-1), 1.0)
