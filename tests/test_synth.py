"""The seeded input generator: reference vector, determinism, offsets,
distribution.  (Inputs only; no method arithmetic lives there.)"""
import numpy as np

from synth import gen
from synth import configs as C


def test_splitmix64_reference_vector():
    # first outputs of the SplitMix64 reference implementation from state
    # 1477776061723855037 (the published splitmix64.c test sequence)
    key = 1477776061723855037
    u = gen.uniform_u16(key, 12)
    words = u.astype(np.uint64).reshape(3, 4)
    r = [int(sum(int(w[j]) << (16 * j) for j in range(4))) for w in words]
    assert r == [1985237415132408290, 2979275885539914483, 13511426838097143398]


def test_stream_offsets_consistent():
    k = gen.tensor_key(3, 7, gen.TENSOR_W1, 5)
    full = gen.uniform_u16(k, 1000)
    for start in (0, 1, 3, 4, 5, 517):
        assert np.array_equal(gen.uniform_u16(k, 100, start), full[start:start + 100])
    a = gen.normal_fp16(1, 2, gen.TENSOR_W2, 3, (10, 64), 0.02)
    b = gen.normal_fp16(1, 2, gen.TENSOR_W2, 3, (4, 64), 0.02, start=3 * 64)
    assert np.array_equal(a[3:7], b)


def test_keys_distinct():
    keys = {gen.tensor_key(s, l, t, e) for s in range(3) for l in range(4)
            for t in range(1, 8) for e in range(16)}
    assert len(keys) == 3 * 4 * 7 * 16


def test_table_quantiles():
    t = gen.normal_table(1.0).astype(np.float64)
    assert np.all(np.diff(t) >= 0)
    assert np.array_equal(t, -t[::-1])             # symmetric quantiles
    assert abs(t.mean()) < 1e-12 and abs(t.std() - 1.0) < 2e-3
    x = gen.normal_fp16(0, 0, gen.TENSOR_X, 0, (200000,), 0.02).astype(np.float64)
    assert abs(x.mean()) < 3e-4 and abs(x.std() - 0.02) < 3e-4


def test_configs_tags_and_inputs():
    assert C.layer_tags(C.TINY, 0).tolist() == [0, 0, 0, 0, 1, 1, 2, 2]
    for layer in range(4):
        t = C.layer_tags(C.MIXTRAL_PREFILL, layer)
        assert sorted(np.bincount(t, minlength=3).tolist()) == [1, 3, 4]
        assert np.bincount(t, minlength=3).tolist() == [4, 3, 1]
        p = C.layer_tags(C.PHI_STACK, layer)
        assert np.bincount(p, minlength=2).tolist() == [8, 8]
    x = C.hidden_states(C.MIXTRAL_T8_SKEW)
    assert x.shape == (8, 4096) and x.dtype == np.float16
    wg = C.router_weight(C.MIXTRAL_T8_SKEW, 0)
    wg1 = gen.normal_fp16(2, 0, gen.TENSOR_WG, 0, (8, 4096), 0.02)
    assert np.array_equal(wg.astype(np.float64), 4 * wg1.astype(np.float64))
    w = C.expert_weight(C.TINY, 0, 3, "w2", 5, 9)
    assert w.shape == (4, 512)
    assert np.array_equal(w, C.expert_weight(C.TINY, 0, 3, "w2")[5:9])
