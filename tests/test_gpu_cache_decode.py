"""The expert cache manager driving the hot path (Section 3.4 with the
Section 3.2 rule), through the C ABI: for every token and layer the cache's
residency gives the layer's tags (resident high copy -> FP16, else the
miss tag, so Eq. 2 decides), the decode step runs on those tags, and the
experts it used are recorded back in the cache (high or low copy; skipped
experts are not loaded).  Every step is checked against the oracle with
the same tags; the cache's counters must equal the uses the steps made."""
import numpy as np
import pytest

from oracle import moe_oracle as O
from synth import configs as C

import gpu_support as S

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2411_01433_amd as P
    P.lib()
    yield


@pytest.mark.parametrize("bits_lo", [4, 2])
def test_cache_tags_drive_decode(bits_lo):
    import paper_2411_01433_amd as P
    L_, E, T = 4, 8, 2
    miss = C.TAG_MISS_INT4 if bits_lo == 4 else C.TAG_MISS_INT2
    wls = [C.Workload(name=f"cache_l{l}", seed=70 + l, d_model=256, d_ff=448, n_experts=E,
                      top_k=2, n_tokens=T, t1=0.5, t2=0.95, fixed_tags=(miss,) * E,
                      router_scale=4)
           for l in range(L_)]
    weights = [S.device_layer_weights(wl, 0) for wl in wls]
    layers = [S.make_layer(wl, [C.TAG_FP16] * E, weights[i]) for i, wl in enumerate(wls)]
    current = [[C.TAG_FP16] * E for _ in range(L_)]
    experts = [S.HostExperts(wl, 0, [miss] * E) for wl in wls]
    cache = P.MoeCache(L_, E, 10, 6, 0.3, 0.2, 0.3, 0.2, bits_hi=16, bits_lo=bits_lo)
    rng = np.random.default_rng(11 + bits_lo)
    uses = hi_uses = 0
    seen_tags, seen_prec = set(), set()
    for tok in range(10):
        cache.begin_token()
        for l, wl in enumerate(wls):
            tags = cache.layer_tags(l).tolist()
            for e in range(E):
                if tags[e] != current[l][e]:
                    layers[l].set_expert_precision(e, int(tags[e]))
                    current[l][e] = tags[e]
            seen_tags |= set(tags)
            x16 = rng.standard_normal((T, wl.d_model)).astype(np.float16)
            y, idx, w, prec = S.run_decode(layers[l], torch.from_numpy(x16).cuda(), T,
                                           wl.d_model, wl.top_k)
            r, _ = S.check_routing(x16, C.router_weight(wl, 0), tags, wl.top_k, wl.t1, wl.t2,
                                   idx, w, prec)
            # the oracle's experts carry the same tag as the device's table
            for e in range(E):
                experts[l][e].tag = int(tags[e])
                experts[l][e].__dict__.pop("_memo", None)
            y_ref = O.layer_output(x16, experts[l], r)
            assert S.normwise(y, y_ref).max() <= S.TOL
            for t in range(T):
                for k in range(wl.top_k):
                    p = int(prec[t, k])
                    seen_prec.add(p)
                    if p == O.PREC_SKIP:
                        continue
                    cache.access(l, int(idx[t, k]), p == O.PREC_HIGH)
                    uses += 1
                    hi_uses += p == O.PREC_HIGH
    pen, hm, lm, nh = cache.stats()
    assert hm + lm + nh == uses
    assert seen_tags == {C.TAG_FP16, miss}
    assert {O.PREC_HIGH, O.PREC_LOW} <= seen_prec
    assert pen == pytest.approx(hm + lm * bits_lo / 16)
    for L in layers:
        L.destroy()
    cache.destroy()
