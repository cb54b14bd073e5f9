"""int8 models (Section 4.1: int2 copies replace int8 experts) through the C
ABI: the int8 high copy, the int8 / int2 / skip decisions of the Eq. 2 rule
at the thresholds quoted for Mixtral (T1 = 0.6, T2 = 0.9), on every kernel
path (one- and two-token decode, matrix-core decode, prefill).

Bar: int8 codes and scales bit-exact; top-k and precisions exact (near
ties resolved as in gpu_support.check_routing); outputs within 2e-3
normwise per token against the oracle, which dequantises the same int8 and
int2 copies in float64."""
import dataclasses

import numpy as np
import pytest

from oracle import moe_oracle as O
from synth import configs as C

import gpu_support as S

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

T1, T2 = 0.6, 0.9


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2411_01433_amd as P
    P.lib()
    yield


# every group kind in one launch: fp16, int8, int4 and int2 copies
MIXED = (C.TAG_INT8, C.TAG_INT8, C.TAG_MISS_INT8_INT2, C.TAG_MISS_INT8_INT2,
         C.TAG_MISS_INT8_INT2, C.TAG_INT2, C.TAG_FP16, C.TAG_MISS_INT4)


def _ragged(T, seed=61):
    # d = 320 and f = 448 end mid-stage for every width (int8 stage: 128
    # columns); the router is scaled by 8 (exact) so that gate gaps reach
    # every Eq. 2 outcome at this small d
    return C.Workload(name=f"int8_ragged_t{T}", seed=seed, d_model=320, d_ff=448,
                      n_experts=8, top_k=2, n_tokens=T, t1=T1, t2=T2, fixed_tags=MIXED,
                      router_scale=8)


def _run(L, x16, d, K, prefill):
    T = x16.shape[0]
    xd = torch.from_numpy(np.ascontiguousarray(x16)).cuda()
    y = torch.empty((T, d), dtype=torch.float32, device="cuda")
    idx = torch.empty((T, K), dtype=torch.int32, device="cuda")
    w = torch.empty((T, K), dtype=torch.float32, device="cuda")
    prec = torch.empty((T, K), dtype=torch.int8, device="cuda")
    (L.prefill if prefill else L.decode_step)(xd, y, idx, w, prec)
    torch.cuda.synchronize()
    return y.cpu().numpy(), idx.cpu().numpy(), w.cpu().numpy(), prec.cpu().numpy()


def _case(wl, x16, prefill=False, rows=None, experts=None):
    tags = list(wl.fixed_tags)
    weights = S.device_layer_weights(wl, 0)
    L = S.make_layer(wl, tags, weights, max_tokens=len(x16))
    y, idx, w, prec = _run(L, x16, wl.d_model, wl.top_k, prefill)
    L.destroy()
    rows = np.arange(len(x16)) if rows is None else np.asarray(rows)
    r, _ = S.check_routing(x16[rows], C.router_weight(wl, 0), tags, wl.top_k, wl.t1, wl.t2,
                           idx[rows], w[rows], prec[rows])
    experts = S.HostExperts(wl, 0, tags) if experts is None else experts
    y_ref = O.layer_output(x16[rows], experts, r)
    err = S.normwise(y[rows], y_ref)
    print(f"{wl.name} prefill={prefill}: max normwise err {err.max():.3e} over {len(rows)} tokens")
    assert err.max() <= S.TOL
    return idx[rows], prec[rows]


def _outcomes(idx, prec, tags):
    """Precision classes the miss-tagged int8 experts took."""
    return {int(p) for e, p in zip(idx.ravel(), prec.ravel())
            if tags[int(e)] == C.TAG_MISS_INT8_INT2}


@pytest.mark.parametrize("T", [1, 2, 3, 4, 9, 17])
def test_decode_paths_ragged(T):
    """T = 1, 2: dot2 kernels; T >= 3: matrix-core kernels (17: more than
    one 16-token pass for a group)."""
    wl = _ragged(T)
    rng = np.random.default_rng(100 + T)
    _case(wl, rng.standard_normal((T, wl.d_model)).astype(np.float16))


def test_decode_rule_outcomes():
    """Over 64 single tokens the miss-tagged experts take every Eq. 2
    outcome: int8, int2 and skip."""
    wl = _ragged(64, seed=62)
    rng = np.random.default_rng(7)
    x16 = rng.standard_normal((64, wl.d_model)).astype(np.float16)
    idx, prec = _case(wl, x16)
    assert _outcomes(idx, prec, wl.fixed_tags) == {O.PREC_HIGH, O.PREC_LOW, O.PREC_SKIP}


@pytest.mark.parametrize("T", [5, 200])
def test_prefill_ragged(T):
    wl = _ragged(T, seed=63)
    rng = np.random.default_rng(200 + T)
    _case(wl, rng.standard_normal((T, wl.d_model)).astype(np.float16), prefill=True)


def test_int8_copy_bit_exact():
    wl = _ragged(1)
    tags = list(wl.fixed_tags)
    weights = S.device_layer_weights(wl, 0)
    L = S.make_layer(wl, tags, weights)
    for e in (0, 2):
        for m, (rows, cols) in enumerate([(wl.d_ff, wl.d_model)] * 2 + [(wl.d_model, wl.d_ff)]):
            codes = torch.empty((rows, cols), dtype=torch.uint8, device="cuda")
            sc = torch.empty((rows, cols // 32), dtype=torch.float16, device="cuda")
            L.export_packed(e, m, 8, codes, sc)
            torch.cuda.synchronize()
            q, s = O.quantize(C.expert_weight(wl, 0, e, ("w1", "w3", "w2")[m]), 8)
            assert np.array_equal(codes.cpu().numpy(), O.pack_codes(q, 8))
            assert np.array_equal(sc.cpu().numpy().view(np.uint16), s.view(np.uint16))
    L.destroy()


def test_mixtral_int8_t1_streams():
    """Full-size Mixtral-shaped int8 layer, one token per step: token streams
    chosen by the oracle's routing so that a miss expert runs from its int8
    copy, from its int2 copy and is skipped."""
    wl = C.MIXTRAL_INT8_T1
    tags = C.layer_tags(wl, 0)
    wg16 = C.router_weight(wl, 0)
    want, streams = {}, []
    for st in range(200):
        xt = C.hidden_states(wl, stream=st)
        r = O.route(xt, wg16, tags, wl.top_k, wl.t1, wl.t2)
        e1, p1 = int(r.idx[0, 1]), int(r.prec[0, 1])
        if tags[e1] == C.TAG_MISS_INT8_INT2 and p1 not in want:
            # keep clear of the thresholds, where either side is accepted
            if min(abs(r.w[0, 0] - wl.t1), abs(r.w[0, 0] - wl.t2)) > 1e-3:
                want[p1] = st
                streams.append(st)
        if len(want) == 3:
            break
    assert set(want) == {O.PREC_HIGH, O.PREC_LOW, O.PREC_SKIP}, want
    weights = S.device_layer_weights(wl, 0)
    L = S.make_layer(wl, tags, weights, max_tokens=1)
    experts = S.HostExperts(wl, 0, tags)
    seen = set()
    for st in streams:
        xt = C.hidden_states(wl, stream=st)
        y, idx, w, prec = S.run_decode(L, torch.from_numpy(xt).cuda(), 1, wl.d_model, wl.top_k)
        r, _ = S.check_routing(xt, wg16, tags, wl.top_k, wl.t1, wl.t2, idx, w, prec)
        err = S.normwise(y, O.layer_output(xt, experts, r)).max()
        print(f"stream {st}: idx {idx[0].tolist()} prec {prec[0].tolist()} err {err:.2e}")
        assert err <= S.TOL
        seen |= _outcomes(idx, prec, tags)
    L.destroy()
    assert seen == {O.PREC_HIGH, O.PREC_LOW, O.PREC_SKIP}


def test_mixtral_int8_matrix_core_and_prefill():
    """The same full-size layer at 8 tokens per decode step and as a
    64-token prefill (sampled rows)."""
    wl = C.MIXTRAL_INT8_T1
    experts = S.HostExperts(wl, 0, C.layer_tags(wl, 0))  # shared: the copies are slow to build
    x8 = np.concatenate([C.hidden_states(wl, stream=s) for s in range(8)])
    _case(dataclasses.replace(wl, n_tokens=8), x8, experts=experts)
    x64 = np.concatenate([C.hidden_states(wl, stream=s) for s in range(64)])
    _case(dataclasses.replace(wl, n_tokens=64), x64, prefill=True, rows=[0, 5, 17, 33],
          experts=experts)
