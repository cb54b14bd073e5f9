"""Stacking Computer (Section 3.3) on the device against the oracle's p
independent routers, through the C ABI.

Bar: predicted experts exact (a near-tied logit pair at the K-th place is
flagged and the device's valid choice accepted, as for the router); gate
values within 1e-5; first_miss and the preload mask exact given the
predicted sets."""
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


def _run(d, E, K, x16, gates16, cached, max_tokens=None):
    import paper_2411_01433_amd as P
    T, p = x16.shape[0], len(gates16)
    gd = [torch.from_numpy(np.ascontiguousarray(g)).cuda() for g in gates16]
    pr = P.MoePredictor(d, E, K, max_tokens or T, gd)
    xd = torch.from_numpy(np.ascontiguousarray(x16)).cuda()
    cd = torch.tensor([np.int64(np.uint64(c).view(np.int64)) for c in cached], dtype=torch.int64,
                      device="cuda")
    idx = torch.full((T, p, K), -1, dtype=torch.int32, device="cuda")
    w = torch.zeros((T, p, K), dtype=torch.float32, device="cuda")
    fm = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    pre = torch.zeros((1,), dtype=torch.int64, device="cuda")
    pr.predict(xd, cd, idx, fm, pre, pred_w=w)
    torch.cuda.synchronize()
    out = (idx.cpu().numpy(), w.cpu().numpy(), int(fm.item()),
           int(np.int64(pre.item()).view(np.uint64)))
    pr.destroy()
    return out


def _check(x16, gates16, cached, K, got):
    g_idx, g_w, g_first, g_pre = got
    T, p = x16.shape[0], len(gates16)
    ref = O.predict_next_layers(x16, gates16, cached, K)
    forced = ref.idx.copy()
    flags = 0
    E = gates16[0].shape[0]
    for t in range(T):
        for j in range(p):
            if np.array_equal(g_idx[t, j], ref.idx[t, j]):
                continue
            srt = np.sort(ref.logits[t, j])[::-1]
            margin = S.TIE_REL * max(1.0, abs(srt[K - 1]))
            amb = (K < E and srt[K - 1] - srt[K] <= margin) or any(
                srt[i] - srt[i + 1] <= margin for i in range(K - 1))
            assert amb, f"token {t} layer +{j + 1}: {g_idx[t, j]} != {ref.idx[t, j]}"
            sel = [int(e) for e in g_idx[t, j]]
            assert len(set(sel)) == K and all(0 <= e < E for e in sel)
            forced[t, j] = sel
            flags += 1
    if flags:
        ref = O.predict_next_layers(x16, gates16, cached, K, forced_idx=forced)
    np.testing.assert_array_equal(g_idx, ref.idx)
    np.testing.assert_allclose(g_w, ref.w, atol=S.W_ATOL, rtol=0)
    assert (g_first, g_pre) == (ref.first_miss, ref.preload)
    return ref


def _masks(rng, E, p):
    return [int(v) for v in rng.integers(0, 1 << min(E, 62), size=p)]


@pytest.mark.parametrize("p", [1, 3, 8])
@pytest.mark.parametrize("T", [1, 4, 64])
def test_predictor_mixtral_gates(p, T):
    """Gates of Mixtral-shaped layers 1..p on a layer-0 gating input."""
    wl = C.MIXTRAL_PREFILL
    gates = [C.router_weight(wl, layer) for layer in range(1, p + 1)]
    x = C.hidden_states(wl)[:T]
    rng = np.random.default_rng(1000 + 10 * p + T)
    full = (1 << wl.n_experts) - 1
    for cached in (_masks(rng, wl.n_experts, p), [full] * p, [0] * p,
                   [full] * (p - 1) + [0]):
        got = _run(wl.d_model, wl.n_experts, wl.top_k, x, gates, cached)
        ref = _check(x, gates, cached, wl.top_k, got)
    assert ref.first_miss == p  # last mask: only the last layer misses


def test_predictor_phi_gates_32_layer_walk():
    """Phi-MoE-shaped gates (16 experts), 4 tokens, p = 3 at several depths."""
    wl = C.PHI_STACK
    rng = np.random.default_rng(7)
    x = C.hidden_states(wl)
    for layer in (0, 10, 28):
        gates = [C.router_weight(wl, layer + j) for j in range(1, 4)]
        cached = _masks(rng, wl.n_experts, 3)
        _check(x, gates, cached, wl.top_k,
               _run(wl.d_model, wl.n_experts, wl.top_k, x, gates, cached))


def test_predictor_ragged_and_wide():
    """d = 192, 5 experts, top-3; and 64 experts, top-8 (the limits)."""
    rng = np.random.default_rng(8)
    x = rng.standard_normal((6, 192)).astype(np.float16)
    gates = [(rng.standard_normal((5, 192)) * 0.3).astype(np.float16) for _ in range(2)]
    cached = _masks(rng, 5, 2)
    _check(x, gates, cached, 3, _run(192, 5, 3, x, gates, cached, max_tokens=9))
    x = rng.standard_normal((3, 256)).astype(np.float16)
    gates = [(rng.standard_normal((64, 256)) * 0.3).astype(np.float16) for _ in range(4)]
    cached = [int(rng.integers(0, 2**62)) | (1 << 63) for _ in range(4)]
    _check(x, gates, cached, 8, _run(256, 64, 8, x, gates, cached))


def test_predictor_prefill_sized():
    """512 tokens (the prefill batch), p = 2."""
    wl = C.MIXTRAL_PREFILL
    gates = [C.router_weight(wl, 1), C.router_weight(wl, 2)]
    x = C.hidden_states(wl)
    cached = [0xFF, 0x0F]
    _check(x, gates, cached, wl.top_k,
           _run(wl.d_model, wl.n_experts, wl.top_k, x, gates, cached))


def test_predictor_repeated_launches():
    """The finish counter resets itself: many launches in a row agree."""
    import paper_2411_01433_amd as P
    wl = C.MIXTRAL_T8_SKEW
    gates = [torch.from_numpy(C.router_weight(wl, 0)).cuda() for _ in range(3)]
    pr = P.MoePredictor(wl.d_model, wl.n_experts, wl.top_k, 8, gates)
    x = torch.from_numpy(C.hidden_states(wl)).cuda()
    cd = torch.tensor([0x0F, 0xFF, 0x00], dtype=torch.int64, device="cuda")
    outs = []
    for _ in range(20):
        idx = torch.empty((8, 3, 2), dtype=torch.int32, device="cuda")
        fm = torch.empty((1,), dtype=torch.int32, device="cuda")
        pre = torch.empty((1,), dtype=torch.int64, device="cuda")
        pr.predict(x, cd, idx, fm, pre)
        outs.append((idx, fm, pre))
    torch.cuda.synchronize()
    for idx, fm, pre in outs[1:]:
        assert torch.equal(idx, outs[0][0]) and torch.equal(fm, outs[0][1])
        assert torch.equal(pre, outs[0][2])
    pr.destroy()
