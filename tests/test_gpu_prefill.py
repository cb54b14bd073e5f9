"""Prefill path (MFMA grouped GEMM) against the oracle, through the C ABI."""
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


def _edge(name, seed, d, f, E, K, T, tags, t1=1.0, t2=1.0):
    return C.Workload(name=name, seed=seed, d_model=d, d_ff=f, n_experts=E,
                      top_k=K, n_tokens=T, t1=t1, t2=t2, fixed_tags=tuple(tags))


def run_prefill(L, x16, d, K, residual_h=None):
    T = x16.shape[0]
    xd = torch.from_numpy(np.ascontiguousarray(x16)).cuda()
    idx = torch.empty((T, K), dtype=torch.int32, device="cuda")
    w = torch.empty((T, K), dtype=torch.float32, device="cuda")
    prec = torch.empty((T, K), dtype=torch.int8, device="cuda")
    if residual_h is None:
        y = torch.empty((T, d), dtype=torch.float32, device="cuda")
        L.prefill(xd, y, idx, w, prec)
        torch.cuda.synchronize()
        return y.cpu().numpy(), idx.cpu().numpy(), w.cpu().numpy(), prec.cpu().numpy()
    xn = torch.empty((T, d), dtype=torch.float16, device="cuda")
    L.prefill_residual(xd, residual_h, xn, idx, w, prec)
    torch.cuda.synchronize()
    return xn.cpu().numpy(), idx.cpu().numpy(), w.cpu().numpy(), prec.cpu().numpy()


def _check(wl, tags, x16, sample=None, t1=None, t2=None, residual=False):
    t1 = wl.t1 if t1 is None else t1
    t2 = wl.t2 if t2 is None else t2
    weights = S.device_layer_weights(wl, 0)
    L = S.make_layer(wl, tags, weights, max_tokens=len(x16), t1=t1, t2=t2)
    K, d = wl.top_k, wl.d_model
    if residual:
        h0 = np.asarray(x16, dtype=np.float32) * np.float32(0.25)
        hd = torch.from_numpy(h0).cuda()
        xn, idx, w, prec = run_prefill(L, x16, d, K, residual_h=hd)
        out = hd.cpu().numpy() - h0
    else:
        out, idx, w, prec = run_prefill(L, x16, d, K)
    L.destroy()
    # routing of every token; the fp64 expert FFN on the sampled rows
    wg16 = C.router_weight(wl, 0)
    r_all, flags = S.check_routing(x16, wg16, tags, K, t1, t2, idx, w, prec)
    rows = np.arange(len(x16)) if sample is None else np.asarray(sample)
    r = O.Routing(idx=r_all.idx[rows], w=r_all.w[rows], prec=r_all.prec[rows],
                  logits=r_all.logits[rows])
    y_ref = O.layer_output(x16[rows], S.HostExperts(wl, 0, tags), r)
    err = S.normwise(out[rows], y_ref)
    print(f"{wl.name}: routing exact on {len(x16)} tokens ({len(flags)} flagged near-ties); "
          f"max normwise err {err.max():.3e} over {len(rows)} tokens")
    assert err.max() <= S.TOL
    if residual:
        h_ref = h0[rows].astype(np.float64) + y_ref
        assert S.normwise(xn[rows], O.rmsnorm(h_ref)).max() <= S.TOL
    return idx, prec


def test_prefill_tiny():
    wl = C.TINY
    _check(wl, C.layer_tags(wl, 0), C.hidden_states(wl))


def test_prefill_tiny_many_tokens_all_tags():
    """Groups of more than one 160-token pass at every width (fp16, int4,
    int2: about 210 tokens each); every tag kind."""
    wl = _edge("prefill_busy", 41, 256, 512, 4, 2, 420,
               [C.TAG_FP16, C.TAG_INT4, C.TAG_INT2, C.TAG_MISS_INT4], t1=0.45, t2=1.0)
    rng = np.random.default_rng(11)
    idx, prec = _check(wl, wl.fixed_tags, rng.standard_normal((420, 256)).astype(np.float16))
    counts = np.bincount(idx.ravel(), minlength=4)
    assert counts[:3].min() > 160, counts


def test_prefill_ragged_shapes():
    wl = _edge("prefill_ragged", 42, 192, 320, 5, 3, 37,
               [C.TAG_FP16, C.TAG_INT4, C.TAG_INT2, C.TAG_MISS_INT4, C.TAG_MISS_INT2],
               t1=0.4, t2=0.8)
    rng = np.random.default_rng(12)
    _check(wl, wl.fixed_tags, rng.standard_normal((37, 192)).astype(np.float16))


def test_prefill_skip_and_residual():
    wl = _edge("prefill_skip", 43, 256, 384, 6, 2, 50, [C.TAG_MISS_INT2] * 6)
    rng = np.random.default_rng(13)
    x = rng.standard_normal((50, 256)).astype(np.float16)
    _check(wl, wl.fixed_tags, x, t1=0.0, t2=0.0, residual=True)
    _check(wl, wl.fixed_tags, x, t1=0.0, t2=1.0)


def test_prefill_max_tokens():
    """The largest step a layer takes (8192 tokens): about 2,000 tokens per
    group, i.e. 13 passes of 160 tokens per weight tile, every tag kind;
    routing of all tokens, the output on 512 evenly spread tokens."""
    T = 8192
    wl = _edge("prefill_max", 44, 256, 512, 8, 2, T,
               [C.TAG_FP16, C.TAG_INT4, C.TAG_INT2, C.TAG_MISS_INT4, C.TAG_MISS_INT2,
                C.TAG_FP16, C.TAG_MISS_INT4, C.TAG_INT4], t1=0.3, t2=0.6)
    rng = np.random.default_rng(14)
    x = rng.standard_normal((T, 256)).astype(np.float16)
    idx, prec = _check(wl, wl.fixed_tags, x, sample=np.linspace(0, T - 1, 512).astype(int))
    counts = np.bincount(idx.ravel(), minlength=8)
    assert counts.min() > 160, counts
    # all three outcomes of Eq. 2 occur on the miss-tagged experts
    assert {0, 1, 2} <= set(np.unique(prec).tolist()), np.unique(prec)


def test_prefill_mixtral_layer_t512():
    """One Mixtral-shaped layer of the 512-token prefill workload (4:3:1
    map of layer 0): routing of all 512 tokens, the layer output on 32
    sampled tokens, against the oracle."""
    wl = C.MIXTRAL_PREFILL
    tags = C.layer_tags(wl, 0)
    x = C.hidden_states(wl)
    sample = np.linspace(0, wl.n_tokens - 1, 32).astype(int)
    _check(wl, tags, x, sample=sample)


def test_prefill_matches_decode():
    wl = C.MIXTRAL_T8_SKEW
    tags = C.layer_tags(wl, 0)
    weights = S.device_layer_weights(wl, 0)
    L = S.make_layer(wl, tags, weights)
    x = C.hidden_states(wl)
    y_p, idx_p, _, prec_p = run_prefill(L, x, wl.d_model, wl.top_k)
    y_d, idx_d, _, prec_d = S.run_decode(L, torch.from_numpy(x).cuda(), wl.n_tokens,
                                         wl.d_model, wl.top_k)
    L.destroy()
    assert np.array_equal(idx_p, idx_d) and np.array_equal(prec_p, prec_d)
    assert S.normwise(y_p, y_d).max() <= S.TOL
