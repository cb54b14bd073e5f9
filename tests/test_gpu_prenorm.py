"""moe_decode_step_prenorm: the decode step that forms its own input
x = fp16(rmsnorm(h)) from the residual stream h, then h += MoE(x).

A stack run with it must equal, bit for bit, the same stack run as
moe_rmsnorm followed by moe_decode_step_residual per layer (the residual
glue of the stack workloads): every layer's x, top-k indices, gate values
and Eq. 2 precisions, and the residual stream after every layer.  Cases
cover the dot2 kernels with the norm formed inside the router, the
matrix-core kernels (more pairs than experts) with the norm in the router,
and steps whose activations do not fit the router's LDS (the norm kernel
runs first): many tokens, and d_model above 4096."""
import dataclasses

import numpy as np
import pytest

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


def _wl(name, seed, d, f, E, K, T, layers, recipe="431"):
    return C.Workload(name=name, seed=seed, d_model=d, d_ff=f, n_experts=E, top_k=K,
                      n_tokens=T, n_layers=layers, residual=True, tag_recipe=recipe)


CASES = [
    # Phi-shaped layers, 4 tokens: dot2 kernels, norm inside the router
    dataclasses.replace(C.PHI_STACK, n_layers=3),
    # 8 tokens over 8 experts (16 pairs): matrix-core kernels, norm in the router
    _wl("prenorm_mc_t8", 61, 1024, 1536, 8, 2, 8, 3),
    # 16 tokens x 4096: activations above the router's LDS, norm kernel first
    _wl("prenorm_t16_d4096", 62, 4096, 512, 8, 2, 16, 2),
    # d_model 8192: above the router's register chunks, norm kernel first
    _wl("prenorm_d8192", 63, 8192, 256, 4, 2, 2, 2, "half"),
    # one token: dot2 one-token kernels
    _wl("prenorm_t1", 64, 2048, 1024, 8, 2, 1, 3),
]


@pytest.mark.parametrize("wl", CASES, ids=[w.name for w in CASES])
def test_prenorm_stack_matches_residual_glue(wl):
    import paper_2411_01433_amd as P
    T, K, d, NL = wl.n_tokens, wl.top_k, wl.d_model, wl.n_layers
    keep, layers = [], []
    for l in range(NL):
        w = S.device_layer_weights(wl, l)
        keep.append(w)
        layers.append(S.make_layer(wl, C.layer_tags(wl, l), w, max_tokens=T))
    h0 = torch.from_numpy(C.hidden_states(wl).astype(np.float32)).cuda()

    def outs():
        return (torch.empty((NL, T, K), dtype=torch.int32, device="cuda"),
                torch.empty((NL, T, K), dtype=torch.float32, device="cuda"),
                torch.empty((NL, T, K), dtype=torch.int8, device="cuda"))

    # residual glue: x_0 = rmsnorm(h), then per layer h += MoE(x_l), x_{l+1} = rmsnorm(h)
    ha = h0.clone()
    xa = torch.empty((NL + 1, T, d), dtype=torch.float16, device="cuda")
    P.rmsnorm(ha, xa[0])
    ia, wa, pa = outs()
    hs_a = []
    for l, L in enumerate(layers):
        L.decode_step_residual(xa[l], ha, xa[l + 1], ia[l], wa[l], pa[l])
        hs_a.append(ha.clone())
    # pre-norm steps on the stream itself
    hb = h0.clone()
    xb = torch.empty((NL, T, d), dtype=torch.float16, device="cuda")
    ib, wb, pb = outs()
    hs_b = []
    for l, L in enumerate(layers):
        L.decode_step_prenorm(hb, xb[l], ib[l], wb[l], pb[l])
        hs_b.append(hb.clone())
    torch.cuda.synchronize()
    for l in range(NL):
        assert torch.equal(xb[l].view(torch.int16), xa[l].view(torch.int16)), f"x of layer {l}"
        assert torch.equal(ib[l], ia[l]) and torch.equal(pb[l], pa[l]), f"routing of layer {l}"
        assert torch.equal(wb[l].view(torch.int32), wa[l].view(torch.int32)), f"gates of layer {l}"
        assert torch.equal(hs_b[l].view(torch.int32), hs_a[l].view(torch.int32)), f"h after layer {l}"
    assert bool(torch.isfinite(hb).all())
    print(f"{wl.name}: {NL} layers x {T} tokens bit-identical")
    for L in layers:
        L.destroy()


def test_prenorm_rejects_bad_arguments():
    import paper_2411_01433_amd as P
    wl = _wl("prenorm_args", 65, 256, 512, 4, 2, 2, 1)
    w = S.device_layer_weights(wl, 0)
    L = S.make_layer(wl, C.layer_tags(wl, 0), w, max_tokens=2)
    h = torch.zeros((2, 256), dtype=torch.float32, device="cuda")
    x = torch.empty((2, 256), dtype=torch.float16, device="cuda")
    with pytest.raises(ValueError):
        L.decode_step_prenorm(h.half(), x)          # h must be fp32
    with pytest.raises(ValueError):
        L.decode_step_prenorm(h, x[:1])             # x shape
    h3 = torch.zeros((3, 256), dtype=torch.float32, device="cuda")
    x3 = torch.empty((3, 256), dtype=torch.float16, device="cuda")
    with pytest.raises(RuntimeError):
        L.decode_step_prenorm(h3, x3)               # above max_tokens
    L.destroy()
