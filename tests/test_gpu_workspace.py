"""Layers of a stack running on one shared workspace
(moe_layer_share_workspace): results bit-identical to per-layer
workspaces on the dot2, matrix-core and prefill paths; the owner cannot
be destroyed while others share it; mismatched layers are refused."""
import numpy as np
import pytest

from synth import configs as C

import gpu_support as S

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

NL = 3


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2411_01433_amd as P
    P.lib()
    yield


def _workload(T, f=512):
    return C.Workload(name=f"ws_t{T}", seed=13, d_model=256, d_ff=f, n_experts=8, top_k=2,
                      n_tokens=T, t1=1.0, t2=1.0,
                      fixed_tags=(C.TAG_FP16,) * 4 + (C.TAG_INT4,) * 2 + (C.TAG_INT2,) * 2)


def _run(layers, wl, prefill):
    import paper_2411_01433_amd as P
    T, d, K = wl.n_tokens, wl.d_model, wl.top_k
    h = torch.from_numpy(C.hidden_states(wl).astype(np.float32)).cuda()
    xb = [torch.empty((T, d), dtype=torch.float16, device="cuda") for _ in range(2)]
    P.rmsnorm(h, xb[0])
    idx = torch.empty((NL, T, K), dtype=torch.int32, device="cuda")
    gw = torch.empty((NL, T, K), dtype=torch.float32, device="cuda")
    prec = torch.empty((NL, T, K), dtype=torch.int8, device="cuda")
    for l, L in enumerate(layers):
        call = L.prefill_residual if prefill else L.decode_step_residual
        call(xb[l % 2], h, xb[(l + 1) % 2], idx[l], gw[l], prec[l])
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in (h, xb[NL % 2], idx, gw, prec)]


@pytest.mark.parametrize("T,prefill", [(1, False), (4, False), (9, False), (37, True)],
                         ids=["decode_t1", "decode_t4_dot2", "decode_t9_matrix_core",
                              "prefill_t37"])
def test_shared_workspace_matches_own(T, prefill):
    wl = _workload(T)
    keep, layers = [], []
    for l in range(NL):
        w = S.device_layer_weights(wl, l)
        keep.append(w)
        layers.append(S.make_layer(wl, C.layer_tags(wl, l), w, max_tokens=T))
    ref = _run(layers, wl, prefill)
    for L in layers[1:]:
        L.share_workspace(layers[0])
    layers[2].share_workspace(layers[0])  # again: a no-op
    for rep in range(2):
        got = _run(layers, wl, prefill)
        for name, a, b in zip(("h", "x_next", "idx", "w", "prec"), got, ref):
            assert np.array_equal(a, b), f"pass {rep}: {name} differs with the shared workspace"
    import paper_2411_01433_amd as P
    with pytest.raises(P.MoeError) as e:
        layers[0].destroy()  # others still run on its workspace
    assert e.value.status == P.binding.MOE_ESTATE
    with pytest.raises(P.MoeError):
        layers[0].share_workspace(layers[1])  # its workspace is shared: cannot move
    for L in layers[1:]:
        L.destroy()
    layers[0].destroy()
    print(f"ws_t{T}{'_prefill' if prefill else ''}: {NL} layers on one workspace, bit-identical")


def test_share_refuses_mismatched_layers():
    import paper_2411_01433_amd as P
    a_wl, b_wl = _workload(4), _workload(4, f=1024)
    wa, wb = S.device_layer_weights(a_wl, 0), S.device_layer_weights(b_wl, 0)
    A = S.make_layer(a_wl, C.layer_tags(a_wl, 0), wa)
    Bl = S.make_layer(b_wl, C.layer_tags(b_wl, 0), wb)
    with pytest.raises(P.MoeError) as e:
        Bl.share_workspace(A)
    assert e.value.status == P.binding.MOE_EINVAL
    Bl.destroy()
    A.destroy()
