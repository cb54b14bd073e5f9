"""A layer stack captured in a HIP graph (torch.cuda.graph over the
library's calls on the capture stream) and replayed: every replay must
give the eager pass's results bit for bit (same kernels, fixed reduction
orders).  Replays are separated by the program's own eager work,
including other calls into the library, and by synchronisations, so a
captured node that depends on state left by an earlier call (a memset, a
stale counter) would show on a later replay."""
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


def _stack(T, prefill):
    import paper_2411_01433_amd as P
    wl = C.Workload(name=f"graph_t{T}", seed=11, d_model=256, d_ff=512, n_experts=8,
                    top_k=2, n_tokens=T, t1=1.0, t2=1.0,
                    fixed_tags=(C.TAG_FP16,) * 4 + (C.TAG_INT4,) * 2 + (C.TAG_INT2,) * 2)
    keep, layers = [], []
    for l in range(NL):
        w = S.device_layer_weights(wl, l)
        keep.append(w)
        layers.append(S.make_layer(wl, C.layer_tags(wl, l), w, max_tokens=T))
    d, K = wl.d_model, wl.top_k
    h0 = torch.from_numpy(C.hidden_states(wl).astype(np.float32)).cuda()
    x0 = torch.empty((T, d), dtype=torch.float16, device="cuda")
    P.rmsnorm(h0, x0)
    h = torch.empty_like(h0)
    xb = [torch.empty_like(x0), torch.empty_like(x0)]
    idx = torch.empty((NL, T, K), dtype=torch.int32, device="cuda")
    gw = torch.empty((NL, T, K), dtype=torch.float32, device="cuda")
    prec = torch.empty((NL, T, K), dtype=torch.int8, device="cuda")

    def step():
        h.copy_(h0)
        xb[0].copy_(x0)
        for l, L in enumerate(layers):
            call = L.prefill_residual if prefill else L.decode_step_residual
            call(xb[l % 2], h, xb[(l + 1) % 2], idx[l], gw[l], prec[l])

    def snapshot():
        torch.cuda.synchronize()
        return [t.cpu().numpy().copy() for t in (h, xb[NL % 2], idx, gw, prec)]

    return wl, layers, keep, step, snapshot


@pytest.mark.parametrize("T,prefill", [(1, False), (4, False), (9, False), (37, True)],
                         ids=["decode_t1", "decode_t4_dot2", "decode_t9_matrix_core",
                              "prefill_t37"])
def test_graph_replay_matches_eager(T, prefill):
    wl, layers, keep, step, snapshot = _stack(T, prefill)
    step()
    ref = snapshot()
    # eager work of the program between replays: another pass of the
    # library on other inputs, and plain torch kernels
    other = torch.from_numpy(C.hidden_states(wl, stream=5)).cuda()
    y_other = torch.empty((T, wl.d_model), dtype=torch.float32, device="cuda")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for r in range(4):
        (layers[0].prefill if prefill else layers[0].decode_step)(other, y_other)
        junk = torch.randn(1 << 16, device="cuda").sum()
        torch.cuda.synchronize()
        g.replay()
        got = snapshot()
        for name, a, b in zip(("h", "x_next", "idx", "w", "prec"), got, ref):
            assert np.array_equal(a, b), f"replay {r}: {name} differs from the eager pass"
        del junk
    print(f"graph_t{T}{'_prefill' if prefill else ''}: 4 replays bit-identical to the eager pass")
    for L in layers:
        L.destroy()
