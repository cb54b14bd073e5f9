"""32-layer stacks with the pre-norm residual glue between layers, checked
teacher-forced: the whole stack runs on the device, and at sampled layers
the oracle takes the device's own layer input (x_l, h_l) and must reproduce
that layer's routing, its increment y_l = h_{l+1} - h_l and the next input
x_{l+1} = fp16(rmsnorm(h_{l+1})).  Free-running agreement over 32 layers is
not a parity bar: top-k is discontinuous, so a near-tie in one layer may
legitimately send the two runs down different experts afterwards."""
import gc

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


def _run_stack(wl, check_layers):
    """Run the stack once; return per checked layer the device's
    (x_l, h_l, h_{l+1}, x_{l+1}, idx, w, prec) on the host."""
    T, K, d, NL = wl.n_tokens, wl.top_k, wl.d_model, wl.n_layers
    layers, keep = [], []
    for l in range(NL):
        w = S.device_layer_weights(wl, l)
        keep.append(w)
        layers.append(S.make_layer(wl, C.layer_tags(wl, l), w, max_tokens=T))
    h0 = C.hidden_states(wl).astype(np.float32)
    h = torch.from_numpy(h0).cuda()
    xb = [torch.from_numpy(O.rmsnorm(h0.astype(np.float64)).astype(np.float16)).cuda(),
          torch.empty((T, d), dtype=torch.float16, device="cuda")]
    idx = torch.empty((T, K), dtype=torch.int32, device="cuda")
    gw = torch.empty((T, K), dtype=torch.float32, device="cuda")
    prec = torch.empty((T, K), dtype=torch.int8, device="cuda")
    seen = {}
    hmax = 0.0
    for l, L in enumerate(layers):
        xi, xo = xb[l % 2], xb[(l + 1) % 2]
        if l in check_layers:
            torch.cuda.synchronize()
            before = (xi.cpu().numpy(), h.cpu().numpy())
        if wl.mode == "prefill":
            L.prefill_residual(xi, h, xo, idx, gw, prec)
        else:
            L.decode_step_residual(xi, h, xo, idx, gw, prec)
        if l in check_layers:
            torch.cuda.synchronize()
            seen[l] = before + (h.cpu().numpy(), xo.cpu().numpy(), idx.cpu().numpy(),
                                gw.cpu().numpy(), prec.cpu().numpy())
    torch.cuda.synchronize()
    hmax = float(h.abs().max().item())
    finite = bool(torch.isfinite(h).all().item())
    for L in layers:
        L.destroy()
    del layers, keep, h, xb
    gc.collect()
    torch.cuda.empty_cache()
    return seen, hmax, finite


def _check_layer(wl, l, rec, rows):
    x_l, h_l, h_n, x_n, idx, w, prec = rec
    tags = C.layer_tags(wl, l)
    r, flags = S.check_routing(x_l[rows], C.router_weight(wl, l), tags, wl.top_k,
                               wl.t1, wl.t2, idx[rows], w[rows], prec[rows])
    y_ref = O.layer_output(x_l[rows], S.HostExperts(wl, l, tags), r)
    h_ref, x_ref = O.residual_step(h_l[rows].astype(np.float64), y_ref, O.RMS_EPS)
    inc = h_n[rows].astype(np.float64) - h_l[rows].astype(np.float64)
    e_inc = S.normwise(inc, y_ref).max()
    e_h = S.normwise(h_n[rows], h_ref).max()
    e_x = S.normwise(x_n[rows], O.rmsnorm(h_ref)).max()
    print(f"{wl.name} layer {l}: increment {e_inc:.2e}, h {e_h:.2e}, x_next {e_x:.2e}, "
          f"flags {len(flags)}")
    assert e_inc <= S.TOL and e_h <= S.TOL and e_x <= S.TOL
    return r


def test_phi_stack32_decode_teacher_forced():
    """Phi-MoE-shaped decode stack: 32 layers, 4 tokens per step, per-layer
    half fp16 / half int4 maps; the multi-token (matrix-core) decode path."""
    wl = C.PHI_STACK
    check = [0, 1, 15, wl.n_layers - 1]
    seen, hmax, finite = _run_stack(wl, set(check))
    print(f"final max|h| {hmax:.3f}")
    assert finite and hmax < 1e3
    for l in check:
        _check_layer(wl, l, seen[l], np.arange(wl.n_tokens))
        gc.collect()


def test_mixtral_stack32_prefill_teacher_forced():
    """Mixtral-shaped prefill stack: 32 layers of 512 tokens, per-layer
    4:3:1 maps; 24 sampled tokens at three layers."""
    wl = C.MIXTRAL_PREFILL
    check = [0, wl.n_layers // 2, wl.n_layers - 1]
    seen, hmax, finite = _run_stack(wl, set(check))
    print(f"final max|h| {hmax:.3f}")
    assert finite and hmax < 1e3
    rows = np.linspace(0, wl.n_tokens - 1, 24).astype(int)
    for l in check:
        r = _check_layer(wl, l, seen[l], rows)
        assert np.all(r.prec != O.PREC_SKIP)
        gc.collect()
