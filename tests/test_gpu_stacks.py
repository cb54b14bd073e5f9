"""32-layer stacks with the pre-norm residual glue between layers.

The whole stack runs on the device once.  Every layer's input x_l and its
routing outputs (top-k indices, gate values, Eq. 2 precisions) are kept,
and the routing of EVERY token of EVERY layer is checked against the
oracle taking the device's own x_l (teacher-forced): indices and
precisions exact up to the flagged near-ties of the comparison rules, gate
values within 1e-5.  The fp64 expert FFN is expensive, so the layer output
(the increment y_l = h_{l+1} - h_l and the next input x_{l+1} =
fp16(rmsnorm(h_{l+1}))) is checked at sampled layers and tokens.
Free-running agreement over 32 layers is not a parity bar: top-k is
discontinuous, so a near-tie in one layer may legitimately send the two
runs down different experts afterwards."""
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


def _run_stack(wl, ffn_layers):
    """Run the stack once.  Returns every layer's device input x_l and
    routing (idx, w, prec) on the host, and for the layers in ffn_layers
    the residual stream before and after the layer."""
    T, K, d, NL = wl.n_tokens, wl.top_k, wl.d_model, wl.n_layers
    layers, keep = [], []
    for l in range(NL):
        w = S.device_layer_weights(wl, l)
        keep.append(w)
        layers.append(S.make_layer(wl, C.layer_tags(wl, l), w, max_tokens=T))
    h = torch.from_numpy(C.hidden_states(wl).astype(np.float32)).cuda()
    # x[l] is layer l's input; the library's own RMSNorm forms x[0]
    xs = torch.empty((NL + 1, T, d), dtype=torch.float16, device="cuda")
    S.rmsnorm_device(h, xs[0])
    idx = torch.empty((NL, T, K), dtype=torch.int32, device="cuda")
    gw = torch.empty((NL, T, K), dtype=torch.float32, device="cuda")
    prec = torch.empty((NL, T, K), dtype=torch.int8, device="cuda")
    h_before, h_after = {}, {}
    for l, L in enumerate(layers):
        if l in ffn_layers:
            h_before[l] = h.clone()
        if wl.mode == "prefill":
            L.prefill_residual(xs[l], h, xs[l + 1], idx[l], gw[l], prec[l])
        else:
            L.decode_step_residual(xs[l], h, xs[l + 1], idx[l], gw[l], prec[l])
        if l in ffn_layers:
            h_after[l] = h.clone()
    torch.cuda.synchronize()
    rec = {"x": xs.cpu().numpy(), "idx": idx.cpu().numpy(), "w": gw.cpu().numpy(),
           "prec": prec.cpu().numpy(),
           "h_before": {l: v.cpu().numpy() for l, v in h_before.items()},
           "h_after": {l: v.cpu().numpy() for l, v in h_after.items()},
           "hmax": float(h.abs().max().item()), "finite": bool(torch.isfinite(h).all().item())}
    for L in layers:
        L.destroy()
    del layers, keep, h, xs, h_before, h_after
    gc.collect()
    torch.cuda.empty_cache()
    return rec


def _check_all_routing(wl, rec):
    """Routing of every token of every layer against the oracle; returns the
    oracle routings (near-ties resolved to the device's choice)."""
    routes, n_flag = [], 0
    for l in range(wl.n_layers):
        r, flags = S.check_routing(rec["x"][l], C.router_weight(wl, l), C.layer_tags(wl, l),
                                   wl.top_k, wl.t1, wl.t2, rec["idx"][l], rec["w"][l],
                                   rec["prec"][l])
        routes.append(r)
        n_flag += len(flags)
    n = wl.n_layers * wl.n_tokens
    print(f"{wl.name}: routing exact on {n} routed token-layers "
          f"({n * wl.top_k} slots), {n_flag} flagged near-ties")
    return routes


def _check_ffn(wl, l, rec, r, rows):
    x_l = rec["x"][l][rows]
    h_l, h_n, x_n = rec["h_before"][l][rows], rec["h_after"][l][rows], rec["x"][l + 1][rows]
    tags = C.layer_tags(wl, l)
    rr = O.Routing(idx=r.idx[rows], w=r.w[rows], prec=r.prec[rows], logits=r.logits[rows])
    y_ref = O.layer_output(x_l, S.HostExperts(wl, l, tags), rr)
    h_ref, _ = O.residual_step(h_l.astype(np.float64), y_ref, O.RMS_EPS)
    inc = h_n.astype(np.float64) - h_l.astype(np.float64)
    e_inc = S.normwise(inc, y_ref).max()
    e_h = S.normwise(h_n, h_ref).max()
    e_x = S.normwise(x_n, O.rmsnorm(h_ref)).max()
    print(f"{wl.name} layer {l}: increment {e_inc:.2e}, h {e_h:.2e}, x_next {e_x:.2e} "
          f"on {len(rows)} tokens")
    assert e_inc <= S.TOL and e_h <= S.TOL and e_x <= S.TOL


def test_phi_stack32_decode_teacher_forced():
    """Phi-MoE-shaped decode stack: 32 layers, 4 tokens per step, per-layer
    half fp16 / half int4 maps; the multi-token (matrix-core) decode path.
    Routing on all 128 token-layers; the FFN at 4 layers, every token."""
    wl = C.PHI_STACK
    ffn = [0, 1, 15, wl.n_layers - 1]
    rec = _run_stack(wl, set(ffn))
    print(f"final max|h| {rec['hmax']:.3f}")
    assert rec["finite"] and rec["hmax"] < 1e3
    routes = _check_all_routing(wl, rec)
    for l in ffn:
        _check_ffn(wl, l, rec, routes[l], np.arange(wl.n_tokens))
        gc.collect()


def test_mixtral_stack32_prefill_teacher_forced():
    """Mixtral-shaped prefill stack: 32 layers of 512 tokens, per-layer
    4:3:1 maps.  Routing on all 16,384 token-layers; the FFN on 24 sampled
    tokens at three layers."""
    wl = C.MIXTRAL_PREFILL
    ffn = [0, wl.n_layers // 2, wl.n_layers - 1]
    rec = _run_stack(wl, set(ffn))
    print(f"final max|h| {rec['hmax']:.3f}")
    assert rec["finite"] and rec["hmax"] < 1e3
    routes = _check_all_routing(wl, rec)
    for r in routes:
        assert np.all(r.prec != O.PREC_SKIP)
    rows = np.linspace(0, wl.n_tokens - 1, 24).astype(int)
    for l in ffn:
        _check_ffn(wl, l, rec, routes[l], rows)
        gc.collect()
