"""Helpers shared by the GPU parity tests, the smoke check and the bench:
device weights from the keyed generator, lazy host experts for the oracle,
and the comparison of the library's outputs with the oracle."""
from __future__ import annotations

import numpy as np

from oracle import moe_oracle as O
from synth import configs as C

TOL = 2e-3          # normwise relative error per token row
W_ATOL = 1e-5       # gate values (fp32 softmax vs float64)
TIE_REL = 1e-4      # logit gap treated as a near-tie
RULE_EPS = 1e-5     # score this close to a threshold: either side accepted


def device_layer_weights(wl: C.Workload, layer: int, device="cuda"):
    """(wg, w1[], w3[], w2[]) of one layer as fp16 device tensors."""
    import torch
    from synth import gpu as G
    wg = torch.from_numpy(C.router_weight(wl, layer)).to(device)
    mats = {}
    for which, shape in (("w1", (wl.d_ff, wl.d_model)), ("w3", (wl.d_ff, wl.d_model)),
                         ("w2", (wl.d_model, wl.d_ff))):
        mats[which] = []
        for e in range(wl.n_experts):
            t = torch.empty(shape, dtype=torch.float16, device=device)
            G.normal_fp16_(t, C.expert_tensor_key(wl, layer, e, which), C.W_STD)
            mats[which].append(t)
    return wg, mats["w1"], mats["w3"], mats["w2"]


def rmsnorm_device(h, x):
    """The library's RMSNorm of the residual glue: x = fp16(rmsnorm(h))."""
    import paper_2411_01433_amd as P
    P.rmsnorm(h, x, O.RMS_EPS)


def make_layer(wl: C.Workload, tags, weights, max_tokens=None, t1=None, t2=None):
    import paper_2411_01433_amd as P
    wg, w1, w3, w2 = weights
    L = P.MoeLayer(wl.d_model, wl.d_ff, wl.n_experts, wl.top_k,
                   max_tokens or wl.n_tokens, wg, w1, w3, w2,
                   t1=wl.t1 if t1 is None else t1, t2=wl.t2 if t2 is None else t2)
    for e, tag in enumerate(tags):
        if int(tag) != C.TAG_FP16:
            L.set_expert_precision(e, int(tag))
    return L


class HostExperts:
    """experts[e] -> oracle Expert of one layer, generated on the host."""

    def __init__(self, wl: C.Workload, layer: int, tags):
        self.wl, self.layer, self.tags = wl, layer, list(tags)
        self._c = {}

    def __getitem__(self, e):
        if e not in self._c:
            w = [C.expert_weight(self.wl, self.layer, e, m) for m in ("w1", "w3", "w2")]
            self._c[e] = O.Expert(w[0], w[1], w[2], int(self.tags[e]))
        return self._c[e]

    def __len__(self):
        return self.wl.n_experts


def normwise(got, ref):
    """max_j |got - ref| / max_j |ref| per row (rows of zeros: absolute)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.abs(ref).max(axis=-1)
    num = np.abs(got - ref).max(axis=-1)
    return np.where(den > 0, num / np.where(den > 0, den, 1), num)


def check_routing(x16, wg16, tags, K, t1, t2, g_idx, g_w, g_prec):
    """Compare routing outputs with the oracle.  Returns the oracle routing
    to evaluate Eq. 1 with (near-ties resolved to the library's choice) and
    the list of flagged (token, reason)."""
    E = wg16.shape[0]
    r = O.route(x16, wg16, tags, K, t1, t2)
    T = r.idx.shape[0]
    forced = r.idx.copy()
    flags = []
    for t in range(T):
        srt = np.sort(r.logits[t])[::-1]
        margin = TIE_REL * max(1.0, abs(srt[K - 1]))
        amb = (K < E and srt[K - 1] - srt[K] <= margin) or any(
            srt[i] - srt[i + 1] <= margin for i in range(K - 1))
        if np.array_equal(g_idx[t], r.idx[t]):
            continue
        assert amb, f"token {t}: top-k {g_idx[t]} != oracle {r.idx[t]} (no near-tie)"
        sel = [int(e) for e in g_idx[t]]
        assert len(set(sel)) == K and all(0 <= e < E for e in sel)
        assert all(r.logits[t, e] >= srt[K - 1] - margin for e in sel)
        forced[t] = sel
        flags.append((t, "topk near-tie"))
    r2 = O.route(x16, wg16, tags, K, t1, t2, forced_idx=forced)
    np.testing.assert_allclose(g_w, r2.w, atol=W_ATOL, rtol=0)
    prec = r2.prec.copy()
    for t in range(T):
        s = O.unimportance_scores(r2.w[t])
        for k in range(K):
            if int(g_prec[t, k]) == int(prec[t, k]):
                continue
            near = min(abs(s[k] - t1), abs(s[k] - t2)) <= RULE_EPS
            assert near, (f"token {t} slot {k}: precision {g_prec[t, k]} != "
                          f"oracle {prec[t, k]} (score {s[k]:.6f})")
            prec[t, k] = int(g_prec[t, k])
            flags.append((t, "threshold near-tie"))
    r2.prec = prec
    return r2, flags


def run_decode(L, x_dev, T, d, K, residual_h=None):
    import torch
    dev = x_dev.device
    idx = torch.empty((T, K), dtype=torch.int32, device=dev)
    w = torch.empty((T, K), dtype=torch.float32, device=dev)
    prec = torch.empty((T, K), dtype=torch.int8, device=dev)
    if residual_h is None:
        y = torch.empty((T, d), dtype=torch.float32, device=dev)
        L.decode_step(x_dev, y, idx, w, prec)
        torch.cuda.synchronize()
        return y.cpu().numpy(), idx.cpu().numpy(), w.cpu().numpy(), prec.cpu().numpy()
    xn = torch.empty((T, d), dtype=torch.float16, device=dev)
    L.decode_step_residual(x_dev, residual_h, xn, idx, w, prec)
    torch.cuda.synchronize()
    return xn.cpu().numpy(), idx.cpu().numpy(), w.cpu().numpy(), prec.cpu().numpy()
