"""moe_decode_step_noalloc (the allocation-free decode step, whose workspace
is a static device array) against moe_decode_step through the C ABI.

Bar: both entry points run the same kernels, so their outputs are
bit-identical; the outputs also match the oracle (routing exact up to the
flagged near-ties, 2e-3 normwise).  Two calls in a row on the shared
scratch, the second with fewer tokens, switch between the matrix-core and
the one/two-token kernels; a step too large for the scratch is refused."""
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


def _outs(T, d, K):
    return (torch.empty((T, d), dtype=torch.float32, device="cuda"),
            torch.empty((T, K), dtype=torch.int32, device="cuda"),
            torch.empty((T, K), dtype=torch.float32, device="cuda"),
            torch.empty((T, K), dtype=torch.int8, device="cuda"))


def _same(a, b):
    return all(torch.equal(u.view(torch.uint8), v.view(torch.uint8)) for u, v in zip(a, b))


def _compare(wl, L, x16, experts):
    T, d, K = x16.shape[0], wl.d_model, wl.top_k
    xd = torch.from_numpy(np.ascontiguousarray(x16)).cuda()
    ref, got = _outs(T, d, K), _outs(T, d, K)
    L.decode_step(xd, *ref)
    L.decode_step_noalloc(xd, *got)
    torch.cuda.synchronize()
    assert _same(ref, got), f"{wl.name} T={T}: noalloc differs from decode_step"
    y, idx, w, prec = (t.cpu().numpy() for t in got)
    r, _ = S.check_routing(x16, C.router_weight(wl, 0), list(wl.fixed_tags or C.layer_tags(wl, 0)),
                           K, wl.t1, wl.t2, idx, w, prec)
    err = S.normwise(y, O.layer_output(x16, experts, r)).max()
    print(f"{wl.name} T={T}: bit-identical to decode_step, max normwise err {err:.2e}")
    assert err <= S.TOL


MIXED = (C.TAG_INT8, C.TAG_MISS_INT8_INT2, C.TAG_FP16, C.TAG_MISS_INT4,
         C.TAG_INT4, C.TAG_INT2, C.TAG_MISS_INT2, C.TAG_FP16)


def test_noalloc_matches_decode_step_ragged():
    wl = C.Workload(name="noalloc_ragged", seed=71, d_model=320, d_ff=448, n_experts=8,
                    top_k=2, n_tokens=9, t1=0.6, t2=0.9, fixed_tags=MIXED, router_scale=8)
    L = S.make_layer(wl, MIXED, S.device_layer_weights(wl, 0), max_tokens=16)
    experts = S.HostExperts(wl, 0, MIXED)
    rng = np.random.default_rng(5)
    for T in (9, 2):      # second call smaller, other kernel family
        _compare(wl, L, rng.standard_normal((T, wl.d_model)).astype(np.float16), experts)
    L.destroy()


def test_noalloc_matches_decode_step_mixtral():
    wl = C.MIXTRAL_T8_SKEW
    tags = C.layer_tags(wl, 0)
    L = S.make_layer(wl, tags, S.device_layer_weights(wl, 0), max_tokens=64)
    experts = S.HostExperts(wl, 0, tags)
    x = np.concatenate([C.hidden_states(wl, stream=s) for s in range(3)])
    for T in (16, 1):
        _compare(wl, L, np.ascontiguousarray(x[:T]), experts)
    L.destroy()


def test_noalloc_refuses_steps_beyond_the_scratch():
    from paper_2411_01433_amd import binding as B
    wl = C.Workload(name="noalloc_big", seed=72, d_model=64, d_ff=8256, n_experts=8,
                    top_k=8, n_tokens=64, fixed_tags=(C.TAG_FP16,) * 8)
    L = S.make_layer(wl, wl.fixed_tags, S.device_layer_weights(wl, 0), max_tokens=64)
    rng = np.random.default_rng(6)
    x16 = rng.standard_normal((64, wl.d_model)).astype(np.float16)
    xd = torch.from_numpy(x16).cuda()
    with pytest.raises(B.MoeError) as ei:
        L.decode_step_noalloc(xd, *_outs(64, wl.d_model, wl.top_k))
    assert ei.value.status == B.MOE_EINVAL and "scratch" in str(ei.value)
    _compare(wl, L, x16[:32], S.HostExperts(wl, 0, wl.fixed_tags))   # fits: 32 tokens
    L.destroy()
