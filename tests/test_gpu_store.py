"""Expert storage in pinned host memory, asynchronous loads of either
precision into device slots, and layers bound to those slots (Dynamic
Expert Loader, Section 3.2 / Fig. 6), through the C ABI.

Bar: loaded fp16 matrices and low-precision codes and scales are bit-exact
(equal to the device weights and to the library's own quantised copies);
a layer decoding through bound slots gives bit-identical outputs to the
same layer with resident copies, and matches the oracle (2e-3 normwise)."""
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


def _edge(bits):
    tags = ([C.TAG_FP16] * 2 + [C.TAG_INT4] * 2 + [C.TAG_MISS_INT4] * 2 if bits == 4 else
            [C.TAG_FP16] * 2 + [C.TAG_INT2] * 2 + [C.TAG_MISS_INT2] * 2)
    return C.Workload(name=f"store_{bits}", seed=40 + bits, d_model=320, d_ff=448, n_experts=6,
                      top_k=2, n_tokens=5, t1=0.4, t2=1.0, fixed_tags=tuple(tags))


@pytest.mark.parametrize("bits", [4, 2])
def test_loaded_copies_are_bit_exact(bits):
    import paper_2411_01433_amd as P
    wl = _edge(bits)
    wg, w1, w3, w2 = S.device_layer_weights(wl, 0)
    st = P.MoeStore(wl.d_model, wl.d_ff, wl.n_experts, bits)
    L = S.make_layer(wl, [C.TAG_INT4 if bits == 4 else C.TAG_INT2] * wl.n_experts,
                     (wg, w1, w3, w2))
    side = torch.cuda.Stream()
    for e in range(wl.n_experts):
        st.put(e, w1[e], w3[e], w2[e])
    for e in (0, 3, 5):
        hi = st.slots(True)
        q, s = st.slots(False)
        st.load(e, True, hi, stream=side)
        st.load(e, False, (q, s), stream=side)
        side.synchronize()
        for m, src in enumerate((w1[e], w3[e], w2[e])):
            assert torch.equal(hi[m].view(torch.int16), src.view(torch.int16))
            rq, rs = torch.empty_like(q[m]), torch.empty_like(s[m])
            L.export_packed(e, m, bits, rq, rs)
            torch.cuda.synchronize()
            assert torch.equal(q[m], rq)
            assert torch.equal(s[m].view(torch.int16), rs.view(torch.int16))
    L.destroy()
    st.destroy()


@pytest.mark.parametrize("bits", [4, 2])
def test_layer_bound_to_loaded_slots(bits):
    """Every expert is loaded into slots on a second stream (fp16 for FP16,
    the low copy for INT, both for MISS tags); an event orders the loads
    before the binds and the decode on the main stream."""
    import paper_2411_01433_amd as P
    wl = _edge(bits)
    tags = list(wl.fixed_tags)
    weights = S.device_layer_weights(wl, 0)
    wg, w1, w3, w2 = weights
    resident = S.make_layer(wl, tags, weights)
    # a second handle whose experts all come from the store
    st = P.MoeStore(wl.d_model, wl.d_ff, wl.n_experts, bits)
    for e in range(wl.n_experts):
        st.put(e, w1[e], w3[e], w2[e])
    side = torch.cuda.Stream()
    slots = []
    for e, tag in enumerate(tags):
        hi = st.slots(True) if tag in (C.TAG_FP16, C.TAG_MISS_INT4, C.TAG_MISS_INT2) else None
        lo = st.slots(False) if tag != C.TAG_FP16 else None
        if hi is not None:
            st.load(e, True, hi, stream=side)
        if lo is not None:
            st.load(e, False, lo, stream=side)
        slots.append((hi, lo))
    done = torch.cuda.Event()
    done.record(side)
    bound = P.MoeLayer(wl.d_model, wl.d_ff, wl.n_experts, wl.top_k, wl.n_tokens, wg, w1, w3, w2,
                       t1=wl.t1, t2=wl.t2)
    torch.cuda.current_stream().wait_event(done)
    for e, ((hi, lo), tag) in enumerate(zip(slots, tags)):
        bound.bind_expert(e, int(tag), w=hi, q=None if lo is None else lo[0],
                          s=None if lo is None else lo[1], low_bits=bits if lo else 0)
    rng = np.random.default_rng(9)
    x16 = rng.standard_normal((wl.n_tokens, wl.d_model)).astype(np.float16)
    xd = torch.from_numpy(x16).cuda()
    a = S.run_decode(resident, xd, wl.n_tokens, wl.d_model, wl.top_k)
    b = S.run_decode(bound, xd, wl.n_tokens, wl.d_model, wl.top_k)
    for u, v in zip(a, b):
        assert np.array_equal(np.asarray(u).view(np.uint8), np.asarray(v).view(np.uint8))
    y, idx, w, prec = b
    r, _ = S.check_routing(x16, C.router_weight(wl, 0), tags, wl.top_k, wl.t1, wl.t2,
                           idx, w, prec)
    y_ref = O.layer_output(x16, S.HostExperts(wl, 0, tags), r)
    assert S.normwise(y, y_ref).max() <= S.TOL
    assert set(np.unique(prec).tolist()) >= {O.PREC_HIGH, O.PREC_LOW}
    for h in (resident, bound):
        h.destroy()
    st.destroy()


def test_store_and_bind_errors():
    import paper_2411_01433_amd as P
    from paper_2411_01433_amd import binding as B
    wl = _edge(4)
    wg, w1, w3, w2 = S.device_layer_weights(wl, 0)
    st = P.MoeStore(wl.d_model, wl.d_ff, wl.n_experts, 4)
    with pytest.raises(B.MoeError) as ei:
        st.load(0, True, st.slots(True))  # never put
    assert ei.value.status == B.MOE_ESTATE
    L = P.MoeLayer(wl.d_model, wl.d_ff, wl.n_experts, wl.top_k, wl.n_tokens, wg, w1, w3, w2)
    q, s = st.slots(False)
    with pytest.raises(B.MoeError):
        L.bind_expert(0, C.TAG_MISS_INT4, q=q, s=s, low_bits=4)  # fp16 missing
    q2 = [torch.empty((r, c // 4), dtype=torch.uint8, device="cuda") for r, c in
          ((wl.d_ff, wl.d_model), (wl.d_ff, wl.d_model), (wl.d_model, wl.d_ff))]
    with pytest.raises(B.MoeError) as ei:
        L.bind_expert(0, C.TAG_INT4, q=q2, s=s, low_bits=2)      # width != the tag's
    assert ei.value.status == B.MOE_EINVAL
    L.bind_expert(0, C.TAG_INT4, q=q, s=s, low_bits=4)
    with pytest.raises(B.MoeError) as ei:
        L.set_expert_precision(0, C.TAG_MISS_INT4)               # no fp16 source left
    assert ei.value.status == B.MOE_ESTATE
    L.destroy()
    st.destroy()


@pytest.mark.parametrize("bits", [4, 2])
def test_rebind_rebuilds_quantised_copies(bits):
    """An expert's library-built low copy is quantised from the fp16 weights
    it had then; after the expert is bound to other fp16 weights, setting a
    low-precision tag again must rebuild the copy from the new weights."""
    wl = _edge(bits)
    wg, w1, w3, w2 = S.device_layer_weights(wl, 0)
    import paper_2411_01433_amd as P
    low = C.TAG_MISS_INT4 if bits == 4 else C.TAG_MISS_INT2
    L = P.MoeLayer(wl.d_model, wl.d_ff, wl.n_experts, wl.top_k, wl.n_tokens, wg, w1, w3, w2)
    L.set_expert_precision(0, low)            # copy of expert 0's weights
    L.bind_expert(0, C.TAG_FP16, w=[w1[1], w3[1], w2[1]])   # expert 0 now holds expert 1's
    L.set_expert_precision(0, low)            # must quantise expert 1's weights
    for m, src in enumerate((w1[1], w3[1], w2[1])):
        rows, cols = src.shape
        q = torch.empty((rows, cols * bits // 8), dtype=torch.uint8, device="cuda")
        s = torch.empty((rows, cols // 32), dtype=torch.float16, device="cuda")
        L.export_packed(0, m, bits, q, s)
        torch.cuda.synchronize()
        qr, sr = O.quantize(src.cpu().numpy(), bits)
        assert np.array_equal(q.cpu().numpy(), O.pack_codes(qr, bits))
        assert np.array_equal(s.cpu().numpy().view(np.uint16), sr.view(np.uint16))
    L.destroy()
