"""rbq_decode_step (the whole decode step in one call) against the five
separate calls it replaces: same inputs, bitwise the same outputs, also when
the call is repeated on the same workspace and when it is replayed from a HIP
graph. The separate calls are checked against the oracle elsewhere; the
end-to-end oracle tests run the fused step."""
import numpy as np
import pytest
import torch

from workloads import gen
import parity_util as pu

pytestmark = pytest.mark.gpu

# (B, Hq, Hkv, n, w, kv dtype, p, flush, seed)
CASES = [
    (1, 32, 8, 5000, 256, "bf16", 0.95, True, 1),     # the 8B-model GQA shape, ragged n
    (2, 8, 2, 3000, 40, "bf16", 0.9, True, 2),
    (1, 16, 1, 2049, 0, "bf16", 0.8, False, 3),       # G = 16, no window
    (1, 1, 1, 700, 33, "f32", 0.9, True, 4),          # fp32 K/V, one head
    (2, 8, 8, 4100, 300, "bf16", 1.0, True, 5),       # p = 1 selects every key
    (1, 8, 2, 0, 64, "bf16", 0.9, True, 6),           # no indexed key: the window only
    (1, 4, 1, 10000, 17, "bf16", 0.5, True, 7),
    (1, 16, 2, 6000, 64, "bf16", 0.9, True, 8),       # G = 8: the matrix-core scan
    (1, 32, 8, 65536, 64, "bf16", 0.9, True, 9),      # G = 4, two keys per lane: the matrix-core scan
]


@pytest.fixture(scope="module")
def pipeline():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2606_31519_amd import pipeline as pl
    return pl


def _state(pipeline, case):
    B, Hq, Hkv, n, w, dt, p, flush, seed = case
    wl = gen.random_case(B, Hq, Hkv, n, seed=seed, kv_dtype=dt, w=w, c_q_scale=0.5)
    st = pipeline.DecodeState.from_workload(wl)
    if n > 0:                 # (a centroid of no keys is undefined: c_k stays zero)
        st.build_index()
    return st


def _outputs(st):
    torch.cuda.synchronize()
    n = st.n
    cnt = st.sel_count.cpu().numpy()
    sel = st.sel_idx.cpu().numpy()
    o = {name: getattr(st, name).cpu().numpy().copy() for name in
         ("qplanes", "qscal", "sel_count", "out", "lse", "codes", "kfac")}
    o["scores"] = st.scores[:, :, :n].cpu().numpy().copy()
    o["sel"] = [sel[b, h, :cnt[b, h]].copy() for b in range(st.B) for h in range(st.Hq)]
    return o


def _same(a, b):
    assert a.keys() == b.keys()
    for k in a:
        if k == "sel":
            assert len(a[k]) == len(b[k]) and all(np.array_equal(x, y) for x, y in zip(a[k], b[k])), k
        else:
            assert a[k].shape == b[k].shape and np.array_equal(a[k].view(np.uint8), b[k].view(np.uint8)), k


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"B{c[0]}-Hq{c[1]}-Hkv{c[2]}-n{c[3]}-w{c[4]}-{c[5]}-p{c[6]}")
def test_fused_step_matches_separate_calls(pipeline, case):
    p, flush = case[6], case[7]
    print("case", case, flush=True)
    ref = _state(pipeline, case)
    ref.step_calls(p, flush=flush)
    want = _outputs(ref)
    st = _state(pipeline, case)
    st.step(p, flush=flush)
    _same(_outputs(st), want)
    if case[3] > 0:
        assert want["sel_count"].min() >= 1
    # the same workspace again: nothing is left over from the first call
    st.step(p, flush=flush)
    _same(_outputs(st), want)


def test_fused_step_graph_replays(pipeline):
    case = CASES[0]
    p = case[6]
    ref = _state(pipeline, case)
    ref.step_calls(p)
    want = _outputs(ref)
    st = _state(pipeline, case)
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        st.step(p)
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=s):
            st.step(p)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for _ in range(3):
        st.out.zero_()
        st.sel_count.zero_()
        torch.cuda.synchronize()
        g.replay()
        _same(_outputs(st), want)
        st.step(p)            # eager work between the replays
        _same(_outputs(st), want)


def test_index_build_beside_prefill_attention(pipeline):
    """The prefill index build on a second stream, started together with a
    causal attention over the same context (as bench.py times it), writes the
    same centroid, codes and factors as a build alone, and those match the
    oracle's encoding of the same keys."""
    from torch.nn.attention import SDPBackend, sdpa_kernel
    case = (1, 8, 2, 4096, 0, "bf16", 0.9, False, 8)
    ref = _state(pipeline, case)
    torch.cuda.synchronize()
    want = [t.cpu().numpy().copy() for t in (ref.c_k, ref.codes, ref.kfac)]
    st = _state(pipeline, case)
    for t in (st.c_k, st.codes, st.kfac):
        t.zero_()
    q = torch.randn(1, st.Hq, st.n, st.D, device="cuda", dtype=torch.bfloat16)
    k = st.K[:, :, :st.n].repeat_interleave(st.Hq // st.Hkv, dim=1).contiguous()
    side, main = torch.cuda.Stream(), torch.cuda.current_stream()
    side.wait_stream(main)
    with sdpa_kernel([SDPBackend.FLASH_ATTENTION]):
        torch.nn.functional.scaled_dot_product_attention(q, k, k, is_causal=True)
    with torch.cuda.stream(side):
        st.build_index()
    main.wait_stream(side)
    torch.cuda.synchronize()
    for a, b in zip(want, (st.c_k, st.codes, st.kfac)):
        assert np.array_equal(a.view(np.uint8), b.cpu().numpy().view(np.uint8))
    # and the build itself against the oracle's Algorithm 1 on the same keys
    B, Hq, Hkv, n, w, dt, p, flush, seed = case
    wl = gen.random_case(B, Hq, Hkv, n, seed=seed, kv_dtype=dt, w=w, c_q_scale=0.5)
    codes, kfac, ck = st.codes.cpu().numpy().view(np.uint32), st.kfac.cpu().numpy(), st.c_k.cpu().numpy()
    for hk in range(Hkv):
        pu.check_encode_group(codes[0, hk, :n], kfac[0, hk, :n], ck[0, hk], wl.K_f32(0, hk, slice(0, n)), wl.P,
                              wl.c_q[0, hk])


def test_fused_step_any_workspace_contents(pipeline):
    """The step's workspace needs no initialisation and carries nothing from
    one call to the next: filled with ones, zeros or random bytes before the
    call, it gives the outputs of the separate calls."""
    case = CASES[0]
    p = case[6]
    ref = _state(pipeline, case)
    ref.step_calls(p)
    want = _outputs(ref)
    st = _state(pipeline, case)
    g = torch.Generator(device="cpu").manual_seed(5)
    for fill in (0xFF, 0x00, None):
        print("workspace fill", fill, flush=True)
        if fill is None:
            st.ws_step.copy_(torch.randint(0, 256, st.ws_step.shape, generator=g, dtype=torch.uint8))
        else:
            st.ws_step.fill_(fill)
        st.step(p)
        _same(_outputs(st), want)


@pytest.mark.parametrize("ci", [0, 4, 7, 8])
def test_fused_step_graph_replays_new_queries(pipeline, ci):
    """Each replay of a captured step quantises the query it finds in the
    buffer: with a new query before every replay (and eager steps between
    the replays) every replay matches the separate calls on that query."""
    case = CASES[ci]
    p = case[6]
    ref = _state(pipeline, case)
    st = _state(pipeline, case)
    q0 = st.q.clone()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        st.step(p)
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=s):
            st.step(p)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    gen_q = torch.Generator(device="cpu").manual_seed(17 + ci)
    for i in range(4):
        print("replay", i, flush=True)
        qn = (q0.cpu() + 0.5 * torch.randn(q0.shape, generator=gen_q)).to(q0.device)
        st.q.copy_(qn)
        ref.q.copy_(qn)
        ref.step_calls(p)
        want = _outputs(ref)
        torch.cuda.synchronize()
        g.replay()
        _same(_outputs(st), want)
        st.step(p)            # eager work between the replays
        _same(_outputs(st), want)
