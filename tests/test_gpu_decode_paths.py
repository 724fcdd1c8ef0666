"""The two ways the sparse attention builds its row lists agree bitwise (Algorithm 2 step 4).

rbq_sparse_decode turns the selection's index lists into per-row bitmaps first
(one pass per row) and builds every split's list of gathered rows from the
bitmap words; the test hook rbq_sparse_decode_debug builds the same lists by
searching each head's index list for the split's range. Both feed the same
attention kernel, so the outputs and log-sum-exps must match bit for bit, over
group sizes 1 to 16, both head dimensions, windows folded into the splits or
absent, and selections from empty to every key. The attention itself is
checked against the oracle by the parity tests of rbq_sparse_decode.
"""
import numpy as np
import pytest
import torch

from workloads import gen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mods():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2606_31519_amd import pipeline as pl
    from paper_2606_31519_amd import rbq
    return pl, rbq


def _both(rbq, st, K_loc, V_loc):
    outs = []
    for call in (rbq.rbq_sparse_decode, rbq.rbq_sparse_decode_debug):
        out, lse = torch.full_like(st.out, float("nan")), torch.full_like(st.lse, float("nan"))
        call(st.B, st.Hq, st.Hkv, st.D, st.q, st.K, st.V, st.cap, st.n, st.sel_idx, st.sel_count, K_loc, V_loc,
             st.cap, st.w, st.sm_scale, out, lse, st.ws_decode)
        outs.append((out, lse))
    torch.cuda.synchronize()
    return [(o.cpu().numpy(), l.cpu().numpy()) for o, l in outs]


@pytest.mark.parametrize("B,Hq,Hkv,n,w,D,p", [
    (2, 8, 2, 3000, 40, 128, 0.9),       # G = 4, a ragged last split
    (1, 32, 8, 20000, 256, 128, 0.95),   # the 128K step's head layout, dense unions
    (2, 16, 1, 5000, 0, 128, 0.9),       # G = 16, no window
    (1, 8, 8, 4097, 17, 128, 0.8),       # G = 1
    (2, 16, 2, 6001, 33, 64, 0.95),      # G = 8, head dimension 64
    (1, 8, 2, 3000, 40, 128, 1.0),       # every key
])
def test_bitmap_lists_match_index_lists(mods, B, Hq, Hkv, n, w, D, p):
    pl, rbq = mods
    print("decode paths", B, Hq, Hkv, n, w, D, p, flush=True)
    wl = gen.random_case(B, Hq, Hkv, n, D=D, seed=n + Hq, kv_dtype="bf16", w=w, c_q_scale=0.3)
    st = pl.DecodeState.from_workload(wl)
    st.build_index()
    st.quantize()
    st.score()
    st.select(p)
    K_loc = st.K[:, :, st.n:] if st.w else None
    V_loc = st.V[:, :, st.n:] if st.w else None
    (oa, la), (ob, lb) = _both(rbq, st, K_loc, V_loc)
    assert np.array_equal(oa.view(np.uint32), ob.view(np.uint32))
    assert np.array_equal(la.view(np.uint32), lb.view(np.uint32))
    assert np.isfinite(oa).all()


def test_bitmap_lists_with_empty_and_out_of_range_rows(mods):
    # rows without a selection (count 0) and entries outside [0, n) are skipped
    # by both paths; the window rows still take part
    pl, rbq = mods
    B, Hq, Hkv, n, w = 1, 8, 2, 2048, 24
    print("decode paths edge rows", flush=True)
    wl = gen.random_case(B, Hq, Hkv, n, seed=77, kv_dtype="bf16", w=w)
    st = pl.DecodeState.from_workload(wl)
    st.build_index()
    st.quantize()
    st.score()
    st.select(0.9)
    torch.cuda.synchronize()
    cnt = st.sel_count.clone()
    cnt[0, 1] = 0
    st.sel_count.copy_(cnt)
    sel = st.sel_idx.view(B, Hq, n)
    c2 = int(cnt[0, 2])
    if c2:
        sel[0, 2, c2 - 1] = n + 5   # past the row: ignored (the list search also stops at n)
    torch.cuda.synchronize()
    (oa, la), (ob, lb) = _both(rbq, st, st.K[:, :, n:], st.V[:, :, n:])
    assert np.array_equal(oa.view(np.uint32), ob.view(np.uint32))
    assert np.array_equal(la.view(np.uint32), lb.view(np.uint32))
