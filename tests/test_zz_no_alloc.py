"""rbq_decode_step_noalloc (the fused step on the library's static scratch
array) against rbq_decode_step on a caller's workspace: the same inputs give
bitwise the same outputs, on two calls in a row, the second one smaller than
the first (so the array still holds the first call's contents), and a size
beyond the array is rejected on the host."""
import numpy as np
import pytest
import torch

from workloads import gen

pytestmark = pytest.mark.gpu

# (B, Hq, Hkv, n, w, kv dtype, p, seed): the larger call first
CALLS = [
    (1, 32, 8, 32768, 256, "bf16", 0.95, 11),   # the 8B-model GQA shape at 32K
    (2, 8, 2, 3001, 40, "bf16", 0.9, 12),       # smaller, ragged n
]


@pytest.fixture(scope="module")
def mods():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2606_31519_amd import pipeline as pl
    from paper_2606_31519_amd import rbq
    return pl, rbq


def _state(pl, case):
    B, Hq, Hkv, n, w, dt, p, seed = case
    wl = gen.random_case(B, Hq, Hkv, n, seed=seed, kv_dtype=dt, w=w, c_q_scale=0.5)
    st = pl.DecodeState.from_workload(wl)
    st.build_index()
    return st


def _noalloc_step(rbq, st, p):
    rbq.rbq_decode_step_noalloc(st.B, st.Hq, st.Hkv, st.D, st.q, st.P, st.c_q, st.c_k, st.K, st.V, st.cap, st.n,
                                st.w, st.codes, st.kfac, True, p, st.sm_scale, st.qplanes, st.qscal, st.scores,
                                st.sel_idx, st.sel_count, st.out, st.lse)


def _outputs(st):
    torch.cuda.synchronize()
    cnt = st.sel_count.cpu().numpy()
    sel = st.sel_idx.cpu().numpy()
    o = {name: getattr(st, name).cpu().numpy().copy() for name in
         ("qplanes", "qscal", "sel_count", "out", "lse", "codes", "kfac")}
    o["scores"] = st.scores[:, :, :st.n].cpu().numpy().copy()
    o["sel"] = [sel[b, h, :cnt[b, h]].copy() for b in range(st.B) for h in range(st.Hq)]
    return o


def test_noalloc_step_matches_workspace_step(mods):
    pl, rbq = mods
    for case in CALLS:
        print("call", case, flush=True)
        p = case[6]
        ref = _state(pl, case)
        ref.step(p, flush=True)        # rbq_decode_step on its own workspace
        want = _outputs(ref)
        del ref
        st = _state(pl, case)
        _noalloc_step(rbq, st, p)
        got = _outputs(st)
        assert got.keys() == want.keys()
        for k in want:
            if k == "sel":
                assert len(got[k]) == len(want[k])
                assert all(np.array_equal(x, y) for x, y in zip(got[k], want[k])), k
            else:
                assert got[k].shape == want[k].shape
                assert np.array_equal(got[k].view(np.uint8), want[k].view(np.uint8)), k
        assert want["sel_count"].min() >= 1
        del st


def test_noalloc_step_rejects_sizes_beyond_the_scratch(mods):
    _, rbq = mods
    B, Hq, Hkv, D, n, w = 4, 64, 8, 128, 131072, 256
    need = rbq.rbq_workspace_bytes(rbq.RBQ_OP_DECODE_STEP, B, Hq, Hkv, D, n, w)
    assert need > rbq.RBQ_NOALLOC_SCRATCH_BYTES
    # rejected before any pointer is read or any kernel is enqueued
    st = rbq.lib.rbq_decode_step_noalloc(B, Hq, Hkv, D, *([None] * 6), rbq.RBQ_BF16, n + w, n, w, None, None, 1,
                                         0.9, 0.1, *([None] * 7), None)
    assert st == rbq.RBQ_EUNSUPPORTED
