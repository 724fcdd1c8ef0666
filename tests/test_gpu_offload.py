"""K/V kept in pinned host memory, the index in HBM: the kernels read the
cache over PCIe through its device address (rbq.MappedHost). The index build,
the fused decode step (whose sparse attention gathers only the selected and
window rows), the same step as separate calls and the dense decode must give
bitwise the results they give with the cache in HBM (the same kernels read the
same bytes), and the mapped run is checked against the oracle as well: the
index, the scores, every head's Top-p set and the sparse and dense attention."""
import math

import numpy as np
import pytest
import torch

from workloads import gen
import parity_util as pu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2606_31519_amd import pipeline, rbq
    return pipeline, rbq


def _pinned(t):
    h = torch.empty(t.shape, dtype=t.dtype, pin_memory=True)
    h.copy_(t)
    return h


@pytest.mark.parametrize("kv_dtype", ["bf16", "f32"])
def test_step_calls_and_dense_decode_with_kv_in_host_memory(env, kv_dtype):
    pipeline, rbq = env
    wl = gen.random_case(2, 8, 2, 5000, seed=41, kv_dtype=kv_dtype, w=64, c_q_scale=0.5)
    ref = pipeline.DecodeState.from_workload(wl)
    Kh, Vh = rbq.MappedHost(_pinned(ref.K)), rbq.MappedHost(_pinned(ref.V))
    st = pipeline.DecodeState(ref.B, ref.Hq, ref.Hkv, ref.D, ref.cap, ref.n, ref.w, Kh, Vh, ref.q, ref.P, ref.c_q)
    outs = []
    for s in (ref, st):
        s.build_index()
        s.step(0.9)          # flushes the window rows (read from the cache) into the index
        dense_out, dense_lse = torch.empty_like(s.out), torch.empty_like(s.lse)
        s.dense_decode(dense_out, dense_lse)
        torch.cuda.synchronize()
        res = [t.cpu().numpy().copy() for t in (s.c_k, s.codes, s.kfac, s.qplanes, s.scores, s.sel_count,
                                                s.out, s.lse, dense_out, dense_lse)]
        # the same step as separate calls: quantize, score, select, sparse decode, flush (reads the window)
        s.step_calls(0.9)
        torch.cuda.synchronize()
        outs.append(res + [t.cpu().numpy().copy() for t in (s.out, s.lse, s.codes, s.kfac)])
    cnt = outs[0][5]
    sel = [x.sel_idx.cpu().numpy() for x in (ref, st)]
    for a, b in zip(*outs):
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8))
    for b_ in range(ref.B):
        for h in range(ref.Hq):
            assert np.array_equal(sel[0][b_, h, :cnt[b_, h]], sel[1][b_, h, :cnt[b_, h]])
    assert cnt.min() >= 1
    # the mapped run against the oracle: index (prefill rows and the flushed window),
    # scores on the GPU's codes, Top-p sets, sparse and dense attention
    c_k, codes, kfac, planes, S = outs[1][0], outs[1][1].view(np.uint32), outs[1][2], outs[1][3].view(np.uint32), outs[1][4]
    qs = st.qscal.cpu().numpy()
    out, lse, dout, dlse = outs[1][6], outs[1][7], outs[1][8], outs[1][9]
    n, w, G, tau = wl.n_index, wl.w, wl.G, 1.0 / math.sqrt(wl.D)
    for b_ in range(wl.B):
        for hk in range(wl.Hkv):
            K, V = wl.K_f32(b_, hk).astype(np.float64), wl.V_f32(b_, hk).astype(np.float64)
            pu.check_encode_group(codes[b_, hk, :n], kfac[b_, hk, :n], c_k[b_, hk], K[:n], wl.P, wl.c_q[b_, hk])
            pu.check_encode_group(codes[b_, hk, n:n + w], kfac[b_, hk, n:n + w], c_k[b_, hk], K[n:n + w], wl.P,
                                  wl.c_q[b_, hk], c_k_given=True)
            for h in range(hk * G, (hk + 1) * G):
                pu.check_qscal(qs[b_, h], planes[b_, h], wl.q[b_, h], wl.P, wl.c_q[b_, hk], c_k[b_, hk])
                pu.check_scores(S[b_, h, :n], codes[b_, hk, :n], kfac[b_, hk, :n], planes[b_, h], qs[b_, h])
                got = sel[1][b_, h, :cnt[b_, h]]
                pu.check_topp(S[b_, h, :n], 0.9, tau, got)
                pu.check_attention(out[b_, h], lse[b_, h], wl.q[b_, h], K[:n], V[:n], got, K[n:n + w], V[n:n + w],
                                   tau)
                pu.check_attention(dout[b_, h], dlse[b_, h], wl.q[b_, h], K[:n], V[:n], np.arange(n), K[n:n + w],
                                   V[n:n + w], tau)
