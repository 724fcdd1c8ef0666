"""A decode loop over a growing cache (pipeline.DecodeSession, the lazy index
update of Section 3.4): one token appended per step, the window flushed into
the index by the step that finds it full. Across three flushes the index rows
of the flushed tokens are the oracle's encoding with the prefill centroid, the
index grows by the window each time, and each checked step's Top-p set and
attention (selection of the current index plus the current window) match the
oracle. Run at D = 128 and 64 on the full index and on the compact index."""
import math

import numpy as np
import pytest
import torch

from oracle import rbq_oracle as orc
from workloads import gen
import parity_util as pu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pipeline():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2606_31519_amd import pipeline as pl
    return pl


def _np(t):
    return t.detach().cpu().numpy()


@pytest.mark.parametrize("D,compact", [(128, False), (64, False), (128, True)])
def test_session_grows_the_index_through_lazy_flushes(pipeline, D, compact):
    print("session D", D, "compact", compact, flush=True)
    B, Hq, Hkv = 1, 8, 2
    n0, window, steps = 3000, 32, 100          # the 32nd, 64th and 96th steps flush (their window is full)
    cap = n0 + 4 * window
    wl = gen.random_case(B, Hq, Hkv, cap, D=D, seed=71, kv_dtype="bf16", q_scale=5.0)
    K = pipeline.to_device_kv(wl.K, wl.kv_dtype, "cuda")
    V = pipeline.to_device_kv(wl.V, wl.kv_dtype, "cuda")
    P = torch.from_numpy(np.ascontiguousarray(wl.P)).cuda()
    # the "generated" tokens are the rows after the prefill, appended one per step
    K_new, V_new = K[:, :, n0:].clone(), V[:, :, n0:].clone()
    K[:, :, n0:] = 0
    V[:, :, n0:] = 0
    ses = pipeline.DecodeSession(B, Hq, Hkv, D, cap, n0, window, K, V, P, compact=compact)
    rng = np.random.default_rng(3)
    tau = 1.0 / math.sqrt(D)
    G = Hq // Hkv
    Kf = np.stack([wl.K_f32(0, hk) for hk in range(Hkv)]).astype(np.float64)   # [Hkv][cap][D]
    Vf = np.stack([wl.V_f32(0, hk) for hk in range(Hkv)]).astype(np.float64)
    ck = None
    flushes = 0
    for t in range(steps):
        ses.append(K_new[:, :, t], V_new[:, :, t])
        q = torch.from_numpy((5.0 * rng.standard_normal((B, Hq, D))).astype(np.float32)).cuda()
        n_before, w_before = ses.n, ses.w
        flushed = ses.step(q, 0.9)
        torch.cuda.synchronize()
        if ck is None:
            ck = _np(ses.state.c_k[0]).astype(np.float64)
        if flushed:
            flushes += 1
            assert ses.n == n_before + window and ses.w == 0
            codes = pu.u32(ses.state.codes[0])
            fac = _np(ses.state.kfac16[0] if compact else ses.state.kfac[0][..., 0]).astype(np.float64)
            for hk in range(Hkv):
                rows = slice(n_before, n_before + window)
                enc = orc.encode_keys(Kf[hk, rows], wl.P, c_k=ck[hk])
                diff = orc.unpack_bits(codes[hk, rows], D) != enc["bits"]
                assert np.all(np.abs(enc["R"][diff]) <= 1e-5 * np.broadcast_to(enc["norm"][:, None], diff.shape)[diff])
                if compact:   # the fp16 factor: the oracle's rounding, or one step off at a near-tie
                    want = orc.compact_factor(enc["f"])
                    assert np.all((fac[hk, rows] == want) | (np.abs(fac[hk, rows] - want) <= 2.0 ** -10 * want))
                else:
                    assert np.all(np.abs(fac[hk, rows] - enc["f"]) <= 1e-5 * enc["f"] + 1e-6)
        if flushed or t in (0, 50):
            n, w = n_before, w_before
            S = _np(ses.state.scores).reshape(-1)[:B * Hq * n].reshape(B, Hq, n)
            cnt = _np(ses.state.sel_count)
            sel = _np(ses.state.sel_idx).reshape(-1)[:B * Hq * n].reshape(B, Hq, n)
            out, lse = _np(ses.state.out), _np(ses.state.lse)
            for h in (0, Hq - 1):
                hk = h // G
                got = sel[0, h, :cnt[0, h]]
                pu.check_topp(S[0, h], 0.9, tau, got)
                pu.check_attention(out[0, h], lse[0, h], _np(q)[0, h].astype(np.float64), Kf[hk, :n], Vf[hk, :n],
                                   got, Kf[hk, n:n + w], Vf[hk, n:n + w], tau)
    assert flushes == 3 and ses.n == n0 + 3 * window


def test_session_steps_after_the_last_flush_with_a_partial_window(pipeline):
    """A capacity that is not the prefill plus a whole number of windows: the
    third flush takes the index to 3096 keys, past cap - window = 3068, and the
    steps after it run with that index and a window that can only grow to the
    4 rows left. The session's buffers must hold every index size it reaches;
    the last steps are checked against the oracle."""
    B, Hq, Hkv, D = 1, 8, 2, 128
    n0, window, cap = 3000, 32, 3100
    wl = gen.random_case(B, Hq, Hkv, cap, D=D, seed=72, kv_dtype="bf16", q_scale=5.0)
    K = pipeline.to_device_kv(wl.K, wl.kv_dtype, "cuda")
    V = pipeline.to_device_kv(wl.V, wl.kv_dtype, "cuda")
    P = torch.from_numpy(np.ascontiguousarray(wl.P)).cuda()
    K_new, V_new = K[:, :, n0:].clone(), V[:, :, n0:].clone()
    K[:, :, n0:] = 0
    V[:, :, n0:] = 0
    ses = pipeline.DecodeSession(B, Hq, Hkv, D, cap, n0, window, K, V, P)
    assert ses.n_max == 3096 and ses.state.scores.numel() >= B * Hq * 3096
    rng = np.random.default_rng(4)
    tau = 1.0 / math.sqrt(D)
    G = Hq // Hkv
    Kf = np.stack([wl.K_f32(0, hk) for hk in range(Hkv)]).astype(np.float64)
    Vf = np.stack([wl.V_f32(0, hk) for hk in range(Hkv)]).astype(np.float64)
    for t in range(cap - n0):
        ses.append(K_new[:, :, t], V_new[:, :, t])
        q = torch.from_numpy((5.0 * rng.standard_normal((B, Hq, D))).astype(np.float32)).cuda()
        n, w = ses.n, ses.w
        ses.step(q, 0.9)
        torch.cuda.synchronize()
        if n < 3096:
            continue
        S = _np(ses.state.scores).reshape(-1)[:B * Hq * n].reshape(B, Hq, n)
        cnt = _np(ses.state.sel_count)
        sel = _np(ses.state.sel_idx).reshape(-1)[:B * Hq * n].reshape(B, Hq, n)
        out, lse = _np(ses.state.out), _np(ses.state.lse)
        for h in range(Hq):
            hk = h // G
            got = sel[0, h, :cnt[0, h]]
            pu.check_topp(S[0, h], 0.9, tau, got)
            pu.check_attention(out[0, h], lse[0, h], _np(q)[0, h].astype(np.float64), Kf[hk, :n], Vf[hk, :n], got,
                               Kf[hk, n:n + w], Vf[hk, n:n + w], tau)
    assert ses.n == 3096 and ses.w == 4
    with pytest.raises(RuntimeError):
        ses.append(K_new[:, :, 0], V_new[:, :, 0])   # the cache is full
