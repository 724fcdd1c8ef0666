"""The compact index (one fp16 factor per key, Appendix C) through the C ABI.

  * rbq_encode_keys_f16: the same sign codes as rbq_encode_keys (bitwise), and
    fp16 factors equal to the oracle's compact_factor of its fp64 f, except
    one binary16 step apart where the fp64 f lies within the fp32 rounding of
    a binary16 tie; they are exactly the full index's fp32 f rounded to fp16;
  * rbq_score_f16 against the oracle's estimate on the stored codes and
    factors (g = 0), and within 2^-11 |A f X| of the full index's scores;
  * rbq_decode_step_f16 against rbq_quantize_query + rbq_score_f16 +
    rbq_topp_select + rbq_sparse_decode + rbq_encode_keys_f16 (bitwise), its
    Top-p sets against the oracle on the same scores and its attention
    against the oracle;
  * the ragged forms against the separate ragged calls and each sequence's
    uniform compact score (bitwise).
"""
import math

import numpy as np
import pytest
import torch

from oracle import rbq_oracle as orc
from workloads import gen
import parity_util as pu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def R():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2606_31519_amd import rbq
    return rbq


@pytest.fixture(scope="module")
def pipeline(R):
    from paper_2606_31519_amd import pipeline as pl
    return pl


def _np(t):
    return t.detach().cpu().numpy()


def _near_binary16_tie(f):
    """fp64 values within 1e-5 relative (the encode's fp32 tolerance on f) of a
    binary16 rounding tie: the GPU's fp32 f may round to the other neighbour there."""
    c = orc.compact_factor(f)
    e = np.floor(np.log2(np.where(c > 0, c, 1.0)))
    step = 2.0 ** (e - 10)
    ties = np.stack([c - step / 2, c + step / 2, c - step / 4])
    return (np.abs(ties - f[None, :]) <= 1e-5 * np.abs(f)[None, :]).any(axis=0)


@pytest.mark.parametrize("kv_dtype,n", [("bf16", 3000), ("f32", 257), ("bf16", 1)])
def test_compact_encode_matches_oracle_and_full_index(R, pipeline, kv_dtype, n):
    print("compact encode", kv_dtype, n, flush=True)
    wl = gen.random_case(2, 4, 2, n, seed=n + 3, kv_dtype=kv_dtype, c_q_scale=0.0, key_offset=2.0)
    full = pipeline.DecodeState.from_workload(wl, c_q=False)
    comp = pipeline.DecodeState.from_workload(wl, compact=True)
    full.build_index()
    comp.build_index()
    torch.cuda.synchronize()
    assert np.array_equal(pu.u32(full.codes), pu.u32(comp.codes))
    assert np.array_equal(_np(full.c_k), _np(comp.c_k))
    f32 = _np(full.kfac)[..., 0]
    f16 = _np(comp.kfac16)
    # the fp32 f rounded to binary16 (saturated), bitwise
    assert np.array_equal(np.minimum(f32, 65504.0).astype(np.float16).view(np.uint16)[..., :n],
                          f16.view(np.uint16)[..., :n])
    for b in range(2):
        for hk in range(2):
            K = wl.K_f32(b, hk, slice(0, n)).astype(np.float64)
            enc = orc.encode_keys(K, wl.P, c_k=_np(comp.c_k[b, hk]).astype(np.float64))
            want = orc.compact_factor(enc["f"])
            got = f16[b, hk, :n].astype(np.float64)
            off = got != want
            assert np.all(_near_binary16_tie(enc["f"])[off]), np.nonzero(off)[0][:8]
            assert off.sum() <= max(2, n // 500)


@pytest.mark.parametrize("B,Hq,Hkv,n", [(1, 4, 1, 4097), (2, 8, 1, 31), (1, 32, 8, 1000), (1, 64, 8, 2500)])
def test_compact_score_parity(R, pipeline, B, Hq, Hkv, n):
    print("compact score", B, Hq, Hkv, n, flush=True)
    wl = gen.random_case(B, Hq, Hkv, n, seed=Hq + n + 1, kv_dtype="bf16", c_q_scale=0.0, key_offset=1.0)
    full = pipeline.DecodeState.from_workload(wl, c_q=False)
    comp = pipeline.DecodeState.from_workload(wl, compact=True)
    for st in (full, comp):
        st.build_index()
        st.quantize()
        st.score()
    torch.cuda.synchronize()
    assert np.array_equal(_np(full.qplanes), _np(comp.qplanes)) and np.array_equal(_np(full.qscal),
                                                                                  _np(comp.qscal))
    S, S_full = _np(comp.scores), _np(full.scores).astype(np.float64)
    codes, f16, f32 = pu.u32(comp.codes), _np(comp.kfac16).astype(np.float64), _np(full.kfac)[..., 0]
    planes, qs = pu.u32(comp.qplanes), _np(comp.qscal)
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hq):
            fac = np.stack([f16[b, h // G, :n], np.zeros(n)], axis=1)
            pu.check_scores(S[b, h, :n], codes[b, h // G, :n], fac, planes[b, h], qs[b, h])
            # against the full index: the factor's rounding bounds the difference
            qc = pu.planes_to_codes(planes[b, h])
            ip, pc = orc.int_dot(orc.unpack_bits(codes[b, h // G, :n], 128), qc)
            X = orc.reconstruct(ip, pc, float(qs[b, h, 0]), float(qs[b, h, 1]), int(qs[b, h, 2]), 128)
            bound = (2.0 ** -11 + 1e-5) * np.abs(float(qs[b, h, 3]) * f32[b, h // G, :n] * X) + \
                1e-5 * abs(float(qs[b, h, 4])) + 1e-6
            assert np.all(np.abs(S[b, h, :n] - S_full[b, h, :n]) <= bound)


@pytest.mark.parametrize("kv_dtype", ["bf16", "f32"])
def test_compact_step_matches_calls_and_oracle(R, pipeline, kv_dtype):
    print("compact step", kv_dtype, flush=True)
    wl = gen.random_case(2, 8, 2, 6000, seed=77, kv_dtype=kv_dtype, w=64, c_q_scale=0.0, q_scale=6.0)
    a = pipeline.DecodeState.from_workload(wl, compact=True)
    b = pipeline.DecodeState.from_workload(wl, compact=True)
    p = 0.9
    for st in (a, b):
        st.build_index()
    a.step(p)
    b.step_calls(p)
    torch.cuda.synchronize()
    for name in ("qplanes", "qscal", "scores", "sel_count", "out", "lse", "codes", "kfac16"):
        x, y = _np(getattr(a, name)), _np(getattr(b, name))
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8)), name
    cnt = _np(a.sel_count)
    sel_a, sel_b = _np(a.sel_idx), _np(b.sel_idx)
    tau = 1.0 / math.sqrt(wl.D)
    S = _np(a.scores)
    G = wl.Hq // wl.Hkv
    for bb in range(wl.B):
        for h in range(wl.Hq):
            s = sel_a[bb, h, :cnt[bb, h]]
            assert np.array_equal(s, sel_b[bb, h, :cnt[bb, h]])
            pu.check_topp(S[bb, h, :wl.n_index], p, tau, s)
            K = wl.K_f32(bb, h // G).astype(np.float64)
            V = wl.V_f32(bb, h // G).astype(np.float64)
            win = np.arange(wl.n_index, wl.n_index + wl.w)
            pu.check_attention(_np(a.out[bb, h]), float(_np(a.lse[bb, h])), wl.q[bb, h].astype(np.float64),
                               K[s], V[s], np.arange(len(s)), K[win], V[win], tau)
    # the flushed window rows: the compact encode of the window with the prefill centroid
    for bb in range(wl.B):
        for hk in range(wl.Hkv):
            Kw = wl.K_f32(bb, hk, slice(wl.n_index, wl.n_index + wl.w)).astype(np.float64)
            enc = orc.encode_keys(Kw, wl.P, c_k=_np(a.c_k[bb, hk]).astype(np.float64))
            got = _np(a.kfac16[bb, hk, wl.n_index:wl.n_index + wl.w]).astype(np.float64)
            off = got != orc.compact_factor(enc["f"])
            assert np.all(_near_binary16_tie(enc["f"])[off])


def test_compact_ragged_step_matches_ragged_calls(R, pipeline):
    seq_n, seq_w, seq_p = [6000, 0, 4097, 1234], [48, 17, 0, 33], [0.9, 0.7, 1.0, 0.95]
    Hq, Hkv, n = 8, 2, 6000
    print("compact ragged", seq_n, seq_w, seq_p, flush=True)
    B, w = len(seq_n), max(seq_w)
    wl = gen.random_case(B, Hq, Hkv, n, seed=19, kv_dtype="bf16", w=w, c_q_scale=0.0)
    a = pipeline.DecodeState.from_workload(wl, compact=True)
    b = pipeline.DecodeState.from_workload(wl, compact=True)
    for st in (a, b):
        st.build_index_ragged(seq_n)
    dev = dict(device="cuda")
    sn = torch.tensor(seq_n, dtype=torch.int32, **dev)
    sw = torch.tensor(seq_w, dtype=torch.int32, **dev)
    sp = torch.tensor(seq_p, dtype=torch.float32, **dev)
    a.step_ragged(sn, sw, sp)
    D, cap = b.D, b.cap
    R.rbq_quantize_query(B, Hq, Hkv, D, b.q, b.P, None, b.c_k, b.qplanes, b.qscal)
    R.rbq_score_varlen_f16(B, Hq, Hkv, D, n, cap, sn, b.codes, b.kfac16, b.qplanes, b.qscal, b.scores)
    R.rbq_topp_select_varlen(B, Hq, n, sn, b.scores, sp, b.sm_scale, b.sel_idx, b.sel_count, b.ws_topp)
    R.rbq_sparse_decode_varlen(B, Hq, Hkv, D, b.q, b.K, b.V, cap, n, w, sn, sw, b.sel_idx, b.sel_count,
                               b.sm_scale, b.out, b.lse, b.ws_decode)
    for s in range(B):   # each sequence's window rows into its index rows [seq_n, seq_n + seq_w)
        if seq_w[s]:
            R.rbq_encode_keys_f16(1, Hkv, D, b.K[s:s + 1, :, seq_n[s]:], cap, seq_w[s], seq_n[s], cap, b.P,
                                  b.c_k[s:s + 1], b.codes[s:s + 1], b.kfac16[s:s + 1], 0, None)
    torch.cuda.synchronize()
    cnt = _np(a.sel_count)
    assert np.array_equal(cnt, _np(b.sel_count))
    for s in range(B):
        for name in ("out", "lse"):
            x, y = _np(getattr(a, name))[s], _np(getattr(b, name))[s]
            assert np.array_equal(x.view(np.uint8), y.view(np.uint8)), (name, s)
        x, y = _np(a.scores)[s, :, :seq_n[s]], _np(b.scores)[s, :, :seq_n[s]]
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8)), s
        for h in range(Hq):
            c = cnt[s, h]
            assert np.array_equal(_np(a.sel_idx)[s, h, :c], _np(b.sel_idx)[s, h, :c])
        rows = slice(0, seq_n[s] + seq_w[s])
        assert np.array_equal(pu.u32(a.codes[s, :, rows]), pu.u32(b.codes[s, :, rows]))
        assert np.array_equal(_np(a.kfac16[s, :, rows]).view(np.uint16), _np(b.kfac16[s, :, rows]).view(np.uint16))
        # the uniform compact score of this sequence alone, bitwise
        if seq_n[s]:
            S1 = torch.zeros(1, Hq, seq_n[s], dtype=torch.float32, **dev)
            R.rbq_score_f16(1, Hq, Hkv, D, seq_n[s], cap, b.codes[s:s + 1], b.kfac16[s:s + 1], b.qplanes[s:s + 1],
                            b.qscal[s:s + 1], S1)
            torch.cuda.synchronize()
            assert np.array_equal(_np(S1)[0].view(np.uint8), x.view(np.uint8))


def test_compact_config3_full_size_sampled(R, pipeline):
    """Config 3's 128K workload on the compact index (the bench's compact_index
    launch shape) through the fused step with the flush: sampled KV groups and
    heads against the oracle (codes, fp16 factors, scores with g = 0, the Top-p
    set, attention)."""
    wl = gen.config3()
    st = pipeline.DecodeState.from_workload(wl, compact=True)
    st.build_index()
    n, w, G = wl.n_index, wl.w, wl.G
    tau = 1.0 / math.sqrt(wl.D)
    for p in (0.9, 0.95):
        print("compact config3 p", p, flush=True)
        st.step(p)
        torch.cuda.synchronize()
        S, codes, f16 = _np(st.scores), pu.u32(st.codes), _np(st.kfac16).astype(np.float64)
        planes, qs, ck = pu.u32(st.qplanes), _np(st.qscal), _np(st.c_k)
        sel, cnt, out, lse = _np(st.sel_idx), _np(st.sel_count), _np(st.out), _np(st.lse)
        for hk in (0, 5):
            K, V = wl.K_f32(0, hk).astype(np.float64), wl.V_f32(0, hk).astype(np.float64)
            enc = orc.encode_keys(K[:n + w], wl.P, c_k=ck[0, hk].astype(np.float64))
            diff = orc.unpack_bits(codes[0, hk, :n + w], wl.D) != enc["bits"]
            assert np.all(np.abs(enc["R"][diff]) <= 1e-5 * np.broadcast_to(enc["norm"][:, None], diff.shape)[diff])
            off = f16[0, hk, :n + w] != orc.compact_factor(enc["f"])
            assert np.all(_near_binary16_tie(enc["f"])[off])
            for h in (hk * G, hk * G + 3):
                pu.check_qscal(qs[0, h], planes[0, h], wl.q[0, h], wl.P, None, ck[0, hk])   # (built without c_q)
                fac = np.stack([f16[0, hk, :n], np.zeros(n)], axis=1)
                pu.check_scores(S[0, h, :n], codes[0, hk, :n], fac, planes[0, h], qs[0, h])
                got = sel[0, h, :cnt[0, h]]
                pu.check_topp(S[0, h, :n], p, tau, got)
                pu.check_attention(out[0, h], lse[0, h], wl.q[0, h], K[:n], V[:n], got, K[n:n + w], V[n:n + w], tau)
