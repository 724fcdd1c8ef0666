"""Head dimension 64 (the D = 64 shape of the paper's kernel ablation) through
the C ABI, uniform batches: every stage against the oracle, and the fused step
against the separate calls.

  * rbq_encode_keys (debug form): the codes are the signs of the GPU's fp32
    rotation (bit-exact), which is within 1e-5 ||x|| of the oracle's; factors,
    alpha and the centroid within 1e-5 relative;
  * rbq_quantize_query (debug form): INT4 codes decided from the GPU's rotated
    query, bit-exact; the integer dot products of rbq_score_ints bit-exact;
    the scores within the score tolerance;
  * rbq_sparse_decode / rbq_dense_decode (bf16 K/V on the matrix cores, fp32 on
    the vector kernel; G = 1 to 16, with a window) against the oracle's attention;
  * rbq_decode_step against the five calls, bitwise, and its Top-p sets against
    the oracle on the same scores.
"""
import math

import numpy as np
import pytest
import torch

from oracle import rbq_oracle as orc
from workloads import gen
import parity_util as pu

pytestmark = pytest.mark.gpu
D = 64


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


@pytest.mark.parametrize("kv_dtype,n", [("bf16", 1000), ("f32", 257), ("bf16", 1)])
def test_d64_encode_stagewise(R, pipeline, kv_dtype, n):
    print("d64 encode", kv_dtype, n, flush=True)
    wl = gen.random_case(2, 4, 2, n, D=D, seed=n + 64, kv_dtype=kv_dtype, c_q_scale=0.5, key_offset=2.0)
    st = pipeline.DecodeState.from_workload(wl)
    rot = torch.empty(2, 2, n, D, device="cuda")
    alpha = torch.empty(2, 2, n, device="cuda")
    st.build_index(rot_out=rot, alpha_out=alpha)
    torch.cuda.synchronize()
    for b in range(2):
        for hk in range(2):
            K = wl.K_f32(b, hk, slice(0, n)).astype(np.float64)
            ck = _np(st.c_k[b, hk]).astype(np.float64)
            assert np.abs(ck - orc.key_centroid(K)).max() <= 1e-5 * (np.abs(K).mean() + 1.0)
            enc = orc.encode_keys(K, wl.P, c_k=ck, c_q=wl.c_q[b, hk])
            codes = pu.u32(st.codes[b, hk, :n])
            r = _np(rot[b, hk]).astype(np.float64)
            assert np.array_equal(codes, orc.pack_bits(orc.sign_bits(r)))
            nrm = enc["norm"]
            assert np.all(np.abs(r - enc["R"]) <= 1e-5 * nrm[:, None] + 1e-30)
            kfac = _np(st.kfac[b, hk, :n]).astype(np.float64)
            assert np.all(np.abs(kfac[:, 0] - enc["f"]) <= 1e-5 * np.abs(enc["f"]) + 1e-6)
            gscale = np.abs(wl.c_q[b, hk]).sum() * np.abs(enc["X"]).max(axis=1)
            assert np.all(np.abs(kfac[:, 1] - enc["g"]) <= 1e-5 * gscale + 1e-6)
            a = _np(alpha[b, hk]).astype(np.float64)
            assert np.all(np.abs(a - enc["alpha"]) <= 1e-5 * enc["alpha"] + 1e-7)


@pytest.mark.parametrize("B,Hq,Hkv,n", [(1, 4, 1, 4097), (2, 8, 2, 31), (1, 32, 8, 1000)])
def test_d64_quantize_and_score(R, pipeline, B, Hq, Hkv, n):
    print("d64 score", B, Hq, Hkv, n, flush=True)
    wl = gen.random_case(B, Hq, Hkv, n, D=D, seed=Hq + n, kv_dtype="bf16", c_q_scale=0.3, key_offset=1.0)
    st = pipeline.DecodeState.from_workload(wl)
    st.build_index()
    qrot = torch.empty(B, Hq, D, device="cuda")
    st.quantize(qrot_out=qrot)
    st.score()
    ip = torch.zeros(B, Hq, n, dtype=torch.int32, device="cuda")
    pc = torch.zeros(B, Hkv, n, dtype=torch.int32, device="cuda")
    R.rbq_score_ints(B, Hq, Hkv, D, n, st.cap, st.codes, st.qplanes, ip, pc)
    torch.cuda.synchronize()
    planes, qs, qr = pu.u32(st.qplanes), _np(st.qscal), _np(qrot)
    codes, kfac, S = pu.u32(st.codes), _np(st.kfac), _np(st.scores)
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hq):
            z = orc.uniform_quantize(qr[b, h], dtype=np.float32)
            qc = pu.planes_to_codes(planes[b, h])
            assert np.array_equal(qc, z["codes"])
            assert qs[b, h, 0] == np.float32(z["ql"]) and qs[b, h, 1] == np.float32(z["delta"])
            assert qs[b, h, 2] == z["s_u"]
            pu.check_qscal(qs[b, h], planes[b, h], wl.q[b, h], wl.P, wl.c_q[b, h // G], _np(st.c_k[b, h // G]), D=D)
            bits = orc.unpack_bits(codes[b, h // G, :n], D)
            ip_or, pc_or = orc.int_dot(bits, qc)
            assert np.array_equal(_np(ip)[b, h], ip_or) and np.array_equal(_np(pc)[b, h // G], pc_or)
            pu.check_scores(S[b, h, :n], codes[b, h // G, :n], kfac[b, h // G, :n].astype(np.float64),
                            planes[b, h], qs[b, h], D=D)


@pytest.mark.parametrize("kv_dtype", ["bf16", "f32"])
@pytest.mark.parametrize("G", [1, 2, 4, 8, 16])
def test_d64_sparse_and_dense_decode(R, pipeline, kv_dtype, G):
    Hkv, n, w = 2, 3000, 40
    print("d64 decode", kv_dtype, G, flush=True)
    wl = gen.random_case(2, G * Hkv, Hkv, n, D=D, seed=G + 5, kv_dtype=kv_dtype, w=w, q_scale=4.0)
    st = pipeline.DecodeState.from_workload(wl)
    rng = np.random.default_rng(G)
    sel = np.zeros((2, G * Hkv, n), np.int32)
    cnt = np.zeros((2, G * Hkv), np.int32)
    for b in range(2):
        for h in range(G * Hkv):
            k = int(rng.integers(0, n // 3))
            s = np.sort(rng.choice(n, k, replace=False)).astype(np.int32)
            sel[b, h, :k], cnt[b, h] = s, k
    st.sel_idx.copy_(torch.from_numpy(sel))
    st.sel_count.copy_(torch.from_numpy(cnt))
    st.sparse_decode()
    d_out, d_lse = torch.empty_like(st.out), torch.empty_like(st.lse)
    st.dense_decode(d_out, d_lse)
    torch.cuda.synchronize()
    out, lse, dout, dlse = _np(st.out), _np(st.lse), _np(d_out), _np(d_lse)
    tau = 1.0 / math.sqrt(D)
    for b in range(2):
        for h in range(G * Hkv):
            K = wl.K_f32(b, h // G).astype(np.float64)
            V = wl.V_f32(b, h // G).astype(np.float64)
            win = np.arange(n, n + w)
            q = wl.q[b, h].astype(np.float64)
            pu.check_attention(out[b, h], float(lse[b, h]), q, K, V, sel[b, h, :cnt[b, h]], K[win], V[win], tau)
            pu.check_attention(dout[b, h], float(dlse[b, h]), q, K, V, np.arange(n), K[win], V[win], tau)


@pytest.mark.parametrize("kv_dtype", ["bf16", "f32"])
def test_d64_step_matches_calls_and_oracle(R, pipeline, kv_dtype):
    print("d64 step", kv_dtype, flush=True)
    wl = gen.random_case(2, 8, 2, 6000, D=D, seed=91, kv_dtype=kv_dtype, w=64, c_q_scale=0.3, q_scale=6.0)
    a = pipeline.DecodeState.from_workload(wl)
    b = pipeline.DecodeState.from_workload(wl)
    p = 0.9
    for st in (a, b):
        st.build_index()
    a.step(p)
    b.step_calls(p)
    torch.cuda.synchronize()
    for name in ("qplanes", "qscal", "scores", "sel_count", "out", "lse", "codes", "kfac"):
        x, y = _np(getattr(a, name)), _np(getattr(b, name))
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8)), name
    cnt, sel_a, sel_b, S = _np(a.sel_count), _np(a.sel_idx), _np(b.sel_idx), _np(a.scores)
    tau = 1.0 / math.sqrt(D)
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
                               K, V, s, K[win], V[win], tau)


def test_d64_ragged_step_matches_ragged_calls_and_each_sequence(R, pipeline):
    """rbq_decode_step_varlen at D = 64 against the separate ragged calls plus
    each sequence's window encode (bitwise), its scores against each sequence's
    uniform score call (bitwise) and its Top-p sets against the oracle."""
    seq_n, seq_w, seq_p = [6000, 0, 4097, 1234], [48, 17, 0, 33], [0.9, 0.7, 1.0, 0.95]
    Hq, Hkv, n = 8, 2, 6000
    print("d64 ragged", seq_n, seq_w, seq_p, flush=True)
    B, w = len(seq_n), max(seq_w)
    wl = gen.random_case(B, Hq, Hkv, n, D=D, seed=23, kv_dtype="bf16", w=w, c_q_scale=0.3)
    a = pipeline.DecodeState.from_workload(wl)
    b = pipeline.DecodeState.from_workload(wl)
    for st in (a, b):
        st.build_index_ragged(seq_n)
    dev = dict(device="cuda")
    sn = torch.tensor(seq_n, dtype=torch.int32, **dev)
    sw = torch.tensor(seq_w, dtype=torch.int32, **dev)
    sp = torch.tensor(seq_p, dtype=torch.float32, **dev)
    a.step_ragged(sn, sw, sp)
    cap = b.cap
    R.rbq_quantize_query(B, Hq, Hkv, D, b.q, b.P, b.c_q, b.c_k, b.qplanes, b.qscal)
    R.rbq_score_varlen(B, Hq, Hkv, D, n, cap, sn, b.codes, b.kfac, b.qplanes, b.qscal, b.scores)
    R.rbq_topp_select_varlen(B, Hq, n, sn, b.scores, sp, b.sm_scale, b.sel_idx, b.sel_count, b.ws_topp)
    R.rbq_sparse_decode_varlen(B, Hq, Hkv, D, b.q, b.K, b.V, cap, n, w, sn, sw, b.sel_idx, b.sel_count,
                               b.sm_scale, b.out, b.lse, b.ws_decode)
    for s in range(B):
        if seq_w[s]:
            R.rbq_encode_keys(1, Hkv, D, b.K[s:s + 1, :, seq_n[s]:], cap, seq_w[s], seq_n[s], cap, b.P,
                              b.c_q[s:s + 1], b.c_k[s:s + 1], b.codes[s:s + 1], b.kfac[s:s + 1], 0, None, None)
    torch.cuda.synchronize()
    cnt = _np(a.sel_count)
    assert np.array_equal(cnt, _np(b.sel_count))
    tau = 1.0 / math.sqrt(D)
    G = Hq // Hkv
    for s in range(B):
        for name in ("out", "lse"):
            x, y = _np(getattr(a, name))[s], _np(getattr(b, name))[s]
            assert np.array_equal(x.view(np.uint8), y.view(np.uint8)), (name, s)
        rows = slice(0, seq_n[s] + seq_w[s])
        assert np.array_equal(pu.u32(a.codes[s, :, rows]), pu.u32(b.codes[s, :, rows]))
        assert np.array_equal(_np(a.kfac[s, :, rows]).view(np.uint32), _np(b.kfac[s, :, rows]).view(np.uint32))
        if not seq_n[s]:
            continue
        x = _np(a.scores)[s, :, :seq_n[s]]
        S1 = torch.zeros(1, Hq, seq_n[s], dtype=torch.float32, **dev)
        R.rbq_score(1, Hq, Hkv, D, seq_n[s], cap, b.codes[s:s + 1], b.kfac[s:s + 1], b.qplanes[s:s + 1],
                    b.qscal[s:s + 1], S1)
        torch.cuda.synchronize()
        assert np.array_equal(_np(S1)[0].view(np.uint8), x.view(np.uint8))
        for h in range(Hq):
            sel = _np(a.sel_idx)[s, h, :cnt[s, h]]
            assert np.array_equal(sel, _np(b.sel_idx)[s, h, :cnt[s, h]])
            p = min(float(np.float32(seq_p[s])), 1.0)   # the device's fp32 p
            if p < 1.0:
                pu.check_topp(x[h], p, tau, sel)
            else:
                assert cnt[s, h] == seq_n[s]
            K = wl.K_f32(s, h // G).astype(np.float64)
            V = wl.V_f32(s, h // G).astype(np.float64)
            win = np.arange(seq_n[s], seq_n[s] + seq_w[s])
            pu.check_attention(_np(a.out[s, h]), float(_np(a.lse[s, h])), wl.q[s, h].astype(np.float64), K, V,
                               sel, K[win], V[win], tau)


def test_d64_compact_index_and_eight_bit_queries(R, pipeline):
    """The compact index at D = 64: codes bitwise those of the full index,
    factors its fp32 f rounded to fp16, the fused step bitwise the separate
    calls; and 8-bit queries at D = 64: integer dots bit-exact, scores within
    the score tolerance."""
    print("d64 compact + q8", flush=True)
    wl = gen.random_case(2, 8, 2, 5000, D=D, seed=29, kv_dtype="bf16", w=32, c_q_scale=0.0, q_scale=6.0)
    full = pipeline.DecodeState.from_workload(wl, c_q=False)
    a = pipeline.DecodeState.from_workload(wl, compact=True)
    b = pipeline.DecodeState.from_workload(wl, compact=True)
    for st in (full, a, b):
        st.build_index()
    torch.cuda.synchronize()
    assert np.array_equal(pu.u32(full.codes), pu.u32(a.codes))
    n = wl.n_index
    f32 = _np(full.kfac)[..., 0][..., :n]
    assert np.array_equal(np.minimum(f32, 65504.0).astype(np.float16).view(np.uint16),
                          _np(a.kfac16)[..., :n].view(np.uint16))
    a.step(0.9)
    b.step_calls(0.9)
    torch.cuda.synchronize()
    for name in ("scores", "sel_count", "out", "lse", "codes", "kfac16"):
        x, y = _np(getattr(a, name)), _np(getattr(b, name))
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8)), name
    # eight-bit queries on the full index
    qp = torch.zeros(2, 8, 8, D // 32, dtype=torch.int32, device="cuda")
    qs = torch.zeros_like(full.qscal)
    R.rbq_quantize_query_bits(2, 8, 2, D, full.q, full.P, None, full.c_k, 8, qp, qs)
    S = torch.zeros_like(full.scores)
    R.rbq_score_q8(2, 8, 2, D, n, full.cap, full.codes, full.kfac, qp, qs, S)
    ip = torch.zeros(2, 8, n, dtype=torch.int32, device="cuda")
    pc = torch.zeros(2, 2, n, dtype=torch.int32, device="cuda")
    R.rbq_score_ints_q8(2, 8, 2, D, n, full.cap, full.codes, qp, ip, pc)
    torch.cuda.synchronize()
    planes, qsn, Sn = pu.u32(qp), _np(qs), _np(S)
    codes, kfac = pu.u32(full.codes), _np(full.kfac)
    for bb in range(2):
        for h in range(8):
            qc = pu.planes_to_codes(planes[bb, h])
            assert qc.max() <= 255
            ip_or, pc_or = orc.int_dot(orc.unpack_bits(codes[bb, h // 4, :n], D), qc)
            assert np.array_equal(_np(ip)[bb, h], ip_or) and np.array_equal(_np(pc)[bb, h // 4], pc_or)
            pu.check_scores(Sn[bb, h, :n], codes[bb, h // 4, :n], kfac[bb, h // 4, :n].astype(np.float64),
                            planes[bb, h], qsn[bb, h], D=D)


def test_d64_config3_full_size_sampled(R, pipeline):
    """Config 3's 128K workload at D = 64 (the bench's head_dim_64 launch shape)
    through the fused step with the flush: sampled KV groups and heads checked
    against the oracle (codes and factors, scores, the Top-p set, attention)."""
    wl = gen.config3_d64()
    st = pipeline.DecodeState.from_workload(wl)
    st.build_index()
    n, w, G = wl.n_index, wl.w, wl.G
    tau = 1.0 / math.sqrt(D)
    for p in (0.9, 0.95):
        print("d64 config3 p", p, flush=True)
        st.step(p)
        torch.cuda.synchronize()
        S, codes, kfac = _np(st.scores), pu.u32(st.codes), _np(st.kfac)
        planes, qs, ck = pu.u32(st.qplanes), _np(st.qscal), _np(st.c_k)
        sel, cnt, out, lse = _np(st.sel_idx), _np(st.sel_count), _np(st.out), _np(st.lse)
        for hk in (0, 5):
            K, V = wl.K_f32(0, hk).astype(np.float64), wl.V_f32(0, hk).astype(np.float64)
            enc = orc.encode_keys(K[:n + w], wl.P, c_k=ck[0, hk].astype(np.float64), c_q=wl.c_q[0, hk])
            diff = orc.unpack_bits(codes[0, hk, :n + w], D) != enc["bits"]
            assert np.all(np.abs(enc["R"][diff]) <= 1e-5 * np.broadcast_to(enc["norm"][:, None], diff.shape)[diff])
            assert np.all(np.abs(kfac[0, hk, :n + w, 0] - enc["f"]) <= 1e-5 * np.abs(enc["f"]) + 1e-6)
            for h in (hk * G, hk * G + 3):
                pu.check_qscal(qs[0, h], planes[0, h], wl.q[0, h], wl.P, wl.c_q[0, hk], ck[0, hk], D=D)
                pu.check_scores(S[0, h, :n], codes[0, hk, :n], kfac[0, hk, :n].astype(np.float64), planes[0, h],
                                qs[0, h], D=D)
                got = sel[0, h, :cnt[0, h]]
                pu.check_topp(S[0, h, :n], p, tau, got)
                pu.check_attention(out[0, h], lse[0, h], wl.q[0, h], K[:n], V[:n], got, K[n:n + w], V[n:n + w], tau)
