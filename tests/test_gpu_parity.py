"""Parity of the HIP path (through the C ABI) with the CPU oracle, stage by stage.

Every test feeds both sides the same seeded inputs; the comparison rules are
in parity_util. Sizes span several tiles with ragged tails; the full-size
workloads are checked on sampled (sequence, head) groups.
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


# ---------------------------------------------------------------- integer path
@pytest.mark.parametrize("B,Hkv,G,cap,n", [(2, 2, 4, 700, 650), (1, 1, 1, 64, 64), (1, 2, 8, 300, 257)])
def test_score_integers_bit_exact(R, B, Hkv, G, cap, n):
    rng = np.random.default_rng(n)
    Hq = Hkv * G
    codes = rng.integers(0, 2 ** 32, (B, Hkv, cap, 4), dtype=np.uint64).astype(np.uint32)
    codes[0, 0, 0] = 0xFFFFFFFF
    codes[0, 0, 1] = 0
    qcodes = rng.integers(0, 16, (B, Hq, 128))
    qcodes[0, 0] = 15
    planes = np.stack([np.stack([orc.query_bit_planes(qcodes[b, h]) for h in range(Hq)]) for b in range(B)])
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int32)).cuda()
    ip = torch.full((B, Hq, n), -1, dtype=torch.int32, device="cuda")
    pc = torch.full((B, Hkv, n), -1, dtype=torch.int32, device="cuda")
    R.rbq_score_ints(B, Hq, Hkv, 128, n, cap, dev(codes), dev(planes), ip, pc)
    torch.cuda.synchronize()
    ip, pc = _np(ip), _np(pc)
    for b in range(B):
        for hk in range(Hkv):
            bits = orc.unpack_bits(codes[b, hk, :n], 128)
            for g in range(G):
                ref_ip, ref_pc = orc.int_dot(bits, qcodes[b, hk * G + g])
                assert np.array_equal(ip[b, hk * G + g], ref_ip)
                assert np.array_equal(pc[b, hk], ref_pc)


# ---------------------------------------------------------------- query quantisation
@pytest.mark.parametrize("case,Hq,Hkv", [("plain", 8, 2), ("centred", 8, 2), ("degenerate", 8, 2),
                                          ("centred", 4, 4), ("centred", 8, 4), ("centred", 64, 8),
                                          ("centred", 16, 1)])
def test_quantize_query_stagewise(R, pipeline, case, Hq, Hkv):
    """Every query head's planes and constants against the oracle, at group
    sizes 1 to 16 with a non-zero query centroid per KV group: head h reads
    c_q and c_k of KV group h / G."""
    w = gen.random_case(2, Hq, Hkv, 64, seed=11, kv_dtype="f32", c_q_scale=0.0 if case == "plain" else 0.7)
    if case == "degenerate":
        w.q[0, 0] = w.c_q[0, 0]          # q == c_q: A = 0
        w.q[1, 3] = 0.0
    G = Hq // Hkv
    st = pipeline.DecodeState.from_workload(w)
    st.c_k.copy_(torch.randn(2, Hkv, 128, generator=torch.Generator().manual_seed(1)).cuda())
    qrot = torch.empty(2, Hq, 128, device="cuda")
    st.quantize(qrot_out=qrot)
    torch.cuda.synchronize()
    planes = pu.u32(st.qplanes)
    qs, qr, ck = _np(st.qscal), _np(qrot), _np(st.c_k)
    for b in range(2):
        for h in range(Hq):
            hk = h // G
            z = orc.uniform_quantize(qr[b, h], dtype=np.float32)      # the decision in fp32, from the GPU's q'
            assert np.array_equal(pu.planes_to_codes(planes[b, h]), z["codes"])
            assert qs[b, h, 0] == np.float32(z["ql"]) and qs[b, h, 1] == np.float32(z["delta"])
            assert qs[b, h, 2] == z["s_u"]
            ref = pu.check_qscal(qs[b, h], planes[b, h], w.q[b, h], w.P, w.c_q[b, hk], ck[b, hk])
            assert np.abs(qr[b, h] - ref["qrot"]).max() <= pu.ROT_ATOL
            # end to end the codes may differ only where the oracle's value sits on a rounding edge
            t = (ref["qrot"] - ref["ql"]) / ref["delta"] if ref["delta"] > 0 else np.zeros(128)
            off = np.nonzero(pu.planes_to_codes(planes[b, h]) != ref["codes"])[0]
            assert np.all(np.abs(t[off] - np.floor(t[off]) - 0.5) <= 1e-4)


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 5, 6, 7, 8])
def test_quantize_query_bits_and_scores(R, pipeline, bits):
    """rbq_quantize_query_bits: the B_q-bit codes decided in fp32 from the GPU's
    rotated query (the same rotation as rbq_quantize_query), bit-exact; B_q = 4
    is rbq_quantize_query bitwise; the scores from those planes match the oracle
    (B_q > 4: eight planes through rbq_score_q8, whose integer dot products are
    bit-exact)."""
    print("query bits", bits, flush=True)
    w = gen.random_case(1, 8, 2, 3000, seed=12, kv_dtype="bf16", c_q_scale=0.5)
    st = pipeline.DecodeState.from_workload(w)
    st.build_index()
    qrot = torch.empty(1, 8, 128, device="cuda")
    st.quantize(qrot_out=qrot)
    planes4, qs4 = pu.u32(st.qplanes).copy(), _np(st.qscal).copy()
    nplanes = 8 if bits > 4 else 4
    qp = torch.zeros(1, 8, nplanes, 4, dtype=torch.int32, device="cuda")
    qs = torch.zeros_like(st.qscal)
    R.rbq_quantize_query_bits(1, 8, 2, 128, st.q, st.P, st.c_q, st.c_k, bits, qp, qs)
    if bits > 4:
        R.rbq_score_q8(1, 8, 2, 128, st.n, st.cap, st.codes, st.kfac, qp, qs, st.scores)
        ip = torch.zeros(1, 8, st.n, dtype=torch.int32, device="cuda")
        pc = torch.zeros(1, 2, st.n, dtype=torch.int32, device="cuda")
        R.rbq_score_ints_q8(1, 8, 2, 128, st.n, st.cap, st.codes, qp, ip, pc)
    else:
        R.rbq_score(1, 8, 2, 128, st.n, st.cap, st.codes, st.kfac, qp, qs, st.scores)
    torch.cuda.synchronize()
    planes, qsb, qr = pu.u32(qp), _np(qs), _np(qrot)
    if bits == 4:
        assert np.array_equal(planes, planes4) and np.array_equal(qsb.view(np.uint32), qs4.view(np.uint32))
    codes, kfac, S = pu.u32(st.codes), _np(st.kfac), _np(st.scores)
    for h in range(8):
        z = orc.uniform_quantize(qr[0, h], dtype=np.float32, bits=bits)
        got = pu.planes_to_codes(planes[0, h])
        assert np.array_equal(got, z["codes"]) and got.max() == (1 << bits) - 1
        assert qsb[0, h, 0] == np.float32(z["ql"]) and qsb[0, h, 1] == np.float32(z["delta"])
        assert qsb[0, h, 2] == z["s_u"]
        if bits > 4:
            ip_or, pc_or = orc.int_dot(orc.unpack_bits(codes[0, h // 4, :st.n], 128), got)
            assert np.array_equal(_np(ip)[0, h], ip_or) and np.array_equal(_np(pc)[0, h // 4], pc_or)
        pu.check_scores(S[0, h, :st.n], codes[0, h // 4, :st.n], kfac[0, h // 4, :st.n].astype(np.float64),
                        planes[0, h], qsb[0, h])


# ---------------------------------------------------------------- index construction
def _check_encode_group(st, w, b, hk, n, rot, alpha, c_k_given=None):
    return pu.check_encode_group(pu.u32(st.codes[b, hk, :n]), _np(st.kfac[b, hk, :n]), _np(st.c_k[b, hk]),
                                 w.K_f32(b, hk, slice(0, n)), w.P, w.c_q[b, hk],
                                 rot=None if rot is None else _np(rot[b, hk]),
                                 alpha=None if alpha is None else _np(alpha[b, hk]), c_k_given=c_k_given is not None)


@pytest.mark.parametrize("kv_dtype,n", [("bf16", 1000), ("f32", 257), ("bf16", 1), ("f32", 128)])
def test_encode_stagewise(R, pipeline, kv_dtype, n):
    w = gen.random_case(2, 4, 2, n, seed=n, kv_dtype=kv_dtype, c_q_scale=0.5, key_offset=2.0)
    st = pipeline.DecodeState.from_workload(w)
    rot = torch.empty(2, 2, n, 128, device="cuda")
    alpha = torch.empty(2, 2, n, device="cuda")
    st.build_index(rot_out=rot, alpha_out=alpha)
    torch.cuda.synchronize()
    for b in range(2):
        for hk in range(2):
            _check_encode_group(st, w, b, hk, n, rot, alpha)


def test_encode_degenerate_key_and_lazy_append(R, pipeline):
    n1, n2 = 300, 77
    w = gen.random_case(1, 4, 1, n1 + n2, seed=5, kv_dtype="bf16", c_q_scale=0.3)
    st = pipeline.DecodeState.from_workload(w)
    st.n = n1
    st.build_index()
    torch.cuda.synchronize()
    ck = _np(st.c_k[0, 0])
    before = pu.u32(st.codes[0, 0, :n1]).copy()
    # lazy append: rows [n1, n1 + n2) encoded with the prefill centroid at offset n1
    R.rbq_encode_keys(1, 1, 128, st.K[:, :, n1:], st.cap, n2, n1, st.cap, st.P, st.c_q, st.c_k, st.codes, st.kfac,
                      0, None, None)
    torch.cuda.synchronize()
    assert np.array_equal(pu.u32(st.codes[0, 0, :n1]), before)
    assert np.array_equal(_np(st.c_k[0, 0]), ck)
    K2 = w.K_f32(0, 0, slice(n1, n1 + n2)).astype(np.float64)
    enc = orc.encode_keys(K2, w.P, c_k=ck.astype(np.float64), c_q=w.c_q[0, 0])
    diff = orc.unpack_bits(pu.u32(st.codes[0, 0, n1:n1 + n2]), 128) != enc["bits"]
    assert np.all(np.abs(enc["R"][diff]) <= 1e-5 * np.broadcast_to(enc["norm"][:, None], diff.shape)[diff])
    # a key equal to the centroid: no bits, f = 0, g = 0
    Kc = torch.from_numpy(np.tile(ck, (3, 1))).to(torch.bfloat16).float().cuda()
    ck_exact = Kc[0].clone()
    st.c_k[0, 0] = ck_exact
    R.rbq_encode_keys(1, 1, 128, Kc, 3, 3, 0, st.cap, st.P, st.c_q, st.c_k, st.codes, st.kfac, 0, None, None)
    torch.cuda.synchronize()
    assert np.all(pu.u32(st.codes[0, 0, :3]) == 0)
    assert np.all(_np(st.kfac[0, 0, :3]) == 0)


# ---------------------------------------------------------------- scores
@pytest.mark.parametrize("B,Hq,Hkv,n,cq", [(1, 4, 1, 4097, 0.0), (2, 8, 1, 31, 0.5), (1, 32, 8, 1000, 0.0),
                                            (2, 16, 2, 1, 0.2), (1, 64, 8, 2500, 0.3)])
def test_score_parity(R, pipeline, B, Hq, Hkv, n, cq):
    w = gen.random_case(B, Hq, Hkv, n, seed=Hq + n, kv_dtype="bf16", c_q_scale=cq, key_offset=1.0)
    st = pipeline.DecodeState.from_workload(w)
    st.build_index()
    st.quantize()
    st.score()
    torch.cuda.synchronize()
    S, codes, kfac = _np(st.scores), pu.u32(st.codes), _np(st.kfac)
    planes, qs = pu.u32(st.qplanes), _np(st.qscal)
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hq):
            pu.check_scores(S[b, h, :n], codes[b, h // G, :n], kfac[b, h // G, :n], planes[b, h], qs[b, h])


# ---------------------------------------------------------------- Top-p
def _topp_rows(R, S: np.ndarray, p: float, sm_scale: float):
    rows, n = S.shape
    dS = torch.from_numpy(np.ascontiguousarray(S, dtype=np.float32)).cuda()
    sel = torch.full((rows, max(n, 1)), -7, dtype=torch.int32, device="cuda")
    cnt = torch.full((rows,), -7, dtype=torch.int32, device="cuda")
    ws = R.workspace(R.RBQ_OP_TOPP, 1, rows, rows, 128, n)
    R.rbq_topp_select(1, rows, n, dS, p, sm_scale, sel, cnt, ws)
    torch.cuda.synchronize()
    return _np(sel), _np(cnt)


@pytest.mark.parametrize("n", [1, 31, 4096, 4097, 20000, 70001])
@pytest.mark.parametrize("p", [0.5, 0.9, 0.95, 0.99, 1.0])
def test_topp_parity_random(R, n, p):
    rng = np.random.default_rng(n)
    S = np.stack([rng.standard_normal(n) * 6.0,                         # spread
                  rng.standard_normal(n) * 0.3,                         # near uniform
                  np.round(rng.standard_normal(n) * 4.0) / 2.0,         # many exact ties
                  np.where(rng.random(n) < 0.01, 30.0, 0.0) + rng.standard_normal(n)])   # peaky
    sel, cnt = _topp_rows(R, S, p, 1 / math.sqrt(128) * 8)
    for r in range(S.shape[0]):
        assert 0 <= cnt[r] <= n
        got = sel[r, :cnt[r]]
        if p >= 1.0:
            assert np.array_equal(got, np.arange(n))
        else:
            pu.check_topp(S[r].astype(np.float32), p, 1 / math.sqrt(128) * 8, got)


def test_topp_degenerate_rows(R):
    n = 5000
    S = np.stack([np.full(n, 0.25), np.full(n, -3.0), np.where(np.arange(n) % 2 == 0, 0.0, -0.0),
                  np.where(np.arange(n) == 1234, 100.0, -100.0)])
    sel, cnt = _topp_rows(R, S, 0.9, 1.0)
    assert cnt[0] == n and cnt[1] == n and cnt[2] == n       # all tied: everything
    assert cnt[3] == 1 and sel[3, 0] == 1234
    sel, cnt = _topp_rows(R, np.zeros((3, 0)), 0.9, 1.0)
    assert np.all(cnt == 0)


def test_topp_large_crossing_bin(R):
    """Rows whose level-1 crossing bin holds most of the keys (far more than the
    candidates kept in registers): the final pass streams the candidate list."""
    n = 70001
    rng = np.random.default_rng(5)
    spread = rng.standard_normal(n) * 5.0
    S = np.stack([np.full(n, 1.5), np.where(rng.random(n) < 0.6, 2.0, spread),
                  2.0 + rng.random(n) * 1e-3])              # one narrow band of distinct values
    for p in (0.5, 0.9, 0.99):
        sel, cnt = _topp_rows(R, S, p, 1.0)
        assert cnt[0] == n
        for r in (1, 2):
            pu.check_topp(S[r].astype(np.float32), p, 1.0, sel[r, :cnt[r]])


def test_topp_rows_past_a_million_keys(R):
    """Rows of more than 64 sub-chunks of 16384 keys: each selection block takes
    several consecutive sub-chunks (the multi-sub-chunk kernels), with a row
    that ends inside a block's span, one with a dense tie at the boundary, and
    one whose first-level crossing bin holds more keys than the candidate
    buffers (the exact full-row fallback)."""
    n = 1_100_001
    rng = np.random.default_rng(9)
    S = np.stack([rng.standard_normal(n) * 5.0,
                  np.where(rng.random(n) < 0.02, 25.0, 0.0) + rng.standard_normal(n),
                  np.round(rng.standard_normal(n) * 2.0) / 4.0])
    for p in (0.5, 0.95):
        sel, cnt = _topp_rows(R, S, p, 1 / math.sqrt(128) * 8)
        for r in range(S.shape[0]):
            pu.check_topp(S[r].astype(np.float32), p, 1 / math.sqrt(128) * 8, sel[r, :cnt[r]])


def test_topp_many_candidates_without_overflow(R):
    """A row whose first-level crossing bin holds more candidates than the final
    pass keeps in LDS, although no single part exceeds its candidate buffer
    (the fallback taken for the row as a whole), beside an ordinary row."""
    n = 131072
    rng = np.random.default_rng(10)
    band = 3.0 + rng.random(n) * 1e-3                     # 20 % of the keys in one narrow band
    S = np.stack([np.where(rng.random(n) < 0.2, band, rng.standard_normal(n) - 4.0),
                  rng.standard_normal(n) * 3.0])
    for p in (0.3, 0.9):
        sel, cnt = _topp_rows(R, S, p, 1.0)
        for r in range(S.shape[0]):
            pu.check_topp(S[r].astype(np.float32), p, 1.0, sel[r, :cnt[r]])


# ---------------------------------------------------------------- attention
def _rand_sel(rng, n, frac, Hq):
    out = []
    for _ in range(Hq):
        k = int(round(frac * n))
        out.append(np.sort(rng.choice(n, size=k, replace=False)) if n else np.zeros(0, np.int64))
    return out


@pytest.mark.parametrize("kv_dtype,G,n,w,frac", [("bf16", 4, 5000, 17, 0.05), ("f32", 1, 3000, 0, 0.3),
                                                 ("bf16", 8, 2049, 256, 0.5), ("bf16", 4, 0, 100, 0.0),
                                                 ("bf16", 2, 700, 0, 0.0), ("bf16", 4, 131, 5, 1.0),
                                                 ("bf16", 16, 1500, 40, 0.2), ("bf16", 1, 2500, 3, 0.1),
                                                 ("bf16", 4, 4100, 300, 0.02)])
def test_sparse_decode_parity(R, pipeline, kv_dtype, G, n, w, frac):
    B, Hkv = 2, 2
    Hq = G * Hkv
    wl = gen.random_case(B, Hq, Hkv, n, seed=n + w, kv_dtype=kv_dtype, w=w)
    st = pipeline.DecodeState.from_workload(wl)
    rng = np.random.default_rng(3)
    sels = [_rand_sel(rng, n, frac, Hq) for _ in range(B)]
    idx = np.zeros((B, Hq, max(n, 1)), np.int32)
    cnt = np.zeros((B, Hq), np.int32)
    for b in range(B):
        for h in range(Hq):
            idx[b, h, :len(sels[b][h])] = sels[b][h]
            cnt[b, h] = len(sels[b][h])
    st.sel_idx.copy_(torch.from_numpy(idx))
    st.sel_count.copy_(torch.from_numpy(cnt))
    st.sparse_decode()
    torch.cuda.synchronize()
    out, lse = _np(st.out), _np(st.lse)
    for b in range(B):
        for h in range(Hq):
            hk = h // G
            K, V = wl.K_f32(b, hk), wl.V_f32(b, hk)
            pu.check_attention(out[b, h], lse[b, h], wl.q[b, h], K[:n], V[:n], sels[b][h], K[n:n + w], V[n:n + w],
                               st.sm_scale)
    # dense: every indexed row plus the window
    st.dense_decode()
    torch.cuda.synchronize()
    out, lse = _np(st.out), _np(st.lse)
    for b in range(B):
        for h in range(Hq):
            hk = h // G
            K, V = wl.K_f32(b, hk), wl.V_f32(b, hk)
            pu.check_attention(out[b, h], lse[b, h], wl.q[b, h], K[:n], V[:n], np.arange(n), K[n:n + w],
                               V[n:n + w], st.sm_scale)


# ---------------------------------------------------------------- end to end
def _end_to_end(R, pipeline, wl, p, groups, rows_per_group=None, flush=False):
    st = pipeline.DecodeState.from_workload(wl)
    st.build_index()
    st.step(p, flush=flush)
    torch.cuda.synchronize()
    n, w, G = wl.n_index, wl.w, wl.G
    S, codes, kfac = _np(st.scores), pu.u32(st.codes), _np(st.kfac)
    planes, qs, ck = pu.u32(st.qplanes), _np(st.qscal), _np(st.c_k)
    sel, cnt, out, lse = _np(st.sel_idx), _np(st.sel_count), _np(st.out), _np(st.lse)
    report = []
    for (b, hk) in groups:
        K, V = wl.K_f32(b, hk), wl.V_f32(b, hk)
        _check_encode_group(st, wl, b, hk, n, None, None)
        heads = range(hk * G, (hk + 1) * G) if rows_per_group is None else [hk * G + g for g in rows_per_group]
        for h in heads:
            ref = pu.check_qscal(qs[b, h], planes[b, h], wl.q[b, h], wl.P, wl.c_q[b, hk], ck[b, hk])
            qc = pu.planes_to_codes(planes[b, h])
            t = (ref["qrot"] - ref["ql"]) / ref["delta"]
            off = np.nonzero(qc != ref["codes"])[0]
            assert np.all(np.abs(t[off] - np.floor(t[off]) - 0.5) <= 1e-4)
            pu.check_scores(S[b, h, :n], codes[b, hk, :n], kfac[b, hk, :n], planes[b, h], qs[b, h])
            got = sel[b, h, :cnt[b, h]]
            res = pu.check_topp(S[b, h, :n], p, st.sm_scale, got)
            pu.check_attention(out[b, h], lse[b, h], wl.q[b, h], K[:n], V[:n], got, K[n:n + w], V[n:n + w],
                               st.sm_scale)
            recall = orc.attention_recall(wl.q[b, h], K[:n], got, st.sm_scale)
            report.append((b, h, int(cnt[b, h]), res["diff"], recall))
    return st, report


def test_end_to_end_config1(R, pipeline):
    wl = gen.config1()
    st, rep = _end_to_end(R, pipeline, wl, wl.p, [(0, 0)])
    print("config1 (b, h, budget, set diff, recall):", rep)


def test_end_to_end_config2(R, pipeline):
    wl = gen.config2()
    st, rep = _end_to_end(R, pipeline, wl, wl.p, [(0, hk) for hk in range(8)])
    budgets = [r[2] for r in rep]
    print(f"config2 budget mean {np.mean(budgets):.0f} of {wl.n_index}, recall mean {np.mean([r[4] for r in rep]):.3f}")


@pytest.mark.slow
def test_end_to_end_config3_full_size_sampled(R, pipeline):
    wl = gen.config3()
    for p in wl.p_sweep:
        st, rep = _end_to_end(R, pipeline, wl, p, [(0, 0), (0, 5)], rows_per_group=[0, 3], flush=True)
        print(f"config3 p={p}: budgets {[r[2] for r in rep]} recall {[round(r[4], 3) for r in rep]}")


def test_end_to_end_config4_batched_varied_sparsity_sampled(R, pipeline):
    """Batch 16 x 32K with per-sequence planted fractions: one launch covers every
    sequence's budget; sampled (sequence, KV head) groups are checked in full."""
    wl = gen.config4()
    st, rep = _end_to_end(R, pipeline, wl, wl.p, [(0, 0), (5, 3), (11, 7), (15, 2)], rows_per_group=[0, 2])
    print("config4 (b, h, budget, set diff, recall):", rep)


@pytest.mark.slow
def test_end_to_end_config5_wide_heads_sampled(R, pipeline):
    """64 query / 8 KV heads, batch 4 x 128K, Student-t keys: the launch shape of
    the standalone scan in the bench; sampled groups and heads checked in full."""
    wl = gen.config5()
    st, rep = _end_to_end(R, pipeline, wl, wl.p, [(0, 0), (3, 6)], rows_per_group=[0, 7])
    print("config5 (b, h, budget, set diff, recall):", rep)


def test_step_is_deterministic(R, pipeline):
    wl = gen.config2(N=8192)
    st = pipeline.DecodeState.from_workload(wl)
    st.build_index()
    outs = []
    for _ in range(2):
        st.step(0.95)
        torch.cuda.synchronize()
        outs.append([_np(t).copy() for t in (st.scores, st.sel_idx, st.sel_count, st.out, st.lse)])
    for a, b in zip(*outs):
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8))
