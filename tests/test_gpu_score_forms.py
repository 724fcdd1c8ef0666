"""The two forms of the score scan (Algorithm 2 step 2) agree bitwise and meet the oracle.

The scan computes the integer part ip = sum_d bit_d q_d either with v_dot8
(one lane per key) or on the matrix cores (one e4m3 x e2m1 product per 16 keys,
taken at G = 8, and at G = 4 with two or four 64-key rounds per wave, when n
and cap are multiples of 4). Each key's score depends on its own code, factors and query
only, so a call over n keys (matrix-core form) and one over n - 1 keys (n - 1
not a multiple of 4: the dot8 form) must give the same bits for the first
n - 1 keys. The matrix-core results are also checked against the oracle's
estimate on sampled (sequence, head) rows, and the ragged and compact-index
calls take the same two routes.
"""
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


def _two_forms(R, st, n, compact, seq_n=None):
    """scores of the first n keys (matrix-core form) and of the first n - 1 keys (dot8 form)"""
    B, Hq, Hkv = st.B, st.Hq, st.Hkv
    fac = st.kfac16 if compact else st.kfac
    out = []
    for m in (n, n - 1):
        S = torch.full((B, Hq, m), float("nan"), device="cuda")
        if seq_n is not None:
            sn = torch.tensor([min(s, m) for s in seq_n], dtype=torch.int32, device="cuda")
            call = R.rbq_score_varlen_f16 if compact else R.rbq_score_varlen
            call(B, Hq, Hkv, 128, m, st.cap, sn, st.codes, fac, st.qplanes, st.qscal, S)
        elif compact:
            R.rbq_score_f16(B, Hq, Hkv, 128, m, st.cap, st.codes, fac, st.qplanes, st.qscal, S)
        else:
            R.rbq_score(B, Hq, Hkv, 128, m, st.cap, st.codes, fac, st.qplanes, st.qscal, S)
        out.append(S)
    torch.cuda.synchronize()
    return _np(out[0]), _np(out[1])


@pytest.mark.parametrize("B,Hq,Hkv,n,compact", [
    (2, 64, 8, 3000, False),     # G = 8, one round per wave, ragged block tails
    (4, 64, 8, 65536, False),    # G = 8, four rounds per wave
    (16, 32, 8, 16384, False),   # G = 4, four rounds per wave
    (1, 32, 8, 65536, False),    # G = 4, two rounds per wave (the shape of the 128K step's scan)
    (2, 64, 8, 3000, True),      # compact index (fp16 factor)
    (1, 32, 8, 65536, True),
    (4, 64, 8, 65536, True),
])
def test_matrix_core_scan_is_bitwise_the_dot8_scan(R, pipeline, B, Hq, Hkv, n, compact):
    print("score forms", B, Hq, Hkv, n, "compact" if compact else "full", flush=True)
    wl = gen.random_case(B, Hq, Hkv, n, seed=B * n + Hq, kv_dtype="bf16", c_q_scale=0.0, key_offset=1.0)
    st = pipeline.DecodeState.from_workload(wl, c_q=False, compact=compact)
    st.build_index()
    st.quantize()
    S4, S3 = _two_forms(R, st, n, compact)
    assert np.array_equal(S4[..., : n - 1].view(np.uint32), S3.view(np.uint32))
    # the oracle on sampled rows of the matrix-core result
    codes, planes, qs = pu.u32(st.codes), pu.u32(st.qplanes), _np(st.qscal)
    G = Hq // Hkv
    rng = np.random.default_rng(n)
    for b, h in {(int(rng.integers(B)), int(rng.integers(Hq))) for _ in range(3)} | {(B - 1, Hq - 1)}:
        if compact:
            fac = np.stack([_np(st.kfac16)[b, h // G, :n].astype(np.float64), np.zeros(n)], axis=1)
        else:
            fac = _np(st.kfac)[b, h // G, :n]
        pu.check_scores(S4[b, h, :n], codes[b, h // G, :n], fac, planes[b, h], qs[b, h])


@pytest.mark.parametrize("B,Hq,Hkv,n,seq,compact", [
    (4, 64, 8, 5000, [4999, 1234, 0, 7], False),                        # G = 8, one round per wave
    (4, 64, 8, 5000, [4999, 1234, 0, 7], True),                         # compact index
    (16, 32, 8, 16384, [16383, 9000, 0, 4097, 1, 16000, 777, 12345,     # G = 4, four rounds per wave
                        16383, 3, 8191, 8192, 100, 15000, 2048, 64], False),
])
def test_matrix_core_scan_ragged(R, pipeline, B, Hq, Hkv, n, seq, compact):
    print("score forms ragged", B, Hq, Hkv, n, "compact" if compact else "full", flush=True)
    wl = gen.random_case(B, Hq, Hkv, n, seed=91 + B, kv_dtype="bf16", c_q_scale=0.0, key_offset=1.0)
    st = pipeline.DecodeState.from_workload(wl, c_q=False, compact=compact)
    st.build_index()
    st.quantize()
    S4, S3 = _two_forms(R, st, n, compact, seq_n=seq)
    codes, planes, qs = pu.u32(st.codes), pu.u32(st.qplanes), _np(st.qscal)
    G = Hq // Hkv
    for b in range(B):
        m = seq[b]   # entries past a sequence's count are unspecified
        assert np.array_equal(S4[b, :, :m].view(np.uint32), S3[b, :, :m].view(np.uint32))
        if m and b < 4:
            for h in (0, Hq - 1):
                if compact:
                    fac = np.stack([_np(st.kfac16)[b, h // G, :m].astype(np.float64), np.zeros(m)], axis=1)
                else:
                    fac = _np(st.kfac)[b, h // G, :m]
                pu.check_scores(S4[b, h, :m], codes[b, h // G, :m], fac, planes[b, h], qs[b, h])


def test_matrix_core_scan_integers_are_exact(R, pipeline):
    # at full-range codes and queries (all bits set, all query codes 15) the
    # integer part reaches its maximum 128 x 15; the reconstruction from the
    # oracle's exact integers must then match the matrix-core scores exactly
    B, Hq, Hkv, n, cap = 1, 64, 8, 1024, 1024
    print("score forms extremes", flush=True)
    rng = np.random.default_rng(5)
    codes = rng.integers(0, 2 ** 32, (B, Hkv, cap, 4), dtype=np.uint64).astype(np.uint32)
    codes[0, :, :16] = 0xFFFFFFFF
    codes[0, :, 16:32] = 0
    qcodes = rng.integers(0, 16, (B, Hq, 128))
    qcodes[0, 0] = 15
    qcodes[0, 1] = 0
    planes = np.stack([np.stack([orc.query_bit_planes(qcodes[b, h]) for h in range(Hq)]) for b in range(B)])
    kfac = np.stack([np.full((B, Hkv, cap), 0.75, np.float32), np.full((B, Hkv, cap), 0.125, np.float32)], -1)
    qs = np.zeros((B, Hq, 8), np.float32)
    qs[..., 0], qs[..., 1], qs[..., 3], qs[..., 4] = -1.0, 0.125, 2.0, 0.5
    qs[..., 2] = qcodes.sum(-1)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    S = torch.empty(B, Hq, n, device="cuda")
    R.rbq_score(B, Hq, Hkv, 128, n, cap, dev(codes.view(np.int32)), dev(kfac), dev(planes.view(np.int32)), dev(qs), S)
    torch.cuda.synchronize()
    S = _np(S)
    for h in range(Hq):
        bits = orc.unpack_bits(codes[0, h // 8, :n], 128)
        ip, pc = orc.int_dot(bits, qcodes[0, h])
        # every quantity here is a small dyadic rational: the fp32 result is exact
        X = 0.125 * (2.0 * ip - qcodes[0, h].sum()) + (-1.0) * (2.0 * pc - 128)
        ref = 2.0 * 0.75 * X + 0.5 + 0.125
        assert np.array_equal(S[0, h], ref.astype(np.float32)), h
