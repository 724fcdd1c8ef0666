"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks an oracle function against something other than itself: the
plain definition (q . k), a brute force over all codewords or subsets, a
closed form derived from the paper's Eq. 31 density, the statistical laws of
Theorem A.1 / Lemma A.5, the deterministic quantiser bound, an independent
library routine (torch's scaled_dot_product_attention, scipy's logsumexp and
beta distribution), or Algorithm 3 (a different selection procedure).
"""
import itertools
import math

import numpy as np
import pytest
import scipy.special
import scipy.stats

from oracle import rbq_oracle as orc
from workloads import gen


def _haar(D, seed):
    return gen.haar_rotations(D, 1, seed)[0]


# ---------------------------------------------------------------- Eq. decomposition
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_decomposition_is_exact_inner_product(seed):
    """Eq. decomposition with the exact <q_c, k_c> reproduces q . k (Section 3.1)."""
    rng = np.random.default_rng(seed)
    D = 128
    q, c_q = rng.standard_normal(D) * 3, rng.standard_normal(D)
    K, c_k = rng.standard_normal((5, D)) + 2.0, rng.standard_normal(D)
    P = _haar(D, seed)
    enc = orc.encode_keys(K, P, c_k=c_k, c_q=c_q)
    qq = orc.quantize_query(q, P, c_q, c_k)
    exact_cos = (enc["X"] / enc["norm"][:, None]) @ qq["u"]
    S = orc.assemble_score(qq["A"], enc["norm"], exact_cos, qq["B0"], enc["g"])
    for i in range(K.shape[0]):
        ref = math.fsum(float(a) * float(b) for a, b in zip(q, K[i]))
        assert abs(S[i] - ref) <= 1e-11 * max(1.0, abs(ref))


def test_centroid_is_mean():
    K = np.arange(12.0).reshape(4, 3)
    assert np.allclose(orc.key_centroid(K), [4.5, 5.5, 6.5])


# ---------------------------------------------------------------- rotation
def test_generator_rotation_is_orthogonal():
    for D in (64, 128):
        P = gen.haar_rotation(D).astype(np.float64)
        assert np.abs(P.T @ P - np.eye(D)).max() <= 1e-6
        assert np.abs(P @ P.T - np.eye(D)).max() <= 1e-6


def test_rotation_direction_and_norm():
    th = 0.3
    P = np.array([[math.cos(th), -math.sin(th)], [math.sin(th), math.cos(th)]])
    # r = P^T x; for x = e0 that is the first row of P
    assert np.allclose(orc.rotate(np.array([[1.0, 0.0]]), P)[0], [math.cos(th), -math.sin(th)])
    rng = np.random.default_rng(3)
    X = rng.standard_normal((50, 128))
    R = orc.rotate(X, _haar(128, 3))
    assert np.allclose(np.linalg.norm(R, axis=1), np.linalg.norm(X, axis=1), rtol=1e-12)


# ---------------------------------------------------------------- Eq. c_bar_eq_sign
@pytest.mark.parametrize("D", [4, 8, 12])
def test_sign_code_is_nearest_rotated_codeword(D):
    """The sign vector is the nearest codeword of the rotated hypercube (Appendix A.2)."""
    rng = np.random.default_rng(D)
    P = _haar(D, 100 + D)
    cands = np.array(list(itertools.product([-1.0, 1.0], repeat=D))) / math.sqrt(D)
    rotated = cands @ P.T                      # rows P c
    for _ in range(5):
        k = rng.standard_normal(D)
        enc = orc.encode_keys(k[None, :], P, c_k=np.zeros(D))
        kc = k / np.linalg.norm(k)
        best = np.argmin(((rotated - kc[None, :]) ** 2).sum(axis=1))
        assert np.array_equal(enc["bits"][0], (cands[best] > 0).astype(np.uint8))


def test_zero_component_gives_zero_bit():
    assert list(orc.sign_bits(np.array([0.0, -0.0, 1e-300, -1e-300]))) == [0, 0, 1, 0]


def test_packing_bit_order_and_roundtrip():
    bits = np.zeros(128, np.uint8)
    for d in (0, 31, 32, 127):
        bits[d] = 1
    w = orc.pack_bits(bits)
    assert list(w) == [1 | (1 << 31), 1, 0, 1 << 31]
    rng = np.random.default_rng(0)
    b = rng.integers(0, 2, (7, 128)).astype(np.uint8)
    assert np.array_equal(orc.unpack_bits(orc.pack_bits(b), 128), b)
    c = orc.codeword(b)
    assert np.allclose(np.abs(c), 1 / math.sqrt(128))
    assert np.array_equal((c > 0).astype(np.uint8), b)


def _golden(name):
    import os
    kv = {}
    with open(os.path.join(os.path.dirname(__file__), "golden", name)) as f:
        for ln in f:
            if ln.strip() and not ln.startswith("#"):
                k, v = ln.split(":", 1)
                kv[k.strip()] = float(v)
    return kv


def test_index_size_matches_appendix_c_case_study():
    """Appendix C prints eta = (D/8 + B_alpha) / (2 D B_data) = 18/512 ~ 3.5 % at D = 128 (FP16):
    the oracle's packed sign codes take exactly D/8 bytes per key."""
    g = _golden("index_overhead_fp16.txt")
    D = int(g["head_dim"])
    rng = np.random.default_rng(3)
    enc = orc.encode_keys(rng.standard_normal((5, D)), _haar(D, 3))
    code_bytes = enc["codes"].astype(np.uint32).nbytes // 5
    assert code_bytes == D // 8
    index = code_bytes + g["bytes_per_alpha"]
    kv = 2 * D * g["bytes_per_kv_element"]
    assert index == g["index_bytes_per_key_per_head"] and kv == g["kv_bytes_per_key_per_head"]
    assert round(100 * index / kv, 1) == g["eta_percent_printed"]


# ---------------------------------------------------------------- correction factor
def test_alpha_special_cases():
    D = 16
    I = np.eye(D)
    # a hypercube-vertex direction: the codeword is exact, alpha = 1
    v = np.where(np.arange(D) % 3 == 0, 1.0, -1.0)
    enc = orc.encode_keys(v[None, :], I, c_k=np.zeros(D))
    assert abs(enc["alpha"][0] - 1.0) < 1e-15
    # an axis direction: alpha = 1 / sqrt(D)
    enc = orc.encode_keys(I[2:3] * 5.0, I, c_k=np.zeros(D))
    assert abs(enc["alpha"][0] - 1 / math.sqrt(D)) < 1e-15
    # the centroid itself: norm 0 -> alpha' = 0 and f = 0
    enc = orc.encode_keys(np.ones((1, D)), I, c_k=np.ones(D))
    assert enc["norm"][0] == 0 and enc["alpha_p"][0] == 0 and enc["f"][0] == 0


@pytest.mark.slow
def test_alpha_mean_matches_eq31_closed_form():
    """E[alpha] = sqrt(D) E|x_1| for x uniform on the sphere, from the density of Eq. 31."""
    D, T = 128, 2000
    rng = np.random.default_rng(11)
    k = rng.standard_normal(D)
    alphas = []
    for chunk in range(4):
        for P in gen.haar_rotations(D, T // 4, 500 + chunk):
            alphas.append(orc.encode_keys(k[None, :], P, c_k=np.zeros(D))["alpha"][0])
    alphas = np.array(alphas)
    e_abs = math.exp(scipy.special.gammaln(D / 2) - scipy.special.gammaln((D + 1) / 2)) / math.sqrt(math.pi)
    expected = math.sqrt(D) * e_abs
    assert abs(expected - 0.79944) < 1e-5
    assert abs(alphas.mean() - expected) < 4 * alphas.std() / math.sqrt(T)
    assert np.all((alphas > 1 / math.sqrt(D)) & (alphas <= 1))


# ---------------------------------------------------------------- Theorem A.1 / Lemma A.5
def _estimates_over_rotations(cos, D, T, seed):
    rng = np.random.default_rng(seed)
    k = rng.standard_normal(D)
    k /= np.linalg.norm(k)
    e = rng.standard_normal(D)
    e -= (e @ k) * k
    e /= np.linalg.norm(e)
    q = cos * k + math.sqrt(1 - cos * cos) * e
    est, alpha = [], []
    for chunk in range(T // 500):
        for P in gen.haar_rotations(D, 500, seed * 100 + chunk):
            enc = orc.encode_keys(k[None, :], P, c_k=np.zeros(D))
            rq = orc.rotate_query(q, P)
            est.append(orc.estimate_unquantized(enc, rq["qrot"])[0])
            alpha.append(enc["alpha"][0])
    return np.array(est), np.array(alpha)


@pytest.mark.slow
def test_estimator_unbiased_and_residual_law():
    """Eq. EandP1 (mean -> true cosine) and Lemma A.5 (scaled residual ~ p_{D-1})."""
    D, T, cos = 128, 3000, 0.6
    est, alpha = _estimates_over_rotations(cos, D, T, seed=5)
    assert abs(est.mean() - cos) < 4 * est.std() / math.sqrt(T)
    z = (est - cos) * alpha / (np.sqrt(1 - alpha ** 2) * math.sqrt(1 - cos * cos))
    assert abs(z.mean()) < 4 / math.sqrt(T * (D - 1))
    assert abs(z.var() * (D - 1) - 1.0) < 0.1
    # (z + 1) / 2 ~ Beta((D-2)/2, (D-2)/2) is the density p_{D-1} of Eq. 31
    a = (D - 2) / 2
    assert scipy.stats.kstest((z + 1) / 2, scipy.stats.beta(a, a).cdf).pvalue > 1e-3
    # Eq. error_bound_P5 with a Gaussian constant: P(|X1| sqrt(D-1) > t) <= 2 exp(-t^2 / 2)
    for t in (1.5, 2.0, 2.5, 3.0):
        frac = np.mean(np.abs(z) * math.sqrt(D - 1) > t)
        bound = 2 * math.exp(-t * t / 2)
        assert frac <= bound + 3 * math.sqrt(bound * (1 - min(bound, 1)) / T) + 1e-9


def test_estimator_is_exact_when_query_equals_key():
    D = 128
    rng = np.random.default_rng(9)
    k = rng.standard_normal(D)
    c = rng.standard_normal(D)
    P = _haar(D, 9)
    enc = orc.encode_keys(k[None, :], P, c_k=c)
    rq = orc.rotate_query(k, P, c_q=c)
    assert abs(orc.estimate_unquantized(enc, rq["qrot"])[0] - 1.0) < 1e-12


# ---------------------------------------------------------------- quantiser (Theorem A.2)
@pytest.mark.parametrize("dtype", [np.float64, np.float32])
def test_quantizer_is_nearest_level_and_bounded(dtype):
    rng = np.random.default_rng(1)
    D = 128
    for _ in range(20):
        x = rng.standard_normal(D)
        x /= np.linalg.norm(x)
        qz = orc.uniform_quantize(x.astype(dtype), dtype=dtype)
        c = qz["codes"]
        assert c.min() == 0 and c.max() == 15
        assert c[np.argmin(x)] == 0 and c[np.argmax(x)] == 15
        levels = qz["ql"] + qz["delta"] * np.arange(16)
        brute = np.argmin(np.abs(x.astype(np.float64)[:, None] - levels[None, :]), axis=1)
        assert np.array_equal(c, brute)
        qbar = orc.dequantize(c, qz["ql"], qz["delta"])
        assert np.all(np.abs(qbar - x) <= qz["delta"] / 2 * (1 + 1e-6))
        signs = rng.choice([-1.0, 1.0], D)
        assert abs(signs @ (x - qbar)) <= D * qz["delta"] / 2


@pytest.mark.parametrize("bits", [1, 2, 3, 5, 6, 7, 8])
def test_quantizer_fewer_bits_is_nearest_level(bits):
    """B_q other than the paper's 4 (Theorem A.2): codes span [0, 2^B_q - 1] and
    each is the nearest of the 2^B_q levels (brute force), within Delta / 2."""
    rng = np.random.default_rng(10 + bits)
    D, top = 128, (1 << bits) - 1
    for _ in range(20):
        x = rng.standard_normal(D)
        x /= np.linalg.norm(x)
        qz = orc.uniform_quantize(x.astype(np.float32), dtype=np.float32, bits=bits)
        c = qz["codes"]
        assert c.min() == 0 and c.max() == top
        levels = qz["ql"] + qz["delta"] * np.arange(top + 1)
        brute = np.argmin(np.abs(x.astype(np.float32).astype(np.float64)[:, None] - levels[None, :]), axis=1)
        assert np.array_equal(c, brute)
        assert np.all(np.abs(orc.dequantize(c, qz["ql"], qz["delta"]) - x) <= qz["delta"] / 2 * (1 + 1e-6))


def test_one_bit_quantizer_is_the_midpoint_sign():
    rng = np.random.default_rng(5)
    x = rng.standard_normal(128)
    qz = orc.uniform_quantize(x, bits=1)
    assert np.array_equal(qz["codes"], (x >= (x.min() + x.max()) / 2).astype(np.int64))


def test_quantization_error_scales_with_the_step():
    """Theorem A.2: the quantisation error of <c_bar, q'> is a sum of D
    near-uniform errors of width Delta = range / (2^B_q - 1), so going from
    B_q = 2 to B_q = 4 divides it by (15 / 3) = 5."""
    D = 128
    rng = np.random.default_rng(6)
    err = {2: [], 4: []}
    for _ in range(400):
        x = rng.standard_normal(D)
        x /= np.linalg.norm(x)
        cbar = rng.choice([-1.0, 1.0], D) / math.sqrt(D)
        for b in err:
            qz = orc.uniform_quantize(x, bits=b)
            err[b].append(cbar @ (x - orc.dequantize(qz["codes"], qz["ql"], qz["delta"])))
    ratio = np.std(err[2]) / np.std(err[4])
    assert 4.0 < ratio < 6.0, ratio


def test_quantizer_degenerate_query():
    qz = orc.uniform_quantize(np.zeros(128))
    assert qz["delta"] == 0 and qz["codes"].sum() == 0
    qq = orc.quantize_query(np.ones(128), np.eye(128), np.ones(128), np.zeros(128))
    assert qq["A"] == 0 and qq["s_u"] == 0


@pytest.mark.slow
def test_quantization_error_below_estimator_error():
    """Theorem A.2 with B_q = 4 at D = 128: the quantisation error of <c_bar, q'> is
    of the same order as, and below, the O(1/sqrt(D)) estimation error."""
    D = 128
    rng = np.random.default_rng(2)
    errs = []
    for P in gen.haar_rotations(D, 300, 77):
        k = rng.standard_normal(D)
        q = rng.standard_normal(D)
        enc = orc.encode_keys(k[None, :], P, c_k=np.zeros(D))
        qq = orc.quantize_query(q, P, None, np.zeros(D))
        cbar = orc.codeword(enc["bits"][0])
        qbar = orc.dequantize(qq["codes"], qq["ql"], qq["delta"])
        errs.append(abs(cbar @ (qq["qrot"] - qbar)))
    assert np.mean(errs) < 1 / math.sqrt(D)


# ---------------------------------------------------------------- Eqs. kc_bar_dot_q_c2 / estk_cq_c
def test_integer_dot_and_reconstruction():
    rng = np.random.default_rng(4)
    D = 128
    bits = rng.integers(0, 2, (9, D)).astype(np.uint8)
    codes = rng.integers(0, 16, D)
    ip, pc = orc.int_dot(bits, codes)
    for i in range(9):
        assert ip[i] == sum(int(bits[i, d]) * int(codes[d]) for d in range(D))
        assert pc[i] == sum(int(b) for b in bits[i])
    # the bit-plane formulation: ip = sum_j 2^j popcount(code_word & plane_j)
    words = orc.pack_bits(bits)
    planes = orc.query_bit_planes(codes)
    for i in range(9):
        acc = 0
        for j in range(4):
            for w in range(D // 32):
                acc += (1 << j) * bin(int(words[i, w]) & int(planes[j, w])).count("1")
        assert acc == ip[i]
    assert np.array_equal(sum((orc.unpack_bits(planes[j], D).astype(np.int64) << j) for j in range(4)), codes)
    # eight planes hold 8-bit codes: ip = sum_{j < 8} 2^j popcount(word & plane_j)
    codes8 = rng.integers(0, 256, D)
    planes8 = orc.query_bit_planes(codes8, planes=8)
    ip8, _ = orc.int_dot(bits, codes8)
    for i in range(9):
        acc = sum((1 << j) * bin(int(words[i, w]) & int(planes8[j, w])).count("1")
                  for j in range(8) for w in range(D // 32))
        assert acc == ip8[i] == sum(int(bits[i, d]) * int(codes8[d]) for d in range(D))
    # the reconstruction equals <2 c_b - 1, Delta q_u + q_l 1> evaluated directly
    ql, delta = -0.21, 0.028
    X = orc.reconstruct(ip, pc, ql, delta, int(codes.sum()), D)
    direct = (2.0 * bits - 1.0) @ (delta * codes + ql)
    assert np.allclose(X, direct, rtol=0, atol=1e-12)


def test_score_paths_agree():
    """estimate_scores == <c_bar, q_bar> / alpha assembled, and == scores_from_codes."""
    w = gen.random_case(1, 4, 1, 200, seed=3, kv_dtype="f32", c_q_scale=0.5, key_offset=1.0)
    K = w.K_f32(0, 0)
    enc = orc.encode_keys(K, w.P, c_q=w.c_q[0, 0])
    for h in range(4):
        qq = orc.quantize_query(w.q[0, h], w.P, w.c_q[0, 0], enc["c_k"])
        est = orc.estimate_scores(enc, qq)
        qbar = orc.dequantize(qq["codes"], qq["ql"], qq["delta"])
        s_norm = (orc.codeword(enc["bits"]) @ qbar) / enc["alpha"]
        S = qq["A"] * enc["norm"] * s_norm + qq["B0"] + enc["g"]
        assert np.allclose(est["S"], S, rtol=1e-12, atol=1e-12)
        alt = orc.scores_from_codes(enc["codes"], enc["f"], enc["g"], qq["codes"], qq["ql"], qq["delta"],
                                    qq["s_u"], qq["A"], qq["B0"])
        assert np.allclose(alt["S"], est["S"], rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- the compact index (Appendix C)
def _is_binary16(v):
    """v (float64) lies in the IEEE binary16 set: 0, or |v| <= 65504 with an
    11-bit significand (normal: 2^(e-10) steps for 2^e <= |v| < 2^(e+1),
    e >= -14; subnormal: multiples of 2^-24)."""
    a = np.abs(np.asarray(v, np.float64))
    ok = a <= 65504.0
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    step = np.where(a >= 2.0 ** -14, 2.0 ** (e - 10), 2.0 ** -24)
    return ok & ((a == 0) | (a / step == np.round(a / step)))


def test_compact_factor_is_ieee_binary16_rounding():
    """Cases worked from the binary16 definition (11-bit significand, round to
    nearest, ties to the even significand), independent of NumPy's float16."""
    u = 2.0 ** -10                       # spacing at [1, 2)
    cases = [
        (1.0, 1.0), (1.0 + u, 1.0 + u),
        (1.0 + u / 2, 1.0),                          # tie -> even significand (1.0)
        (1.0 + 3 * u / 2, 1.0 + 2 * u),              # tie between odd 1+u and even 1+2u
        (1.0 + u / 2 + 2.0 ** -30, 1.0 + u),         # just above the tie
        (2049.0, 2048.0), (2051.0, 2052.0),          # spacing 2 on [2048, 4096): ties to even
        (2050.9, 2050.0), (2051.1, 2052.0),
        (65504.0, 65504.0), (65519.0, 65504.0), (65520.0, 65504.0), (1e9, 65504.0),   # saturation
        (0.0, 0.0), (2.0 ** -24, 2.0 ** -24),        # zero, the smallest subnormal
        (2.0 ** -25, 0.0),                           # tie between 0 (even) and 2^-24 (odd)
        (3 * 2.0 ** -25, 2.0 ** -23),                # tie between 2^-24 (odd) and 2^-23 (even)
        (1.0 / 3.0, 1365 * 2.0 ** -12),              # 0x3555: 1.0101010101b x 2^-2
    ]
    for x, want in cases:
        assert orc.compact_factor(np.array([x]))[0] == want, x
    # random normal-range factors: in the binary16 set, within half a spacing (2^-11 relative)
    rng = np.random.default_rng(8)
    f = np.exp(rng.uniform(np.log(1e-3), np.log(6e4), 20000))
    c = orc.compact_factor(f)
    assert _is_binary16(c).all()
    assert np.all(np.abs(c - f) <= 2.0 ** -11 * np.abs(f))
    # nearest: no binary16 neighbour of c is closer to f
    e = np.floor(np.log2(c))
    step = 2.0 ** (e - 10)
    assert (_is_binary16(c - step) & _is_binary16(c + step)).all()
    for nb in (c - step, c - step / 2, c + step):   # neighbours below (half a step below a power of two) and above
        ok = _is_binary16(nb) & (nb != c)
        assert np.all(np.abs(nb - f)[ok] >= np.abs(c - f)[ok])


def test_compact_index_scores_and_size():
    """Appendix C's index: D/8 bytes of codes + one 2-byte factor per key and
    head, 18 bytes at D = 128 (the printed eta = 18/512 ~ 3.5 %). Its scores
    are the full estimate with g = 0 and f rounded to binary16, so each stays
    within 2^-11 |A f X| of the fp64 estimate, and the Top-p sets stay close."""
    g = _golden("index_overhead_fp16.txt")
    D = int(g["head_dim"])
    assert D // 8 + np.dtype(np.float16).itemsize == g["index_bytes_per_key_per_head"]
    w = gen.random_case(1, 4, 1, 3000, seed=9, kv_dtype="f32", c_q_scale=0.0, key_offset=1.0, q_scale=6.0)
    K = w.K_f32(0, 0)
    enc = orc.encode_keys(K, w.P)
    f16 = orc.compact_factor(enc["f"])
    assert np.all(f16 > 0)
    same = 0
    for h in range(4):
        qq = orc.quantize_query(w.q[0, h], w.P, None, enc["c_k"])
        full = orc.scores_from_codes(enc["codes"], enc["f"], enc["g"], qq["codes"], qq["ql"], qq["delta"],
                                     qq["s_u"], qq["A"], qq["B0"])
        comp = orc.scores_from_codes(enc["codes"], f16, np.zeros_like(f16), qq["codes"], qq["ql"], qq["delta"],
                                     qq["s_u"], qq["A"], qq["B0"])
        bound = 2.0 ** -11 * np.abs(qq["A"] * enc["f"] * full["X"]) + 1e-12
        assert np.all(np.abs(comp["S"] - full["S"]) <= bound)
        a = orc.topp_select(full["S"], 0.9, 1 / np.sqrt(D))["idx"]
        b = orc.topp_select(comp["S"], 0.9, 1 / np.sqrt(D))["idx"]
        same += np.intersect1d(a, b).size / max(a.size, b.size)
    assert same / 4 > 0.95


def test_estimate_tracks_true_scores():
    """On keys shaped like an LLM's, the estimate correlates strongly with q . k."""
    w = gen.config1()
    K = w.K_f32(0, 0)
    enc = orc.encode_keys(K, w.P)
    qq = orc.quantize_query(w.q[0, 0], w.P, None, enc["c_k"])
    S = orc.estimate_scores(enc, qq)["S"]
    true = K.astype(np.float64) @ w.q[0, 0].astype(np.float64)
    assert np.corrcoef(S, true)[0, 1] > 0.9


# ---------------------------------------------------------------- Top-p
def _brute_min_sets(pi, p):
    n = len(pi)
    best, sets = None, []
    for r in range(1, n + 1):
        for comb in itertools.combinations(range(n), r):
            if sum(pi[list(comb)]) >= p:
                sets.append(set(comb))
        if sets:
            return sets
    return [set(range(n))]


@pytest.mark.parametrize("seed", range(6))
def test_topp_is_minimal_set(seed):
    rng = np.random.default_rng(seed)
    n = 9
    S = rng.standard_normal(n) * 3
    pi = orc.softmax(S)
    for p in (0.3, 0.6, 0.9, 0.99):
        sel = set(orc.topp_select(S, p, 1.0)["idx"].tolist())
        assert sel in _brute_min_sets(pi, p)


def test_topp_ties_and_limits():
    S = np.array([3.0, 2.0, 2.0, 1.0, 0.0])
    pi = orc.softmax(S)
    p = pi[0] + 0.5 * pi[1]
    assert orc.topp_select(S, p, 1.0)["idx"].tolist() == [0, 1, 2]
    assert orc.topp_select(S, 1.0, 1.0)["idx"].tolist() == [0, 1, 2, 3, 4]
    assert orc.topp_select(S, 1e-9, 1.0)["idx"].tolist() == [0]
    assert orc.topp_select(np.full(6, 0.5), 0.4, 1.0)["idx"].tolist() == list(range(6))
    assert orc.topp_select(np.zeros(0), 0.5, 1.0)["idx"].size == 0


@pytest.mark.parametrize("seed", range(4))
def test_topp_agrees_with_algorithm3(seed):
    rng = np.random.default_rng(seed)
    S = rng.standard_normal(2000) * 4
    tau = 1 / math.sqrt(128) * 8
    for p in (0.5, 0.8, 0.9, 0.95):
        sel = orc.topp_select(S, p, tau)
        cum = sel["cum"]
        m = sel["m_star"]
        if abs(cum[m - 1] - p) < 1e-9 or (m > 1 and abs(cum[m - 2] - p) < 1e-9):
            continue
        alg3 = orc.topp_threshold_alg3(orc.softmax(S * tau), p)
        assert np.array_equal(np.nonzero(alg3["mask"])[0], sel["idx"])


# ---------------------------------------------------------------- attention
def test_attention_matches_torch_sdpa():
    import torch
    rng = np.random.default_rng(8)
    D, n, w = 128, 300, 20
    K, V = rng.standard_normal((n, D)), rng.standard_normal((n, D))
    Kl, Vl = rng.standard_normal((w, D)), rng.standard_normal((w, D))
    q = rng.standard_normal(D) * 2
    sel = np.sort(rng.choice(n, 40, replace=False))
    scale = 1 / math.sqrt(D)
    got = orc.sparse_decode(q, K, V, sel, Kl, Vl, scale)
    Kall, Vall = np.concatenate([K, Kl]), np.concatenate([V, Vl])
    mask = np.zeros(n + w, bool)
    mask[sel] = True
    mask[n:] = True
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))
    ref = torch.nn.functional.scaled_dot_product_attention(
        t(q)[None, None, None], t(Kall)[None, None], t(Vall)[None, None], attn_mask=t(mask)[None, None, None],
        scale=scale)[0, 0, 0].numpy()
    assert np.allclose(got["out"], ref, rtol=0, atol=1e-12)
    lse = scipy.special.logsumexp((Kall[mask] @ q) * scale)
    assert abs(got["lse"] - lse) < 1e-12
    # identical keys: plain mean of the values; empty set: zeros and -inf
    same = orc.attention(q, np.tile(K[:1], (5, 1)), V[:5], scale)
    assert np.allclose(same["out"], V[:5].mean(axis=0), atol=1e-13)
    empty = orc.attention(q, np.zeros((0, D)), np.zeros((0, D)), scale)
    assert np.all(empty["out"] == 0) and empty["lse"] == -np.inf


def test_end_to_end_budget_and_recall_trends():
    """Budget grows with p; the selection recovers most of the exact attention mass."""
    w = gen.config2(N=4096)
    b, hk = 0, 3
    K = w.K_f32(b, hk)
    V = w.V_f32(b, hk)
    Q = w.q[b, hk * w.G:(hk + 1) * w.G]
    budgets, mean_recalls = [], []
    for p in (0.5, 0.8, 0.9, 0.99):
        res = orc.decode_group(K, V, K[:0], V[:0], Q, w.P, p)
        sizes = [h["sel"]["idx"].size for h in res["heads"]]
        budgets.append(sum(sizes))
        recalls = [orc.attention_recall(Q[g], K, res["heads"][g]["sel"]["idx"], 1 / math.sqrt(128))
                   for g in range(w.G)]
        mean_recalls.append(float(np.mean(recalls)))
        if p >= 0.8:   # tiny sets (p = 0.5: a few keys per head) lose more to estimator noise
            assert mean_recalls[-1] > p - 0.2
    assert budgets == sorted(budgets)
    assert mean_recalls == sorted(mean_recalls)
