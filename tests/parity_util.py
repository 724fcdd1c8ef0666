"""Comparison rules between the HIP path and the oracle (used by the GPU tests).

  * integers (popcounts, binary x INT4 dots, packed codes given the same fp32
    inputs, quantised query codes given the same rotated query): bit-exact.
  * sign codes from independent rotations: every differing bit has a rotated
    component |r_oracle| <= 1e-5 * ||k - c_k||.
  * scores: |S_gpu - S_oracle| <= 1e-5 * (sum of the magnitudes of the terms the
    fp32 kernel adds) + 1e-6, where the terms are |A f Delta (2 ip - S_u)|,
    |A f q_l (2 pc - D)|, |B0| and |g|.
  * Top-p sets: equal, except for keys whose score lies inside the boundary
    band: the scores at sorted positions whose oracle cumulative mass is within
    MASS_BAND of p (plus the boundary key), widened by 1e-6 relative. The GPU set
    must also be a valid threshold set (every key above its lowest selected
    score is selected).
  * attention outputs (fp32): 2e-3 absolute; log-sum-exp 1e-3 absolute.
"""
from __future__ import annotations

import numpy as np

from oracle import rbq_oracle as orc

# The GPU's cumulative softmax mass differs from the fp64 one by the 2^-40
# truncation of each mass (<= n 2^-40 of the top mass: 1.2e-7 at n = 2^17), the
# hardware exp2's ~1 ulp (1.2e-7 relative), and above all the fp32 rounding of
# the exponent's argument x = (S - m) tau log2(e): each of its two roundings is
# 2^-24 |x|, which moves a mass by ln2 2^-23 |x| relative, so the total moves by
# ln2 2^-23 times the mass-weighted mean of |x| (up to ~20 on the flat rows of
# the tests): ~2e-6 in all. The band is that with a margin for the exp2's ulps.
MASS_BAND = 5e-6
OUT_ATOL = 2e-3
LSE_ATOL = 1e-3
# The log-sum-exp inherits the rounding of the fp32 logits: a 128-term dot product
# accumulated in fp32 is off by at most ~128 * 2^-24 = 2^-17 of sum_i |q_i k_i|
# (the standard bound for n-term summation), and a common shift of the logits
# shifts the log-sum-exp by as much. Once |lse| passes 2^13, one fp32 ulp of it
# alone exceeds LSE_ATOL.
LSE_ACC_REL = 2.0 ** -17


def u32(t) -> np.ndarray:
    return t.detach().cpu().numpy().view(np.uint32)


def planes_to_codes(planes: np.ndarray) -> np.ndarray:
    """[planes][D/32] uint32 bit-planes (4, or 8 for B_q > 4) -> [D] query codes."""
    D = planes.shape[-1] * 32
    return sum(orc.unpack_bits(planes[j], D).astype(np.int64) << j for j in range(planes.shape[0]))


# The GPU rotates the unit query in fp32: each component is a D-term dot product
# of a column of P with u, whose fp32 rounding is at most D * 2^-24 * sum_j |P_jd u_j|
# <= D * 2^-24 (Cauchy-Schwarz, unit vectors): 7.6e-6 at D = 128. q_l and q_r are
# the minimum and maximum of those components, so each is within that of the
# oracle's, and Delta = (q_r - q_l) / 15 within 2/15 of it plus its own rounding.
ROT_ATOL = 1e-5


def check_qscal(qs, planes, q, P, c_q, c_k, D=128):
    """The per-head constants rbq_quantize_query wrote ({q_l, Delta, S_u, A, B0,
    q_r}) against the oracle's Algorithm 2 step 1 for the same query and
    centroids: A and B0 within fp32 rounding of their sums, q_l / q_r / Delta
    within the rotation bound above, and S_u exactly the sum of the GPU's codes."""
    ref = orc.quantize_query(np.asarray(q, np.float64), P, None if c_q is None else np.asarray(c_q, np.float64),
                             np.asarray(c_k, np.float64))
    qs = np.asarray(qs, np.float64)
    assert abs(qs[3] - ref["A"]) <= 1e-5 * ref["A"] + 1e-6, ("A", qs[3], ref["A"])
    assert abs(qs[4] - ref["B0"]) <= 1e-5 * float(np.abs(q) @ np.abs(c_k)) + 1e-6, ("B0", qs[4], ref["B0"])
    assert abs(qs[0] - ref["ql"]) <= ROT_ATOL, ("q_l", qs[0], ref["ql"])
    assert abs(qs[5] - ref["qr"]) <= ROT_ATOL, ("q_r", qs[5], ref["qr"])
    assert abs(qs[1] - ref["delta"]) <= 2 * ROT_ATOL / 15 + 2.0 ** -23 * abs(ref["delta"]), ("Delta", qs[1], ref["delta"])
    assert qs[2] == planes_to_codes(planes).sum(), ("S_u", qs[2])
    assert qs[6] == 0.0 and qs[7] == 0.0
    return ref


def check_encode_group(codes, kfac, c_k, K, P, c_q, rot=None, alpha=None, c_k_given=False):
    """Index rows of one (sequence, KV head) against the oracle's Algorithm 1 on
    the same keys: the centroid (unless it was given), the sign codes (bit-exact
    given the GPU's rotated values when `rot` is passed; end to end, every
    flipped bit lies within 1e-5 * ||x|| of zero), f and g to 1e-5 relative.
    codes [n][D/32] uint32, kfac [n][2], c_k [D], K [n][D] float64; returns the
    number of flipped bits."""
    K = np.asarray(K, np.float64)
    ck = np.asarray(c_k, np.float64)
    D = K.shape[1]
    if not c_k_given:
        assert np.abs(ck - orc.key_centroid(K)).max() <= 1e-5 * (np.abs(K).mean() + 1.0)
    enc = orc.encode_keys(K, P, c_k=ck, c_q=c_q)
    kfac = np.asarray(kfac, np.float64)
    nrm = enc["norm"]
    if rot is not None:
        r = np.asarray(rot, np.float64)
        assert np.array_equal(codes, orc.pack_bits(orc.sign_bits(r)))        # stage-wise exact
        assert np.all(np.abs(r - enc["R"]) <= 1e-5 * nrm[:, None] + 1e-30)
    diff = orc.unpack_bits(codes, D) != enc["bits"]
    assert np.all(np.abs(enc["R"][diff]) <= 1e-5 * np.broadcast_to(nrm[:, None], diff.shape)[diff])
    assert np.all(np.abs(kfac[:, 0] - enc["f"]) <= 1e-5 * np.abs(enc["f"]) + 1e-6)
    cq = np.zeros(D) if c_q is None else np.asarray(c_q, np.float64)
    gscale = np.abs(cq).sum() * np.abs(enc["X"]).max(axis=1)
    assert np.all(np.abs(kfac[:, 1] - enc["g"]) <= 1e-5 * gscale + 1e-6)
    if alpha is not None:
        a = np.asarray(alpha, np.float64)
        assert np.all(np.abs(a - enc["alpha"]) <= 1e-5 * enc["alpha"] + 1e-7)
    return int(diff.sum())


def score_tolerance(codes, f, g, qcodes, qs, D=128):
    bits = orc.unpack_bits(codes, D)
    ip, pc = orc.int_dot(bits, qcodes)
    ql, delta, su, A, B0 = (float(qs[i]) for i in range(5))
    terms = (np.abs(A * f * delta * (2 * ip - su)) + np.abs(A * f * ql * (2 * pc - D)) + abs(B0) + np.abs(g))
    return 1e-5 * terms + 1e-6


def check_scores(S_gpu, codes, kfac, qplanes, qs, D=128):
    """Scores of one query head against the keys of its group, on the GPU's codes."""
    qcodes = planes_to_codes(qplanes)
    f, g = kfac[:, 0].astype(np.float64), kfac[:, 1].astype(np.float64)
    ref = orc.scores_from_codes(codes, f, g, qcodes, float(qs[0]), float(qs[1]), int(qs[2]), float(qs[3]),
                                float(qs[4]))["S"]
    tol = score_tolerance(codes, f, g, qcodes, qs, D)
    err = np.abs(S_gpu.astype(np.float64) - ref)
    bad = np.nonzero(err > tol)[0]
    assert bad.size == 0, f"{bad.size} scores off, worst {err.max():.3e} at {int(np.argmax(err - tol))}"
    return ref


def check_topp(S_gpu_row: np.ndarray, p: float, sm_scale: float, sel_gpu: np.ndarray) -> dict:
    """GPU selection of one row vs the oracle's selection on the same fp32 scores."""
    S = S_gpu_row.astype(np.float64)
    o = orc.topp_select(S, p, sm_scale)
    got = np.asarray(sel_gpu, np.int64)
    assert np.all(np.diff(got) > 0), "GPU selection is not strictly ascending"
    if got.size:
        assert got[0] >= 0 and got[-1] < S.size
    if S.size == 0:
        assert got.size == 0
        return dict(oracle=o, diff=0)
    # a valid threshold set: nothing outside it scores above its lowest member
    if got.size and got.size < S.size:
        inside = np.zeros(S.size, bool)
        inside[got] = True
        assert S[inside].min() >= S[~inside].max(), "GPU selection is not a threshold set"
    diff = np.setxor1d(got, o["idx"])
    if diff.size:
        cum, order, m = o["cum"], o["order"], o["m_star"]
        band_pos = set(np.nonzero(np.abs(cum - p) <= MASS_BAND)[0].tolist()) | {m - 1}
        band_scores = S[order[sorted(band_pos)]]
        lo, hi = band_scores.min(), band_scores.max()
        slack = 1e-6 * max(abs(lo), abs(hi)) + 1e-12
        outside = diff[(S[diff] < lo - slack) | (S[diff] > hi + slack)]
        assert outside.size == 0, (f"{diff.size} keys differ, {outside.size} outside the tie band "
                                   f"(gpu {got.size}, oracle {o['idx'].size})")
    return dict(oracle=o, diff=int(diff.size))


def check_attention(out_gpu, lse_gpu, q, K, V, sel, K_loc, V_loc, sm_scale):
    ref = orc.sparse_decode(q, K, V, sel, K_loc, V_loc, sm_scale)
    err = np.abs(out_gpu.astype(np.float64) - ref["out"]).max() if ref["out"].size else 0.0
    assert err <= OUT_ATOL, f"attention output off by {err:.3e}"
    if lse_gpu is not None:
        if ref["lse"] == -np.inf:
            assert lse_gpu == -np.inf
        else:
            rows = [np.asarray(K, np.float64)[np.asarray(sel, np.int64)]]
            if K_loc is not None and len(K_loc):
                rows.append(np.asarray(K_loc, np.float64))
            mag = sm_scale * float((np.abs(np.concatenate(rows)) @ np.abs(np.asarray(q, np.float64))).max())
            tol = LSE_ATOL + LSE_ACC_REL * mag
            assert abs(float(lse_gpu) - ref["lse"]) <= tol, (float(lse_gpu), ref["lse"], tol)
    return err
