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
