"""CPU oracle for RaBitQCache's decode path -- TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 NumPy implementation of what the paper computes at a
decode step, written from the paper: index construction (Algorithm 1),
query rotation and INT4 quantisation (Section 3.3, Appendix A.3.2), the
binary x INT4 score estimate (Eq. estimator_core, Eqs. kc_bar_dot_q_c2 and
estk_cq_c, Eq. decomposition), adaptive Top-p selection (Algorithm 2 step 3,
Section 4.1) and attention over the selected keys plus the local window
(Algorithm 2 step 4, Section 3.4).

Only the tests, the package's smoke check and the bench's CPU-baseline leg
may import this module. It shares no code, table or helper with the HIP
library, and the library never calls it.

Conventions (readings of the paper where it is silent or inconsistent):
  * rotation: r = P^T x, i.e. the row vector x @ P, for keys and queries alike
    (Section 3.1 writes sign(P^T k_c) and q' = P^T q_c; Algorithm 1 writes
    (K - c_k) P^T in one place and (K - c_k) P in the text; the P^T form of
    Section 3.1 / Appendix A.2 is taken).
  * sign bit: 1 iff the rotated component is strictly positive (Appendix
    A.2), so +-0 gives 0.
  * packed codes: dimension d lives in 32-bit word d // 32 at bit d % 32.
  * correction factor: alpha' = <c_bar', P^T k_c> = sum_j |r_j| / ||x||
    (Appendix A.2's stored quantity); the paper-unit alpha = alpha' / sqrt(D).
  * quantiser step: Delta = (q_r - q_l) / (2^B_q - 1) with no rounding of the
    step (Appendix A.3.2); deterministic rounding floor(t + 1/2).
  * degenerate vectors: ||x|| = 0 gives f = 0; ||q - c_q|| = 0 gives u = 0,
    Delta = 0 and all codes 0.
  * compact index: f stored as IEEE binary16, saturated at 65504, rounded
    to nearest with ties to even; no g, hence c_q = 0 (Appendix C).
  * Top-p: the smallest prefix of keys sorted by estimated score whose
    softmax(S / sqrt(D)) mass reaches p, extended to every key tied with the
    last one; p >= 1 keeps every key.
  * parity unpinned: none. Every function below is pinned by a test in
    tests/test_oracle_pins.py against a closed form, a brute force, a
    textbook/library routine or a statistical law the paper states.
"""
from __future__ import annotations

import numpy as np

B_Q = 4                      # query bits, Section 3.3 / Theorem A.2 (B_q = 4)
Q_LEVELS = (1 << B_Q) - 1    # 15


# ---------------------------------------------------------------------------
# Index construction (Algorithm 1; Section 3.2; Appendix A.2)
# ---------------------------------------------------------------------------
def key_centroid(K: np.ndarray) -> np.ndarray:
    """Algorithm 1, step 1: the centroid c_k of a batch of keys [n][D]."""
    K = np.asarray(K, dtype=np.float64)
    return K.sum(axis=0) / K.shape[0]


def rotate(X: np.ndarray, P: np.ndarray) -> np.ndarray:
    """P^T x for every row x of X (Section 3.1, Appendix A.2): the rows of X @ P."""
    return np.asarray(X, np.float64) @ np.asarray(P, np.float64)


def sign_bits(R: np.ndarray) -> np.ndarray:
    """Nearest hypercube codeword as bits: 1 iff the component is > 0 (Eq. c_bar_eq_sign)."""
    return (np.asarray(R) > 0).astype(np.uint8)


def pack_bits(bits: np.ndarray) -> np.ndarray:
    """[..., D] 0/1 -> [..., D/32] uint32, dimension d at word d // 32, bit d % 32."""
    bits = np.asarray(bits, np.uint64)
    D = bits.shape[-1]
    assert D % 32 == 0
    b = bits.reshape(bits.shape[:-1] + (D // 32, 32))
    weights = np.uint64(1) << np.arange(32, dtype=np.uint64)
    return (b * weights).sum(axis=-1).astype(np.uint32)


def unpack_bits(words: np.ndarray, D: int) -> np.ndarray:
    """Inverse of pack_bits."""
    words = np.asarray(words, np.uint32)
    sh = np.arange(32, dtype=np.uint32)
    b = (words[..., :, None] >> sh) & np.uint32(1)
    return b.reshape(words.shape[:-1] + (D,)).astype(np.uint8)


def codeword(bits: np.ndarray) -> np.ndarray:
    """c_bar = (2 c_b - 1) / sqrt(D) (Appendix A.2)."""
    bits = np.asarray(bits, np.float64)
    return (2.0 * bits - 1.0) / np.sqrt(bits.shape[-1])


def encode_keys(K: np.ndarray, P: np.ndarray, c_k: np.ndarray | None = None,
                c_q: np.ndarray | None = None) -> dict:
    """Algorithm 1 for one (sequence, KV head): keys K [n][D].

    If c_k is None the centroid of K is computed (prefill); otherwise the given
    prefill centroid is reused (Section 3.1: centroids from the prefill stay
    valid for later tokens). Returns the centred keys, their norms, the
    rotated keys, the sign bits and packed codes, alpha' and the paper-unit
    alpha, and the per-key factors f = ||x|| / alpha' and g = <c_q, x>.
    """
    K = np.asarray(K, np.float64)
    n, D = K.shape
    if c_k is None:
        c_k = key_centroid(K) if n > 0 else np.zeros(D)
    c_k = np.asarray(c_k, np.float64)
    c_q = np.zeros(D) if c_q is None else np.asarray(c_q, np.float64)
    X = K - c_k[None, :]                              # Algorithm 1, centring
    norm = np.sqrt((X * X).sum(axis=1))               # ||k - c_k||
    R = rotate(X, P)                                  # Algorithm 1, step 2
    bits = sign_bits(R)                               # Algorithm 1, step 3
    # alpha' = <c_bar', P^T k_c> with c_bar' = 2 c_b - 1 and k_c = x / ||x||
    cbar_p = 2.0 * bits.astype(np.float64) - 1.0
    with np.errstate(invalid="ignore", divide="ignore"):
        alpha_p = np.where(norm > 0, (cbar_p * R).sum(axis=1) / norm, 0.0)
        f = np.where(alpha_p > 0, norm / alpha_p, 0.0)
    g = X @ c_q                                       # <c_q, k> - <c_q, c_k>
    return dict(c_k=c_k, X=X, norm=norm, R=R, bits=bits, codes=pack_bits(bits) if D % 32 == 0 else None,
                alpha_p=alpha_p, alpha=alpha_p / np.sqrt(D), f=f, g=g)


def compact_factor(f) -> np.ndarray:
    """The per-key factor f as the compact index keeps it: the paper stores the
    one scalar per key and head in FP16 (Appendix C, the correction factor's
    storage; B_alpha = 2 bytes). Saturated at 65504, the largest finite IEEE
    binary16 value (a reading: the paper does not treat values beyond the
    range), then rounded to the nearest binary16 value with ties to even
    (NumPy's float64 -> float16 conversion); returned as float64. The compact
    index keeps no g, so it goes with c_q = 0."""
    f = np.minimum(np.asarray(f, np.float64), 65504.0)
    return f.astype(np.float16).astype(np.float64)


# ---------------------------------------------------------------------------
# Query pre-processing and INT4 quantisation (Algorithm 2 step 1; Section 3.3;
# Appendix A.3.2)
# ---------------------------------------------------------------------------
def rotate_query(q: np.ndarray, P: np.ndarray, c_q: np.ndarray | None = None) -> dict:
    """q_c = (q - c_q) / ||q - c_q||, q' = P^T q_c (Algorithm 2, step 1)."""
    q = np.asarray(q, np.float64)
    c_q = np.zeros_like(q) if c_q is None else np.asarray(c_q, np.float64)
    y = q - c_q
    A = float(np.sqrt((y * y).sum()))
    u = y / A if A > 0 else np.zeros_like(y)
    return dict(A=A, u=u, qrot=rotate(u[None, :], P)[0])


def uniform_quantize(qrot: np.ndarray, dtype=np.float64, bits: int = B_Q) -> dict:
    """Uniform scalar quantiser of Appendix A.3.2 with B_q = `bits` (4 in the paper).

    [q_l, q_r] is the value range of q', Delta = (q_r - q_l) / (2^B_q - 1) and
    q_u = Round((q' - q_l) / Delta) with Round(t) = floor(t + 1/2), kept in
    [0, 2^B_q - 1]. Every operation is evaluated in `dtype`: float64 for the
    oracle's own path, float32 where the decision has to be taken in the
    kernel's precision (the quantised code is an integer decided by floating
    point).
    """
    levels = (1 << bits) - 1
    x = np.asarray(qrot, dtype=dtype)
    ql, qr = x.min(), x.max()
    delta = dtype((qr - ql) / dtype(levels))
    if delta > 0:
        t = (x - ql) / delta + dtype(0.5)
        codes = np.clip(np.floor(t), 0, levels).astype(np.int64)
    else:
        codes = np.zeros(x.shape, np.int64)
    return dict(ql=float(ql), qr=float(qr), delta=float(delta), codes=codes, s_u=int(codes.sum()))


def dequantize(codes: np.ndarray, ql: float, delta: float) -> np.ndarray:
    """q_bar = Delta * q_u + q_l * 1 (Appendix A.3.2)."""
    return delta * np.asarray(codes, np.float64) + ql


def quantize_query(q: np.ndarray, P: np.ndarray, c_q: np.ndarray | None, c_k: np.ndarray,
                   bits: int = B_Q) -> dict:
    """Rotation, B_q-bit (INT4 by default) quantisation and the per-query
    constants of Eq. decomposition.

    Returns A = ||q - c_q||, q', the quantiser (q_l, Delta, codes, S_u = sum q_u)
    and B0 = <q, c_k>.
    """
    rq = rotate_query(q, P, c_q)
    qz = uniform_quantize(rq["qrot"], bits=bits)
    return dict(A=rq["A"], u=rq["u"], qrot=rq["qrot"], ql=qz["ql"], qr=qz["qr"], delta=qz["delta"],
                codes=qz["codes"], s_u=qz["s_u"],
                B0=float(np.asarray(q, np.float64) @ np.asarray(c_k, np.float64)))


def query_bit_planes(codes: np.ndarray, planes: int = B_Q) -> np.ndarray:
    """Bit-plane j of the query codes, packed like the key codes: [planes][D/32]
    uint32 (4 planes for the INT4 codes of Section 3.3; 8 hold codes of up to
    8 bits)."""
    codes = np.asarray(codes, np.int64)
    return np.stack([pack_bits(((codes >> j) & 1).astype(np.uint8)) for j in range(planes)])


# ---------------------------------------------------------------------------
# Score estimation (Algorithm 2 step 2; Eqs. estimator_core, kc_bar_dot_q_c2,
# estk_cq_c, decomposition)
# ---------------------------------------------------------------------------
def int_dot(bits: np.ndarray, codes: np.ndarray) -> tuple:
    """<c_b, q_u> and popcount(c_b) per key, from unpacked bits (exact integers)."""
    b = np.asarray(bits, np.int64)
    return b @ np.asarray(codes, np.int64), b.sum(axis=-1)


def reconstruct(ip, pc, ql: float, delta: float, s_u: int, D: int):
    """<c_bar', q_bar> = 2 Delta <c_b, q_u> + 2 q_l sum c_b - Delta sum q_u - D q_l."""
    ip = np.asarray(ip, np.float64)
    pc = np.asarray(pc, np.float64)
    return 2.0 * delta * ip + 2.0 * ql * pc - delta * s_u - D * ql


def normalized_estimate(X_rec, alpha_p):
    """Eq. estk_cq_c: <q_c, k_c> ~ <c_bar', q_bar> / <c_bar', P^T k_c> (0 where alpha' = 0)."""
    X_rec = np.asarray(X_rec, np.float64)
    alpha_p = np.asarray(alpha_p, np.float64)
    with np.errstate(invalid="ignore", divide="ignore"):
        return np.where(alpha_p > 0, X_rec / alpha_p, 0.0)


def assemble_score(A: float, norm, s_norm, B0: float, g):
    """Eq. decomposition: <q,k> = ||q-c_q|| ||k-c_k|| <q_c,k_c> + <q,c_k> + <c_q,k> - <c_q,c_k>,
    with <c_q,k> - <c_q,c_k> = g = <c_q, k - c_k>."""
    return A * np.asarray(norm, np.float64) * np.asarray(s_norm, np.float64) + B0 + np.asarray(g, np.float64)


def estimate_scores(enc: dict, qq: dict) -> dict:
    """All of Algorithm 2 step 2 for one query against the encoded keys."""
    D = enc["bits"].shape[-1]
    ip, pc = int_dot(enc["bits"], qq["codes"])
    X_rec = reconstruct(ip, pc, qq["ql"], qq["delta"], qq["s_u"], D)
    s_norm = normalized_estimate(X_rec, enc["alpha_p"])
    S = assemble_score(qq["A"], enc["norm"], s_norm, qq["B0"], enc["g"])
    return dict(ip=ip, pc=pc, X=X_rec, s_norm=s_norm, S=S)


def scores_from_codes(codes: np.ndarray, f: np.ndarray, g: np.ndarray, q_codes: np.ndarray, ql: float,
                      delta: float, s_u: int, A: float, B0: float) -> dict:
    """The same estimate starting from packed codes and the stored per-key
    factors f = ||x|| / alpha' and g (A * ||x|| * X / alpha' = A * f * X)."""
    D = codes.shape[-1] * 32
    bits = unpack_bits(codes, D)
    ip, pc = int_dot(bits, q_codes)
    X_rec = reconstruct(ip, pc, ql, delta, s_u, D)
    S = A * np.asarray(f, np.float64) * X_rec + B0 + np.asarray(g, np.float64)
    return dict(ip=ip, pc=pc, X=X_rec, S=S)


def estimate_unquantized(enc: dict, qrot: np.ndarray) -> np.ndarray:
    """Eq. estimator_core without query quantisation: <c_bar, q'> / alpha."""
    cbar = codeword(enc["bits"])
    with np.errstate(invalid="ignore", divide="ignore"):
        return np.where(enc["alpha"] > 0, (cbar @ np.asarray(qrot, np.float64)) / enc["alpha"], 0.0)


# ---------------------------------------------------------------------------
# Adaptive Top-p selection (Algorithm 2 step 3; Section 4.1)
# ---------------------------------------------------------------------------
def softmax(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, np.float64)
    e = np.exp(x - x.max())
    return e / e.sum()


def topp_select(S: np.ndarray, p: float, sm_scale: float) -> dict:
    """I = the smallest set of keys whose softmax(S * sm_scale) mass is >= p.

    Keys are ranked by S (descending); m* is the shortest prefix whose
    cumulative mass reaches p; s* is the score at that position; every key
    with S >= s* is kept (ties at the boundary included). p >= 1 keeps all.
    Returns the ascending indices plus s*, m* and the sorted cumulative mass
    (the latter for judging near-ties).
    """
    S = np.asarray(S, np.float64)
    n = S.shape[0]
    if n == 0:
        return dict(idx=np.zeros(0, np.int64), s_star=np.inf, m_star=0, cum=np.zeros(0), order=np.zeros(0, np.int64))
    pi = softmax(S * sm_scale)
    order = np.argsort(-S, kind="stable")
    cum = np.cumsum(pi[order])
    if p >= 1.0:
        m_star = n
    else:
        hit = np.nonzero(cum >= p)[0]
        m_star = int(hit[0]) + 1 if hit.size else n
    s_star = S[order[m_star - 1]]
    idx = np.nonzero(S >= s_star)[0]
    return dict(idx=idx, s_star=float(s_star), m_star=m_star, cum=cum, order=order)


def topp_threshold_alg3(probs: np.ndarray, p: float, max_iter: int = 500) -> dict:
    """Algorithm 3's ternary search on probabilities, with an iteration cap.

    Two pivots split (low, high]; the masses above each pivot and the tightest
    data bounds inside the interval decide which third to drop, until one
    distinct value is left in (low, high]. The mask is probs > low.
    """
    s = np.asarray(probs, np.float64)
    low, high = 0.0, float(s.max())
    it = 0
    while it < max_iter:
        it += 1
        pv0 = (high + 2.0 * low) / 3.0
        pv1 = (2.0 * high + low) / 3.0
        g0 = s[s > pv0].sum()
        g1 = s[s > pv1].sum()
        above = s[s > low]
        below = s[s <= high]
        v_min = above.min() if above.size else np.inf
        v_max = below.max() if below.size else -np.inf
        if g1 >= p:
            low = pv1
        elif g0 >= p:
            low = pv0
            high = min(pv1, v_max)
        else:
            high = min(pv0, v_max)
        if v_min == v_max:
            break
    return dict(theta=low, mask=s > low, iters=it)


# ---------------------------------------------------------------------------
# Hybrid sparse attention (Algorithm 2 step 4; Section 3.4)
# ---------------------------------------------------------------------------
def attention(q: np.ndarray, Krows: np.ndarray, Vrows: np.ndarray, sm_scale: float) -> dict:
    """softmax(q K^T * sm_scale) V over the given rows (Section 2.1), with its log-sum-exp.

    With no rows the output is 0 and lse is -inf.
    """
    Krows = np.asarray(Krows, np.float64)
    Vrows = np.asarray(Vrows, np.float64)
    if Krows.shape[0] == 0:
        return dict(out=np.zeros(Vrows.shape[-1] if Vrows.ndim == 2 else np.asarray(q).shape[-1]), lse=-np.inf)
    logits = (Krows @ np.asarray(q, np.float64)) * sm_scale
    m = logits.max()
    e = np.exp(logits - m)
    z = e.sum()
    return dict(out=(e @ Vrows) / z, lse=float(m + np.log(z)))


def sparse_decode(q: np.ndarray, K: np.ndarray, V: np.ndarray, sel: np.ndarray, K_loc: np.ndarray,
                  V_loc: np.ndarray, sm_scale: float) -> dict:
    """Attn(q, K[I] u K_local, V[I] u V_local) (Algorithm 2 step 4): the selected
    rows of the indexed cache together with every row of the local window."""
    sel = np.asarray(sel, np.int64)
    Kr = np.concatenate([np.asarray(K, np.float64)[sel], np.asarray(K_loc, np.float64)], axis=0)
    Vr = np.concatenate([np.asarray(V, np.float64)[sel], np.asarray(V_loc, np.float64)], axis=0)
    return attention(q, Kr, Vr, sm_scale)


def attention_recall(q: np.ndarray, K: np.ndarray, sel: np.ndarray, sm_scale: float) -> float:
    """Share of the exact attention over the indexed keys held by the selected ones (Table 1)."""
    pi = softmax((np.asarray(K, np.float64) @ np.asarray(q, np.float64)) * sm_scale)
    return float(pi[np.asarray(sel, np.int64)].sum())


# ---------------------------------------------------------------------------
# One decode step for one (sequence, KV head) group
# ---------------------------------------------------------------------------
def decode_group(K_index: np.ndarray, V_index: np.ndarray, K_loc: np.ndarray, V_loc: np.ndarray,
                 Q: np.ndarray, P: np.ndarray, p: float, c_q: np.ndarray | None = None,
                 sm_scale: float | None = None, c_k: np.ndarray | None = None) -> dict:
    """Algorithms 1 and 2 end to end for the G query heads Q [G][D] of one KV group."""
    D = K_index.shape[-1]
    sm_scale = 1.0 / np.sqrt(D) if sm_scale is None else sm_scale
    enc = encode_keys(K_index, P, c_k=c_k, c_q=c_q)
    outs = []
    for q in np.asarray(Q, np.float64):
        qq = quantize_query(q, P, c_q, enc["c_k"])
        est = estimate_scores(enc, qq)
        sel = topp_select(est["S"], p, sm_scale)
        att = sparse_decode(q, K_index, V_index, sel["idx"], K_loc, V_loc, sm_scale)
        outs.append(dict(qq=qq, est=est, sel=sel, att=att))
    return dict(enc=enc, heads=outs)
