"""Seeded synthetic inputs shaped like RaBitQCache's decode workloads.

Both sides of every parity check draw their inputs from here: the HIP
library (through its binding) and the CPU oracle. This module only draws
random numbers, shapes them and casts them; it holds none of the method's
arithmetic (no centring, rotation, sign coding, query quantisation, score
estimation, Top-p selection or sparse attention).

What the paper fixes and what is stood in for:
  * The paper measures on LongBench / RULER / GSM8K with LongChat-7B and
    LLaMA-3.1-8B/70B (Section 5.2). None of those datasets or weights are
    used here; seeded synthetic keys, values and queries of the same shapes
    stand in for them: grouped-query attention with 32 query heads over 8 KV
    heads and head_dim 128 (the LLaMA-3.1-8B shape), contexts 4K..128K, and a
    peaky attention pattern that gives Top-p budgets in the paper's range
    (Tables 1 and 8: 5-25 % of the context at p = 0.9-0.95).
  * The random orthogonal matrix P is drawn once (Section 3.2: generated
    once at model initialisation) from the Haar measure that the proof of
    Theorem A.1 assumes (Lemma A.4), by QR of a Gaussian matrix with the
    sign fix Q * diag(sign(diag R)).

Every array is produced in a fixed order from numpy's PCG64 generator, so the
same seed gives the same bytes on any machine with the same numpy.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

P_SEED = 1234
DATA_SEED_BASE = 20260000


# --------------------------------------------------------------------------
# dtype helpers (bf16 is carried as its uint16 bit pattern)
# --------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even).

    Returns the 16-bit patterns as uint16. Inputs are finite by construction.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


# --------------------------------------------------------------------------
# the rotation matrix
# --------------------------------------------------------------------------
def haar_rotation(D: int, seed: int = P_SEED, dtype=np.float32) -> np.ndarray:
    """A D x D orthogonal matrix drawn from the Haar measure, cast to `dtype`."""
    rng = np.random.default_rng(seed)
    g = rng.standard_normal((D, D))
    q, r = np.linalg.qr(g)
    q = q * np.sign(np.diag(r))[None, :]
    return np.ascontiguousarray(q.astype(dtype))


def haar_rotations(D: int, count: int, seed: int) -> np.ndarray:
    """`count` independent Haar matrices in float64, [count][D][D]."""
    rng = np.random.default_rng(seed)
    g = rng.standard_normal((count, D, D))
    q, r = np.linalg.qr(g)
    s = np.sign(np.diagonal(r, axis1=1, axis2=2))
    return q * s[:, None, :]


# --------------------------------------------------------------------------
# workload container
# --------------------------------------------------------------------------
@dataclasses.dataclass
class Workload:
    """One decode workload.

    K, V   : [B][Hkv][N][D]; float32 when kv_dtype == "f32", else uint16 bf16 bits.
             Rows [0, n_index) are indexed; rows [n_index, n_index + w) are the
             local window (the newest keys, attended in full precision).
    q      : [B][Hq][D] float32, the decode-step query.
    c_q    : [B][Hkv][D] float32 query centroid per KV group (zeros: no query centring).
    P      : [D][D] float32 rotation.
    """
    name: str
    B: int
    Hq: int
    Hkv: int
    D: int
    N: int
    n_index: int
    w: int
    kv_dtype: str
    K: np.ndarray
    V: np.ndarray
    q: np.ndarray
    c_q: np.ndarray
    P: np.ndarray
    p: float
    planted: Optional[list] = None   # per (b, q-head): planted key indices
    p_sweep: tuple = ()

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    def K_f32(self, b: int, hk: int, rows: slice = slice(None)) -> np.ndarray:
        k = self.K[b, hk, rows]
        return k if self.kv_dtype == "f32" else bf16_bits_to_f32(k)

    def V_f32(self, b: int, hk: int, rows: slice = slice(None)) -> np.ndarray:
        v = self.V[b, hk, rows]
        return v if self.kv_dtype == "f32" else bf16_bits_to_f32(v)


def _cast_kv(x32: np.ndarray, kv_dtype: str) -> np.ndarray:
    return x32.astype(np.float32) if kv_dtype == "f32" else f32_to_bf16_bits(x32)


def _widen(x: np.ndarray, kv_dtype: str) -> np.ndarray:
    return x if kv_dtype == "f32" else bf16_bits_to_f32(x)


# --------------------------------------------------------------------------
# planted-direction queries
# --------------------------------------------------------------------------
def _softmax_share(s: np.ndarray, planted: np.ndarray, gamma: float, inv_sqrt_d: float) -> float:
    """Share of exp(gamma * s_i / sqrt(D)) carried by the planted rows.

    Used only to calibrate synthetic queries so that the exact attention of a
    query is concentrated on its planted keys to a chosen degree.
    """
    z = gamma * inv_sqrt_d * s
    z = z - z.max()
    e = np.exp(z)
    return float(e[planted].sum() / e.sum())


def _calibrate_gamma(s: np.ndarray, planted: np.ndarray, rho: float, D: int) -> float:
    inv = 1.0 / np.sqrt(D)
    lo, hi = 0.0, 1.0
    while _softmax_share(s, planted, hi, inv) < rho and hi < 1e4:
        hi *= 2.0
    for _ in range(48):
        mid = 0.5 * (lo + hi)
        if _softmax_share(s, planted, mid, inv) < rho:
            lo = mid
        else:
            hi = mid
    return 0.5 * (lo + hi)


def _plant_group(rng, Kg: np.ndarray, G: int, frac: float, n_draw: int) -> tuple:
    """Plant one random unit direction per query head of a KV group.

    Adds beta * w_h (beta = median key norm) to round(frac * n_draw) keys drawn
    without replacement from rows [0, n_draw). Returns (directions, planted sets).
    """
    N, D = Kg.shape
    beta = float(np.median(np.linalg.norm(Kg.astype(np.float64), axis=1)))
    dirs, sets = [], []
    m = max(1, int(round(frac * n_draw)))
    for _ in range(G):
        w = rng.standard_normal(D)
        w /= np.linalg.norm(w)
        idx = np.sort(rng.choice(n_draw, size=m, replace=False))
        Kg[idx] += (beta * w).astype(Kg.dtype)
        dirs.append(w)
        sets.append(idx)
    return dirs, sets


def _lowrank_keys(rng, N: int, D: int, rank: int = 16, noise: float = 0.5, n_outlier: int = 4,
                  outlier_scale: float = 8.0) -> np.ndarray:
    z = rng.standard_normal((N, rank), dtype=np.float32)
    wl = rng.standard_normal((rank, D), dtype=np.float32) * np.float32(1.0 / np.sqrt(rank))
    e = rng.standard_normal((N, D), dtype=np.float32)
    s = np.ones(D, dtype=np.float32)
    s[rng.choice(D, size=n_outlier, replace=False)] = outlier_scale
    return (z @ wl + np.float32(noise) * e) * s[None, :]


def _student_t_keys(rng, N: int, D: int, nu: float = 3.0) -> np.ndarray:
    z = rng.standard_normal((N, D), dtype=np.float32)
    g = rng.standard_gamma(nu / 2.0, size=(N, D), dtype=np.float32)
    return z / np.sqrt(np.float32(2.0 / nu) * g)


def _planted_gqa(name, B, Hq, Hkv, D, N, n_index, w, seed, p, key_fn, frac_fn, rho=0.9,
                 p_sweep=()) -> Workload:
    """Each (sequence, KV head) group draws from its own generator, spawned from
    `seed` in group order, so the groups can be generated by parallel threads
    (numpy releases the GIL while it fills arrays) with a result that does not
    depend on the thread count or scheduling."""
    import concurrent.futures
    import os

    rng = np.random.default_rng(seed)
    G = Hq // Hkv
    fracs = [frac_fn(rng, b) for b in range(B)]
    children = np.random.SeedSequence(seed).spawn(B * Hkv)
    K = np.empty((B, Hkv, N, D), dtype=np.uint16)
    V = np.empty((B, Hkv, N, D), dtype=np.uint16)
    q = np.empty((B, Hq, D), dtype=np.float32)
    planted = [None] * (B * Hq)

    def group(idx):
        b, hk = divmod(idx, Hkv)
        grng = np.random.default_rng(children[idx])
        Kg = key_fn(grng, N, D)
        dirs, sets = _plant_group(grng, Kg, G, fracs[b], N)
        K[b, hk] = f32_to_bf16_bits(Kg)
        V[b, hk] = f32_to_bf16_bits(grng.standard_normal((N, D), dtype=np.float32))
        kw = bf16_bits_to_f32(K[b, hk]).astype(np.float64)
        for g in range(G):
            s = kw @ dirs[g]
            gamma = _calibrate_gamma(s, sets[g], rho, D)
            q[b, hk * G + g] = (gamma * dirs[g]).astype(np.float32)
            planted[b * Hq + hk * G + g] = sets[g]

    workers = max(1, min(16, len(os.sched_getaffinity(0)), B * Hkv))
    with concurrent.futures.ThreadPoolExecutor(max_workers=workers) as ex:
        list(ex.map(group, range(B * Hkv)))
    return Workload(name=name, B=B, Hq=Hq, Hkv=Hkv, D=D, N=N, n_index=n_index, w=w, kv_dtype="bf16",
                    K=K, V=V, q=q, c_q=np.zeros((B, Hkv, D), np.float32), P=haar_rotation(D),
                    p=p, planted=planted, p_sweep=tuple(p_sweep))


# --------------------------------------------------------------------------
# the five workload presets
# --------------------------------------------------------------------------
def config1(seed: int = DATA_SEED_BASE + 1) -> Workload:
    """Single head, D=128, N=4096 fp32 keys ~ N(0,1) with 4 outlier channels x8.

    The query is the mean of 8 planted keys plus N(0, 0.1^2) noise; values
    ~ N(0,1); p = 0.9; no local window.
    """
    rng = np.random.default_rng(seed)
    N, D = 4096, 128
    K = rng.standard_normal((N, D))
    K[:, rng.choice(D, size=4, replace=False)] *= 8.0
    planted = np.sort(rng.choice(N, size=8, replace=False))
    q = K[planted].mean(axis=0) + 0.1 * rng.standard_normal(D)
    V = rng.standard_normal((N, D))
    return Workload(name="single-head N=4096 fp32", B=1, Hq=1, Hkv=1, D=D, N=N, n_index=N, w=0,
                    kv_dtype="f32", K=K.astype(np.float32)[None, None], V=V.astype(np.float32)[None, None],
                    q=q.astype(np.float32)[None, None], c_q=np.zeros((1, 1, D), np.float32),
                    P=haar_rotation(D), p=0.9, planted=[planted])


def config2(seed: int = DATA_SEED_BASE + 2, N: int = 32768) -> Workload:
    """GQA 32/8 heads, D=128, context 32K, batch 1, bf16; low-rank keys, 1 % planted, p=0.95."""
    return _planted_gqa("gqa 32q/8kv ctx=32K b=1 bf16", 1, 32, 8, 128, N, N, 0, seed, 0.95,
                        _lowrank_keys, lambda rng, b: 0.01)


def config3(seed: int = DATA_SEED_BASE + 3, N: int = 131072, w: int = 256) -> Workload:
    """Config 2's generator at 128K context; the newest `w` keys form the local window."""
    return _planted_gqa("gqa 32q/8kv ctx=128K b=1 bf16 window=256", 1, 32, 8, 128, N, N - w, w, seed, 0.95,
                        _lowrank_keys, lambda rng, b: 0.01, p_sweep=(0.8, 0.9, 0.95, 0.99))


def config3_d64(seed: int = DATA_SEED_BASE + 3, N: int = 131072, w: int = 256) -> Workload:
    """Config 3 at head dimension 64 (the D = 64 shape of the kernel ablation):
    the same generator, 32 / 8 heads, 128K context, bf16, 256-key window."""
    return _planted_gqa("gqa 32q/8kv ctx=128K b=1 bf16 window=256 D=64", 1, 32, 8, 64, N, N - w, w, seed, 0.95,
                        _lowrank_keys, lambda rng, b: 0.01, p_sweep=(0.8, 0.9, 0.95, 0.99))


def config4(seed: int = DATA_SEED_BASE + 4, B: int = 16, N: int = 32768) -> Workload:
    """Batch 16 x 32K, 32/8 heads, bf16; per-sequence planted fraction ~ U(0.1 %, 10 %)."""
    return _planted_gqa("gqa 32q/8kv ctx=32K b=16 bf16 varied sparsity", B, 32, 8, 128, N, N, 0, seed, 0.95,
                        _lowrank_keys, lambda rng, b: float(rng.uniform(0.001, 0.1)))


def config5(seed: int = DATA_SEED_BASE + 5, B: int = 4, N: int = 131072) -> Workload:
    """64 q-heads over 8 KV heads, batch 4 x 128K, bf16, Student-t (nu=3) keys, 1 % planted."""
    return _planted_gqa("gqa 64q/8kv ctx=128K b=4 bf16 student-t", B, 64, 8, 128, N, N, 0, seed, 0.95,
                        _student_t_keys, lambda rng, b: 0.01)


def random_case(B: int, Hq: int, Hkv: int, N: int, D: int = 128, seed: int = 0, kv_dtype: str = "bf16",
                w: int = 0, p: float = 0.9, outliers: int = 4, c_q_scale: float = 0.0,
                key_offset: float = 0.0, q_scale: float = 3.0) -> Workload:
    """Small generic case: Gaussian keys with outlier channels and an optional
    common offset, Gaussian values and queries, optional non-zero c_q."""
    rng = np.random.default_rng(seed)
    K = rng.standard_normal((B, Hkv, N + w, D)).astype(np.float32)
    if outliers:
        K[..., rng.choice(D, size=outliers, replace=False)] *= 8.0
    K += np.float32(key_offset) * rng.standard_normal(D).astype(np.float32)
    V = rng.standard_normal((B, Hkv, N + w, D)).astype(np.float32)
    q = (q_scale * rng.standard_normal((B, Hq, D))).astype(np.float32)
    c_q = (c_q_scale * rng.standard_normal((B, Hkv, D))).astype(np.float32)
    return Workload(name=f"random B={B} Hq={Hq} Hkv={Hkv} N={N} w={w}", B=B, Hq=Hq, Hkv=Hkv, D=D, N=N + w,
                    n_index=N, w=w, kv_dtype=kv_dtype, K=_cast_kv(K, kv_dtype), V=_cast_kv(V, kv_dtype),
                    q=q, c_q=c_q, P=haar_rotation(D, seed=P_SEED + seed), p=p)


CONFIGS = {1: config1, 2: config2, 3: config3, 4: config4, 5: config5}
