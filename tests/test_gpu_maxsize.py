"""One sequence near the path's size limits: 4,193,792 indexed keys of one KV
head (4 query heads) plus a 512-row window, bf16, through rbq_decode_step.
The selection then spans 256 sub-chunks of 16384 keys per row (64 parts of
4 sub-chunks), its bitmaps 65,536 words per row, and the decode's 32-bit byte
offsets reach 1 GiB.

Inputs are seeded on the device (Gaussian keys with four outlier channels
x8, Gaussian values, a scaled Gaussian query). The oracle checks the
centroid, sampled codes and factors (including flushed window rows), sampled
scores, every head's whole Top-p set, and the attention over each head's
selection plus the window."""
import math

import numpy as np
import pytest
import torch

from oracle import rbq_oracle as orc
from workloads import gen
import parity_util as pu

pytestmark = pytest.mark.gpu

N = (1 << 22) - 512
W = 512
HQ, HKV, D = 4, 1, 128


@pytest.fixture(scope="module")
def pipeline():
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2606_31519_amd import pipeline as pl
    return pl


def _rows(t, idx):
    """Rows idx of a [cap][D] device tensor, as float64 on the host."""
    return t[torch.as_tensor(idx, device=t.device, dtype=torch.long)].double().cpu().numpy()


def test_largest_sequence_end_to_end(pipeline):
    cap = N + W
    print("max size: n", N, "window", W, flush=True)
    g = torch.Generator(device="cuda").manual_seed(31)
    K = torch.randn(1, HKV, cap, D, generator=g, device="cuda")
    K[..., :4] *= 8.0
    K = K.to(torch.bfloat16)
    V = torch.randn(1, HKV, cap, D, generator=g, device="cuda").to(torch.bfloat16)
    q = 1.5 * torch.randn(1, HQ, D, generator=g, device="cuda")   # logits of std ~2.6: budgets of 10^4 to 3.10^5 keys
    P = torch.from_numpy(gen.haar_rotation(D)).cuda()
    st = pipeline.DecodeState(1, HQ, HKV, D, cap, N, W, K, V, q, P, None)
    st.build_index()
    p = 0.9
    st.step(p)          # also flushes the window into index rows [N, N + W)
    torch.cuda.synchronize()
    tau = 1.0 / math.sqrt(D)
    Kd = st.K[0, 0]

    # centroid over every indexed key, summed in fp64 on the host
    acc = np.zeros(D)
    for r0 in range(0, N, 1 << 19):
        acc += Kd[r0:min(N, r0 + (1 << 19))].double().sum(0).cpu().numpy()
    ck = st.c_k[0, 0].double().cpu().numpy()
    assert np.abs(ck - acc / N).max() <= 1e-5 * (np.abs(acc / N).max() + 1.0)

    # codes and factors of sampled rows: the first, the last indexed, the flushed window, random ones
    rng = np.random.default_rng(5)
    idx = np.unique(np.concatenate([np.arange(64), np.arange(N - 64, N + W), rng.integers(0, N, 4000)]))
    enc = orc.encode_keys(_rows(Kd, idx), st.P.cpu().numpy().astype(np.float64), c_k=ck)
    codes = pu.u32(st.codes[0, 0])[idx]
    kfac = st.kfac[0, 0].cpu().numpy().astype(np.float64)[idx]
    diff = orc.unpack_bits(codes, D) != enc["bits"]
    assert np.all(np.abs(enc["R"][diff]) <= 1e-5 * np.broadcast_to(enc["norm"][:, None], diff.shape)[diff])
    assert np.all(np.abs(kfac[:, 0] - enc["f"]) <= 1e-5 * enc["f"] + 1e-6)

    # scores of the sampled indexed keys; the whole Top-p set of every head; the attention
    S = st.scores[0].cpu().numpy()
    sel, cnt = st.sel_idx[0].cpu().numpy(), st.sel_count[0].cpu().numpy()
    planes, qs = pu.u32(st.qplanes[0]), st.qscal[0].cpu().numpy()
    out, lse = st.out[0].cpu().numpy(), st.lse[0].cpu().numpy()
    ix = idx[idx < N]
    P64 = st.P.cpu().numpy().astype(np.float64)
    for h in range(HQ):
        pu.check_qscal(qs[h], planes[h], q[0, h].double().cpu().numpy(), P64, None, ck)
        pu.check_scores(S[h, ix], codes[idx < N], kfac[idx < N], planes[h], qs[h])
        s_h = sel[h, :cnt[h]]
        res = pu.check_topp(S[h, :N], p, tau, s_h)
        print(f"head {h}: budget {cnt[h]}, set diff {res['diff']}", flush=True)
        Ksel, Vsel = _rows(Kd, s_h), _rows(st.V[0, 0], s_h)
        Kw, Vw = _rows(Kd, np.arange(N, N + W)), _rows(st.V[0, 0], np.arange(N, N + W))
        pu.check_attention(out[h], lse[h], q[0, h].double().cpu().numpy(), Ksel, Vsel, np.arange(len(s_h)),
                           Kw, Vw, tau)
