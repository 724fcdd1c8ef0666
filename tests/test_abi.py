"""The C ABI without a GPU: the library loads, exports every declared entry
point, and rejects invalid arguments on the host before enqueuing anything."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rbq.h")
HEADERS = sorted(os.path.join(ROOT, "include", f) for f in os.listdir(os.path.join(ROOT, "include"))
                 if f.endswith(".h"))
LIB = os.path.join(ROOT, "paper_2606_31519_amd", "librbq.so")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        from paper_2606_31519_amd import build
        build.build()
    from paper_2606_31519_amd import rbq
    return rbq


def declared_symbols(headers=None):
    text = "".join(open(h).read() for h in (headers or HEADERS))
    return sorted(set(re.findall(r"^(?:rbq_status|size_t|const char\*|int32_t)\s+(rbq_\w+)\(", text, re.M)))


def test_test_hooks_are_not_in_the_product_header():
    product = declared_symbols([HEADER])
    testing = declared_symbols([os.path.join(ROOT, "include", "rbq_testing.h")])
    assert testing and not set(testing) & set(product)
    assert all(n.endswith(("_debug", "_ints", "_ints_q8")) for n in testing)


def test_header_declares_the_five_calls():
    names = declared_symbols()
    for n in ("rbq_encode_keys", "rbq_quantize_query", "rbq_score", "rbq_topp_select", "rbq_sparse_decode"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    cdll = ctypes.CDLL(LIB)
    for n in declared_symbols():
        assert hasattr(cdll, n), n
    assert set(declared_symbols()) <= set(lib.EXPORTED)


def test_status_strings_and_version(lib):
    assert lib.status_string(0) == "ok"
    assert lib.status_string(1) == "invalid argument"
    assert lib.rbq_version() >= 100


def test_index_footprint_matches_the_space_model(lib):
    # Appendix C: eta = (D/8 + B_alpha) / (2 D B_data); with FP16 alpha and FP16
    # KV at D = 128 the paper states 18/512 ~ 3.5 %. This layout stores 8 bytes of
    # factors per key instead of B_alpha = 2.
    D, B_data = 128, 2
    assert abs((D / 8 + 2) / (2 * D * B_data) - 0.035) < 0.001
    per_key = lib.rbq_index_bytes(1, 1, D, 1)
    assert per_key == D // 8 + 8
    assert abs(per_key / (2 * D * B_data) - 0.046875) < 1e-12
    assert lib.rbq_index_bytes(4, 8, D, 131072) == 4 * 8 * 131072 * 24


def test_workspace_sizes(lib):
    assert lib.rbq_workspace_bytes(lib.RBQ_OP_TOPP, 1, 32, 8, 128, 131072) > 32 * 8448 * 8
    assert lib.rbq_workspace_bytes(lib.RBQ_OP_SPARSE_DECODE, 1, 32, 8, 128, 130816, 256) > 0
    assert lib.rbq_workspace_bytes(lib.RBQ_OP_ENCODE, 1, 8, 8, 128, 4096, 0) >= 8 * 4 * 128 * 4
    assert lib.rbq_workspace_bytes(99, 1, 32, 8, 128, 100) == 0
    assert lib.rbq_workspace_bytes(lib.RBQ_OP_TOPP, 0, 32, 8, 128, 100) == 0


FAKE = 1 << 40   # never dereferenced: every call below fails validation first


def _status(fn, *args):
    return fn(*args)


def test_invalid_arguments_are_rejected_on_the_host(lib):
    L = lib.lib
    EINVAL, EUNSUP = lib.RBQ_EINVAL, lib.RBQ_EUNSUPPORTED
    # encode: offset + n_new > cap, null P, bad flags, centroid of zero keys, bad dtype, D unsupported
    enc = lambda **k: L.rbq_encode_keys(k.get("B", 1), k.get("H", 1), k.get("D", 128), FAKE, k.get("dt", 1),
                                        k.get("ld", 10), k.get("n", 10), k.get("off", 0), k.get("cap", 10),
                                        k.get("P", FAKE), None, FAKE, FAKE, FAKE, k.get("flags", 0), None,
                                        k.get("ws", FAKE), k.get("wsb", 1 << 20), 0)
    assert enc(off=1) == EINVAL
    assert enc(P=None) == EINVAL
    assert enc(flags=4) == EINVAL
    assert enc(n=0, flags=1) == EINVAL
    assert enc(flags=1, ws=None) == EINVAL
    assert enc(flags=1, wsb=16) == EINVAL
    assert enc(dt=7) == EUNSUP
    assert enc(D=96) == EUNSUP
    assert enc(D=100) == EINVAL
    assert enc(ld=5) == EINVAL
    assert enc(B=0) == EINVAL
    # quantize: Hq not a multiple of Hkv, null c_k
    assert L.rbq_quantize_query(1, 6, 4, 128, FAKE, FAKE, None, FAKE, FAKE, FAKE, 0) == EINVAL
    assert L.rbq_quantize_query(1, 8, 4, 128, FAKE, FAKE, None, None, FAKE, FAKE, 0) == EINVAL
    # score: n > cap
    assert L.rbq_score(1, 8, 4, 128, 11, 10, FAKE, FAKE, FAKE, FAKE, FAKE, 0) == EINVAL
    assert L.rbq_score(1, 8, 4, 128, -1, 10, FAKE, FAKE, FAKE, FAKE, FAKE, 0) == EINVAL
    # top-p: p outside (0, 1], non-finite or non-positive scale, short workspace
    tp = lambda p=0.9, s=0.1, wsb=1 << 30: L.rbq_topp_select(1, 8, 100, FAKE, p, s, FAKE, FAKE, FAKE, wsb, 0)
    assert tp(p=0.0) == EINVAL
    assert tp(p=1.5) == EINVAL
    assert tp(p=float("nan")) == EINVAL
    assert tp(s=float("inf")) == EINVAL
    assert tp(s=-1.0) == EINVAL
    assert tp(wsb=8) == EINVAL
    # rows of 2^24 keys or more would overflow the 64-bit fixed-point mass sums
    big = lambda n: L.rbq_topp_select(1, 1, n, FAKE, 0.9, 0.1, FAKE, FAKE, FAKE, 1 << 40, 0)
    assert big(1 << 24) == EUNSUP
    assert big((1 << 31) - 1) == EUNSUP
    assert L.rbq_topp_select_varlen(1, 1, 1 << 24, FAKE, FAKE, FAKE, 0.1, FAKE, FAKE, FAKE, 1 << 40, 0) == EUNSUP
    # decode: window above the limit, window without buffers, G not a power of two, n > cap
    dec = lambda **k: L.rbq_sparse_decode(1, k.get("Hq", 8), 4 if k.get("Hq", 8) % 4 == 0 else 3, 128, FAKE, FAKE,
                                          FAKE, 1, k.get("cap", 100), k.get("n", 100), FAKE, FAKE,
                                          k.get("kl", FAKE), FAKE, k.get("ld", 300), k.get("w", 10), 0.1, FAKE,
                                          None, FAKE, 1 << 30, 0)
    assert dec(w=5000, ld=5000) == EINVAL
    assert dec(kl=None) == EINVAL
    assert dec(ld=5) == EINVAL
    assert dec(n=101) == EINVAL
    assert dec(Hq=12) == EUNSUP
    assert L.rbq_dense_decode(1, 8, 4, 128, FAKE, FAKE, FAKE, 3, 100, 100, None, None, 0, 0, 0.1, FAKE, None,
                              FAKE, 1 << 30, 0) == EUNSUP
    # device pointers must be 16-byte aligned (the kernels use 16-byte vector loads)
    assert L.rbq_score(1, 8, 4, 128, 10, 10, FAKE + 4, FAKE, FAKE, FAKE, FAKE, 0) == EINVAL
    assert L.rbq_quantize_query(1, 8, 4, 128, FAKE + 8, FAKE, None, FAKE, FAKE, FAKE, 0) == EINVAL
    assert dec(kl=FAKE + 2) == EINVAL
    # the fused step: n + w beyond the capacity, a short workspace
    step = lambda **k: L.rbq_decode_step(1, 8, 4, 128, FAKE, FAKE, None, FAKE, FAKE, FAKE, 1, k.get("cap", 200),
                                         100, k.get("w", 10), FAKE, FAKE, 1, 0.9, 0.1, FAKE, FAKE, FAKE, FAKE, FAKE,
                                         FAKE, None, FAKE, k.get("wsb", 1 << 30), 0)
    assert step(cap=105) == EINVAL
    assert step(wsb=64) == EINVAL


def test_ragged_calls_reject_invalid_arguments_on_the_host(lib):
    L = lib.lib
    EINVAL = lib.RBQ_EINVAL
    # score: the per-sequence counts are required and aligned; n > cap
    sc = lambda **k: L.rbq_score_varlen(1, 8, 4, 128, k.get("n", 10), k.get("cap", 10), k.get("sn", FAKE), FAKE,
                                        FAKE, FAKE, FAKE, FAKE, 0)
    assert sc(sn=None) == EINVAL
    assert sc(sn=FAKE + 4) == EINVAL
    assert sc(n=11) == EINVAL
    # top-p: per-sequence p required; the workspace is needed whatever the device p values are
    tp = lambda **k: L.rbq_topp_select_varlen(2, 8, 100, k.get("sn", FAKE), FAKE, k.get("sp", FAKE),
                                              k.get("s", 0.1), FAKE, FAKE, FAKE, k.get("wsb", 1 << 30), 0)
    assert tp(sp=None) == EINVAL
    assert tp(sp=FAKE + 8) == EINVAL
    assert tp(sn=None) == EINVAL
    assert tp(s=0.0) == EINVAL
    assert tp(wsb=8) == EINVAL
    # decode: every sequence's window must fit at the tail (n + w <= cap); aligned seq_w when given
    dec = lambda **k: L.rbq_sparse_decode_varlen(2, 8, 4, 128, FAKE, FAKE, FAKE, 1, k.get("cap", 200), 100,
                                                 k.get("w", 10), k.get("sn", FAKE), k.get("sw", None), FAKE, FAKE,
                                                 0.1, FAKE, None, FAKE, 1 << 30, 0)
    assert dec(cap=105) == EINVAL
    assert dec(sn=None) == EINVAL
    assert dec(sw=FAKE + 4) == EINVAL
    assert dec(w=5000, cap=10000) == EINVAL   # above the window limit
    assert L.rbq_dense_decode_varlen(2, 8, 4, 128, FAKE, FAKE, FAKE, 1, 105, 100, 10, FAKE, None, 0.1, FAKE, None,
                                     FAKE, 1 << 30, 0) == EINVAL
    # the fused step: short workspace, missing p, window past the capacity
    step = lambda **k: L.rbq_decode_step_varlen(2, 8, 4, 128, FAKE, FAKE, None, FAKE, FAKE, FAKE, 1,
                                                k.get("cap", 200), 100, 10, FAKE, None, FAKE, FAKE, 1,
                                                k.get("sp", FAKE), 0.1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None,
                                                FAKE, k.get("wsb", 1 << 30), 0)
    assert step(cap=105) == EINVAL
    assert step(sp=None) == EINVAL
    assert step(wsb=64) == EINVAL


def test_query_bits_range_is_checked_on_the_host(lib):
    L = lib.lib
    qb = lambda bits: L.rbq_quantize_query_bits(1, 8, 4, 128, FAKE, FAKE, None, FAKE, bits, FAKE, FAKE, 0)
    assert qb(0) == lib.RBQ_EINVAL
    assert qb(9) == lib.RBQ_EINVAL
    for bits in (5, 8):   # in range, then rejected for the missing c_k before anything is launched
        assert L.rbq_quantize_query_bits(1, 8, 4, 128, FAKE, FAKE, None, None, bits, FAKE, FAKE, 0) == lib.RBQ_EINVAL
    assert L.rbq_score_q8(1, 8, 4, 128, 11, 10, FAKE, FAKE, FAKE, FAKE, FAKE, 0) == lib.RBQ_EINVAL
    assert L.rbq_score_q8(1, 8, 4, 128, 10, 10, FAKE, FAKE, FAKE + 4, FAKE, FAKE, 0) == lib.RBQ_EINVAL
    assert L.rbq_score_ints_q8(1, 8, 4, 128, 10, 10, FAKE, None, FAKE, FAKE, 0) == lib.RBQ_EINVAL
    assert L.rbq_quantize_query_bits(1, 8, 4, 128, FAKE, FAKE, None, None, 2, FAKE, FAKE, 0) == lib.RBQ_EINVAL


def test_compact_index_calls_reject_invalid_arguments_on_the_host(lib):
    L = lib.lib
    EINVAL, EUNSUP = lib.RBQ_EINVAL, lib.RBQ_EUNSUPPORTED
    enc = lambda **k: L.rbq_encode_keys_f16(1, 1, k.get("D", 128), FAKE, 1, 10, 10, k.get("off", 0), 10, FAKE,
                                            FAKE, FAKE, k.get("kf", FAKE), k.get("flags", 0), FAKE, 1 << 20, 0)
    assert enc(kf=None) == EINVAL
    assert enc(kf=FAKE + 2) == EINVAL
    assert enc(off=1) == EINVAL
    assert enc(flags=4) == EINVAL
    assert enc(D=96) == EUNSUP
    sc = lambda n=10, kf=FAKE: L.rbq_score_f16(1, 8, 4, 128, n, 10, FAKE, kf, FAKE, FAKE, FAKE, 0)
    assert sc(n=11) == EINVAL
    assert sc(kf=None) == EINVAL
    assert sc(kf=FAKE + 4) == EINVAL
    assert sc(n=0, kf=None) == lib.RBQ_OK          # nothing to score: nothing read, nothing enqueued
    step = lambda **k: L.rbq_decode_step_f16(1, 8, 4, 128, FAKE, FAKE, FAKE, FAKE, FAKE, 1, k.get("cap", 200), 100,
                                             10, FAKE, k.get("kf", FAKE), 1, 0.9, 0.1, FAKE, FAKE, FAKE, FAKE,
                                             FAKE, FAKE, None, FAKE, k.get("wsb", 1 << 30), 0)
    assert step(cap=105) == EINVAL
    assert step(wsb=64) == EINVAL
    assert step(kf=None) == EINVAL
    sv = L.rbq_score_varlen_f16(1, 8, 4, 128, 10, 10, None, FAKE, FAKE, FAKE, FAKE, FAKE, 0)
    assert sv == EINVAL                              # seq_n is required
    stv = L.rbq_decode_step_varlen_f16(1, 8, 4, 128, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 200, 100, 10, FAKE, None,
                                       FAKE, None, 1, FAKE, 0.1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE,
                                       1 << 30, 0)
    assert stv == EINVAL                             # no factor array


def test_every_call_validates_at_head_dim_64(lib):
    """D = 64 runs every call; invalid arguments are still rejected on the host
    (nothing here reaches a launch), and an unsupported D gives RBQ_EUNSUPPORTED."""
    L = lib.lib
    EINVAL, EUNSUP = lib.RBQ_EINVAL, lib.RBQ_EUNSUPPORTED
    assert L.rbq_score_varlen(1, 8, 4, 64, 10, 10, None, FAKE, FAKE, FAKE, FAKE, FAKE, 0) == EINVAL   # no seq_n
    assert L.rbq_score_varlen(1, 8, 4, 96, 10, 10, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0) == EUNSUP
    assert L.rbq_score_varlen_f16(1, 8, 4, 64, 11, 10, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0) == EINVAL
    assert L.rbq_sparse_decode_varlen(1, 8, 4, 64, FAKE, FAKE, FAKE, 1, 105, 100, 10, FAKE, None, FAKE, FAKE, 0.1,
                                      FAKE, None, FAKE, 1 << 30, 0) == EINVAL      # n + w > cap
    assert L.rbq_dense_decode_varlen(1, 8, 4, 64, FAKE, FAKE, FAKE, 1, 200, 100, 10, None, None, 0.1, FAKE, None,
                                     FAKE, 1 << 30, 0) == EINVAL                    # no seq_n
    assert L.rbq_decode_step_varlen(1, 8, 4, 64, FAKE, FAKE, None, FAKE, FAKE, FAKE, 1, 200, 100, 10, FAKE, None,
                                    FAKE, FAKE, 1, FAKE, 0.1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE,
                                    64, 0) == EINVAL                                # short workspace
    assert L.rbq_encode_keys_f16(1, 1, 64, FAKE, 1, 10, 10, 1, 10, FAKE, FAKE, FAKE, FAKE, 0, FAKE, 1 << 20,
                                 0) == EINVAL                                       # offset + n_new > cap
    assert L.rbq_encode_keys_f16(1, 1, 96, FAKE, 1, 10, 10, 0, 10, FAKE, FAKE, FAKE, FAKE, 0, FAKE, 1 << 20,
                                 0) == EUNSUP
    assert L.rbq_score_f16(1, 8, 4, 64, 10, 10, FAKE, None, FAKE, FAKE, FAKE, 0) == EINVAL
    assert L.rbq_decode_step_f16(1, 8, 4, 64, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 105, 100, 10, FAKE, FAKE, 1, 0.9,
                                 0.1, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, 1 << 30, 0) == EINVAL
    assert L.rbq_score_q8(1, 8, 4, 64, 11, 10, FAKE, FAKE, FAKE, FAKE, FAKE, 0) == EINVAL
    assert L.rbq_score_ints_q8(1, 8, 4, 64, 10, 10, FAKE, None, FAKE, FAKE, 0) == EINVAL
    assert L.rbq_score(1, 8, 4, 64, 11, 10, FAKE, FAKE, FAKE, FAKE, FAKE, 0) == EINVAL
    assert lib.rbq_workspace_bytes(lib.RBQ_OP_DECODE_STEP, 1, 8, 4, 64, 1000, 16) < \
        lib.rbq_workspace_bytes(lib.RBQ_OP_DECODE_STEP, 1, 8, 4, 128, 1000, 16)


def test_mapped_device_pointer_rejects_null_arguments(lib):
    out = ctypes.c_void_p(123)
    assert lib.lib.rbq_mapped_device_pointer(None, ctypes.byref(out)) == lib.RBQ_EINVAL
    assert lib.lib.rbq_mapped_device_pointer(ctypes.c_void_p(FAKE), None) == lib.RBQ_EINVAL


def test_noalloc_step_rejects_sizes_beyond_its_scratch_on_the_host(lib):
    """rbq_decode_step_noalloc returns RBQ_EUNSUPPORTED for sizes whose step
    workspace exceeds its static scratch, before any pointer is read or any
    device call is made (so it runs without a GPU)."""
    B, Hq, Hkv, D, n, w = 4, 64, 8, 128, 131072, 256
    assert lib.rbq_workspace_bytes(lib.RBQ_OP_DECODE_STEP, B, Hq, Hkv, D, n, w) > lib.RBQ_NOALLOC_SCRATCH_BYTES
    st = lib.lib.rbq_decode_step_noalloc(B, Hq, Hkv, D, *([None] * 6), lib.RBQ_BF16, n + w, n, w, None, None, 1,
                                         0.9, 0.1, *([None] * 7), None)
    assert st == lib.RBQ_EUNSUPPORTED
