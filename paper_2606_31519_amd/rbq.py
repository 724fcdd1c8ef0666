"""Thin Python binding of librbq.so (argument marshalling only).

Every function has the name of the C entry point it calls and takes torch
tensors where the C call takes device pointers; the work is enqueued on
torch's current HIP stream. Nothing here computes any part of the method:
the library's kernels do. A missing library raises ImportError; there is no
fallback.
"""
from __future__ import annotations

import ctypes
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librbq.so")

RBQ_OK, RBQ_EINVAL, RBQ_EUNSUPPORTED, RBQ_EDEVICE = 0, 1, 2, 3
RBQ_F32, RBQ_BF16 = 0, 1
RBQ_ENCODE_SET_CENTROID = 1
RBQ_OP_ENCODE, RBQ_OP_TOPP, RBQ_OP_SPARSE_DECODE, RBQ_OP_DENSE_DECODE, RBQ_OP_DECODE_STEP = 1, 2, 3, 4, 5
QSCAL_STRIDE = 8
RBQ_MAX_WINDOW = 4096   # largest local window accepted by the decode calls
RBQ_NOALLOC_SCRATCH_BYTES = 16 << 20   # the static scratch of rbq_decode_step_noalloc

EXPORTED = [
    "rbq_encode_keys", "rbq_quantize_query", "rbq_score", "rbq_topp_select", "rbq_sparse_decode",
    "rbq_dense_decode", "rbq_decode_step", "rbq_workspace_bytes", "rbq_index_bytes", "rbq_status_string", "rbq_version",
    "rbq_encode_keys_debug", "rbq_quantize_query_debug", "rbq_score_ints",
    "rbq_score_varlen", "rbq_topp_select_varlen", "rbq_sparse_decode_varlen", "rbq_dense_decode_varlen",
    "rbq_decode_step_varlen", "rbq_quantize_query_bits",
    "rbq_score_q8", "rbq_score_ints_q8", "rbq_mapped_device_pointer",
    "rbq_encode_keys_f16", "rbq_score_f16", "rbq_decode_step_f16", "rbq_score_varlen_f16", "rbq_decode_step_varlen_f16",
    "rbq_decode_step_noalloc",
]


class RbqError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed: {status} ({status_string(status)})")
        self.status = status


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run paper_2606_31519_amd.build.build() first")
    lib = ctypes.CDLL(LIB_PATH)
    i32, i64, u32, sz, vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_size_t, ctypes.c_void_p
    f32 = ctypes.c_float
    sig = {
        "rbq_encode_keys": [i32, i32, i32, vp, i32, i64, i32, i32, i32, vp, vp, vp, vp, vp, u32, vp, vp, sz, vp],
        "rbq_encode_keys_debug": [i32, i32, i32, vp, i32, i64, i32, i32, i32, vp, vp, vp, vp, vp, u32, vp, vp, sz,
                                  vp, vp],
        "rbq_quantize_query": [i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp],
        "rbq_quantize_query_debug": [i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp],
        "rbq_score": [i32, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp],
        "rbq_score_ints": [i32, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp],
        "rbq_topp_select": [i32, i32, i32, vp, f32, f32, vp, vp, vp, sz, vp],
        "rbq_sparse_decode": [i32, i32, i32, i32, vp, vp, vp, i32, i32, i32, vp, vp, vp, vp, i64, i32, f32, vp, vp,
                              vp, sz, vp],
        "rbq_dense_decode": [i32, i32, i32, i32, vp, vp, vp, i32, i32, i32, vp, vp, i64, i32, f32, vp, vp, vp, sz,
                             vp],
        "rbq_decode_step": [i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, vp, vp, i32, f32, f32,
                            vp, vp, vp, vp, vp, vp, vp, vp, sz, vp],
        "rbq_decode_step_noalloc": [i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, vp, vp, i32, f32,
                                    f32, vp, vp, vp, vp, vp, vp, vp, vp],
        "rbq_quantize_query_bits": [i32, i32, i32, i32, vp, vp, vp, vp, i32, vp, vp, vp],
        "rbq_score_varlen": [i32, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp],
        "rbq_topp_select_varlen": [i32, i32, i32, vp, vp, vp, f32, vp, vp, vp, sz, vp],
        "rbq_sparse_decode_varlen": [i32, i32, i32, i32, vp, vp, vp, i32, i32, i32, i32, vp, vp, vp, vp, f32, vp,
                                     vp, vp, sz, vp],
        "rbq_dense_decode_varlen": [i32, i32, i32, i32, vp, vp, vp, i32, i32, i32, i32, vp, vp, f32, vp, vp, vp, sz,
                                    vp],
        "rbq_decode_step_varlen": [i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, vp, vp, vp, vp,
                                   i32, vp, f32, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp],
        "rbq_score_q8": [i32, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp],
        "rbq_mapped_device_pointer": [vp, ctypes.POINTER(vp)],
        "rbq_score_ints_q8": [i32, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp],
        # the compact index (fp16 factors, no c_q)
        "rbq_encode_keys_f16": [i32, i32, i32, vp, i32, i64, i32, i32, i32, vp, vp, vp, vp, u32, vp, sz, vp],
        "rbq_score_f16": [i32, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp],
        "rbq_decode_step_f16": [i32, i32, i32, i32, vp, vp, vp, vp, vp, i32, i32, i32, i32, vp, vp, i32, f32, f32,
                                vp, vp, vp, vp, vp, vp, vp, vp, sz, vp],
        "rbq_score_varlen_f16": [i32, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp],
        "rbq_decode_step_varlen_f16": [i32, i32, i32, i32, vp, vp, vp, vp, vp, i32, i32, i32, i32, vp, vp, vp, vp,
                                       i32, vp, f32, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.rbq_workspace_bytes.argtypes = [i32] * 7
    lib.rbq_workspace_bytes.restype = sz
    lib.rbq_index_bytes.argtypes = [i32] * 4
    lib.rbq_index_bytes.restype = sz
    lib.rbq_status_string.argtypes = [i32]
    lib.rbq_status_string.restype = ctypes.c_char_p
    lib.rbq_version.argtypes = []
    lib.rbq_version.restype = i32
    return lib


lib = _load()


def status_string(s: int) -> str:
    return lib.rbq_status_string(s).decode()


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream=None):
    if stream is not None:
        return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream
    return torch.cuda.current_stream().cuda_stream


def _check(name, st):
    if st != RBQ_OK:
        raise RbqError(name, st)


def _need(name, **sizes):
    """Refuse a tensor smaller than what the call reads or writes through it:
    the C ABI takes bare pointers and cannot see buffer sizes. Each keyword is
    name=(tensor or None, elements needed)."""
    for arg, (t, count) in sizes.items():
        if isinstance(t, torch.Tensor) and t.numel() < count:
            raise ValueError(f"{name}: {arg} holds {t.numel()} elements, the call needs {count}")


class MappedHost:
    """A pinned host tensor handed to the kernels by its device address
    (hipHostGetDevicePointer), so that they read it over PCIe: a K/V cache kept
    in host memory while the index (codes, factors, centroids) stays in HBM.
    Only the rows a call touches cross the bus (the selected and window rows for
    the sparse attention). Usable wherever a call takes K / V (or a K_loc / V_loc
    from rows()), with the dtype of the wrapped tensor."""

    def __init__(self, t: torch.Tensor, _base=None, _offset=0):
        if t.device.type != "cpu" or not t.is_pinned() or not t.is_contiguous():
            raise ValueError("a host K/V buffer must be a contiguous pinned CPU tensor (pin_memory=True)")
        if _base is None:
            dev = ctypes.c_void_p()
            _check("rbq_mapped_device_pointer", lib.rbq_mapped_device_pointer(ctypes.c_void_p(t.data_ptr()),
                                                                              ctypes.byref(dev)))
            _base = dev.value
        self.tensor, self.dtype, self._base, self._offset = t, t.dtype, _base, _offset

    def data_ptr(self) -> int:
        return self._base + self._offset

    def rows(self, first_row: int, head_dim: int) -> "MappedHost":
        """The same buffer from row `first_row` of every block on (K + n*D: a cache tail)."""
        return MappedHost(self.tensor, self._base, self._offset + first_row * head_dim * self.tensor.element_size())


def kv_dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return RBQ_BF16
    if t.dtype == torch.float32:
        return RBQ_F32
    raise ValueError(f"unsupported key/value dtype {t.dtype}")


def rbq_workspace_bytes(op, batch, heads_q, heads_kv, head_dim, n, w=0) -> int:
    return int(lib.rbq_workspace_bytes(op, batch, heads_q, heads_kv, head_dim, n, w))


def rbq_index_bytes(batch, heads_kv, head_dim, cap) -> int:
    return int(lib.rbq_index_bytes(batch, heads_kv, head_dim, cap))


def rbq_version() -> int:
    return int(lib.rbq_version())


def workspace(op, batch, heads_q, heads_kv, head_dim, n, w=0, device="cuda") -> torch.Tensor:
    nbytes = max(rbq_workspace_bytes(op, batch, heads_q, heads_kv, head_dim, n, w), 256)
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def rbq_encode_keys(batch, heads_kv, head_dim, keys, keys_ld, n_new, offset, cap, P, c_q, c_k, codes, kfac,
                    flags, alpha_out=None, ws=None, stream=None, rot_out=None):
    """rbq_encode_keys (rbq_encode_keys_debug when rot_out is given)."""
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    args = (batch, heads_kv, head_dim, _ptr(keys), kv_dtype_code(keys), keys_ld, n_new, offset, cap, _ptr(P),
            _ptr(c_q), _ptr(c_k), _ptr(codes), _ptr(kfac), flags, _ptr(alpha_out), _ptr(ws), ws_bytes)
    if rot_out is None:
        _check("rbq_encode_keys", lib.rbq_encode_keys(*args, _stream(stream)))
    else:
        _check("rbq_encode_keys_debug", lib.rbq_encode_keys_debug(*args, _ptr(rot_out), _stream(stream)))


def rbq_quantize_query(batch, heads_q, heads_kv, head_dim, q, P, c_q, c_k, qplanes, qscal, stream=None,
                       qrot_out=None):
    _need("rbq_quantize_query", qplanes=(qplanes, batch * heads_q * 4 * (head_dim // 32)),
          qscal=(qscal, batch * heads_q * QSCAL_STRIDE))
    args = (batch, heads_q, heads_kv, head_dim, _ptr(q), _ptr(P), _ptr(c_q), _ptr(c_k), _ptr(qplanes), _ptr(qscal))
    if qrot_out is None:
        _check("rbq_quantize_query", lib.rbq_quantize_query(*args, _stream(stream)))
    else:
        _check("rbq_quantize_query_debug", lib.rbq_quantize_query_debug(*args, _ptr(qrot_out), _stream(stream)))


def rbq_quantize_query_bits(batch, heads_q, heads_kv, head_dim, q, P, c_q, c_k, bits, qplanes, qscal, stream=None):
    _check("rbq_quantize_query_bits", lib.rbq_quantize_query_bits(
        batch, heads_q, heads_kv, head_dim, _ptr(q), _ptr(P), _ptr(c_q), _ptr(c_k), bits, _ptr(qplanes), _ptr(qscal),
        _stream(stream)))


def rbq_score(batch, heads_q, heads_kv, head_dim, n, cap, codes, kfac, qplanes, qscal, scores, stream=None):
    _need("rbq_score", scores=(scores, batch * heads_q * n))
    _check("rbq_score", lib.rbq_score(batch, heads_q, heads_kv, head_dim, n, cap, _ptr(codes), _ptr(kfac),
                                      _ptr(qplanes), _ptr(qscal), _ptr(scores), _stream(stream)))


def rbq_score_q8(batch, heads_q, heads_kv, head_dim, n, cap, codes, kfac, qplanes8, qscal, scores, stream=None):
    """rbq_score for queries of up to 8 bits (eight bit-planes per head)."""
    _need("rbq_score_q8", scores=(scores, batch * heads_q * n))
    _check("rbq_score_q8", lib.rbq_score_q8(batch, heads_q, heads_kv, head_dim, n, cap, _ptr(codes), _ptr(kfac),
                                            _ptr(qplanes8), _ptr(qscal), _ptr(scores), _stream(stream)))


def rbq_score_ints_q8(batch, heads_q, heads_kv, head_dim, n, cap, codes, qplanes8, ip_out, pc_out, stream=None):
    _need("rbq_score_ints_q8", ip_out=(ip_out, batch * heads_q * n), pc_out=(pc_out, batch * heads_kv * n))
    _check("rbq_score_ints_q8", lib.rbq_score_ints_q8(batch, heads_q, heads_kv, head_dim, n, cap, _ptr(codes),
                                                      _ptr(qplanes8), _ptr(ip_out), _ptr(pc_out), _stream(stream)))


def rbq_score_ints(batch, heads_q, heads_kv, head_dim, n, cap, codes, qplanes, ip_out, pc_out, stream=None):
    _need("rbq_score_ints", ip_out=(ip_out, batch * heads_q * n), pc_out=(pc_out, batch * heads_kv * n))
    _check("rbq_score_ints", lib.rbq_score_ints(batch, heads_q, heads_kv, head_dim, n, cap, _ptr(codes),
                                                _ptr(qplanes), _ptr(ip_out), _ptr(pc_out), _stream(stream)))


def rbq_topp_select(batch, heads_q, n, scores, p, sm_scale, sel_idx, sel_count, ws, stream=None):
    _need("rbq_topp_select", scores=(scores, batch * heads_q * n), sel_idx=(sel_idx, batch * heads_q * n),
          sel_count=(sel_count, batch * heads_q))
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("rbq_topp_select", lib.rbq_topp_select(batch, heads_q, n, _ptr(scores), p, sm_scale, _ptr(sel_idx),
                                                  _ptr(sel_count), _ptr(ws), ws_bytes, _stream(stream)))


def rbq_sparse_decode(batch, heads_q, heads_kv, head_dim, q, K, V, cap, n, sel_idx, sel_count, K_loc, V_loc,
                      loc_ld, w, sm_scale, out, lse, ws, stream=None):
    _need("rbq_sparse_decode", sel_idx=(sel_idx, batch * heads_q * n), sel_count=(sel_count, batch * heads_q),
          out=(out, batch * heads_q * head_dim), lse=(lse, batch * heads_q))
    ws_bytes = ws.numel() * ws.element_size()
    _check("rbq_sparse_decode", lib.rbq_sparse_decode(
        batch, heads_q, heads_kv, head_dim, _ptr(q), _ptr(K), _ptr(V), kv_dtype_code(K), cap, n, _ptr(sel_idx),
        _ptr(sel_count), _ptr(K_loc), _ptr(V_loc), loc_ld, w, sm_scale, _ptr(out), _ptr(lse), _ptr(ws), ws_bytes,
        _stream(stream)))


def rbq_dense_decode(batch, heads_q, heads_kv, head_dim, q, K, V, cap, n, K_loc, V_loc, loc_ld, w, sm_scale, out,
                     lse, ws, stream=None):
    _need("rbq_dense_decode", out=(out, batch * heads_q * head_dim), lse=(lse, batch * heads_q))
    ws_bytes = ws.numel() * ws.element_size()
    _check("rbq_dense_decode", lib.rbq_dense_decode(
        batch, heads_q, heads_kv, head_dim, _ptr(q), _ptr(K), _ptr(V), kv_dtype_code(K), cap, n, _ptr(K_loc),
        _ptr(V_loc), loc_ld, w, sm_scale, _ptr(out), _ptr(lse), _ptr(ws), ws_bytes, _stream(stream)))


def rbq_decode_step(batch, heads_q, heads_kv, head_dim, q, P, c_q, c_k, K, V, cap, n, w, codes, kfac, flush, p,
                    sm_scale, qplanes, qscal, scores, sel_idx, sel_count, out, lse, ws, stream=None):
    _need("rbq_decode_step", qplanes=(qplanes, batch * heads_q * 4 * (head_dim // 32)),
          qscal=(qscal, batch * heads_q * QSCAL_STRIDE), scores=(scores, batch * heads_q * n),
          sel_idx=(sel_idx, batch * heads_q * n), sel_count=(sel_count, batch * heads_q),
          out=(out, batch * heads_q * head_dim), lse=(lse, batch * heads_q))
    ws_bytes = ws.numel() * ws.element_size()
    _check("rbq_decode_step", lib.rbq_decode_step(
        batch, heads_q, heads_kv, head_dim, _ptr(q), _ptr(P), _ptr(c_q), _ptr(c_k), _ptr(K), _ptr(V),
        kv_dtype_code(K), cap, n, w, _ptr(codes), _ptr(kfac), int(bool(flush)), p, sm_scale, _ptr(qplanes),
        _ptr(qscal), _ptr(scores), _ptr(sel_idx), _ptr(sel_count), _ptr(out), _ptr(lse), _ptr(ws), ws_bytes,
        _stream(stream)))


def rbq_decode_step_noalloc(batch, heads_q, heads_kv, head_dim, q, P, c_q, c_k, K, V, cap, n, w, codes, kfac, flush,
                            p, sm_scale, qplanes, qscal, scores, sel_idx, sel_count, out, lse, stream=None):
    _need("rbq_decode_step_noalloc", qplanes=(qplanes, batch * heads_q * 4 * (head_dim // 32)),
          qscal=(qscal, batch * heads_q * QSCAL_STRIDE), scores=(scores, batch * heads_q * n),
          sel_idx=(sel_idx, batch * heads_q * n), sel_count=(sel_count, batch * heads_q),
          out=(out, batch * heads_q * head_dim), lse=(lse, batch * heads_q))
    _check("rbq_decode_step_noalloc", lib.rbq_decode_step_noalloc(
        batch, heads_q, heads_kv, head_dim, _ptr(q), _ptr(P), _ptr(c_q), _ptr(c_k), _ptr(K), _ptr(V),
        kv_dtype_code(K), cap, n, w, _ptr(codes), _ptr(kfac), int(bool(flush)), p, sm_scale, _ptr(qplanes),
        _ptr(qscal), _ptr(scores), _ptr(sel_idx), _ptr(sel_count), _ptr(out), _ptr(lse), _stream(stream)))

# ---- ragged batches: per-sequence key counts (seq_n), window rows (seq_w) and p (seq_p), device tensors


def rbq_score_varlen(batch, heads_q, heads_kv, head_dim, n, cap, seq_n, codes, kfac, qplanes, qscal, scores,
                     stream=None):
    _need("rbq_score_varlen", scores=(scores, batch * heads_q * n), seq_n=(seq_n, batch))
    _check("rbq_score_varlen", lib.rbq_score_varlen(batch, heads_q, heads_kv, head_dim, n, cap, _ptr(seq_n),
                                                    _ptr(codes), _ptr(kfac), _ptr(qplanes), _ptr(qscal),
                                                    _ptr(scores), _stream(stream)))


def rbq_topp_select_varlen(batch, heads_q, n, seq_n, scores, seq_p, sm_scale, sel_idx, sel_count, ws, stream=None):
    _need("rbq_topp_select_varlen", scores=(scores, batch * heads_q * n), sel_idx=(sel_idx, batch * heads_q * n),
          sel_count=(sel_count, batch * heads_q), seq_n=(seq_n, batch), seq_p=(seq_p, batch))
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("rbq_topp_select_varlen", lib.rbq_topp_select_varlen(
        batch, heads_q, n, _ptr(seq_n), _ptr(scores), _ptr(seq_p), sm_scale, _ptr(sel_idx), _ptr(sel_count),
        _ptr(ws), ws_bytes, _stream(stream)))


def rbq_sparse_decode_varlen(batch, heads_q, heads_kv, head_dim, q, K, V, cap, n, w, seq_n, seq_w, sel_idx,
                             sel_count, sm_scale, out, lse, ws, stream=None):
    _need("rbq_sparse_decode_varlen", sel_idx=(sel_idx, batch * heads_q * n), sel_count=(sel_count, batch * heads_q),
          out=(out, batch * heads_q * head_dim), lse=(lse, batch * heads_q), seq_n=(seq_n, batch),
          seq_w=(seq_w, batch))
    ws_bytes = ws.numel() * ws.element_size()
    _check("rbq_sparse_decode_varlen", lib.rbq_sparse_decode_varlen(
        batch, heads_q, heads_kv, head_dim, _ptr(q), _ptr(K), _ptr(V), kv_dtype_code(K), cap, n, w, _ptr(seq_n),
        _ptr(seq_w), _ptr(sel_idx), _ptr(sel_count), sm_scale, _ptr(out), _ptr(lse), _ptr(ws), ws_bytes,
        _stream(stream)))


def rbq_dense_decode_varlen(batch, heads_q, heads_kv, head_dim, q, K, V, cap, n, w, seq_n, seq_w, sm_scale, out,
                            lse, ws, stream=None):
    _need("rbq_dense_decode_varlen", out=(out, batch * heads_q * head_dim), lse=(lse, batch * heads_q),
          seq_n=(seq_n, batch), seq_w=(seq_w, batch))
    ws_bytes = ws.numel() * ws.element_size()
    _check("rbq_dense_decode_varlen", lib.rbq_dense_decode_varlen(
        batch, heads_q, heads_kv, head_dim, _ptr(q), _ptr(K), _ptr(V), kv_dtype_code(K), cap, n, w, _ptr(seq_n),
        _ptr(seq_w), sm_scale, _ptr(out), _ptr(lse), _ptr(ws), ws_bytes, _stream(stream)))


def rbq_decode_step_varlen(batch, heads_q, heads_kv, head_dim, q, P, c_q, c_k, K, V, cap, n, w, seq_n, seq_w, codes,
                           kfac, flush, seq_p, sm_scale, qplanes, qscal, scores, sel_idx, sel_count, out, lse, ws,
                           stream=None):
    _need("rbq_decode_step_varlen", qplanes=(qplanes, batch * heads_q * 4 * (head_dim // 32)),
          qscal=(qscal, batch * heads_q * QSCAL_STRIDE), scores=(scores, batch * heads_q * n),
          sel_idx=(sel_idx, batch * heads_q * n), sel_count=(sel_count, batch * heads_q),
          out=(out, batch * heads_q * head_dim), lse=(lse, batch * heads_q),
          seq_n=(seq_n, batch), seq_w=(seq_w, batch), seq_p=(seq_p, batch))
    ws_bytes = ws.numel() * ws.element_size()
    _check("rbq_decode_step_varlen", lib.rbq_decode_step_varlen(
        batch, heads_q, heads_kv, head_dim, _ptr(q), _ptr(P), _ptr(c_q), _ptr(c_k), _ptr(K), _ptr(V),
        kv_dtype_code(K), cap, n, w, _ptr(seq_n), _ptr(seq_w), _ptr(codes), _ptr(kfac), int(bool(flush)),
        _ptr(seq_p), sm_scale, _ptr(qplanes), _ptr(qscal), _ptr(scores), _ptr(sel_idx), _ptr(sel_count), _ptr(out),
        _ptr(lse), _ptr(ws), ws_bytes, _stream(stream)))


# ---- the compact index: one fp16 factor per key ([B][Hkv][cap] torch.float16), built and read with c_q = 0


def rbq_encode_keys_f16(batch, heads_kv, head_dim, keys, keys_ld, n_new, offset, cap, P, c_k, codes, kfac16, flags,
                        ws=None, stream=None):
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("rbq_encode_keys_f16", lib.rbq_encode_keys_f16(
        batch, heads_kv, head_dim, _ptr(keys), kv_dtype_code(keys), keys_ld, n_new, offset, cap, _ptr(P), _ptr(c_k),
        _ptr(codes), _ptr(kfac16), flags, _ptr(ws), ws_bytes, _stream(stream)))


def rbq_score_f16(batch, heads_q, heads_kv, head_dim, n, cap, codes, kfac16, qplanes, qscal, scores, stream=None):
    _need("rbq_score_f16", scores=(scores, batch * heads_q * n))
    _check("rbq_score_f16", lib.rbq_score_f16(batch, heads_q, heads_kv, head_dim, n, cap, _ptr(codes), _ptr(kfac16),
                                              _ptr(qplanes), _ptr(qscal), _ptr(scores), _stream(stream)))


def rbq_decode_step_f16(batch, heads_q, heads_kv, head_dim, q, P, c_k, K, V, cap, n, w, codes, kfac16, flush, p,
                        sm_scale, qplanes, qscal, scores, sel_idx, sel_count, out, lse, ws, stream=None):
    _need("rbq_decode_step_f16", qplanes=(qplanes, batch * heads_q * 4 * (head_dim // 32)),
          qscal=(qscal, batch * heads_q * QSCAL_STRIDE), scores=(scores, batch * heads_q * n),
          sel_idx=(sel_idx, batch * heads_q * n), sel_count=(sel_count, batch * heads_q),
          out=(out, batch * heads_q * head_dim), lse=(lse, batch * heads_q))
    ws_bytes = ws.numel() * ws.element_size()
    _check("rbq_decode_step_f16", lib.rbq_decode_step_f16(
        batch, heads_q, heads_kv, head_dim, _ptr(q), _ptr(P), _ptr(c_k), _ptr(K), _ptr(V), kv_dtype_code(K), cap, n,
        w, _ptr(codes), _ptr(kfac16), int(bool(flush)), p, sm_scale, _ptr(qplanes), _ptr(qscal), _ptr(scores),
        _ptr(sel_idx), _ptr(sel_count), _ptr(out), _ptr(lse), _ptr(ws), ws_bytes, _stream(stream)))


def rbq_score_varlen_f16(batch, heads_q, heads_kv, head_dim, n, cap, seq_n, codes, kfac16, qplanes, qscal, scores,
                         stream=None):
    _need("rbq_score_varlen_f16", scores=(scores, batch * heads_q * n), seq_n=(seq_n, batch))
    _check("rbq_score_varlen_f16", lib.rbq_score_varlen_f16(
        batch, heads_q, heads_kv, head_dim, n, cap, _ptr(seq_n), _ptr(codes), _ptr(kfac16), _ptr(qplanes),
        _ptr(qscal), _ptr(scores), _stream(stream)))


def rbq_decode_step_varlen_f16(batch, heads_q, heads_kv, head_dim, q, P, c_k, K, V, cap, n, w, seq_n, seq_w, codes,
                               kfac16, flush, seq_p, sm_scale, qplanes, qscal, scores, sel_idx, sel_count, out, lse,
                               ws, stream=None):
    _need("rbq_decode_step_varlen_f16", qplanes=(qplanes, batch * heads_q * 4 * (head_dim // 32)),
          qscal=(qscal, batch * heads_q * QSCAL_STRIDE), scores=(scores, batch * heads_q * n),
          sel_idx=(sel_idx, batch * heads_q * n), sel_count=(sel_count, batch * heads_q),
          out=(out, batch * heads_q * head_dim), lse=(lse, batch * heads_q),
          seq_n=(seq_n, batch), seq_w=(seq_w, batch), seq_p=(seq_p, batch))
    ws_bytes = ws.numel() * ws.element_size()
    _check("rbq_decode_step_varlen_f16", lib.rbq_decode_step_varlen_f16(
        batch, heads_q, heads_kv, head_dim, _ptr(q), _ptr(P), _ptr(c_k), _ptr(K), _ptr(V), kv_dtype_code(K), cap, n,
        w, _ptr(seq_n), _ptr(seq_w), _ptr(codes), _ptr(kfac16), int(bool(flush)), _ptr(seq_p), sm_scale,
        _ptr(qplanes), _ptr(qscal), _ptr(scores), _ptr(sel_idx), _ptr(sel_count), _ptr(out), _ptr(lse), _ptr(ws),
        ws_bytes, _stream(stream)))
