"""Device buffers of one decode workload and the calls of one decode step.

The KV cache of a (sequence, KV head) holds `cap` rows: rows [0, n) are
indexed (Algorithm 1), rows [n, n + w) are the local window of newest keys
that decode attends in full precision and that a lazy flush later appends to
the index (Section 3.4). torch only allocates memory and supplies the stream;
every step of the method runs in librbq.so's kernels.
"""
from __future__ import annotations

import math

import numpy as np
import torch

from . import rbq


def to_device_kv(arr: np.ndarray, kv_dtype: str, device) -> torch.Tensor:
    """Upload keys/values given as float32 or as bf16 bit patterns (uint16)."""
    if kv_dtype == "f32":
        return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).to(device)
    t = torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).to(device)
    return t.view(torch.bfloat16)


class DecodeState:
    """Index + cache + per-step buffers for B sequences x Hkv KV heads."""

    def __init__(self, B, Hq, Hkv, D, cap, n, w, K, V, q, P, c_q=None, device="cuda", compact=False):
        """compact: the compact index (one fp16 factor per key in kfac16, no
        query centroid) and the *_f16 calls instead of the fp32 (f, g) index."""
        if compact and c_q is not None:
            raise ValueError("the compact index is built and read without a query centroid")
        self.compact = compact
        self.B, self.Hq, self.Hkv, self.D = B, Hq, Hkv, D
        self.cap, self.n, self.w = cap, n, w
        self.device = device
        self.K, self.V = K, V                       # [B][Hkv][cap][D]
        self.q = q                                  # [B][Hq][D] fp32
        self.P = P                                  # [D][D] fp32
        self.c_q = c_q                              # [B][Hkv][D] fp32 or None
        f32 = dict(dtype=torch.float32, device=device)
        self.c_k = torch.zeros(B, Hkv, D, **f32)
        self.codes = torch.zeros(B, Hkv, cap, D // 32, dtype=torch.int32, device=device)
        self.kfac = None if compact else torch.zeros(B, Hkv, cap, 2, **f32)
        self.kfac16 = torch.zeros(B, Hkv, cap, dtype=torch.float16, device=device) if compact else None
        self.qplanes = torch.zeros(B, Hq, 4, D // 32, dtype=torch.int32, device=device)
        self.qscal = torch.zeros(B, Hq, rbq.QSCAL_STRIDE, **f32)
        self.scores = torch.zeros(B, Hq, max(n, 1), **f32)
        self.sel_idx = torch.zeros(B, Hq, max(n, 1), dtype=torch.int32, device=device)
        self.sel_count = torch.zeros(B, Hq, dtype=torch.int32, device=device)
        self.out = torch.zeros(B, Hq, D, **f32)
        self.lse = torch.zeros(B, Hq, **f32)
        self.ws_encode = rbq.workspace(rbq.RBQ_OP_ENCODE, B, Hq, Hkv, D, max(n, w, 1), 0, device)
        self.ws_topp = rbq.workspace(rbq.RBQ_OP_TOPP, B, Hq, Hkv, D, n, 0, device)
        self.ws_decode = rbq.workspace(rbq.RBQ_OP_SPARSE_DECODE, B, Hq, Hkv, D, n, w, device)
        self.ws_step = rbq.workspace(rbq.RBQ_OP_DECODE_STEP, B, Hq, Hkv, D, n, w, device)
        self.sm_scale = 1.0 / math.sqrt(D)

    @classmethod
    def from_workload(cls, wl, device="cuda", c_q: bool = True, compact: bool = False):
        K = to_device_kv(wl.K, wl.kv_dtype, device)
        V = to_device_kv(wl.V, wl.kv_dtype, device)
        q = torch.from_numpy(np.ascontiguousarray(wl.q)).to(device)
        P = torch.from_numpy(np.ascontiguousarray(wl.P)).to(device)
        cq = torch.from_numpy(np.ascontiguousarray(wl.c_q)).to(device) if c_q and not compact else None
        return cls(wl.B, wl.Hq, wl.Hkv, wl.D, wl.N, wl.n_index, wl.w, K, V, q, P, cq, device, compact)

    def _window(self, t):
        """Rows [n, cap) of a cache (the local window), in HBM or mapped host memory."""
        return t.rows(self.n, self.D) if isinstance(t, rbq.MappedHost) else t[:, :, self.n:]

    # ---------------------------------------------------------------- the five calls
    def build_index(self, stream=None, rot_out=None, alpha_out=None):
        """Prefill index construction over rows [0, n), setting c_k (Algorithm 1)."""
        if self.compact:
            rbq.rbq_encode_keys_f16(self.B, self.Hkv, self.D, self.K, self.cap, self.n, 0, self.cap, self.P,
                                    self.c_k, self.codes, self.kfac16, rbq.RBQ_ENCODE_SET_CENTROID, self.ws_encode,
                                    stream)
            return
        rbq.rbq_encode_keys(self.B, self.Hkv, self.D, self.K, self.cap, self.n, 0, self.cap, self.P, self.c_q,
                            self.c_k, self.codes, self.kfac, rbq.RBQ_ENCODE_SET_CENTROID, alpha_out,
                            self.ws_encode, stream, rot_out=rot_out)

    def flush_window(self, stream=None):
        """Lazy update: encode the w window rows into index rows [n, n + w) with
        the prefill centroid (Section 3.4). The index size used by scoring is
        left at n, so repeated steps stay identical."""
        if self.w == 0:
            return
        K_win = self._window(self.K)
        if self.compact:
            rbq.rbq_encode_keys_f16(self.B, self.Hkv, self.D, K_win, self.cap, self.w, self.n, self.cap, self.P,
                                    self.c_k, self.codes, self.kfac16, 0, None, stream)
            return
        rbq.rbq_encode_keys(self.B, self.Hkv, self.D, K_win, self.cap, self.w, self.n, self.cap, self.P, self.c_q,
                            self.c_k, self.codes, self.kfac, 0, None, None, stream)

    def quantize(self, stream=None, qrot_out=None):
        rbq.rbq_quantize_query(self.B, self.Hq, self.Hkv, self.D, self.q, self.P, self.c_q, self.c_k,
                               self.qplanes, self.qscal, stream, qrot_out=qrot_out)

    def score(self, stream=None):
        if self.compact:
            rbq.rbq_score_f16(self.B, self.Hq, self.Hkv, self.D, self.n, self.cap, self.codes, self.kfac16,
                              self.qplanes, self.qscal, self.scores, stream)
            return
        rbq.rbq_score(self.B, self.Hq, self.Hkv, self.D, self.n, self.cap, self.codes, self.kfac, self.qplanes,
                      self.qscal, self.scores, stream)

    def select(self, p, stream=None):
        rbq.rbq_topp_select(self.B, self.Hq, self.n, self.scores, p, self.sm_scale, self.sel_idx, self.sel_count,
                            self.ws_topp, stream)

    def sparse_decode(self, stream=None):
        K_loc = self._window(self.K) if self.w else None
        V_loc = self._window(self.V) if self.w else None
        rbq.rbq_sparse_decode(self.B, self.Hq, self.Hkv, self.D, self.q, self.K, self.V, self.cap, self.n,
                              self.sel_idx, self.sel_count, K_loc, V_loc, self.cap, self.w, self.sm_scale, self.out,
                              self.lse, self.ws_decode, stream)

    def dense_decode(self, out=None, lse=None, stream=None):
        K_loc = self._window(self.K) if self.w else None
        V_loc = self._window(self.V) if self.w else None
        rbq.rbq_dense_decode(self.B, self.Hq, self.Hkv, self.D, self.q, self.K, self.V, self.cap, self.n, K_loc,
                             V_loc, self.cap, self.w, self.sm_scale, self.out if out is None else out,
                             self.lse if lse is None else lse, self.ws_decode, stream)

    def step(self, p, stream=None, flush=True):
        """One decode step of the whole path with rbq_decode_step: quantize ->
        score -> Top-p -> sparse attention (index selection + window), and the
        lazy flush of the window into index rows [n, n + w) (which this step's
        scoring does not read), in one call with fewer launches."""
        if self.compact:
            rbq.rbq_decode_step_f16(self.B, self.Hq, self.Hkv, self.D, self.q, self.P, self.c_k, self.K, self.V,
                                    self.cap, self.n, self.w, self.codes, self.kfac16, flush, p, self.sm_scale,
                                    self.qplanes, self.qscal, self.scores, self.sel_idx, self.sel_count, self.out,
                                    self.lse, self.ws_step, stream)
            return
        rbq.rbq_decode_step(self.B, self.Hq, self.Hkv, self.D, self.q, self.P, self.c_q, self.c_k, self.K, self.V,
                            self.cap, self.n, self.w, self.codes, self.kfac, flush, p, self.sm_scale, self.qplanes,
                            self.qscal, self.scores, self.sel_idx, self.sel_count, self.out, self.lse, self.ws_step,
                            stream)

    def step_calls(self, p, stream=None, flush=True):
        """The same step as the five separate calls (bitwise the same outputs)."""
        self.quantize(stream)
        self.score(stream)
        self.select(p, stream)
        self.sparse_decode(stream)
        if flush:
            self.flush_window(stream)

    # ---------------------------------------------------------------- ragged batches
    # seq_n / seq_w / seq_p: per-sequence indexed keys, window rows (the cache
    # tail after them) and p, as int32 / int32 / float32 device tensors [B]; the
    # state's n and w are the largest counts (n + w <= cap).
    def build_index_ragged(self, seq_n_host, stream=None):
        """Index construction of a ragged batch: sequence b over its rows
        [0, seq_n_host[b]) with its own centroid (a sequence without keys keeps a
        zero centroid)."""
        for b, nb in enumerate(seq_n_host):
            nb = min(int(nb), self.n)
            if nb > 0 and self.compact:
                rbq.rbq_encode_keys_f16(1, self.Hkv, self.D, self.K[b:b + 1], self.cap, nb, 0, self.cap, self.P,
                                        self.c_k[b:b + 1], self.codes[b:b + 1], self.kfac16[b:b + 1],
                                        rbq.RBQ_ENCODE_SET_CENTROID, self.ws_encode, stream)
            elif nb > 0:
                rbq.rbq_encode_keys(1, self.Hkv, self.D, self.K[b:b + 1], self.cap, nb, 0, self.cap, self.P,
                                    None if self.c_q is None else self.c_q[b:b + 1], self.c_k[b:b + 1],
                                    self.codes[b:b + 1], self.kfac[b:b + 1], rbq.RBQ_ENCODE_SET_CENTROID, None,
                                    self.ws_encode, stream)

    def step_ragged(self, seq_n, seq_w, seq_p, stream=None, flush=True):
        """One decode step of a ragged batch (rbq_decode_step_varlen)."""
        if self.compact:
            rbq.rbq_decode_step_varlen_f16(self.B, self.Hq, self.Hkv, self.D, self.q, self.P, self.c_k, self.K,
                                           self.V, self.cap, self.n, self.w, seq_n, seq_w, self.codes, self.kfac16,
                                           flush, seq_p, self.sm_scale, self.qplanes, self.qscal, self.scores,
                                           self.sel_idx, self.sel_count, self.out, self.lse, self.ws_step, stream)
            return
        rbq.rbq_decode_step_varlen(self.B, self.Hq, self.Hkv, self.D, self.q, self.P, self.c_q, self.c_k, self.K,
                                   self.V, self.cap, self.n, self.w, seq_n, seq_w, self.codes, self.kfac, flush,
                                   seq_p, self.sm_scale, self.qplanes, self.qscal, self.scores, self.sel_idx,
                                   self.sel_count, self.out, self.lse, self.ws_step, stream)

    def sparse_decode_ragged(self, seq_n, seq_w, stream=None):
        rbq.rbq_sparse_decode_varlen(self.B, self.Hq, self.Hkv, self.D, self.q, self.K, self.V, self.cap, self.n,
                                     self.w, seq_n, seq_w, self.sel_idx, self.sel_count, self.sm_scale, self.out,
                                     self.lse, self.ws_decode, stream)

    def dense_decode_ragged(self, seq_n, seq_w, out=None, lse=None, stream=None):
        rbq.rbq_dense_decode_varlen(self.B, self.Hq, self.Hkv, self.D, self.q, self.K, self.V, self.cap, self.n,
                                    self.w, seq_n, seq_w, self.sm_scale, self.out if out is None else out,
                                    self.lse if lse is None else lse, self.ws_decode, stream)


class DecodeSession:
    """A decode loop over one growing cache: the lazy index update of Section
    3.4 as a serving loop would run it. The cache holds `cap` rows per (sequence,
    KV head). The prefill rows [0, n) are indexed once (with their centroid);
    each generated token's key and value are appended to the window after the
    indexed rows, each step attends over the Top-p selection of the index plus
    the whole window (one rbq_decode_step), and the step that finds the window
    full also flushes it into the index (encoded with the prefill centroid), so
    the next step scores n + window keys. Buffers and workspaces are sized once,
    for the largest index the cache can hold.

    K, V: [B][Hkv][cap][D] device tensors holding the prefill rows; P: the
    rotation; c_q: query centroids or None; compact: the fp16-factor index
    (then without c_q)."""

    def __init__(self, B, Hq, Hkv, D, cap, n_prefill, window, K, V, P, c_q=None, device="cuda", compact=False):
        if not 0 < window <= rbq.RBQ_MAX_WINDOW or n_prefill + window > cap:
            raise ValueError("the window must fit after the prefill rows (n_prefill + window <= cap)")
        q = torch.zeros(B, Hq, D, dtype=torch.float32, device=device)
        # Every flush adds a whole window to the index, and append() keeps
        # n + w <= cap, so the index sizes a step can see are n_prefill + k * window
        # up to cap (the last one may leave less than a window of room, and the
        # steps after it run with that index and a partial window).
        self.n_sizes = list(range(n_prefill, cap + 1, window))
        self.n_max = self.n_sizes[-1]
        # sized for the largest index: the scores, selections and per-row workspaces grow with n
        self.state = DecodeState(B, Hq, Hkv, D, cap, self.n_max, window, K, V, q, P, c_q, device, compact)
        self.n, self.w, self.window = n_prefill, 0, window
        st = self.state
        # the step workspace is not monotonic in n (smaller indexes may take more,
        # shorter decode splits): size it for every index size the loop will pass;
        # for a given n it grows with the window rows, so the full window bounds it
        need = max(rbq.rbq_workspace_bytes(rbq.RBQ_OP_DECODE_STEP, B, Hq, Hkv, D, m, window)
                   for m in self.n_sizes)
        if need > st.ws_step.numel():
            st.ws_step = torch.empty(need, dtype=torch.uint8, device=device)
        if compact:
            rbq.rbq_encode_keys_f16(B, Hkv, D, K, cap, n_prefill, 0, cap, P, st.c_k, st.codes, st.kfac16,
                                    rbq.RBQ_ENCODE_SET_CENTROID, st.ws_encode)
        else:
            rbq.rbq_encode_keys(B, Hkv, D, K, cap, n_prefill, 0, cap, P, c_q, st.c_k, st.codes, st.kfac,
                                rbq.RBQ_ENCODE_SET_CENTROID, None, st.ws_encode)

    def append(self, k: torch.Tensor, v: torch.Tensor):
        """Append one token's key and value ([B][Hkv][D]) to the window."""
        if self.w == self.window:
            raise RuntimeError("the window is full: run step() first (it flushes the window)")
        if self.n + self.w >= self.state.cap:
            raise RuntimeError("the cache is full")
        r = self.n + self.w
        self.state.K[:, :, r].copy_(k)
        self.state.V[:, :, r].copy_(v)
        self.w += 1

    def step(self, q: torch.Tensor, p: float, stream=None) -> bool:
        """One decode step for the query q [B][Hq][D] at Top-p p; returns whether
        the window was flushed into the index. The outputs are state.out and
        state.lse; the selection is state.sel_idx / state.sel_count (row stride:
        the n of this step, self.n before a flush)."""
        st = self.state
        if self.n > self.n_max or self.n + self.w > st.cap:
            raise RuntimeError(f"index of {self.n} keys + {self.w} window rows exceeds the session's buffers "
                               f"({self.n_max} keys, cap {st.cap})")
        st.q.copy_(q)
        flush = self.w == self.window
        if st.compact:
            rbq.rbq_decode_step_f16(st.B, st.Hq, st.Hkv, st.D, st.q, st.P, st.c_k, st.K, st.V, st.cap, self.n,
                                    self.w, st.codes, st.kfac16, flush, p, st.sm_scale, st.qplanes, st.qscal,
                                    st.scores, st.sel_idx, st.sel_count, st.out, st.lse, st.ws_step, stream)
        else:
            rbq.rbq_decode_step(st.B, st.Hq, st.Hkv, st.D, st.q, st.P, st.c_q, st.c_k, st.K, st.V, st.cap, self.n,
                                self.w, st.codes, st.kfac, flush, p, st.sm_scale, st.qplanes, st.qscal, st.scores,
                                st.sel_idx, st.sel_count, st.out, st.lse, st.ws_step, stream)
        self.last_n, self.last_w = self.n, self.w
        if flush:
            self.n += self.w
            self.w = 0
        return flush
