"""Python binding of the MI355X greedy speculative-verification library.

A thin ctypes layer over the C ABI of ``include/ee.h``: it allocates device
memory with PyTorch (weights, packed-weight arena, KV pool, workspace),
passes raw pointers and the current HIP stream, and converts arguments and
results.  Every step of the verification path runs in the HIP kernels of
``libee.so``; nothing here computes any part of it.  If the library has not
been built, importing this package raises.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np
import torch  # loaded first so the HIP runtime it ships is the one libee.so binds to

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libee.so")

EE_OK, EE_EINVAL, EE_ECAPACITY, EE_ESTATE, EE_EHIP = 0, -1, -2, -3, -4
EE_F32, EE_BF16 = 0, 1

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -c 'import __graft_entry__ as g; g.build()'`")
_lib = ctypes.CDLL(LIB_PATH)

_i32, _vp, _sz = ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t
_pi32 = ctypes.POINTER(ctypes.c_int32)


class EEModelConfig(ctypes.Structure):
    _fields_ = [("n_layers", _i32), ("d_model", _i32), ("n_heads", _i32), ("n_kv_heads", _i32),
                ("head_dim", _i32), ("ffn", _i32), ("vocab", _i32), ("dtype", _i32),
                ("rms_eps", ctypes.c_float), ("rope_theta", ctypes.c_float),
                ("max_ctx", _i32), ("max_seqs", _i32), ("k_max", _i32), ("page_size", _i32)]


class EEWeights(ctypes.Structure):
    _fields_ = [("embed", _vp), ("lm_head", _vp), ("final_gain", _vp),
                ("wq", ctypes.POINTER(_vp)), ("wk", ctypes.POINTER(_vp)), ("wv", ctypes.POINTER(_vp)),
                ("wo", ctypes.POINTER(_vp)), ("w_gate", ctypes.POINTER(_vp)),
                ("w_up", ctypes.POINTER(_vp)), ("w_down", ctypes.POINTER(_vp)),
                ("attn_gain", ctypes.POINTER(_vp)), ("ffn_gain", ctypes.POINTER(_vp))]


def _sig(name, res, args):
    f = getattr(_lib, name)
    f.restype, f.argtypes = res, args
    return f


ee_packed_weight_bytes = _sig("ee_packed_weight_bytes", _sz, [ctypes.POINTER(EEModelConfig)])
ee_kv_pool_bytes = _sig("ee_kv_pool_bytes", _sz, [ctypes.POINTER(EEModelConfig)])
ee_workspace_bytes = _sig("ee_workspace_bytes", _sz, [ctypes.POINTER(EEModelConfig)])
ee_create = _sig("ee_create", _i32, [ctypes.POINTER(EEModelConfig), ctypes.POINTER(EEWeights),
                                     _vp, _vp, _vp, _vp, ctypes.POINTER(_vp)])
ee_destroy = _sig("ee_destroy", _i32, [_vp])
ee_prefill = _sig("ee_prefill", _i32, [_vp, _i32, _pi32, _i32, _pi32])
ee_verify = _sig("ee_verify", _i32, [_vp, _i32, _pi32, _i32, _pi32, _pi32, _pi32, _pi32])
ee_verify_noalloc = _sig("ee_verify_noalloc", _i32, [_vp, _i32, _pi32, _i32, _pi32, _pi32, _pi32, _pi32])
ee_verify_batch = _sig("ee_verify_batch", _i32, [_vp, _i32, _pi32, _pi32, _i32, _pi32, _pi32, _pi32, _pi32])
ee_verify_topk = _sig("ee_verify_topk", _i32, [_vp, _i32, _pi32, _pi32, _i32, _i32, _i32, _pi32, _pi32, _pi32])
_pf32 = ctypes.POINTER(ctypes.c_float)
ee_verify_sample = _sig("ee_verify_sample", _i32, [_vp, _i32, _pi32, _i32, _vp, _pf32, _pf32, ctypes.c_float, _i32,
                                                   _pi32, _pi32])
ee_extend = _sig("ee_extend", _i32, [_vp, _i32, _pi32, _i32, _pi32])
ee_kv_rollback = _sig("ee_kv_rollback", _i32, [_vp, _i32, _i32, _i32])
ee_seq_state = _sig("ee_seq_state", _i32, [_vp, _i32, _pi32, _pi32])
ee_match_reuse_c = _sig("ee_match_reuse", _i32, [_pi32, _i32, _pi32, _i32, _i32, _i32, _i32, _pi32, _pi32])
ee_get_logits = _sig("ee_get_logits", _i32, [_vp, ctypes.POINTER(ctypes.c_float), _i32])
ee_read_kv = _sig("ee_read_kv", _i32, [_vp, _i32, _i32, _vp, _vp])
ee_load_kv = _sig("ee_load_kv", _i32, [_vp, _i32, _i32, _i32, _vp, _vp])
ee_capture_bytes = _sig("ee_capture_bytes", _sz, [ctypes.POINTER(EEModelConfig), _i32])
ee_capture = _sig("ee_capture", _i32, [_vp, _vp, _sz])
ee_last_error = _sig("ee_last_error", ctypes.c_char_p, [_vp])
ee_profile = _sig("ee_profile", _i32, [_vp, ctypes.c_uint32])
ee_use_graphs = _sig("ee_use_graphs", _i32, [_vp, _i32])
ee_time_gemm = _sig("ee_time_gemm", _i32, [_vp, ctypes.c_uint32, _i32, _i32, ctypes.POINTER(ctypes.c_double)])
ee_time_stream_read = _sig("ee_time_stream_read", _i32, [_vp, _vp, _sz, _i32, ctypes.POINTER(ctypes.c_double)])
ee_profile_read = _sig("ee_profile_read", _i32, [_vp, ctypes.POINTER(ctypes.c_double),
                                                 ctypes.POINTER(ctypes.c_int64), _i32])

PROF_CLASSES = ("norm", "qkv", "attn", "combine", "oproj", "gateup", "down", "lmhead", "argmax",
                "accept", "compact", "finish")


EE_PHASE_REUSE, EE_PHASE_GENERATE = 0, 1


class EEEditParams(ctypes.Structure):
    _fields_ = [("k_reuse", _i32), ("gamma", _i32), ("top_k", _i32), ("dynamic", _i32),
                ("min_match", _i32), ("max_match", _i32)]


class EEEditState(ctypes.Structure):
    _fields_ = [("phase", _i32), ("cursor", _i32), ("last_phase", _i32), ("last_accept", _i32),
                ("steps", ctypes.c_int64 * 2), ("emitted", ctypes.c_int64 * 2),
                ("draft_tokens", ctypes.c_int64), ("draft_forwards", ctypes.c_int64)]


ee_edit_begin = _sig("ee_edit_begin", _i32, [_vp, _i32, _vp, _i32, ctypes.POINTER(EEEditState)])
ee_edit_step = _sig("ee_edit_step", _i32, [_vp, _i32, _vp, _i32, _pi32, _i32, ctypes.POINTER(EEEditParams),
                                           ctypes.POINTER(EEEditState), _pi32, _i32, _i32, _pi32])


class EEError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"ee error {code}: {msg}")
        self.code = code


def _check(rc: int, ctx=None):
    if rc != EE_OK:
        raise EEError(rc, ee_last_error(ctx).decode())


def _i32arr(x):
    a = np.ascontiguousarray(np.asarray(x, dtype=np.int32))
    return a, a.ctypes.data_as(_pi32)


def make_config(shape, max_ctx: int, max_seqs: int = 1, k_max: int = 64) -> EEModelConfig:
    return EEModelConfig(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads,
                         shape.head_dim, shape.ffn, shape.vocab,
                         EE_BF16 if shape.dtype == "bf16" else EE_F32,
                         shape.rms_eps, shape.rope_theta, max_ctx, max_seqs, k_max, 64)


def match_reuse(generated, original, cursor: int, min_ngram: int = 1, max_ngram: int = 8):
    """Reuse-phase matcher: (draft_start, match_len), (-1, 0) if nothing matches."""
    g, gp = _i32arr(generated)
    o, op = _i32arr(original)
    ds, ml = ctypes.c_int32(), ctypes.c_int32()
    _check(ee_match_reuse_c(gp, len(g), op, len(o), cursor, min_ngram, max_ngram,
                            ctypes.byref(ds), ctypes.byref(ml)))
    return ds.value, ml.value


def _to_device(a: np.ndarray, device) -> torch.Tensor:
    if a.dtype == np.uint16:
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16))
    else:
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(device, non_blocking=False)


class Engine:
    """One library context: packed weights, a paged KV pool, one workspace.

    ``weights`` provides numpy arrays in the model dtype (``embed``,
    ``lm_head``, ``final_gain``, ``layer(l)`` mapping), as drawn by
    ``workloads.gen_weights``.
    """

    def __init__(self, shape, weights, max_ctx: int, max_seqs: int = 1, k_max: int = 64,
                 device: str = "cuda:0"):
        if not torch.cuda.is_available():
            raise RuntimeError("the verification library needs a ROCm GPU")
        self.shape, self.device = shape, torch.device(device)
        self.cfg = make_config(shape, max_ctx, max_seqs, k_max)
        cfgp = ctypes.byref(self.cfg)
        nb_packed, nb_kv, nb_ws = ee_packed_weight_bytes(cfgp), ee_kv_pool_bytes(cfgp), ee_workspace_bytes(cfgp)
        if not (nb_packed and nb_kv and nb_ws):
            raise EEError(EE_EINVAL, "invalid model config for the library")
        with torch.cuda.device(self.device):
            self.packed = torch.empty(nb_packed, dtype=torch.uint8, device=self.device)
            self.kv_pool = torch.empty(nb_kv, dtype=torch.uint8, device=self.device)
            self.workspace = torch.empty(nb_ws, dtype=torch.uint8, device=self.device)
            self.stream = torch.cuda.current_stream(self.device)
            keep = []

            def dev(a):
                t = _to_device(a, self.device)
                keep.append(t)
                return t.data_ptr()

            L = shape.n_layers
            arr = lambda: (_vp * L)()
            ptrs = {k: arr() for k in ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down",
                                       "attn_gain", "ffn_gain")}
            for l in range(L):
                lw = weights.layer(l)
                for k in ptrs:
                    ptrs[k][l] = dev(lw[k])
            w = EEWeights(dev(weights.embed), dev(weights.lm_head), dev(weights.final_gain),
                          *[ctypes.cast(ptrs[k], ctypes.POINTER(_vp)) for k in
                            ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down", "attn_gain", "ffn_gain")])
            torch.cuda.synchronize(self.device)
            ctx = _vp()
            _check(ee_create(cfgp, ctypes.byref(w), self.packed.data_ptr(), self.kv_pool.data_ptr(),
                             self.workspace.data_ptr(), self.stream.cuda_stream, ctypes.byref(ctx)))
            self.ctx = ctx
            del keep
        self._last_rows = 0

    # -- calls ---------------------------------------------------------------
    def prefill(self, seq: int, tokens) -> int:
        t, tp = _i32arr(tokens)
        nxt = ctypes.c_int32()
        _check(ee_prefill(self.ctx, seq, tp, len(t), ctypes.byref(nxt)), self.ctx)
        self._last_rows = min(len(t) - (len(t) - 1) // (self.cfg.k_max + 1) * (self.cfg.k_max + 1),
                              self.cfg.k_max + 1)
        return nxt.value

    def extend(self, seq: int, tokens) -> int:
        """Commit [pending, tokens...] without verification; returns the new
        pending token (the greedy token after the last one)."""
        t, tp = _i32arr(tokens)
        nxt = ctypes.c_int32()
        _check(ee_extend(self.ctx, seq, tp if len(t) else None, len(t), ctypes.byref(nxt)), self.ctx)
        self._last_rows = (len(t) + 1) - len(t) // (self.cfg.k_max + 1) * (self.cfg.k_max + 1)
        return nxt.value

    def verify(self, seq: int, draft, parent=None):
        """Returns (accept_len, next_token, accepted_nodes or None)."""
        d, dp = _i32arr(draft)
        k = len(d)
        a, nxt = ctypes.c_int32(), ctypes.c_int32()
        if parent is not None:
            p, pp = _i32arr(parent)
            if len(p) != k:
                raise EEError(EE_EINVAL, "parent must have one entry per draft node")
            nodes = np.zeros(max(k, 1), dtype=np.int32)
            _check(ee_verify(self.ctx, seq, dp, k, pp, ctypes.byref(a), ctypes.byref(nxt),
                             nodes.ctypes.data_as(_pi32)), self.ctx)
            self._last_rows = k + 1
            return a.value, nxt.value, nodes[:a.value].copy()
        _check(ee_verify(self.ctx, seq, dp, k, None, ctypes.byref(a), ctypes.byref(nxt), None), self.ctx)
        self._last_rows = k + 1
        return a.value, nxt.value, None

    def verify_noalloc(self, seq: int, draft, parent=None):
        """ee_verify_noalloc: ee_verify with the step's scratch in the
        library's static device array (no allocation, no graph).  Returns
        (accept_len, next_token, accepted_nodes or None)."""
        d, dp = _i32arr(draft)
        k = len(d)
        a, nxt = ctypes.c_int32(), ctypes.c_int32()
        pp, nodes = None, None
        if parent is not None:
            p, pp = _i32arr(parent)
            if len(p) != k:
                raise EEError(EE_EINVAL, "parent must have one entry per draft node")
            nodes = np.zeros(max(k, 1), dtype=np.int32)
        _check(ee_verify_noalloc(self.ctx, seq, dp, k, pp, ctypes.byref(a), ctypes.byref(nxt),
                                 nodes.ctypes.data_as(_pi32) if nodes is not None else None), self.ctx)
        self._last_rows = k + 1
        return a.value, nxt.value, (nodes[:a.value].copy() if nodes is not None else None)

    def verify_batch(self, seqs, drafts, parents=None):
        """One block for several sequences; drafts (and parents) are equal-length
        lists, one per sequence.  Returns [(accept_len, next_token,
        accepted_nodes or None)] in the order of ``seqs``."""
        n = len(seqs)
        k = len(drafts[0]) if n else 0
        if len(drafts) != n or any(len(d) != k for d in drafts):
            raise EEError(EE_EINVAL, "one draft per sequence, all of the same length")
        sq, sp = _i32arr(seqs)
        d, dp = _i32arr(np.concatenate([np.asarray(x, dtype=np.int32).reshape(-1) for x in drafts])
                        if n else np.zeros(0, np.int32))
        acc = np.zeros(max(n, 1), dtype=np.int32)
        nxt = np.zeros(max(n, 1), dtype=np.int32)
        nodes = np.zeros(max(n * k, 1), dtype=np.int32)
        pp = None
        if parents is not None:
            if len(parents) != n or any(len(p) != k for p in parents):
                raise EEError(EE_EINVAL, "parents must match the drafts")
            p, pp = _i32arr(np.concatenate([np.asarray(x, dtype=np.int32).reshape(-1) for x in parents]))
        _check(ee_verify_batch(self.ctx, n, sp, dp, k, pp, acc.ctypes.data_as(_pi32), nxt.ctypes.data_as(_pi32),
                               nodes.ctypes.data_as(_pi32) if parents is not None else None), self.ctx)
        self._last_rows = n * (k + 1)
        out = []
        for b in range(n):
            a = int(acc[b])
            out.append((a, int(nxt[b]), nodes[b * k:b * k + a].copy() if parents is not None else None))
        return out

    def verify_sample(self, seq: int, draft, eps, u, q=None, temperature: float = 1.0, residual: bool = True):
        """Stochastic verification (Eq. 4).  ``q``: None (greedy draft) or a
        [K, vocab] float32 array of draft distributions (uploaded to the
        device here); ``eps`` (K) and ``u`` (K + 1) are uniform draws.
        Returns (accept_len, next_token)."""
        d, dp = _i32arr(draft)
        k = len(d)
        e = np.ascontiguousarray(np.asarray(eps, dtype=np.float32).reshape(-1))
        uu = np.ascontiguousarray(np.asarray(u, dtype=np.float32).reshape(-1))
        if len(e) != k or len(uu) != k + 1:
            raise EEError(EE_EINVAL, "eps needs K values and u K + 1")
        qdev = None
        if q is not None:
            qa = np.ascontiguousarray(np.asarray(q, dtype=np.float32))
            if qa.shape != (k, self.shape.vocab):
                raise EEError(EE_EINVAL, "q must be [K, vocab]")
            qdev = torch.from_numpy(qa).to(self.device)
            torch.cuda.synchronize(self.device)
        a, nxt = ctypes.c_int32(), ctypes.c_int32()
        _check(ee_verify_sample(self.ctx, seq, dp if k else None, k, qdev.data_ptr() if qdev is not None else None,
                                e.ctypes.data_as(_pf32), uu.ctypes.data_as(_pf32), float(temperature),
                                int(bool(residual)), ctypes.byref(a), ctypes.byref(nxt)), self.ctx)
        self._last_rows = k + 1
        return a.value, nxt.value

    def verify_topk(self, seqs, drafts, top_k: int, dynamic: bool = True):
        """Entropy-aware (``dynamic``) or fixed top-k verification of linear
        drafts, one per sequence, all of the same length.  Returns
        [(accept_len, next_token, thresholds)] in the order of ``seqs``, where
        thresholds[i] is the tau applied to draft token i."""
        n = len(seqs)
        k = len(drafts[0]) if n else 0
        if len(drafts) != n or any(len(d) != k for d in drafts):
            raise EEError(EE_EINVAL, "one draft per sequence, all of the same length")
        sq, sp = _i32arr(seqs)
        d, dp = _i32arr(np.concatenate([np.asarray(x, dtype=np.int32).reshape(-1) for x in drafts])
                        if n else np.zeros(0, np.int32))
        acc = np.zeros(max(n, 1), dtype=np.int32)
        nxt = np.zeros(max(n, 1), dtype=np.int32)
        thr = np.zeros(max(n * k, 1), dtype=np.int32)
        _check(ee_verify_topk(self.ctx, n, sp, dp, k, int(top_k), int(bool(dynamic)), acc.ctypes.data_as(_pi32),
                              nxt.ctypes.data_as(_pi32), thr.ctypes.data_as(_pi32)), self.ctx)
        self._last_rows = n * (k + 1)
        return [(int(acc[b]), int(nxt[b]), thr[b * k:(b + 1) * k].copy()) for b in range(n)]

    def rollback(self, seq: int, new_len: int, pending: int):
        _check(ee_kv_rollback(self.ctx, seq, new_len, pending), self.ctx)

    def seq_state(self, seq: int):
        n, p = ctypes.c_int32(), ctypes.c_int32()
        _check(ee_seq_state(self.ctx, seq, ctypes.byref(n), ctypes.byref(p)), self.ctx)
        return n.value, p.value

    def logits(self) -> np.ndarray:
        rows = self._last_rows
        out = np.empty((rows, self.shape.vocab), dtype=np.float32)
        _check(ee_get_logits(self.ctx, out.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), rows), self.ctx)
        return out

    def read_kv(self, seq: int, layer: int):
        n, _ = self.seq_state(seq)
        s = self.shape
        dt = np.uint16 if s.dtype == "bf16" else np.float32
        k = np.empty((n, s.n_kv_heads, s.head_dim), dtype=dt)
        v = np.empty_like(k)
        _check(ee_read_kv(self.ctx, seq, layer, k.ctypes.data, v.ctypes.data), self.ctx)
        return k, v

    def load_kv(self, seq: int, k, v, pending: int):
        """Install a committed cache in the empty sequence `seq`: k and v are
        [n_layers, n, n_kv_heads, head_dim] in the model dtype (bf16 bit
        patterns as uint16, or float32); `pending` starts the next block."""
        s = self.shape
        dt = np.uint16 if s.dtype == "bf16" else np.float32
        k = np.ascontiguousarray(k, dtype=dt)
        v = np.ascontiguousarray(v, dtype=dt)
        if k.shape != v.shape or k.ndim != 4 or k.shape[0] != s.n_layers or k.shape[2:] != (s.n_kv_heads, s.head_dim):
            raise EEError(EE_EINVAL, "k and v must be [n_layers, n, n_kv_heads, head_dim]")
        _check(ee_load_kv(self.ctx, seq, k.shape[1], int(pending), k.ctypes.data, v.ctypes.data), self.ctx)

    def capture(self, rows: int | None):
        """Start (rows: the row count of the blocks to capture) or end (None)
        recording every rounding site's values (ee_capture) into a device
        buffer of this engine; ``captured()`` reads the last block's."""
        if rows is None:     # the buffer stays readable until the next capture
            _check(ee_capture(self.ctx, None, 0), self.ctx)
            return
        nb = ee_capture_bytes(ctypes.byref(self.cfg), int(rows))
        if not nb:
            raise EEError(EE_EINVAL, "invalid capture row count")
        self._cap = torch.empty(nb, dtype=torch.uint8, device=self.device)
        self._cap_rows = int(rows)
        _check(ee_capture(self.ctx, self._cap.data_ptr(), nb), self.ctx)

    def captured(self):
        """{(site, layer): array} of the last captured block, in the model
        dtype (bf16 bit patterns as uint16): x_attn, o, x_ffn, z [rows, cols]
        and q [rows, n_heads, head_dim], k, v [rows, n_kv_heads, head_dim]
        per layer; x_final [rows, d_model] at layer n_layers."""
        s, R = self.shape, self._cap_rows
        torch.cuda.synchronize(self.device)
        raw = self._cap.cpu().numpy()
        dt, esz, ks = (np.uint16, 2, 32) if s.dtype == "bf16" else (np.float32, 4, 16)
        R16 = (R + 15) // 16 * 16
        off = 0

        def take(n):
            nonlocal off
            a = raw[off:off + n * esz].view(dt)
            off += n * esz
            return a

        def packed(cols):
            # fragments [R16/16][cols/KS][4 lane groups][16 lanes][KS/4 elements]
            a = take(R16 * cols).reshape(R16 // 16, cols // ks, 4, 16, ks // 4)
            return a.transpose(0, 3, 1, 2, 4).reshape(R16, cols)[:R]

        out = {}
        qd, kd = s.n_heads * s.head_dim, s.n_kv_heads * s.head_dim
        for l in range(s.n_layers):
            out[("x_attn", l)] = packed(s.d_model)
            out[("q", l)] = take(R * qd).reshape(R, s.n_heads, s.head_dim)
            out[("k", l)] = take(R * kd).reshape(R, s.n_kv_heads, s.head_dim)
            out[("v", l)] = take(R * kd).reshape(R, s.n_kv_heads, s.head_dim)
            out[("o", l)] = packed(qd)
            out[("x_ffn", l)] = packed(s.d_model)
            out[("z", l)] = packed(s.ffn)
        out[("x_final", s.n_layers)] = packed(s.d_model)
        assert off == len(raw)
        return out

    def use_graphs(self, on: bool):
        """Replay captured HIP graphs per block shape and attention split count
        (default) or launch eagerly."""
        _check(ee_use_graphs(self.ctx, int(bool(on))), self.ctx)

    def profile(self, classes=()):
        """Bracket launches of the named kernel classes with HIP events."""
        mask = 0
        for c in classes:
            mask |= 1 << PROF_CLASSES.index(c)
        _check(ee_profile(self.ctx, mask), self.ctx)

    def profile_read(self, reset: bool = True):
        """{class: (total ms, launches)} accumulated since the last reset."""
        ms = (ctypes.c_double * len(PROF_CLASSES))()
        n = (ctypes.c_int64 * len(PROF_CLASSES))()
        _check(ee_profile_read(self.ctx, ms, n, int(reset)), self.ctx)
        return {c: (ms[i], n[i]) for i, c in enumerate(PROF_CLASSES)}

    def time_gemm(self, cls: str, rows: int, reps: int = 3) -> float:
        """Microseconds per launch of one projection's GEMM, launched for every
        layer in turn, back to back (ee_time_gemm)."""
        us = ctypes.c_double()
        _check(ee_time_gemm(self.ctx, PROF_CLASSES.index(cls), rows, reps, ctypes.byref(us)), self.ctx)
        return us.value

    def time_stream_read(self, buf: torch.Tensor, reps: int = 10) -> float:
        """Microseconds per pass of a plain streaming read of the device
        tensor ``buf`` (ee_time_stream_read)."""
        us = ctypes.c_double()
        nb = buf.numel() * buf.element_size() // 16 * 16
        _check(ee_time_stream_read(self.ctx, buf.data_ptr(), nb, int(reps), ctypes.byref(us)), self.ctx)
        return us.value

    def close(self):
        if getattr(self, "ctx", None):
            _check(ee_destroy(self.ctx))
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class EditSession:
    """An edit session over a target engine's sequence and, optionally, a
    draft engine's sequence holding the same prompt (ee_edit_begin /
    ee_edit_step).  ``output`` is the emitted token stream so far."""

    def __init__(self, target: Engine, seq: int, original, draft: Engine | None = None, draft_seq: int = 0,
                 k_reuse: int = 32, gamma: int = 7, top_k: int = 0, dynamic: bool = True,
                 min_match: int = 3, max_match: int = 8, capacity: int = 1 << 16):
        self.target, self.seq, self.draft, self.draft_seq = target, seq, draft, draft_seq
        self.original, self._op = _i32arr(original)
        self.params = EEEditParams(k_reuse, gamma, top_k, int(bool(dynamic)), min_match, max_match)
        self.state = EEEditState()
        _check(ee_edit_begin(target.ctx, seq, draft.ctx if draft else None, draft_seq,
                             ctypes.byref(self.state)), target.ctx)
        self._out = np.zeros(capacity, dtype=np.int32)
        self._out[0] = target.seq_state(seq)[1]
        self.n = 1

    @property
    def output(self):
        return self._out[:self.n].tolist()

    def step(self):
        """One Reuse or Generate step; returns (phase, new tokens)."""
        nn = ctypes.c_int32()
        _check(ee_edit_step(self.target.ctx, self.seq, self.draft.ctx if self.draft else None, self.draft_seq,
                            self._op, len(self.original), ctypes.byref(self.params), ctypes.byref(self.state),
                            self._out.ctypes.data_as(_pi32), self.n, len(self._out), ctypes.byref(nn)),
               self.target.ctx)
        new = self._out[self.n:self.n + nn.value].tolist()
        self.n += nn.value
        return self.state.last_phase, new
