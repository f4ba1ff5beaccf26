"""ctypes binding of libmetro.so (include/metro.h, include/metro_ops.h, include/metro_sched.h).

Argument marshalling only: every step of the forward pass runs in the HIP
library.  PyTorch serves as the source of device buffers (``tensor.data_ptr()``)
and of the current HIP stream.  Importing this module raises ImportError when
the library has not been built -- there is no fallback.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmetro.so")
if not os.path.exists(_LIB_PATH):
    raise ImportError(f"{_LIB_PATH} is not built; run `python -m paper_2411_03519_amd.build`")
lib = ctypes.CDLL(_LIB_PATH)

ABI_VERSION = 2

STATUS = {0: "METRO_OK", -1: "METRO_E_INVAL", -2: "METRO_E_NOMEM", -3: "METRO_E_NOPAGES", -4: "METRO_E_SEQ",
          -5: "METRO_E_CAPACITY", -6: "METRO_E_HIP"}

WEIGHT_ID = {"embed": 0, "final_norm": 1, "lm_head": 2, "attn_norm": 3, "wq": 4, "wk": 5, "wv": 6, "wo": 7,
             "ffn_norm": 8, "wgate": 9, "wup": 10, "wdown": 11}

EPI_STORE_F32, EPI_ADD_F32, EPI_SWIGLU = 0, 1, 2

KERNEL_CLASS = {"embed": 0, "rmsnorm": 1, "gemm_qkv": 2, "rope_kv": 3, "attention": 4,
                "gemm_o": 6, "gemm_gate_up": 7, "gemm_down": 8, "lm_head": 9, "argmax": 10}
PHASE = {"any": 0, "prefill": 1, "decode": 2}


class Config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rope_base", ctypes.c_float), ("rms_eps", ctypes.c_float),
                ("page_size", ctypes.c_int32), ("max_batch", ctypes.c_int32), ("max_tokens", ctypes.c_int32),
                ("max_context", ctypes.c_int32), ("max_seqs", ctypes.c_int32), ("kv_pool_bytes", ctypes.c_int64)]


class PrefixCacheStats(ctypes.Structure):
    _fields_ = [("pages", ctypes.c_int32), ("limit", ctypes.c_int32), ("lookup_tokens", ctypes.c_int64),
                ("hit_tokens", ctypes.c_int64), ("inserted", ctypes.c_int64), ("evicted", ctypes.c_int64)]


class ModelInfo(ctypes.Structure):
    _fields_ = [("weight_bytes", ctypes.c_int64), ("scratch_bytes", ctypes.c_int64),
                ("kv_pool_bytes", ctypes.c_int64), ("kv_bytes_per_token", ctypes.c_int64),
                ("n_pages", ctypes.c_int32), ("free_pages", ctypes.c_int32), ("open_seqs", ctypes.c_int32),
                ("device", ctypes.c_int32)]


_vp, _i32, _i64, _u64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
_SIGS = {
    "metro_abi_version": (_i32, []),
    "metro_last_error": (ctypes.c_char_p, []),
    "metro_status_name": (ctypes.c_char_p, [_i32]),
    "metro_create_model": (_i32, [ctypes.POINTER(Config), _u64, ctypes.POINTER(_vp)]),
    "metro_destroy_model": (None, [_vp]),
    "metro_load_weight": (_i32, [_vp, _i32, _i32, _vp, _i64]),
    "metro_model_get_info": (_i32, [_vp, ctypes.POINTER(ModelInfo)]),
    "metro_seq_open": (_i32, [_vp, ctypes.POINTER(_i64)]),
    "metro_seq_open_cached": (_i32, [_vp, _vp, _i32, ctypes.POINTER(_i64), ctypes.POINTER(_i32)]),
    "metro_prefix_cache": (_i32, [_vp, _i32]),
    "metro_prefix_cache_get_stats": (_i32, [_vp, ctypes.POINTER(PrefixCacheStats)]),
    "metro_seq_fork": (_i32, [_vp, _i64, _i32, _vp, ctypes.POINTER(_i64)]),
    "metro_seq_close": (_i32, [_vp, _i64]),
    "metro_seq_length": (_i32, [_vp, _i64, ctypes.POINTER(_i32)]),
    "metro_seq_pages": (_i32, [_vp, _i64, _vp, _i32, ctypes.POINTER(_i32)]),
    "metro_prefill_chunk": (_i32, [_vp, _i32, _vp, _vp, _vp, _vp, _vp, _vp]),
    "metro_decode_step": (_i32, [_vp, _i32, _vp, _vp, _vp, _vp, _vp]),
    "metro_profile_start": (_i32, [_vp, _i32, _i32]),
    "metro_profile_stop": (_i32, [_vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_i64)]),
    "metro_op_pack_weight": (_i32, [_vp, _i32, _i32, _i32, _i32, _vp, _vp]),
    "metro_op_gemm": (_i32, [_vp, _i32, _vp, _i32, _i32, _i32, _i32, _vp, _vp, _i32, _vp, _vp]),
    "metro_op_gemm_plan": (_i32, [_i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp]),
    "metro_op_rmsnorm": (_i32, [_vp, _vp, ctypes.c_float, _vp, _i32, _i32, _vp]),
    "metro_op_argmax": (_i32, [_vp, _i32, _i32, _vp, _vp]),
    "metro_op_attn_decode": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp]),
    "metro_op_attn_prefill": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp]),
    "metro_op_attn_decode_noalloc": (_i32, [_vp, _vp, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _vp]),
    "metro_sched_create": (_i32, [_vp, _vp, ctypes.POINTER(_vp)]),
    "metro_sched_destroy": (None, [_vp]),
    "metro_sched_next": (_i32, [_vp, ctypes.POINTER(_i32), ctypes.POINTER(_i32), _vp, _i32, ctypes.POINTER(_i32)]),
    "metro_sched_ack": (_i32, [_vp, _i32, _vp]),
    "metro_sched_state": (_i32, [_vp, _vp, _vp, _vp, ctypes.POINTER(_i32), ctypes.POINTER(_i32)]),
    "metro_engine_create": (_i32, [_vp, _vp, ctypes.POINTER(_vp)]),
    "metro_engine_destroy": (None, [_vp]),
    "metro_engine_submit": (_i32, [_vp, _i64, _i32, _vp, _i32, _i32]),
    "metro_engine_step": (_i32, [_vp, _vp, ctypes.POINTER(_i32)]),
    "metro_engine_last_plan": (_i32, [_vp, _vp, _vp, _vp, _i32, ctypes.POINTER(_i32)]),
    "metro_engine_finished": (_i32, [_vp, _vp, _i32, ctypes.POINTER(_i32)]),
    "metro_engine_result": (_i32, [_vp, _i64, _vp, _i32, ctypes.POINTER(_i32)]),
    "metro_engine_get_stats": (_i32, [_vp, _vp]),
}
for _name, (_res, _args) in _SIGS.items():
    _f = getattr(lib, _name)
    _f.restype = _res
    _f.argtypes = _args

if lib.metro_abi_version() != ABI_VERSION:
    raise ImportError(f"libmetro.so ABI {lib.metro_abi_version()} != binding ABI {ABI_VERSION}")


class MetroError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status
        self.name = STATUS.get(status, str(status))


def check(status: int) -> None:
    if status != 0:
        raise MetroError(status, lib.metro_last_error().decode())


def _ptr(t) -> int | None:
    """Device address of a torch tensor (None passes NULL)."""
    if t is None:
        return None
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("expected a contiguous device tensor")
    return t.data_ptr()


def _stream(stream) -> int | None:
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def _host_i64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int64))


def _host_i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


class Model:
    """One Llama-style model on the current HIP device (see metro_create_model)."""

    def __init__(self, shape: dict, *, max_batch: int, max_tokens: int, max_context: int, max_seqs: int | None = None,
                 kv_pool_bytes: int = 0, seed: int = 0):
        self.shape = dict(shape)
        cfg = Config(n_layers=shape["n_layers"], d_model=shape["d_model"], n_heads=shape["n_heads"],
                     n_kv_heads=shape["n_kv_heads"], head_dim=shape["head_dim"], ffn_dim=shape["ffn_dim"],
                     vocab=shape["vocab"], rope_base=shape["rope_base"], rms_eps=shape["rms_eps"], page_size=16,
                     max_batch=max_batch, max_tokens=max_tokens, max_context=max_context,
                     max_seqs=max_seqs if max_seqs is not None else max(max_batch, 1),
                     kv_pool_bytes=kv_pool_bytes)
        h = _vp()
        check(lib.metro_create_model(ctypes.byref(cfg), seed, ctypes.byref(h)))
        self._h = h
        self.vocab = shape["vocab"]

    # -- lifetime --------------------------------------------------------------
    def close(self) -> None:
        if getattr(self, "_h", None) and self._h.value:
            lib.metro_destroy_model(self._h)
            self._h = _vp()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    # -- weights -----------------------------------------------------------------
    def load_weight(self, name: str, layer: int, bits: np.ndarray) -> None:
        a = np.ascontiguousarray(bits, dtype=np.uint16)
        check(lib.metro_load_weight(self._h, WEIGHT_ID[name], layer, a.ctypes.data, a.size))

    def load_weights(self, weights: dict) -> None:
        """Weights as produced by ``synth.llama_weights`` (bf16 bit arrays)."""
        for name in ("embed", "final_norm", "lm_head"):
            self.load_weight(name, -1, weights[name])
        for li, lw in enumerate(weights["layers"]):
            for name, arr in lw.items():
                self.load_weight(name, li, arr)

    def info(self) -> ModelInfo:
        inf = ModelInfo()
        check(lib.metro_model_get_info(self._h, ctypes.byref(inf)))
        return inf

    # -- sequences ---------------------------------------------------------------
    def seq_open(self) -> int:
        s = _i64()
        check(lib.metro_seq_open(self._h, ctypes.byref(s)))
        return s.value

    def seq_open_cached(self, tokens) -> tuple[int, int]:
        """Open a sequence for a prompt; returns (seq, n_cached): the leading
        tokens attached from the prefix cache, the rest to be prefilled."""
        t = _host_i32(tokens)
        s, n = _i64(), _i32()
        check(lib.metro_seq_open_cached(self._h, t.ctypes.data if t.size else None, t.size, ctypes.byref(s),
                                        ctypes.byref(n)))
        return s.value, n.value

    def prefix_cache(self, max_pages: int) -> None:
        check(lib.metro_prefix_cache(self._h, max_pages))

    def prefix_cache_stats(self) -> dict:
        st = PrefixCacheStats()
        check(lib.metro_prefix_cache_get_stats(self._h, ctypes.byref(st)))
        return {f: getattr(st, f) for f, _ in PrefixCacheStats._fields_}

    def seq_fork(self, src: int, n_tokens: int, stream=None) -> int:
        s = _i64()
        check(lib.metro_seq_fork(self._h, src, n_tokens, _stream(stream), ctypes.byref(s)))
        return s.value

    def seq_close(self, seq: int) -> None:
        check(lib.metro_seq_close(self._h, seq))

    def seq_length(self, seq: int) -> int:
        n = _i32()
        check(lib.metro_seq_length(self._h, seq, ctypes.byref(n)))
        return n.value

    def seq_pages(self, seq: int) -> np.ndarray:
        n = _i32()
        check(lib.metro_seq_pages(self._h, seq, None, 0, ctypes.byref(n)))
        out = np.zeros(n.value, dtype=np.int32)
        check(lib.metro_seq_pages(self._h, seq, out.ctypes.data, n.value, ctypes.byref(n)))
        return out

    # -- forward -----------------------------------------------------------------
    def prefill_chunk(self, seqs, chunks, logits=None, next_tok=None, stream=None) -> None:
        """Append ``chunks[i]`` (host token ids) to ``seqs[i]``; fills ``logits``
        (device fp32 [n, vocab]) and ``next_tok`` (device int32 [n]) if given."""
        s = _host_i64(seqs)
        lens = [len(c) for c in chunks]
        cu = _host_i32(np.concatenate([[0], np.cumsum(lens)]))
        toks = _host_i32(np.concatenate([np.asarray(c) for c in chunks]) if chunks else [])
        check(lib.metro_prefill_chunk(self._h, len(s), s.ctypes.data, cu.ctypes.data, toks.ctypes.data,
                                      _ptr(logits), _ptr(next_tok), _stream(stream)))

    def decode_step(self, seqs, tokens_dev, logits=None, next_tok=None, stream=None) -> None:
        """One token per sequence: ``tokens_dev`` is a device int32 [batch]
        (e.g. the previous step's ``next_tok``).  Host tokens (a list, numpy
        array or CPU tensor) are copied to the device first, on the call's
        stream; the library itself reads device memory only."""
        s = _host_i64(seqs)
        import torch
        if not (isinstance(tokens_dev, torch.Tensor) and tokens_dev.is_cuda):
            host = torch.as_tensor(np.ascontiguousarray(np.asarray(tokens_dev, dtype=np.int32)))
            st = (torch.cuda.current_stream() if stream is None
                  else torch.cuda.ExternalStream(stream) if isinstance(stream, int) else stream)
            with torch.cuda.stream(st):
                tokens_dev = host.to("cuda")
        check(lib.metro_decode_step(self._h, len(s), s.ctypes.data, _ptr(tokens_dev), _ptr(logits), _ptr(next_tok),
                                    _stream(stream)))

    # -- launch timing ------------------------------------------------------------
    def profile_start(self, kernel_class: str, phase: str = "any") -> None:
        check(lib.metro_profile_start(self._h, KERNEL_CLASS[kernel_class], PHASE[phase]))

    def profile_stop(self):
        """(total GPU ms between the bracketing events, number of launches)."""
        ms, n = ctypes.c_double(), _i64()
        check(lib.metro_profile_stop(self._h, ctypes.byref(ms), ctypes.byref(n)))
        return ms.value, n.value


# -- single-op entry points -------------------------------------------------------

def op_pack_weight(W, ld: int, N: int, K: int, Kp: int, out, stream=None):
    """Row-major bf16 W [N, ld] (first K columns) -> out, the [N, Kp] matrix in
    the matrix-core operand order op_gemm reads (columns K .. Kp-1 zero)."""
    check(lib.metro_op_pack_weight(_ptr(W), ld, N, K, Kp, _ptr(out), _stream(stream)))


def op_gemm(X, W, M: int, N: int, Kp: int, epilogue: int, out, ldo: int, ldx: int | None = None, workspace=None,
            stream=None):
    """W is packed (op_pack_weight)."""
    f32 = out if epilogue != EPI_SWIGLU else None
    b16 = out if epilogue == EPI_SWIGLU else None
    check(lib.metro_op_gemm(_ptr(X), ldx if ldx is not None else Kp, _ptr(W), Kp, M, N, epilogue, _ptr(f32),
                            _ptr(b16), ldo, _ptr(workspace), _stream(stream)))


GEMM_KINDS = ("decode", "tile128x128", "tile256x128", "tile256x256")


def op_gemm_plan(M: int, N: int, Kp: int, epilogue: int, workspace: bool = False):
    """(kernel kind name, k slices, tail split) that op_gemm would use; host only."""
    kind, ks, tail = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
    check(lib.metro_op_gemm_plan(M, N, Kp, epilogue, int(bool(workspace)), ctypes.byref(kind), ctypes.byref(ks),
                                 ctypes.byref(tail)))
    return GEMM_KINDS[kind.value], ks.value, tail.value


def op_rmsnorm(x, g, eps: float, h, rows: int, d: int, stream=None):
    check(lib.metro_op_rmsnorm(_ptr(x), _ptr(g), eps, _ptr(h), rows, d, _stream(stream)))


def op_argmax(logits, rows: int, vocab: int, out, stream=None):
    check(lib.metro_op_argmax(_ptr(logits), rows, vocab, _ptr(out), _stream(stream)))


def op_attn_decode(q, kv, n_pages: int, nq: int, nkv: int, hd: int, ctx, block_tables, out, stream=None):
    """Decode attention on caller buffers: q [rows, nq, hd] bf16, kv the page
    array, ctx and block_tables host ints (see metro_ops.h), out [rows, nq*hd]."""
    c = _host_i32(ctx)
    bt = _host_i32(block_tables)
    check(lib.metro_op_attn_decode(_ptr(q), _ptr(kv), n_pages, nq, nkv, hd, len(c), c.ctypes.data, bt.ctypes.data,
                                   _ptr(out), _stream(stream)))


def op_attn_decode_noalloc(q, kv, n_pages: int, nq: int, nkv: int, hd: int, ctx, block_tables, out, stream=None):
    """op_attn_decode without device allocation (the library's fixed scratch
    array; asynchronous on the stream)."""
    c = _host_i32(ctx)
    bt = _host_i32(block_tables)
    check(lib.metro_op_attn_decode_noalloc(_ptr(q), _ptr(kv), n_pages, nq, nkv, hd, len(c), c.ctypes.data,
                                           bt.ctypes.data, _ptr(out), _stream(stream)))


def op_attn_prefill(q, kv, n_pages: int, nq: int, nkv: int, hd: int, cu_q, ctx_before, block_tables, out,
                    stream=None):
    """Chunked-prefill attention on caller buffers (see metro_ops.h)."""
    cu = _host_i32(cu_q)
    cb = _host_i32(ctx_before)
    bt = _host_i32(block_tables)
    check(lib.metro_op_attn_prefill(_ptr(q), _ptr(kv), n_pages, nq, nkv, hd, len(cb), cu.ctypes.data,
                                    cb.ctypes.data, bt.ctypes.data, _ptr(out), _stream(stream)))


# ----------------------------------------------------------------------------
# Out-of-order agent scheduler (include/metro_sched.h); host only, no device
# ----------------------------------------------------------------------------

DIST_CHEBYSHEV, DIST_EUCLIDEAN = 0, 1


class SchedConfig(ctypes.Structure):
    _fields_ = [("n_agents", ctypes.c_int32), ("radius_p", ctypes.c_float), ("max_vel", ctypes.c_float),
                ("metric", ctypes.c_int32), ("target_step", ctypes.c_int32), ("sync", ctypes.c_int32)]


class Scheduler:
    """metro_sched_*: ``next()`` -> (cluster, step, members) or None;
    ``ack(cluster, positions)`` with each member's new (x, y)."""

    def __init__(self, positions, radius_p: float, max_vel: float, metric: int = DIST_CHEBYSHEV,
                 target_step: int = 10, sync: bool = False):
        self._h = ctypes.c_void_p()
        xy = np.ascontiguousarray(np.asarray(positions, dtype=np.int32).reshape(-1, 2))
        self.n = xy.shape[0]
        cfg = SchedConfig(self.n, radius_p, max_vel, metric, target_step, 1 if sync else 0)
        h = ctypes.c_void_p()
        check(lib.metro_sched_create(ctypes.byref(cfg), xy.ctypes.data, ctypes.byref(h)))
        self._h = h
        self._buf = np.zeros(self.n, dtype=np.int32)

    def close(self):
        if self._h and lib is not None:   # lib is gone during interpreter shutdown
            lib.metro_sched_destroy(self._h)
        self._h = ctypes.c_void_p()

    def __del__(self):
        self.close()

    def next(self, cap: int | None = None):
        cid, step, n = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        cap = self.n if cap is None else cap
        buf = self._buf if cap <= self.n else np.zeros(cap, dtype=np.int32)
        check(lib.metro_sched_next(self._h, ctypes.byref(cid), ctypes.byref(step), buf.ctypes.data, cap,
                                    ctypes.byref(n)))
        if n.value == 0:
            return None
        return cid.value, step.value, [int(a) for a in buf[:n.value]]

    def ack(self, cluster: int, positions):
        xy = np.ascontiguousarray(np.asarray(positions, dtype=np.int32).reshape(-1, 2))
        check(lib.metro_sched_ack(self._h, cluster, xy.ctypes.data))

    def state(self):
        steps = np.zeros(self.n, np.int32)
        xy = np.zeros((self.n, 2), np.int32)
        st = np.zeros(self.n, np.int32)
        running, done = ctypes.c_int32(), ctypes.c_int32()
        check(lib.metro_sched_state(self._h, steps.ctypes.data, xy.ctypes.data, st.ctypes.data,
                                     ctypes.byref(running), ctypes.byref(done)))
        return {"steps": steps, "xy": xy, "state": st, "running": running.value, "done": bool(done.value)}


# ----------------------------------------------------------------------------
# Mixed continuous batching engine (include/metro_sched.h)
# ----------------------------------------------------------------------------

class EngineConfig(ctypes.Structure):
    _fields_ = [("max_tokens", ctypes.c_int32), ("chunk", ctypes.c_int32), ("max_items", ctypes.c_int32),
                ("priority", ctypes.c_int32)]


class EngineStats(ctypes.Structure):
    _fields_ = [("forwards", ctypes.c_int64), ("items", ctypes.c_int64), ("prompt_tokens", ctypes.c_int64),
                ("decode_tokens", ctypes.c_int64), ("live", ctypes.c_int32), ("waiting", ctypes.c_int32),
                ("page_retries", ctypes.c_int64)]


class Engine:
    """metro_engine_*: requests in (``submit``), one forward per ``step()``,
    finished request ids from ``finished()``, their tokens from ``result()``.
    ``model`` None: planning only (no device work)."""

    def __init__(self, model, max_tokens: int, chunk: int, max_items: int, priority: bool = True):
        self._h = ctypes.c_void_p()
        self.max_items = max_items
        cfg = EngineConfig(max_tokens, chunk, max_items, 1 if priority else 0)
        h = ctypes.c_void_p()
        check(lib.metro_engine_create(model._h if model is not None else None, ctypes.byref(cfg), ctypes.byref(h)))
        self._h = h
        self._model = model

    def close(self):
        if self._h and lib is not None:
            lib.metro_engine_destroy(self._h)
        self._h = ctypes.c_void_p()

    def __del__(self):
        self.close()

    def submit(self, request: int, step: int, prompt, n_out: int) -> None:
        p = _host_i32(prompt)
        check(lib.metro_engine_submit(self._h, request, step, p.ctypes.data, len(p), n_out))

    def step(self, stream=None) -> int:
        n = ctypes.c_int32()
        s = _stream(stream) if self._model is not None else None
        check(lib.metro_engine_step(self._h, s, ctypes.byref(n)))
        return n.value

    def last_plan(self):
        """[(request, tokens, is_decode)] of the last step, in forward order."""
        cap = self.max_items
        ids = np.zeros(cap, np.int64)
        tok = np.zeros(cap, np.int32)
        dec = np.zeros(cap, np.int32)
        n = ctypes.c_int32()
        check(lib.metro_engine_last_plan(self._h, ids.ctypes.data, tok.ctypes.data, dec.ctypes.data, cap,
                                         ctypes.byref(n)))
        return [(int(ids[i]), int(tok[i]), bool(dec[i])) for i in range(n.value)]

    def finished(self):
        out = []
        buf = np.zeros(256, np.int64)
        while True:
            n = ctypes.c_int32()
            check(lib.metro_engine_finished(self._h, buf.ctypes.data, len(buf), ctypes.byref(n)))
            out += [int(x) for x in buf[:n.value]]
            if n.value < len(buf):
                return out

    def result(self, request: int):
        n = ctypes.c_int32()
        check(lib.metro_engine_result(self._h, request, None, 0, ctypes.byref(n)))
        buf = np.zeros(max(1, n.value), np.int32)
        check(lib.metro_engine_result(self._h, request, buf.ctypes.data, len(buf), ctypes.byref(n)))
        return buf[:n.value].copy()

    def stats(self) -> dict:
        st = EngineStats()
        check(lib.metro_engine_get_stats(self._h, ctypes.byref(st)))
        return {k: getattr(st, k) for k, _ in EngineStats._fields_}
