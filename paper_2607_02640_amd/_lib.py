"""ctypes binding of libmtn (include/mtn.h).

Argument marshalling only: every step of the attention path runs in the HIP
library.  Device buffers are passed as torch tensors (their data pointers) and
the stream as torch's current HIP stream.  Loading fails loudly when the
library has not been built; there is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
# MTN_LIB selects another build of the same library (e.g. a tuning variant)
LIB_PATH = os.environ.get("MTN_LIB") or os.path.join(_HERE, "libmtn.so")

MTN_OK = 0
MTN_ERR_INVALID_ARG = -1
MTN_ERR_BAD_SESSION = -2
MTN_ERR_CHUNK_TOO_LARGE = -3
MTN_ERR_NO_SESSION_SLOT = -4
MTN_ERR_POOL_EXHAUSTED = -5
MTN_ERR_SESSION_FULL = -6
MTN_ERR_DEVICE = -7
MTN_ERR_BAD_STATE = -8
MTN_ERR_UNSUPPORTED = -9
MTN_ERR_HOST_MEMORY = -10

MTN_F32 = 0
MTN_BF16 = 1
MTN_FP8_E4M3 = 2
# pool dtype name -> (kv_dtype, io_dtype); "fp8" keeps E4M3 codes with bf16 io
DTYPES = {"f32": (MTN_F32, MTN_F32), "bf16": (MTN_BF16, MTN_BF16),
          "fp8": (MTN_FP8_E4M3, MTN_BF16)}
MTN_WINDOW_UNBOUNDED = -1
MTN_POOL_HOST_ONLY = 1

# every symbol include/mtn.h declares
EXPORTS = [
    "mtn_pool_required_bytes", "mtn_pool_create", "mtn_pool_destroy",
    "mtn_session_open", "mtn_session_close", "mtn_plan_begin", "mtn_plan_commit",
    "mtn_plan_abort",
    "mtn_frame_append_kv", "mtn_attend_chunk_prefill", "mtn_attend_decode",
    "mtn_attend_decode_append", "mtn_attend_decode_noalloc",
    "mtn_frame_step", "mtn_pool_stats", "mtn_session_info", "mtn_session_block_table",
    "mtn_plan_info", "mtn_debug_poison_dead", "mtn_pool_set_timing", "mtn_pool_set_prefill_pass_rows",
    "mtn_pool_kernel_times", "mtn_hbm_copy", "mtn_hbm_read", "mtn_status_string", "mtn_pool_last_error",
    "mtn_pool_set_decode_kernel", "mtn_pool_last_split", "mtn_debug_inject_failure",
    "mtn_admission_create", "mtn_admission_destroy", "mtn_admission_offer",
    "mtn_admission_release", "mtn_admission_observe", "mtn_admission_get",
]


class PoolConfig(C.Structure):
    _fields_ = [
        ("n_layers", C.c_int32), ("n_q_heads", C.c_int32), ("n_kv_heads", C.c_int32),
        ("head_dim", C.c_int32), ("block_size", C.c_int32), ("n_sink", C.c_int32),
        ("window", C.c_int32), ("max_chunk", C.c_int32), ("max_sessions", C.c_int32),
        ("max_len", C.c_int32), ("n_blocks", C.c_int64), ("kv_dtype", C.c_int32),
        ("io_dtype", C.c_int32), ("rope_theta", C.c_double), ("softmax_scale", C.c_float),
        ("flags", C.c_uint32),
    ]


class PoolStats(C.Structure):
    _fields_ = [
        ("capacity", C.c_int64), ("assigned", C.c_int64), ("reserved", C.c_int64),
        ("open_sessions", C.c_int32), ("blocks_per_session", C.c_int32),
        ("ring_tokens", C.c_int32), ("sink_blocks", C.c_int32),
    ]


class AdmissionConfig(C.Structure):
    _fields_ = [
        ("target_ms", C.c_double), ("backoff", C.c_double), ("increase", C.c_int32),
        ("initial_cap", C.c_int32), ("min_cap", C.c_int32), ("max_cap", C.c_int32),
        ("hold_ticks", C.c_int32),
    ]


class AdmissionState(C.Structure):
    _fields_ = [
        ("cap", C.c_int32), ("admitted", C.c_int32), ("hold", C.c_int32),
        ("offered", C.c_int64), ("rejected", C.c_int64), ("ticks", C.c_int64),
        ("decreases", C.c_int64), ("increases", C.c_int64),
    ]


class FrameBatch(C.Structure):
    _fields_ = [
        ("n_seq", C.c_int32),
        ("sids", C.POINTER(C.c_int32)), ("chunk_len", C.POINTER(C.c_int32)),
        ("n_decode", C.POINTER(C.c_int32)),
        ("q_chunk", C.c_void_p), ("k_chunk", C.c_void_p), ("v_chunk", C.c_void_p),
        ("out_chunk", C.c_void_p), ("lse_chunk", C.c_void_p),
        ("q_dec", C.c_void_p), ("k_dec", C.c_void_p), ("v_dec", C.c_void_p),
        ("out_dec", C.c_void_p), ("lse_dec", C.c_void_p),
        ("n_split", C.c_int32),
    ]


_lib = None


def load() -> C.CDLL:
    """Load libmtn.so (built by paper_2607_02640_amd.build); raise if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is missing: build it with paper_2607_02640_amd.build.build() "
            "(the attention path has no non-HIP fallback)")
    lib = C.CDLL(LIB_PATH)
    i32, i64, vp = C.c_int32, C.c_int64, C.c_void_p
    P32, P64 = C.POINTER(C.c_int32), C.POINTER(C.c_int64)
    sig = {
        "mtn_pool_required_bytes": (i32, [C.POINTER(PoolConfig), C.POINTER(C.c_size_t)]),
        "mtn_pool_create": (i32, [C.POINTER(PoolConfig), vp, C.c_size_t, vp, C.POINTER(vp)]),
        "mtn_pool_destroy": (None, [vp]),
        "mtn_session_open": (i32, [vp, P32]),
        "mtn_session_close": (i32, [vp, i32]),
        "mtn_plan_begin": (i32, [vp, i32, P32, P32, vp]),
        "mtn_plan_commit": (i32, [vp]),
        "mtn_plan_abort": (i32, [vp]),
        "mtn_pool_set_decode_kernel": (i32, [vp, i32]),
        "mtn_pool_last_split": (i32, [vp, P32]),
        "mtn_debug_inject_failure": (i32, [vp, i64]),
        "mtn_frame_append_kv": (i32, [vp, i32, vp, vp, vp]),
        "mtn_attend_chunk_prefill": (i32, [vp, i32, vp, vp, vp, vp]),
        "mtn_attend_decode": (i32, [vp, i32, vp, vp, vp, i32, vp]),
        "mtn_attend_decode_append": (i32, [vp, i32, vp, vp, vp, vp, vp, i32, vp]),
        "mtn_attend_decode_noalloc": (i32, [vp, i32, vp, vp, vp, i32, vp]),
        "mtn_frame_step": (i32, [vp, C.POINTER(FrameBatch), vp]),
        "mtn_pool_stats": (i32, [vp, C.POINTER(PoolStats)]),
        "mtn_session_info": (i32, [vp, i32, P64, P32]),
        "mtn_session_block_table": (i32, [vp, i32, P32, i32, P32]),
        "mtn_plan_info": (i32, [vp, P64, P32, P32, i32, P64, P64, P32]),
        "mtn_debug_poison_dead": (i32, [vp, vp]),
        "mtn_pool_set_timing": (i32, [vp, i32]),
        "mtn_pool_set_prefill_pass_rows": (i32, [vp, i32]),
        "mtn_pool_kernel_times": (i32, [vp, P64, C.POINTER(C.c_double)]),
        "mtn_hbm_copy": (i32, [vp, vp, C.c_size_t, vp]),
        "mtn_hbm_read": (i32, [vp, C.c_size_t, vp]),
        "mtn_admission_create": (i32, [C.POINTER(AdmissionConfig), C.POINTER(vp)]),
        "mtn_admission_destroy": (None, [vp]),
        "mtn_admission_offer": (i32, [vp, P32]),
        "mtn_admission_release": (i32, [vp]),
        "mtn_admission_observe": (i32, [vp, C.c_double]),
        "mtn_admission_get": (i32, [vp, C.POINTER(AdmissionState)]),
        "mtn_status_string": (C.c_char_p, [i32]),
        "mtn_pool_last_error": (C.c_char_p, [vp]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


class MtnError(RuntimeError):
    def __init__(self, code: int, where: str, detail: str = ""):
        lib = load()
        super().__init__(f"{where}: {lib.mtn_status_string(code).decode()} ({code})"
                         + (f": {detail}" if detail else ""))
        self.code = code


def _arr32(xs: Sequence[int]):
    return (C.c_int32 * len(xs))(*[int(x) for x in xs])


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is not None:
        return stream
    import torch
    if torch.cuda.is_available():
        return torch.cuda.current_stream().cuda_stream
    return None


class Pool:
    """A KV pool (mtn_pool) with the C ABI's calls as methods.

    ``kv`` is a caller-owned device tensor of at least ``required_bytes``;
    pass ``host_only=True`` to exercise planning without a device.
    """

    def __init__(self, *, n_layers, n_q_heads, n_kv_heads, head_dim, n_sink, window,
                 max_chunk, max_sessions, n_blocks, dtype="bf16", max_len=0,
                 rope_theta=10000.0, softmax_scale=0.0, block_size=16, host_only=False,
                 kv=None, stream=None):
        self.lib = load()
        kvt, iot = DTYPES[dtype]
        self.cfg = PoolConfig(
            n_layers, n_q_heads, n_kv_heads, head_dim, block_size, n_sink,
            MTN_WINDOW_UNBOUNDED if window is None else window, max_chunk, max_sessions,
            max_len, n_blocks, kvt, iot, rope_theta, softmax_scale,
            MTN_POOL_HOST_ONLY if host_only else 0)
        self.dtype = dtype
        self.host_only = host_only
        nbytes = C.c_size_t()
        self._check(self.lib.mtn_pool_required_bytes(C.byref(self.cfg), C.byref(nbytes)),
                    "required_bytes")
        self.required_bytes = nbytes.value
        self.kv = kv
        h = C.c_void_p()
        st = self.lib.mtn_pool_create(C.byref(self.cfg), _ptr(kv) if kv is not None else None,
                                      C.c_size_t(kv.numel() * kv.element_size() if kv is not None else 0),
                                      None if host_only else _stream(stream), C.byref(h))
        self._check(st, "pool_create")
        self.h = h

    @staticmethod
    def required(**kw) -> int:
        lib = load()
        kvt, iot = DTYPES[kw.get("dtype", "bf16")]
        w = kw["window"]
        cfg = PoolConfig(kw["n_layers"], kw["n_q_heads"], kw["n_kv_heads"], kw["head_dim"],
                         kw.get("block_size", 16), kw["n_sink"],
                         MTN_WINDOW_UNBOUNDED if w is None else w, kw["max_chunk"],
                         kw["max_sessions"], kw.get("max_len", 0), kw["n_blocks"], kvt, iot,
                         kw.get("rope_theta", 1e4), 0.0, 0)
        n = C.c_size_t()
        st = lib.mtn_pool_required_bytes(C.byref(cfg), C.byref(n))
        if st:
            raise MtnError(st, "required_bytes")
        return n.value

    # -- helpers -------------------------------------------------------------
    def _check(self, st, where):
        if st != MTN_OK:
            detail = ""
            if getattr(self, "h", None) is not None:
                detail = (self.lib.mtn_pool_last_error(self.h) or b"").decode()
            raise MtnError(st, where, detail)

    def close(self):
        if getattr(self, "h", None) is not None and self.h.value:
            self.lib.mtn_pool_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- C ABI ---------------------------------------------------------------
    def session_open(self) -> int:
        sid = C.c_int32()
        self._check(self.lib.mtn_session_open(self.h, C.byref(sid)), "session_open")
        return sid.value

    def session_close(self, sid: int) -> None:
        self._check(self.lib.mtn_session_close(self.h, sid), "session_close")

    def plan_begin(self, sids, n_tok, stream=None) -> None:
        st = self.lib.mtn_plan_begin(self.h, len(sids), _arr32(sids), _arr32(n_tok),
                                     None if self.host_only else _stream(stream))
        self._check(st, "plan_begin")

    def plan_commit(self) -> None:
        self._check(self.lib.mtn_plan_commit(self.h), "plan_commit")

    def plan_abort(self) -> None:
        self._check(self.lib.mtn_plan_abort(self.h), "plan_abort")

    def set_decode_kernel(self, kind: int) -> None:
        """0 = by shape, 1 = vector kernel, 2 = matrix-core kernel."""
        self._check(self.lib.mtn_pool_set_decode_kernel(self.h, kind), "set_decode_kernel")

    def last_split(self) -> int:
        n = C.c_int32()
        self._check(self.lib.mtn_pool_last_split(self.h, C.byref(n)), "last_split")
        return n.value

    def inject_failure(self, launch_index: int) -> None:
        self._check(self.lib.mtn_debug_inject_failure(self.h, launch_index), "inject_failure")

    def frame_append_kv(self, layer, k, v, stream=None) -> None:
        self._check(self.lib.mtn_frame_append_kv(self.h, layer, _ptr(k), _ptr(v), _stream(stream)),
                    "frame_append_kv")

    def attend_chunk_prefill(self, layer, q, out, lse=None, stream=None) -> None:
        self._check(self.lib.mtn_attend_chunk_prefill(self.h, layer, _ptr(q), _ptr(out), _ptr(lse),
                                                      _stream(stream)), "attend_chunk_prefill")

    def attend_decode(self, layer, q, out, lse=None, n_split=0, stream=None) -> None:
        self._check(self.lib.mtn_attend_decode(self.h, layer, _ptr(q), _ptr(out), _ptr(lse),
                                               n_split, _stream(stream)), "attend_decode")

    def attend_decode_noalloc(self, layer, q, out, lse=None, n_split=0, stream=None) -> None:
        self._check(self.lib.mtn_attend_decode_noalloc(self.h, layer, _ptr(q), _ptr(out),
                                                       _ptr(lse), n_split, _stream(stream)),
                    "attend_decode_noalloc")

    def attend_decode_append(self, layer, k, v, q, out, lse=None, n_split=0,
                             stream=None) -> None:
        self._check(self.lib.mtn_attend_decode_append(self.h, layer, _ptr(k), _ptr(v), _ptr(q),
                                                      _ptr(out), _ptr(lse), n_split,
                                                      _stream(stream)), "attend_decode_append")

    def frame_step(self, sids, chunk_len, n_decode, q_chunk, k_chunk, v_chunk, out_chunk,
                   q_dec=None, k_dec=None, v_dec=None, out_dec=None, lse_chunk=None,
                   lse_dec=None, n_split=0, stream=None) -> None:
        b = FrameBatch()
        b.n_seq = len(sids)
        self._keep = (_arr32(sids), _arr32(chunk_len), _arr32(n_decode))
        b.sids, b.chunk_len, b.n_decode = (C.cast(a, C.POINTER(C.c_int32)) for a in self._keep)
        b.q_chunk, b.k_chunk, b.v_chunk = _ptr(q_chunk), _ptr(k_chunk), _ptr(v_chunk)
        b.out_chunk, b.lse_chunk = _ptr(out_chunk), _ptr(lse_chunk)
        b.q_dec, b.k_dec, b.v_dec = _ptr(q_dec), _ptr(k_dec), _ptr(v_dec)
        b.out_dec, b.lse_dec = _ptr(out_dec), _ptr(lse_dec)
        b.n_split = n_split
        self._check(self.lib.mtn_frame_step(self.h, C.byref(b),
                                            None if self.host_only else _stream(stream)),
                    "frame_step")

    def stats(self) -> dict:
        s = PoolStats()
        self._check(self.lib.mtn_pool_stats(self.h, C.byref(s)), "pool_stats")
        return {k: getattr(s, k) for k, _ in PoolStats._fields_}

    def session_info(self, sid):
        ln, na = C.c_int64(), C.c_int32()
        self._check(self.lib.mtn_session_info(self.h, sid, C.byref(ln), C.byref(na)), "session_info")
        return ln.value, na.value

    def block_table(self, sid):
        n = self.stats()["blocks_per_session"]
        buf = (C.c_int32 * n)()
        cnt = C.c_int32()
        self._check(self.lib.mtn_session_block_table(self.h, sid, buf, n, C.byref(cnt)),
                    "session_block_table")
        return list(buf[:cnt.value])

    def plan_info(self, n_seq: int, cap: int = 1 << 16):
        pos = (C.c_int64 * cap)()
        blk = (C.c_int32 * cap)()
        off = (C.c_int32 * cap)()
        lo = (C.c_int64 * cap)()
        hi = (C.c_int64 * cap)()
        n = C.c_int32()
        self._check(self.lib.mtn_plan_info(self.h, pos, blk, off, cap, lo, hi, C.byref(n)),
                    "plan_info")
        return (list(pos[:n.value]), list(blk[:n.value]), list(off[:n.value]),
                list(lo[:n_seq]), list(hi[:n_seq]))

    def poison_dead(self, stream=None) -> None:
        self._check(self.lib.mtn_debug_poison_dead(self.h, _stream(stream)), "debug_poison_dead")

    def set_prefill_pass_rows(self, rows: int) -> None:
        """Query rows per chunk-prefill pass: 0 = per plan, or 128 / 256."""
        self._check(self.lib.mtn_pool_set_prefill_pass_rows(self.h, rows), "set_prefill_pass_rows")

    def set_timing(self, on: bool) -> None:
        self._check(self.lib.mtn_pool_set_timing(self.h, 1 if on else 0), "set_timing")

    def kernel_times(self):
        n = (C.c_int64 * 4)()
        ms = (C.c_double * 4)()
        self._check(self.lib.mtn_pool_kernel_times(self.h, n, ms), "kernel_times")
        names = ("append", "prefill", "decode", "merge")
        return {names[i]: (n[i], ms[i]) for i in range(4)}


def hbm_copy(src, dst, nbytes: int, stream=None) -> None:
    lib = load()
    st = lib.mtn_hbm_copy(_ptr(src), _ptr(dst), C.c_size_t(nbytes), _stream(stream))
    if st != MTN_OK:
        raise MtnError(st, "hbm_copy")


def hbm_read(src, nbytes: int, stream=None) -> None:
    lib = load()
    st = lib.mtn_hbm_read(_ptr(src), C.c_size_t(nbytes), _stream(stream))
    if st != MTN_OK:
        raise MtnError(st, "hbm_read")


class Admission:
    """AIMD admission controller on the per-frame latency (host only; see
    mtn_admission_* in include/mtn.h)."""

    def __init__(self, *, target_ms, backoff, increase, initial_cap, min_cap, max_cap,
                 hold_ticks):
        self._lib = load()
        cfg = AdmissionConfig(float(target_ms), float(backoff), int(increase), int(initial_cap),
                              int(min_cap), int(max_cap), int(hold_ticks))
        h = C.c_void_p()
        st = self._lib.mtn_admission_create(C.byref(cfg), C.byref(h))
        if st != MTN_OK:
            raise MtnError(st, "mtn_admission_create")
        self._h = h

    def close(self):
        if getattr(self, "_h", None):
            self._lib.mtn_admission_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def offer(self) -> bool:
        out = C.c_int32()
        st = self._lib.mtn_admission_offer(self._h, C.byref(out))
        if st != MTN_OK:
            raise MtnError(st, "mtn_admission_offer")
        return bool(out.value)

    def release(self) -> None:
        st = self._lib.mtn_admission_release(self._h)
        if st != MTN_OK:
            raise MtnError(st, "mtn_admission_release")

    def observe(self, tick_ms: float) -> None:
        st = self._lib.mtn_admission_observe(self._h, C.c_double(tick_ms))
        if st != MTN_OK:
            raise MtnError(st, "mtn_admission_observe")

    def state(self) -> dict:
        s = AdmissionState()
        st = self._lib.mtn_admission_get(self._h, C.byref(s))
        if st != MTN_OK:
            raise MtnError(st, "mtn_admission_get")
        return {k: getattr(s, k) for k, _ in AdmissionState._fields_}
