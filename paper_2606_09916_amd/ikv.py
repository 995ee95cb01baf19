"""Python binding of libikv.so (include/ikv.h): argument marshalling only.

Every function here hands raw device pointers of torch tensors to the C ABI and
raises IkvError on a non-zero status. All arithmetic runs in the HIP kernels; if
the library is not built, loading it raises instead of falling back to anything.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import c_float, c_int32, c_int64, c_size_t, c_uint32, c_void_p

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libikv.so")

IKV_BF16, IKV_F32 = 0, 1
IKV_RESIDUAL, IKV_NO_XATTN, IKV_POOL7, IKV_TWO_PASS = 1, 2, 4, 8
CALL_SCORE, CALL_SELECT, CALL_REDIRECT, CALL_DECODE, CALL_COMPACT, CALL_PREFILL = 1, 2, 3, 4, 5, 6
STATUS = {0: "IKV_OK", -1: "IKV_EINVAL", -2: "IKV_ESHAPE", -3: "IKV_EWORKSPACE", -4: "IKV_EUNSUPPORTED",
          -5: "IKV_EHIP"}

# Every symbol include/ikv.h declares.
SYMBOLS = ("ikv_init_dead_slot", "ikv_qm_update", "ikv_score_history", "ikv_select_budget", "ikv_select_budget_static",
           "ikv_redirect_slots", "ikv_decode_attend_slotmap", "ikv_workspace_bytes", "ikv_last_error",
           "ikv_timing", "ikv_timing_read", "ikv_memstore_create", "ikv_memstore_destroy", "ikv_memstore_acquire",
           "ikv_memstore_release", "ikv_memstore_trigger", "ikv_memstore_size", "ikv_resolve_span",
           "ikv_compact_apply", "ikv_prefill_span")
IKV_KEY_EXPLICIT, IKV_KEY_SPAN, IKV_KEY_PREFIX, IKV_KEY_LOCAL = 1, 2, 3, 4


class IkvError(RuntimeError):
    def __init__(self, status: int, func: str, msg: str):
        super().__init__(f"{func}: {STATUS.get(status, status)}: {msg}")
        self.status = status


class Pool(ctypes.Structure):
    _fields_ = [("L", c_int32), ("Hq", c_int32), ("Hkv", c_int32), ("D", c_int32),
                ("num_slots", c_int64), ("dead_slot", c_int32), ("kv_dtype", c_int32),
                ("k_pool", c_void_p), ("v_pool", c_void_p)]


class Session(ctypes.Structure):
    _fields_ = [("slot_off", c_int64), ("mem_off", c_int64), ("qspan_off", c_int64), ("qpos_off", c_int64),
                ("N", c_int32), ("pi", c_int32), ("qs", c_int32), ("qe", c_int32), ("C", c_int32),
                ("radix_prefix", c_int32), ("R", c_int32), ("nq", c_int32)]


class KeySource(ctypes.Structure):
    _fields_ = [("session_id", ctypes.c_char_p), ("session_id_len", c_int32), ("n_tokens", c_int32),
                ("tokens", c_void_p), ("span_start", c_int32), ("span_end", c_int32)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libikv.so once; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_09916_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, S = ctypes.POINTER(Pool), ctypes.POINTER(Session)
        sig = {
            "ikv_init_dead_slot": [P, c_void_p],
            "ikv_qm_update": [P, S, c_void_p, c_int32, c_void_p, c_void_p, c_float, c_void_p],
            "ikv_score_history": [P, S, c_void_p, c_int32, c_void_p, c_void_p, c_void_p, c_void_p, c_uint32,
                                  c_void_p, c_void_p, c_size_t, c_void_p],
            "ikv_select_budget": [S, c_void_p, c_int32, c_void_p, c_int32, c_void_p, c_void_p, c_void_p, c_void_p,
                                  c_void_p, c_size_t, c_void_p],
            "ikv_select_budget_static": [S, c_void_p, c_int32, c_void_p, c_int32, c_void_p, c_void_p, c_void_p,
                                         c_void_p, c_void_p],
            "ikv_redirect_slots": [S, c_void_p, c_int32, c_int64, c_void_p, c_int32, c_void_p, c_void_p, c_void_p,
                                   c_void_p, c_void_p, c_void_p, c_size_t, c_void_p],
            "ikv_decode_attend_slotmap": [P, S, c_void_p, c_int32, c_void_p, c_void_p, c_void_p, c_void_p,
                                          c_void_p, c_size_t, c_void_p],
            "ikv_workspace_bytes": [P, S, c_int32, c_int32, c_uint32, ctypes.POINTER(c_size_t)],
            "ikv_compact_apply": [P, S, c_void_p, c_int32, c_void_p, c_void_p, c_void_p, ctypes.c_double, c_void_p,
                                  c_void_p, c_size_t, c_void_p],
            "ikv_prefill_span": [P, S, c_void_p, c_int32, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                 ctypes.c_double, c_float, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_size_t,
                                 c_void_p],
            "ikv_timing": [c_int32],
            "ikv_memstore_create": [c_int32, ctypes.POINTER(c_void_p)],
            "ikv_memstore_acquire": [c_void_p, ctypes.POINTER(KeySource), ctypes.POINTER(c_int32),
                                     ctypes.POINTER(c_int32), ctypes.POINTER(c_int32)],
            "ikv_memstore_release": [c_void_p, c_int32],
            "ikv_memstore_trigger": [c_void_p, c_int32, c_int32, c_int32, c_int32, ctypes.POINTER(c_int32)],
            "ikv_memstore_size": [c_void_p, ctypes.POINTER(c_int32)],
            "ikv_resolve_span": [c_int32, c_void_p, c_void_p, c_void_p, c_int32, c_int32, ctypes.POINTER(c_int32),
                                 ctypes.POINTER(c_int32)],
            "ikv_timing_read": [ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(c_float), c_int32],
        }
        for name, args in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = c_int32
        L.ikv_memstore_destroy.argtypes = [c_void_p]
        L.ikv_memstore_destroy.restype = None
        L.ikv_last_error.argtypes = []
        L.ikv_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _check(status: int, func: str) -> None:
    if status != 0:
        raise IkvError(status, func, lib().ikv_last_error().decode())


def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


def _stream(stream) -> int | None:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


# ----------------------------------------------------------------------------- descriptors

def make_pool(k_pool, v_pool, L, Hq, Hkv, D, num_slots, dead_slot=0) -> Pool:
    """Pool descriptor over two device tensors [L][num_slots][Hkv][D] (bfloat16 or float32)."""
    import torch
    dt = {torch.bfloat16: IKV_BF16, torch.float32: IKV_F32}[k_pool.dtype]
    return Pool(L, Hq, Hkv, D, num_slots, dead_slot, dt, k_pool.data_ptr(), v_pool.data_ptr())


class Sessions:
    """Host array of session descriptors plus its device copy (same bytes)."""

    def __init__(self, rows, device):
        import torch
        self.B = len(rows)
        self.host = (Session * max(1, self.B))()
        for i, r in enumerate(rows):
            for k, v in r.items():
                setattr(self.host[i], k, int(v))
        raw = bytes(memoryview(self.host).cast("B"))[: self.B * ctypes.sizeof(Session)]
        self.dev = torch.frombuffer(bytearray(raw or b"\0"), dtype=torch.uint8).to(device)

    @property
    def host_ptr(self):
        return ctypes.cast(self.host, ctypes.POINTER(Session))

    @property
    def dev_ptr(self) -> int:
        return self.dev.data_ptr()

    def __getitem__(self, i) -> Session:
        return self.host[i]


class Workspace:
    """Reusable device scratch, grown on demand and kept 256-byte aligned."""

    def __init__(self, device):
        self.device = device
        self.buf = None
        self.nbytes = 0

    def get(self, nbytes: int):
        import torch
        if nbytes == 0:
            return None, 0
        if self.buf is None or self.nbytes < nbytes:
            self.buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
            self.nbytes = nbytes
        p = self.buf.data_ptr()
        return (p + 255) & ~255, nbytes


def workspace_bytes(pool: Pool | None, sess: Sessions, call: int, flags: int = 0) -> int:
    n = c_size_t(0)
    _check(lib().ikv_workspace_bytes(ctypes.byref(pool) if pool is not None else None, sess.host_ptr, sess.B,
                                     call, flags, ctypes.byref(n)), "ikv_workspace_bytes")
    return n.value


# ----------------------------------------------------------------------------- calls

def init_dead_slot(pool: Pool, stream=None) -> None:
    _check(lib().ikv_init_dead_slot(ctypes.byref(pool), _stream(stream)), "ikv_init_dead_slot")


def qm_update(pool: Pool, sess: Sessions, M, q_span, lam: float = 0.5, stream=None) -> None:
    _check(lib().ikv_qm_update(ctypes.byref(pool), sess.host_ptr, sess.dev_ptr, sess.B, _ptr(M), _ptr(q_span),
                               float(lam), _stream(stream)), "ikv_qm_update")


def score_history(pool: Pool, sess: Sessions, slot_maps, M, scores, ws: Workspace, qpos=None, residual=None,
                  flags: int = 0, stream=None) -> None:
    wp, wn = ws.get(workspace_bytes(pool, sess, CALL_SCORE, flags))
    _check(lib().ikv_score_history(ctypes.byref(pool), sess.host_ptr, sess.dev_ptr, sess.B, _ptr(slot_maps),
                                   _ptr(M), _ptr(qpos), _ptr(residual), flags, _ptr(scores), wp, wn,
                                   _stream(stream)), "ikv_score_history")


def select_budget(sess: Sessions, slot_maps, dead_slot: int, scores, keep, n_keep, tau, ws: Workspace,
                  stream=None) -> None:
    wp, wn = ws.get(workspace_bytes(None, sess, CALL_SELECT))
    _check(lib().ikv_select_budget(sess.host_ptr, sess.dev_ptr, sess.B, _ptr(slot_maps), dead_slot, _ptr(scores),
                                   _ptr(keep), _ptr(n_keep), _ptr(tau), wp, wn, _stream(stream)),
           "ikv_select_budget")


def select_budget_static(sess: Sessions, slot_maps, dead_slot: int, scores, keep, n_keep, tau, stream=None) -> None:
    """ikv_select_budget on the library's static scratch: no workspace, nothing allocated."""
    _check(lib().ikv_select_budget_static(sess.host_ptr, sess.dev_ptr, sess.B, _ptr(slot_maps), dead_slot,
                                          _ptr(scores), _ptr(keep), _ptr(n_keep), _ptr(tau), _stream(stream)),
           "ikv_select_budget_static")


def redirect_slots(sess: Sessions, num_slots: int, slot_maps, dead_slot: int, keep, freed, n_freed, live, n_live,
                   ws: Workspace, stream=None) -> None:
    pool = Pool()
    pool.num_slots = num_slots
    wp, wn = ws.get(workspace_bytes(pool, sess, CALL_REDIRECT))
    _check(lib().ikv_redirect_slots(sess.host_ptr, sess.dev_ptr, sess.B, num_slots, _ptr(slot_maps), dead_slot,
                                    _ptr(keep), _ptr(freed), _ptr(n_freed), _ptr(live), _ptr(n_live), wp, wn,
                                    _stream(stream)), "ikv_redirect_slots")


def decode_attend_slotmap(pool: Pool, sess: Sessions, q, live, n_live, out, ws: Workspace, stream=None) -> None:
    wp, wn = ws.get(workspace_bytes(pool, sess, CALL_DECODE))
    _check(lib().ikv_decode_attend_slotmap(ctypes.byref(pool), sess.host_ptr, sess.dev_ptr, sess.B, _ptr(q),
                                           _ptr(live), _ptr(n_live), _ptr(out), wp, wn, _stream(stream)),
           "ikv_decode_attend_slotmap")


def compact_apply(pool: Pool, sess: Sessions, slot_maps, keep, dst_slots, n_keep, ws: Workspace,
                  rope_base: float = 1.0e6, stream=None) -> None:
    """Left-pack the kept rows into dst_slots with RoPE re-rotation (the compact layout)."""
    wp, wn = ws.get(workspace_bytes(pool, sess, CALL_COMPACT))
    _check(lib().ikv_compact_apply(ctypes.byref(pool), sess.host_ptr, sess.dev_ptr, sess.B, _ptr(slot_maps),
                                   _ptr(keep), _ptr(dst_slots), float(rope_base), _ptr(n_keep), wp, wn,
                                   _stream(stream)), "ikv_compact_apply")


def prefill_span(pool: Pool, sess: Sessions, slot_maps, q_raw, k_raw, v_raw, hist, n_hist, q_out, out, kq,
                 ws: Workspace, M=None, lam: float = 0.5, rope_base: float = 1.0e6, stream=None) -> None:
    """RoPE, pool write, causal span attention, Enc and memory update, and key means of the span."""
    wp, wn = ws.get(workspace_bytes(pool, sess, CALL_PREFILL))
    _check(lib().ikv_prefill_span(ctypes.byref(pool), sess.host_ptr, sess.dev_ptr, sess.B, _ptr(slot_maps),
                                  _ptr(q_raw), _ptr(k_raw), _ptr(v_raw), _ptr(hist), _ptr(n_hist), float(rope_base),
                                  float(lam), _ptr(M), _ptr(q_out), _ptr(out), _ptr(kq), wp, wn, _stream(stream)),
           "ikv_prefill_span")


# ----------------------------------------------------------------------------- timing

def timing(enable: bool) -> None:
    """Record (or stop recording) a HIP event pair around every kernel the calls launch."""
    _check(lib().ikv_timing(1 if enable else 0), "ikv_timing")


def timing_read(cap: int = 65536) -> list[tuple[str, float]]:
    """Wait for the recorded kernels and return [(kernel name, ms)] in launch order."""
    names = (ctypes.c_char_p * max(1, cap))()
    ms = (c_float * max(1, cap))()
    n = lib().ikv_timing_read(names, ms, cap)
    if n < 0:
        _check(n, "ikv_timing_read")
    return [(names[i].decode(), float(ms[i])) for i in range(min(n, cap))]


# ----------------------------------------------------------------------------- session management (host)

class MemStore:
    """The QueryMemory store of one compressor (ikv_memstore_*): session keys to rows of a
    caller-owned device arena, least recently used rows reused first."""

    def __init__(self, capacity: int = 1024):
        h = c_void_p()
        _check(lib().ikv_memstore_create(capacity, ctypes.byref(h)), "ikv_memstore_create")
        self._h = h
        self.capacity = capacity

    def close(self) -> None:
        if self._h:
            lib().ikv_memstore_destroy(self._h)
            self._h = c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def acquire(self, session_id: bytes | None = None, tokens=None, span: tuple[int, int] | None = None):
        """(slot, fresh, kind) of the session the sources identify."""
        import numpy as np
        src = KeySource()
        keep = []
        if session_id:
            src.session_id = session_id
            src.session_id_len = len(session_id)
        if tokens is not None and len(tokens):
            t = np.ascontiguousarray(tokens, dtype=np.int32)
            keep.append(t)
            src.tokens = t.ctypes.data
            src.n_tokens = len(t)
            if span is not None:
                src.span_start, src.span_end = int(span[0]), int(span[1])
        slot, fresh, kind = c_int32(), c_int32(), c_int32()
        _check(lib().ikv_memstore_acquire(self._h, ctypes.byref(src), ctypes.byref(slot), ctypes.byref(fresh),
                                          ctypes.byref(kind)), "ikv_memstore_acquire")
        return slot.value, bool(fresh.value), kind.value

    def release(self, slot: int) -> None:
        _check(lib().ikv_memstore_release(self._h, slot), "ikv_memstore_release")

    def trigger(self, slot: int, N: int, C: int, trigger: int = 512) -> bool:
        fire = c_int32()
        _check(lib().ikv_memstore_trigger(self._h, slot, N, C, trigger, ctypes.byref(fire)), "ikv_memstore_trigger")
        return bool(fire.value)

    def __len__(self) -> int:
        n = c_int32()
        _check(lib().ikv_memstore_size(self._h, ctypes.byref(n)), "ikv_memstore_size")
        return n.value


def resolve_span(N: int, messages, tail_w: int = 32) -> tuple[int, int]:
    """[qs, qe) from the rendered messages [(start, end, actionable)], or the tail fallback."""
    import numpy as np
    m = list(messages)
    st = np.ascontiguousarray([a for a, _, _ in m] or [0], dtype=np.int32)
    en = np.ascontiguousarray([b for _, b, _ in m] or [0], dtype=np.int32)
    ac = np.ascontiguousarray([1 if c else 0 for _, _, c in m] or [0], dtype=np.uint8)
    qs, qe = c_int32(), c_int32()
    _check(lib().ikv_resolve_span(N, st.ctypes.data, en.ctypes.data, ac.ctypes.data, len(m), tail_w,
                                  ctypes.byref(qs), ctypes.byref(qe)), "ikv_resolve_span")
    return qs.value, qe.value
