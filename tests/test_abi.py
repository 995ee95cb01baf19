"""C-ABI checks that need no GPU: the library loads, exports every symbol that
include/ikv.h declares, its struct layouts match the binding, and argument
validation rejects bad calls before anything touches the device."""
import ctypes
import os
import re

import pytest

import paper_2606_09916_amd as ikv
from paper_2606_09916_amd import ikv as raw

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ikv.h")


def declared_symbols():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ikv_[a-z_]+)\s*\(", src)))


def test_header_symbols_match_binding_and_library():
    syms = declared_symbols()
    assert syms == sorted(raw.SYMBOLS)
    lib = ikv.lib()
    for s in syms:
        assert hasattr(lib, s), s


def test_struct_layouts():
    assert ctypes.sizeof(ikv.Session) == 64
    assert ctypes.sizeof(ikv.Pool) == 48
    assert ikv.Session.N.offset == 32 and ikv.Session.nq.offset == 60
    assert ikv.Pool.num_slots.offset == 16 and ikv.Pool.k_pool.offset == 32


def _pool(**kw):
    p = ikv.Pool(L=2, Hq=8, Hkv=2, D=64, num_slots=100, dead_slot=0, kv_dtype=ikv.IKV_F32,
                 k_pool=0x1000, v_pool=0x2000)
    for k, v in kw.items():
        setattr(p, k, v)
    return p


def _sess(**kw):
    s = (ikv.Session * 1)()
    base = dict(slot_off=0, mem_off=0, qspan_off=0, qpos_off=0, N=50, pi=0, qs=40, qe=50, C=20, radix_prefix=0,
                R=4, nq=10)
    base.update(kw)
    for k, v in base.items():
        setattr(s[0], k, v)
    return s


def _ws(pool, sess, call, flags=0):
    n = ctypes.c_size_t(0)
    st = ikv.lib().ikv_workspace_bytes(ctypes.byref(pool) if pool is not None else None,
                                       ctypes.cast(sess, ctypes.POINTER(ikv.Session)), 1, call, flags,
                                       ctypes.byref(n))
    return st, n.value


@pytest.mark.parametrize("field,value,code", [
    ("Hq", 7, -2), ("D", 96, -4), ("Hq", 32 * 2, -4), ("dead_slot", 100, -2), ("kv_dtype", 5, -1),
    ("k_pool", None, -1), ("L", 0, -2), ("num_slots", 0, -2),
])
def test_pool_validation(field, value, code):
    st, _ = _ws(_pool(**{field: value}), _sess(), ikv.CALL_SCORE)
    assert st == code, ikv.lib().ikv_last_error()
    assert ikv.lib().ikv_last_error()


@pytest.mark.parametrize("field,value", [
    ("N", -1), ("pi", 51), ("qs", 45), ("qe", 60), ("C", -3), ("R", 0), ("R", 300), ("nq", 257),
    ("radix_prefix", -1), ("slot_off", -5),
])
def test_session_validation(field, value):
    kw = {field: value}
    if field == "qs":
        kw["qe"] = 44
    st, _ = _ws(_pool(), _sess(**kw), ikv.CALL_SCORE)
    assert st == -2


def test_workspace_sizes_are_consistent():
    p = _pool()
    st, plain = _ws(p, _sess(), ikv.CALL_SCORE)
    assert st == 0 and plain > 0 and plain % 256 == 0
    st, resid = _ws(p, _sess(), ikv.CALL_SCORE, ikv.IKV_RESIDUAL)
    assert st == 0 and resid > plain
    # selection: per chunk of 4096 positions a 2048-bin histogram + counts (2112 words),
    # one key per position, then 4 result words per session, padded to 64 words; then per
    # session the cooperative path's block: 128 barrier flags of 64 bits, 128 x 4 partial
    # count words and five 2048-bin histograms
    coop = 2 * 128 + 4 * 128 + 5 * 2048

    def pad(w):
        return (w + 63) // 64 * 64
    assert _ws(None, _sess(), ikv.CALL_SELECT) == (0, (pad(2112 + 50 + 4) + coop) * 4)
    assert _ws(None, _sess(slot_off=1000), ikv.CALL_SELECT) == (0, (pad(2112 + 1050 + 4) + coop) * 4)
    assert _ws(None, _sess(N=4097, qs=4000, qe=4097), ikv.CALL_SELECT) == (0, (pad(2 * 2112 + 4097 + 4) + coop) * 4)
    st, red = _ws(p, _sess(), ikv.CALL_REDIRECT)
    assert st == 0 and red == 2 * 64 * 4          # two 100-slot bitsets, each padded to 64 words
    st, dec = _ws(p, _sess(), ikv.CALL_DECODE)
    assert st == 0 and dec == 2 * 8 * 1 * (64 + 2) * 4
    assert _ws(p, _sess(), 99)[0] == -1


def test_calls_reject_bad_arguments_before_launch():
    L = ikv.lib()
    p = _pool()
    s = _sess()
    sp = ctypes.cast(s, ctypes.POINTER(ikv.Session))
    fake = 0x10000
    # unknown flag bits
    assert L.ikv_score_history(ctypes.byref(p), sp, fake, 1, fake, fake, fake, fake, 16, fake, fake, 1 << 30,
                               None) == -1
    # residual flag without weights
    assert L.ikv_score_history(ctypes.byref(p), sp, fake, 1, fake, fake, fake, None, 1, fake, fake, 1 << 30,
                               None) == -1
    # workspace too small / misaligned
    assert L.ikv_score_history(ctypes.byref(p), sp, fake, 1, fake, fake, fake, None, 0, fake, fake, 16, None) == -3
    assert L.ikv_score_history(ctypes.byref(p), sp, fake, 1, fake, fake, fake, None, 0, fake, fake + 4, 1 << 30,
                               None) == -3
    # memory rows must be 16-byte aligned
    assert L.ikv_score_history(ctypes.byref(p), ctypes.cast(_sess(mem_off=1), ctypes.POINTER(ikv.Session)), fake,
                               1, fake, fake, fake, None, 0, fake, fake, 1 << 30, None) == -1
    # selection workspace too small
    assert L.ikv_select_budget(sp, fake, 1, fake, 0, fake, fake, fake, fake, fake, 16, None) == -3
    # null outputs
    assert L.ikv_select_budget(sp, fake, 1, fake, 0, fake, None, fake, fake, None, 0, None) == -1
    assert L.ikv_redirect_slots(sp, fake, 1, 100, fake, 0, fake, fake, fake, None, fake, fake, 1 << 20,
                                None) == -1
    assert L.ikv_redirect_slots(sp, fake, 1, 100, fake, 100, fake, fake, fake, fake, fake, fake, 1 << 20,
                                None) == -2
    assert L.ikv_decode_attend_slotmap(ctypes.byref(p), sp, fake, 1, None, fake, fake, fake, fake, 1 << 20,
                                       None) == -1
    assert L.ikv_qm_update(ctypes.byref(p), sp, fake, 1, fake, fake, -1.0, None) == -1
    assert L.ikv_qm_update(ctypes.byref(p), sp, None, 1, fake, fake, 0.5, None) == -1
    # span rows and memory rows must be 16-byte aligned (float32 pool: offsets a multiple of 4)
    assert L.ikv_qm_update(ctypes.byref(p), ctypes.cast(_sess(qspan_off=2), ctypes.POINTER(ikv.Session)), fake, 1,
                           fake, fake, 0.5, None) == -1
    assert L.ikv_qm_update(ctypes.byref(p), ctypes.cast(_sess(mem_off=2), ctypes.POINTER(ikv.Session)), fake, 1,
                           fake, fake, 0.5, None) == -1
    assert L.ikv_qm_update(ctypes.byref(p), sp, fake, 1, fake + 8, fake, 0.5, None) == -1
    # B = 0 is a no-op
    assert L.ikv_select_budget(sp, fake, 0, None, 0, None, None, None, None, None, 0, None) == 0


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(raw, "_lib", None)
    monkeypatch.setattr(raw, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="missing"):
        raw.lib()


def test_timing_toggle_and_empty_read():
    # no kernel launched: switching timing on and reading touches no device
    assert ikv.lib().ikv_timing(1) == 0
    assert ikv.timing_read() == []
    assert ikv.lib().ikv_timing_read(None, None, 0) == 0
    assert ikv.lib().ikv_timing_read(None, None, 5) == -1
    assert ikv.lib().ikv_timing(0) == 0
