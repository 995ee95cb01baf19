"""IntentKV per-step retention hot path on MI355X (gfx950).

The HIP library ``libikv.so`` (C ABI in ``include/ikv.h``) holds every step:
QueryMemory update, rule + residual scoring, budgeted selection, slot-map
redirect and slot-map decode attention. This package is its Python binding.
"""
from .ikv import (CALL_DECODE, CALL_REDIRECT, CALL_SCORE, CALL_SELECT, IKV_BF16, IKV_F32,  # noqa: F401
                  IKV_NO_XATTN, IKV_RESIDUAL, SYMBOLS, IkvError, Pool, Session, Sessions, Workspace,
                  decode_attend_slotmap, init_dead_slot, lib, make_pool, qm_update, redirect_slots,
                  score_history, select_budget, timing, timing_read, workspace_bytes)
