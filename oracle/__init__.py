"""Float64 CPU oracle of the IntentKV retention path -- test infrastructure only.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. It shares no code with the HIP library.
"""
from .ikv_oracle import *  # noqa: F401,F403
from .ikv_oracle import (FLAG_NO_XATTN, FLAG_RESIDUAL, decode, kbar, mbar, qm_update,  # noqa: F401
                         redirect, residual_param_count, residual_scores, residual_unpack,
                         row_lse, rule_scores, scores, select_budget, sets, step, widen)
