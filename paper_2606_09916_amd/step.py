"""Device state of one retention step and the five C-ABI calls in order.

``RetentionStep`` uploads a batch of sessions (numpy arrays in the layouts of
include/ikv.h) into torch device tensors and runs qm_update -> score_history ->
select_budget -> redirect_slots -> decode_attend_slotmap through the binding.
It only moves memory; every step of the path runs in libikv.so.
"""
from __future__ import annotations

import numpy as np

from . import ikv


def _t(a, device, dtype=None):
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:                     # bf16 bit patterns
        return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
    t = torch.from_numpy(a).to(device)
    return t if dtype is None else t.to(dtype)


class RetentionStep:
    """One step over a batch.

    ``batch`` needs the fields of the generator's Batch: shape (L, Hq, Hkv, D),
    sessions (N, C, pi, qs, qe, R, radix_prefix, query positions), num_slots,
    k_pool, v_pool, slot_maps, slot_off, M, mem_off, q_span, qspan_off, qpos,
    qpos_off, q_dec.
    """

    def __init__(self, batch, device, residual=None, flags: int = 0, lam: float = 0.5, dead_slot: int = 0,
                 k_dev=None, v_dev=None):
        import torch
        self.device = device
        sh = batch.shape
        self.L, self.Hq, self.Hkv, self.D = sh.L, sh.Hq, sh.Hkv, sh.D
        self.num_slots = batch.num_slots
        self.dead = dead_slot
        self.lam = lam
        self.flags = flags
        # pools already on the device (too large to draw on the host) or uploaded here
        self.k_pool = k_dev if k_dev is not None else _t(batch.k_pool, device)
        self.v_pool = v_dev if v_dev is not None else _t(batch.v_pool, device)
        self.pool = ikv.make_pool(self.k_pool, self.v_pool, sh.L, sh.Hq, sh.Hkv, sh.D, batch.num_slots, dead_slot)
        self.S0 = _t(batch.slot_maps.astype(np.int32), device)
        self.S = self.S0.clone()
        self.M0 = _t(batch.M.astype(np.float32), device)
        self.M = self.M0.clone()
        self.q_span = _t(batch.q_span, device)
        self.qpos = _t(batch.qpos.astype(np.int32), device) if len(batch.qpos) else None
        self.q_dec = _t(batch.q_dec, device)
        self.residual = None if residual is None else _t(np.asarray(residual, np.float32), device)
        rows = []
        for b, s in enumerate(batch.sessions):
            rows.append(dict(slot_off=batch.slot_off[b], mem_off=batch.mem_off[b], qspan_off=batch.qspan_off[b],
                             qpos_off=batch.qpos_off[b], N=s.N, pi=s.pi, qs=s.qs, qe=s.qe, C=s.C,
                             radix_prefix=s.radix_prefix, R=s.R, nq=len(s.query_positions())))
        self.sess = ikv.Sessions(rows, device)
        self.B = len(rows)
        total = int(batch.slot_maps.shape[0])
        self.scores = torch.empty(total, dtype=torch.float32, device=device)
        self.keep = torch.empty(total, dtype=torch.uint8, device=device)
        self.freed = torch.empty(total, dtype=torch.int32, device=device)
        self.live = torch.empty(total, dtype=torch.int32, device=device)
        self.n_keep = torch.empty(self.B, dtype=torch.int32, device=device)
        self.tau = torch.empty(self.B, dtype=torch.float32, device=device)
        self.n_freed = torch.empty(self.B, dtype=torch.int32, device=device)
        self.n_live = torch.empty(self.B, dtype=torch.int32, device=device)
        self.out = torch.empty_like(self.q_dec)
        self.ws = ikv.Workspace(device)

    # ---------------------------------------------------------------- calls
    def reset(self):
        """Restore the slot maps and the QueryMemory to their initial state."""
        self.S.copy_(self.S0)
        self.M.copy_(self.M0)

    def init_dead_slot(self):
        ikv.init_dead_slot(self.pool)

    def qm_update(self, lam=None):
        ikv.qm_update(self.pool, self.sess, self.M, self.q_span, self.lam if lam is None else lam)

    def score(self, flags=None):
        f = self.flags if flags is None else flags
        ikv.score_history(self.pool, self.sess, self.S, self.M, self.scores, self.ws, qpos=self.qpos,
                          residual=self.residual if f & ikv.IKV_RESIDUAL else None, flags=f)

    def select(self):
        ikv.select_budget(self.sess, self.S, self.dead, self.scores, self.keep, self.n_keep, self.tau, self.ws)

    def redirect(self):
        ikv.redirect_slots(self.sess, self.num_slots, self.S, self.dead, self.keep, self.freed, self.n_freed,
                           self.live, self.n_live, self.ws)

    def decode(self):
        ikv.decode_attend_slotmap(self.pool, self.sess, self.q_dec, self.live, self.n_live, self.out, self.ws)

    def step(self, update_memory: bool = True):
        if update_memory:
            self.qm_update()
        self.score()
        self.select()
        self.redirect()
        self.decode()

    # ---------------------------------------------------------------- readback
    def host(self, name):
        t = getattr(self, name)
        import torch
        if t.dtype == torch.bfloat16:
            return t.view(torch.int16).cpu().numpy().view(np.uint16)
        return t.cpu().numpy()
