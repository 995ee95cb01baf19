"""Selection (Eq. 1) and redirect (Eq. 7, Sec. 3.4) on sizes the tiny end-to-end
cases do not reach: sessions longer than the workgroup's key cache, heavy ties
spread over every wave's range, batched sessions of different lengths, and pools
whose slot bitsets do not fit in LDS. Every result is compared with the oracle
exactly (these are integer and comparison results)."""
import math

import numpy as np
import pytest

import oracle
import synth
from paper_2606_09916_amd import ikv

pytestmark = pytest.mark.gpu
DEAD = synth.DEAD_SLOT


def _torch():
    import torch
    return torch


def _sets(S, row):
    return oracle.sets(S, row["pi"], row["qs"], row["qe"], row["C"], DEAD)


def _rows(lengths, **kw):
    rows, off = [], 0
    for n in lengths:
        r = dict(slot_off=off, mem_off=0, qspan_off=0, qpos_off=0, N=n, pi=0, qs=max(0, n - 64), qe=n,
                 C=max(1, n // 4), radix_prefix=0, R=16, nq=0)
        r.update(kw)
        rows.append(r)
        off += n
    return rows


def _select(dev, rows, S_all, sc_all):
    torch = _torch()
    sess = ikv.Sessions(rows, dev)
    B, tot = len(rows), len(S_all)
    S_d = torch.from_numpy(S_all).to(dev)
    sc_d = torch.from_numpy(sc_all).to(dev)
    keep = torch.zeros(tot, dtype=torch.uint8, device=dev)
    n_keep = torch.zeros(B, dtype=torch.int32, device=dev)
    tau = torch.zeros(B, dtype=torch.float32, device=dev)
    ikv.select_budget(sess, S_d, DEAD, sc_d, keep, n_keep, tau, ikv.Workspace(dev))
    torch.cuda.synchronize()
    return keep.cpu().numpy(), n_keep.cpu().numpy(), tau.cpu().numpy()


@pytest.mark.parametrize("lengths,ties", [((40000,), True), ((40000,), False), ((32768, 40001, 5000), True),
                                          ((70000,), False)])
def test_select_long_sessions_exact(dev, lengths, ties):
    rows = _rows(lengths)
    Ss, scs = [], []
    for b, n in enumerate(lengths):
        Ss.append(synth.slot_map(n, 2 * n + 1, seed=100 + b))
        scs.append(synth.score_vector(n, seed=200 + b, ties=ties))
    S_all, sc_all = np.concatenate(Ss), np.concatenate(scs)
    keep, n_keep, tau = _select(dev, rows, S_all, sc_all)
    for b, r in enumerate(rows):
        o, n = r["slot_off"], r["N"]
        k_o, n_o, t_o = oracle.select_budget(scs[b].astype(np.float64), _sets(Ss[b], r))
        assert np.array_equal(keep[o:o + n].astype(bool), k_o), f"session {b}"
        assert int(n_keep[b]) == n_o
        assert tau[b] == t_o or (math.isnan(tau[b]) and math.isnan(t_o))


@pytest.mark.parametrize("lengths,ties,coop", [((140000, 3000), False, True), ((200000,), True, True),
                                               ((32768, 20000, 7), True, False), ((40000, 9000), False, False)])
def test_select_paths_exact(dev, lengths, ties, coop, monkeypatch):
    """Sessions past the cooperative path's limit (131,072 positions) take the
    three-kernel path; with IKV_NO_COOP=1 sessions up to 32,768 positions take the
    one-workgroup kernel and longer ones the three-kernel path."""
    if not coop:
        monkeypatch.setenv("IKV_NO_COOP", "1")
    test_select_long_sessions_exact(dev, lengths, ties)


@pytest.mark.parametrize("n,C,coop", [(50000, 20000, True), (3000, 1000, True), (40000, 39990, True),
                                      (3000, 1000, False), (50000, 20000, False), (150000, 60000, True)])
def test_select_all_scores_equal(dev, n, C, coop, monkeypatch):
    # every candidate ties at the threshold: the budget fills in position order
    if not coop:
        monkeypatch.setenv("IKV_NO_COOP", "1")
    rows = _rows((n,), C=C, pi=7)
    S = synth.slot_map(n, n + 1, seed=5, dead_frac=0.2)
    sc = np.full(n, 0.375, np.float32)
    keep, n_keep, tau = _select(dev, rows, S, sc)
    k_o, n_o, t_o = oracle.select_budget(sc.astype(np.float64), _sets(S, rows[0]))
    assert np.array_equal(keep.astype(bool), k_o)
    assert int(n_keep[0]) == n_o and tau[0] == t_o


def _redirect(dev, rows, num_slots, S_all, keep_all):
    torch = _torch()
    sess = ikv.Sessions(rows, dev)
    B, tot = len(rows), len(S_all)
    S_d = torch.from_numpy(S_all.copy()).to(dev)
    keep_d = torch.from_numpy(keep_all).to(dev)
    freed = torch.full((tot,), -7, dtype=torch.int32, device=dev)
    live = torch.full((tot,), -7, dtype=torch.int32, device=dev)
    n_freed = torch.zeros(B, dtype=torch.int32, device=dev)
    n_live = torch.zeros(B, dtype=torch.int32, device=dev)
    ws = ikv.Workspace(dev)
    ikv.redirect_slots(sess, num_slots, S_d, DEAD, keep_d, freed, n_freed, live, n_live, ws)
    torch.cuda.synchronize()
    return (S_d.cpu().numpy(), freed.cpu().numpy(), n_freed.cpu().numpy(), live.cpu().numpy(),
            n_live.cpu().numpy())


@pytest.mark.parametrize("num_slots", [524288, 600000])
def test_redirect_large_pools_exact(dev, num_slots):
    # 524288 slots: the last pool size whose bitsets sit in LDS; 600000: the workspace path
    lengths = (40000, 9000)
    rows = _rows(lengths, radix_prefix=0)
    rows[1]["radix_prefix"] = 500
    Ss, keeps = [], []
    for b, n in enumerate(lengths):
        S = synth.slot_map(n, num_slots, seed=300 + b, dead_frac=0.15)
        S = synth.alias_slots(S, seed=310 + b, pairs=n // 20)
        Ss.append(S)
        keeps.append(synth.keep_mask(S, seed=320 + b))
    S_d, freed, n_freed, live, n_live = _redirect(dev, rows, num_slots, np.concatenate(Ss), np.concatenate(keeps))
    for b, r in enumerate(rows):
        o, n = r["slot_off"], r["N"]
        S_o, freed_o, live_o = oracle.redirect(Ss[b], keeps[b].astype(bool), DEAD, r["radix_prefix"])
        assert np.array_equal(S_d[o:o + n], S_o), f"session {b}"
        assert int(n_freed[b]) == len(freed_o) and int(n_live[b]) == len(live_o)
        assert np.array_equal(freed[o:o + len(freed_o)], freed_o)
        assert np.array_equal(live[o:o + len(live_o)], live_o)


def test_select_barrier_give_up_is_reported(dev, monkeypatch):
    """The cooperative selection's grid barriers wait a bounded number of polls. Forced
    from the host to give up at once (IKV_SELECT_SPINS=0, so every kernel still runs to
    its end), the call's outputs are not valid and the library's next call returns
    IKV_EHIP; the call after that selects exactly again."""
    torch = _torch()
    monkeypatch.delenv("IKV_NO_COOP", raising=False)
    n = 40000
    rows = _rows((n,))
    S = synth.slot_map(n, 2 * n + 1, seed=101)
    sc = synth.score_vector(n, seed=201, ties=False)
    ikv.timing(True)
    try:
        monkeypatch.setenv("IKV_SELECT_SPINS", "0")
        _select(dev, rows, S, sc)
        names = [name for name, _ in ikv.timing_read()]
    finally:
        ikv.timing(False)
    if "k_select_coop" not in names:
        pytest.skip(f"the cooperative selection did not run here ({names})")
    monkeypatch.delenv("IKV_SELECT_SPINS")
    with pytest.raises(ikv.IkvError) as e:
        _select(dev, rows, S, sc)
    assert e.value.status == -5 and "gave up" in str(e.value)
    keep, n_keep, tau = _select(dev, rows, S, sc)
    k_o, n_o, t_o = oracle.select_budget(sc.astype(np.float64), _sets(S, rows[0]))
    assert np.array_equal(keep.astype(bool), k_o) and int(n_keep[0]) == n_o
    torch.cuda.synchronize()
