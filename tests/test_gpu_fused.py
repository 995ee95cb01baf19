"""The one-key-pass score at 16 < R <= 64 (k_score_fused): one session whose candidate
list tiles are all resident, the keys read once, the row normalisers of Eq. 3 exchanged
between the tiles' workgroups while the pass runs. Its scores are checked against the
float64 oracle and against the two-pass form (without IKV_FUSED=1) on the same inputs, with
the rule path's closed form (every memory row's softmax sums to 1, so the rule scores sum
to L * Hkv * R); ragged, nearly empty and empty tiles; the residual head on top; and the
exchange's bounded waits forced from the host to give up."""
import math

import numpy as np
import pytest

import oracle
import synth
from paper_2606_09916_amd import ikv
from paper_2606_09916_amd.step import RetentionStep
from parity import RESID_MFMA_FLOOR, SCORE_FLOOR, check_keep, check_scores

# The form is switched off in the library (fused_tiles returns 0): on some runs one row
# normaliser came out wrong (test_fused_unit_counts[5-1-8300-24]: relative score errors of
# 6e-4 to 8e-4 in about one run in three), and the cause is not found.
pytestmark = [pytest.mark.gpu,
              pytest.mark.skip(reason="one-key-pass form switched off: intermittent wrong row normaliser, cause not found")]


def _batch(N, R, dead_frac, seed, L=2, Hkv=2, dead_range=None):
    s = synth.SessionSpec(N=N, C=N // 4, pi=8, qs=N - 24, qe=N, R=R, dead_frac=dead_frac)
    batch = synth.make_batch(synth.Shape(L=L, Hq=Hkv * 4, Hkv=Hkv, D=128), [s], seed=seed, kv_dtype=synth.BF16,
                             layout="paged")
    if dead_range is not None:                       # whole list tiles without a candidate
        a, b = dead_range
        batch.slot_maps[a:b] = synth.DEAD_SLOT
    return batch


def _sets(batch):
    s = batch.sessions[0]
    return oracle.sets(batch.S(0), s.pi, s.qs, s.qe, s.C, synth.DEAD_SLOT)


def _score(dev, batch, flags, blob, monkeypatch, fused):
    import torch
    monkeypatch.setenv("IKV_FUSED", "1" if fused else "0")
    st = RetentionStep(batch, dev, residual=blob, flags=flags)
    st.init_dead_slot()
    ikv.timing(True)
    try:
        st.score()
        torch.cuda.synchronize()
        names = [n for n, _ in ikv.timing_read()]
    finally:
        ikv.timing(False)
    return st, names


@pytest.mark.parametrize("N,R,dead,flags,dead_range", [
    (9000, 64, 0.1, 0, None),
    (9000, 33, 0.0, 0, None),
    (12000, 17, 0.3, 0, None),
    (16500, 64, 0.5, 0, (2000, 5000)),
    (20000, 48, 0.1, ikv.IKV_RESIDUAL, None),
    (10000, 64, 0.2, ikv.IKV_RESIDUAL | ikv.IKV_NO_XATTN, (128, 1024)),
])
def test_fused_scores_against_oracle_and_two_pass(dev, monkeypatch, N, R, dead, flags, dead_range):
    batch = _batch(N, R, dead, seed=N + R, dead_range=dead_range)
    blob = synth.residual_blob(128, seed=R, variant="scaled", units=4, out_std=0.03) if flags else None
    st, names = _score(dev, batch, flags, blob, monkeypatch, fused=True)
    assert "k_score_fused" in names, names
    sets = _sets(batch)
    want = oracle.scores(batch.k_pool, batch.S(0), sets, batch.M_of(0), 2, R, blob, flags, batch.qpos_of(0),
                         synth.DEAD_SLOT)
    cand = sets["cand"]
    floor = RESID_MFMA_FLOOR if flags else SCORE_FLOOR
    got = st.host("scores")
    rel = check_scores(got, want, cand, floor=floor)
    if not flags:
        assert rel < 1e-5, rel
        assert math.isclose(float(got[cand].astype(np.float64).sum()), 2 * 2 * R, rel_tol=1e-5)
    st.select()
    keep_o, n_o, tau_o = oracle.select_budget(want, sets)
    check_keep(st.host("keep"), int(st.host("n_keep")[0]), keep_o, n_o, want, tau_o, cand)
    # the two-pass form on the same inputs agrees within the same rule
    st2, names2 = _score(dev, batch, flags, blob, monkeypatch, fused=False)
    assert "k_score_fused" not in names2, names2
    check_scores(st2.host("scores"), want, cand, floor=floor)
    print(f"N={N} R={R}: worst relative score error {rel:.2e}")


@pytest.mark.parametrize("L,Hkv,N,R", [(3, 3, 9500, 40), (1, 1, 16000, 64), (5, 1, 8300, 24)])
def test_fused_unit_counts(dev, monkeypatch, L, Hkv, N, R):
    """Unit counts that are not a multiple of a head pair (odd KV heads, one layer): the
    owner of row r of unit x is workgroup (x * R16 + r) mod G whatever the count, and
    the units past the last one only finish. Rule path against the oracle and its
    closed form, and against the two-pass form."""
    batch = _batch(N, R, 0.2, seed=L * 100 + Hkv * 10 + R, L=L, Hkv=Hkv)
    st, names = _score(dev, batch, 0, None, monkeypatch, fused=True)
    assert "k_score_fused" in names, names
    sets = _sets(batch)
    want = oracle.scores(batch.k_pool, batch.S(0), sets, batch.M_of(0), Hkv, R, None, 0, batch.qpos_of(0),
                         synth.DEAD_SLOT)
    cand = sets["cand"]
    got = st.host("scores")
    rel = check_scores(got, want, cand, floor=SCORE_FLOOR)
    assert rel < 1e-5, rel
    assert math.isclose(float(got[cand].astype(np.float64).sum()), L * Hkv * R, rel_tol=1e-5)
    st2, _ = _score(dev, batch, 0, None, monkeypatch, fused=False)
    check_scores(st2.host("scores"), want, cand, floor=SCORE_FLOOR)


def test_fused_is_deterministic(dev, monkeypatch):
    batch = _batch(9000, 64, 0.1, seed=77)
    a, _ = _score(dev, batch, 0, None, monkeypatch, fused=True)
    b, _ = _score(dev, batch, 0, None, monkeypatch, fused=True)
    assert np.array_equal(a.host("scores"), b.host("scores"))


def test_fused_exchange_give_up_is_reported(dev, monkeypatch):
    """The exchange's waits are bounded. Forced from the host to give up at once
    (IKV_EXCHANGE_SPINS=0: the rows of the last two units are always combined after the
    unit loop, where an owner only waits, so they time out, and every kernel still runs
    to its end), the call's scores are not valid and the library's next call returns
    IKV_EHIP; the call after that scores exactly again."""
    batch = _batch(9000, 64, 0.1, seed=78)
    monkeypatch.setenv("IKV_EXCHANGE_SPINS", "0")
    st, names = _score(dev, batch, 0, None, monkeypatch, fused=True)
    assert "k_score_fused" in names
    monkeypatch.delenv("IKV_EXCHANGE_SPINS")
    with pytest.raises(ikv.IkvError) as e:
        st.score()
    assert e.value.status == -5 and "gave up" in str(e.value)
    st.score()
    sets = _sets(batch)
    want = oracle.scores(batch.k_pool, batch.S(0), sets, batch.M_of(0), 2, 64, None, 0, batch.qpos_of(0),
                         synth.DEAD_SLOT)
    check_scores(st.host("scores"), want, sets["cand"])
