"""The one-key-pass form of the score (every session at most 16 memory rows, one 16-row
slice; Sec. 3.2 with R = G, Eq. 3): the logits of one pass over the keys are stashed
and normalised afterwards. It must meet the same bar against the float64 oracle as the
two-pass form (IKV_TWO_PASS), and agree with it to float32 rounding order."""
import numpy as np
import pytest

import oracle
import synth
from paper_2606_09916_amd import ikv
from paper_2606_09916_amd.step import RetentionStep
from parity import RESID_MFMA_FLOOR, SCORE_FLOOR, check_keep, check_scores
from test_gpu_parity import _compare_step, oracle_scores

pytestmark = pytest.mark.gpu


def _batch(R, N, Hkv, dead, seed, C=None, pi=4):
    spec = synth.SessionSpec(N=N, C=min(C or 300, N // 3), pi=pi, qs=N - 16, qe=N, R=R, dead_frac=dead)
    return synth.make_batch(synth.Shape(L=2, Hq=Hkv * 2, Hkv=Hkv, D=128), [spec], seed=seed, kv_dtype=synth.BF16,
                            layout="paged")


@pytest.mark.parametrize("R,N,Hkv,resid,dead", [(1, 700, 2, False, 0.1), (4, 1000, 2, True, 0.1),
                                                (5, 1300, 2, True, 0.0), (13, 900, 3, True, 0.2),
                                                (16, 1500, 2, False, 0.05), (4, 129, 2, True, 0.0),
                                                (8, 2100, 1, True, 0.3)])
def test_one_key_pass_against_oracle_and_two_passes(dev, R, N, Hkv, resid, dead):
    batch = _batch(R, N, Hkv, dead, seed=5 * R + N)
    blob = synth.residual_blob(128, seed=R) if resid else None
    flags = ikv.IKV_RESIDUAL if resid else 0
    st = RetentionStep(batch, dev, residual=blob, flags=flags)
    st.init_dead_slot()
    want, sets = oracle_scores(batch, 0, blob, flags)
    st.score(flags=flags | ikv.IKV_TWO_PASS)
    two = st.host("scores").copy()
    st.score(flags=flags)
    one = st.host("scores").copy()
    c = sets["cand"]
    for name, got in (("two passes", two), ("one pass", one)):
        err = np.abs(got[c] - want[c])
        k = int(np.argmax(err)) if c.any() else 0
        print(f"{name}: worst |error| {err.max() if c.any() else 0:.3e} at a score of "
              f"{want[c][k] if c.any() else 0:.3e}; largest |score| {np.abs(want[c]).max() if c.any() else 0:.3e}")
    floor = RESID_MFMA_FLOOR if resid else SCORE_FLOOR
    check_scores(two, want, c, floor=floor)
    check_scores(one, want, c, floor=floor)
    st.select()
    keep_o, n_o, tau_o = oracle.select_budget(want, sets)
    check_keep(st.host("keep"), int(st.host("n_keep")[0]), keep_o, n_o, want, tau_o, c)
    rel = np.abs(one[c] - two[c]).max() / np.abs(two[c]).max() if c.any() else 0.0
    print(f"R={R}: one pass vs two passes, max difference {rel:.2e} of the largest score")
    assert rel < 2e-6


def test_one_key_pass_batched_rows_up_to_16(dev):
    """A batch of sessions with 1 to 16 memory rows: one at its budget (skipped), one
    shorter than a list tile, dead positions, a forced prefix and a protected radix
    prefix; the whole step against the oracle, with the QueryMemory update."""
    shape = synth.Shape(L=2, Hq=8, Hkv=2, D=128)
    sessions = [synth.SessionSpec(N=1100, C=300, pi=8, qs=1080, qe=1100, R=4, dead_frac=0.1),
                synth.SessionSpec(N=700, C=200, pi=0, qs=650, qe=700, R=13),
                synth.SessionSpec(N=400, C=400, pi=0, qs=380, qe=400, R=16),
                synth.SessionSpec(N=1500, C=150, pi=16, qs=1440, qe=1500, R=1, radix_prefix=16),
                synth.SessionSpec(N=100, C=30, pi=0, qs=90, qe=100, R=5, dead_frac=0.2),
                synth.SessionSpec(N=900, C=500, pi=0, qs=860, qe=900, R=16, dead_frac=0.2)]
    batch = synth.make_batch(shape, sessions, seed=61, kv_dtype=synth.BF16, layout="paged", spare_pages=4)
    blob = synth.residual_blob(128, seed=62)
    st = RetentionStep(batch, dev, residual=blob, flags=ikv.IKV_RESIDUAL)
    st.init_dead_slot()
    st.step(update_memory=True)
    for b in range(len(sessions)):
        _compare_step(st, batch, b, blob, ikv.IKV_RESIDUAL, True)


def test_one_key_pass_qwen3_8b_32k_rows_per_query_head(dev):
    """The paper's own memory shape (one row per query head, R = G = 4) at the
    Qwen3-8B 32k step, full size, against the full oracle; the residual head's
    cross-attention must visibly move the scores and the kept set."""
    batch = synth.qwen3_8b_32k(R=4)
    blob = synth.residual_blob(128, seed=25, variant="scaled", units=36 * 8, out_std=2e-3)
    st = RetentionStep(batch, dev, residual=blob, flags=ikv.IKV_RESIDUAL)
    st.init_dead_slot()
    st.step(update_memory=False)
    ndiff = _compare_step(st, batch, 0, blob, ikv.IKV_RESIDUAL, False, xattn_check=True)
    print(f"kept-set differences inside the band: {ndiff}")
