"""Many sessions in one call: the one-GPU share of a Qwen2.5-14B tensor-parallel pair
(48 layers, 20 query / 4 KV heads, D = 128), ragged sessions sharing one paged pool,
memory rows per KV head drawn from 32..128 (any count, not only whole 16-row slices),
budget a quarter of each session, residual head on with weights under which its
cross-attention visibly moves every session's scores and kept set. Every session is
compared with the full oracle; the sum of each session's rule scores must also equal
its row count (every softmax sums to one)."""
import numpy as np
import pytest

import oracle
import synth
from paper_2606_09916_amd import ikv
from paper_2606_09916_amd.step import RetentionStep
from parity import (RESID_MFMA_FLOOR, check_attention, check_keep, check_scores, check_xattn_visible,
                    oracle_scores_pair)

pytestmark = pytest.mark.gpu
SEED = 5
SHAPE = synth.Shape(L=48, Hq=20, Hkv=4, D=128)


@pytest.fixture(scope="module")
def share_batch():
    g = synth.stream(SEED, synth.T_TURNS, 1)
    B = 16
    Ns = g.integers(1024, 8193, B)
    Rs = g.integers(32, 129, B)
    sessions = [synth.SessionSpec(N=int(n), C=int(n) // 4, pi=0, qs=int(n) - 64, qe=int(n), R=int(r))
                for n, r in zip(Ns, Rs)]
    return synth.make_batch(SHAPE, sessions, seed=SEED, kv_dtype=synth.BF16, layout="paged", spare_pages=37)


def _check_batch(st, batch, blob, xattn=True):
    sc, keep, S_all = st.host("scores"), st.host("keep"), st.host("S")
    live_all, n_live = st.host("live"), st.host("n_live")
    out = st.host("out")
    sh = batch.shape
    for b, s in enumerate(batch.sessions):
        o = int(batch.slot_off[b])
        sl = slice(o, o + s.N)
        M = oracle.qm_update(batch.M_of(b), batch.q_span_of(b))
        sets = oracle.sets(batch.S(b), s.pi, s.qs, s.qe, s.C, synth.DEAD_SLOT)
        want, nox = oracle_scores_pair(batch.k_pool, batch.S(b), sets, M, sh.Hkv, s.R, blob, batch.qpos_of(b),
                                       synth.DEAD_SLOT)
        if xattn:
            ratio, nd = check_xattn_visible(want, nox, sets)
        rel = check_scores(sc[sl], want, sets["cand"], floor=RESID_MFMA_FLOOR)
        rule = oracle.rule_scores(batch.k_pool, batch.S(b), sets["cand"], M, sh.Hkv, s.R)
        assert abs(rule[sets["cand"]].sum() - sh.L * sh.Hkv * s.R) < 1e-6 * sh.L * sh.Hkv * s.R
        keep_o, n_o, tau_o = oracle.select_budget(want, sets)
        keep_g = keep[sl].astype(bool)
        nband = check_keep(keep_g, int(st.host("n_keep")[b]), keep_o, n_o, want, tau_o, sets["cand"])
        S_o, freed_o, live_o = oracle.redirect(batch.S(b), keep_g, synth.DEAD_SLOT, s.radix_prefix)
        assert np.array_equal(S_all[sl], S_o)
        assert np.array_equal(live_all[o:o + int(n_live[b])], live_o)
        o_o = oracle.decode(batch.q_dec[b], batch.k_pool, batch.v_pool, live_o)
        err = check_attention(synth.widen(out[b]), o_o, bf16=True)
        print(f"session {b}: N={s.N} R={s.R} score err {rel:.1e} attention err {err:.1e} band diffs {nband}"
              + (f" x-attn {ratio:.0f}x tol, {nd} kept" if xattn else ""), flush=True)


def test_batched_share_step(dev, share_batch):
    batch = share_batch
    blob = synth.residual_blob(128, seed=25, variant="scaled", units=SHAPE.L * SHAPE.Hkv, out_std=0.03)
    st = RetentionStep(batch, dev, residual=blob, flags=ikv.IKV_RESIDUAL)
    st.init_dead_slot()
    st.step(update_memory=True)
    _check_batch(st, batch, blob)


def test_batched_share_ragged_row_counts(dev):
    """Sessions whose memory-row counts fill no whole 16-row slice (33, 47, 100, 127),
    one call each for scoring, selection, redirect and decode, at the share's shape."""
    specs = [synth.SessionSpec(N=n, C=n // 4, pi=0, qs=n - 64, qe=n, R=r, dead_frac=d)
             for n, r, d in ((2100, 33, 0.0), (3300, 47, 0.1), (1700, 100, 0.0), (2900, 127, 0.05))]
    batch = synth.make_batch(SHAPE, specs, seed=SEED + 1, kv_dtype=synth.BF16, layout="paged", spare_pages=5)
    blob = synth.residual_blob(128, seed=27, variant="scaled", units=SHAPE.L * SHAPE.Hkv, out_std=0.03)
    st = RetentionStep(batch, dev, residual=blob, flags=ikv.IKV_RESIDUAL)
    st.init_dead_slot()
    st.step(update_memory=True)
    _check_batch(st, batch, blob)
    # the rule score alone (no residual): every session's scores sum to its row count
    st.score(flags=0)
    sc = st.host("scores").astype(np.float64)
    for b, s in enumerate(batch.sessions):
        o = int(batch.slot_off[b])
        x = sc[o:o + s.N]
        assert abs(x[np.isfinite(x)].sum() - SHAPE.L * SHAPE.Hkv * s.R) < 1e-4 * SHAPE.L * SHAPE.Hkv * s.R
