"""Many sessions in one call: the one-GPU share of a Qwen2.5-14B tensor-parallel pair
(48 layers, 20 query / 4 KV heads, D = 128), 16 ragged sessions of 1k-8k positions
with 32-128 memory rows each (multiples of 16), sharing one paged pool, budget a
quarter of each session, residual head on. Every session is compared with the full
oracle; the sum of each session's rule scores must also equal its row count
(every softmax sums to one)."""
import numpy as np
import pytest

import oracle
import synth
from paper_2606_09916_amd import ikv
from paper_2606_09916_amd.step import RetentionStep
from parity import check_attention, check_keep, check_scores

pytestmark = pytest.mark.gpu
SEED = 5


@pytest.fixture(scope="module")
def share_batch():
    g = synth.stream(SEED, synth.T_TURNS, 1)
    B = 16
    Ns = g.integers(1024, 8193, B)
    Rs = 16 * g.integers(2, 9, B)
    sessions = [synth.SessionSpec(N=int(n), C=int(n) // 4, pi=0, qs=int(n) - 64, qe=int(n), R=int(r))
                for n, r in zip(Ns, Rs)]
    shape = synth.Shape(L=48, Hq=20, Hkv=4, D=128)
    return synth.make_batch(shape, sessions, seed=SEED, kv_dtype=synth.BF16, layout="paged", spare_pages=37)


def test_batched_share_step(dev, share_batch):
    batch = share_batch
    blob = synth.residual_blob(128, seed=25)
    st = RetentionStep(batch, dev, residual=blob, flags=ikv.IKV_RESIDUAL)
    st.init_dead_slot()
    st.step(update_memory=True)
    sc, keep, S_all = st.host("scores"), st.host("keep"), st.host("S")
    live_all, n_live = st.host("live"), st.host("n_live")
    out = st.host("out")
    sh = batch.shape
    for b, s in enumerate(batch.sessions):
        o = int(batch.slot_off[b])
        sl = slice(o, o + s.N)
        M = oracle.qm_update(batch.M_of(b), batch.q_span_of(b))
        sets = oracle.sets(batch.S(b), s.pi, s.qs, s.qe, s.C, synth.DEAD_SLOT)
        want = oracle.scores(batch.k_pool, batch.S(b), sets, M, sh.Hkv, s.R, blob, oracle.FLAG_RESIDUAL,
                             batch.qpos_of(b), synth.DEAD_SLOT)
        check_scores(sc[sl], want, sets["cand"])
        rule = oracle.rule_scores(batch.k_pool, batch.S(b), sets["cand"], M, sh.Hkv, s.R)
        assert abs(rule[sets["cand"]].sum() - sh.L * sh.Hkv * s.R) < 1e-6 * sh.L * sh.Hkv * s.R
        keep_o, n_o, tau_o = oracle.select_budget(want, sets)
        keep_g = keep[sl].astype(bool)
        check_keep(keep_g, int(st.host("n_keep")[b]), keep_o, n_o, want, tau_o, sets["cand"])
        S_o, freed_o, live_o = oracle.redirect(batch.S(b), keep_g, synth.DEAD_SLOT, s.radix_prefix)
        assert np.array_equal(S_all[sl], S_o)
        assert np.array_equal(live_all[o:o + int(n_live[b])], live_o)
        o_o = oracle.decode(batch.q_dec[b], batch.k_pool, batch.v_pool, live_o)
        check_attention(synth.widen(out[b]), o_o, bf16=True)
