"""The test-side helpers that compose the oracle's steps agree with the oracle's own
composition (CPU)."""
import numpy as np

import oracle
import synth
from parity import check_xattn_visible, oracle_scores_pair


def test_scores_pair_matches_oracle_scores():
    batch = synth.make_batch(synth.Shape(L=2, Hq=8, Hkv=2, D=64),
                             [synth.SessionSpec(N=600, C=150, pi=4, qs=580, qe=600, R=5, dead_frac=0.2)],
                             seed=31, kv_dtype=synth.BF16, layout="paged")
    s, S = batch.sessions[0], batch.S(0)
    qpos = np.concatenate([np.flatnonzero(S == 0)[:5], np.arange(570, 600)]).astype(np.int32)
    st = oracle.sets(S, s.pi, s.qs, s.qe, s.C, 0)
    blob = synth.residual_blob(64, seed=4, variant="scaled", units=4, out_std=0.01)
    full, nox = oracle_scores_pair(batch.k_pool, S, st, batch.M_of(0), 2, s.R, blob, qpos, 0)
    np.testing.assert_array_equal(full, oracle.scores(batch.k_pool, S, st, batch.M_of(0), 2, s.R, blob,
                                                      oracle.FLAG_RESIDUAL, qpos, 0))
    np.testing.assert_array_equal(nox, oracle.scores(batch.k_pool, S, st, batch.M_of(0), 2, s.R, blob,
                                                     oracle.FLAG_RESIDUAL | oracle.FLAG_NO_XATTN, qpos, 0))
    check_xattn_visible(full, nox, st)


def test_scaled_blob_shape_and_layout():
    for D in (64, 128):
        blob = synth.residual_blob(D, seed=1, variant="scaled", units=288, out_std=0.005, alpha=1.0)
        assert blob.dtype == np.float32 and len(blob) == oracle.residual_param_count(D)
        W = oracle.residual_unpack(blob, D)
        assert W["alpha"][0] == 1.0
        # the key-mean columns carry the sqrt(units) factor: about sqrt(288 / 1) larger than the rule column
        assert np.abs(W["W_Q"][:, :D]).mean() > 8 * np.abs(W["W_Q"][:, 3 * D]).mean()
