"""Comparison rules between the HIP path and the float64 oracle.

* scores: |s_gpu - s_o| <= 1e-3 |s_o| + f max|s_o| on candidates, -inf elsewhere, with
  the floor f = 1e-6 for float32 arithmetic (the rule path, and the residual head on the
  vector units); with the residual head on the matrix cores f = 1e-5: its products take
  each float32 operand as a bf16 hi + lo pair, about 2^-18 relative, so a score carries
  an absolute error set by the size of the head's terms rather than by the score, which
  the residual can bring near zero (measured up to 3.5e-6 max|s_o| with one layer pair
  and one KV head, where the mean key rows are largest);
* kept sets: identical except at positions whose oracle score lies within
  1e-5 |tau_o| of the oracle threshold tau_o; the kept counts are identical;
* attention outputs: |o_gpu - o_o| <= 2e-3 plus half a bf16 ulp of o_o for bf16
  outputs (the output is rounded to bf16), 2e-3 for float32 outputs.
"""
import math

import numpy as np

SCORE_RTOL = 1e-3
SCORE_FLOOR = 1e-6
RESID_MFMA_FLOOR = 1e-5
BAND = 1e-5
ATTN_ATOL = 2e-3


def check_scores(s_gpu, s_o, cand, floor=SCORE_FLOOR):
    s_gpu = np.asarray(s_gpu, np.float64)
    assert np.all(np.isneginf(s_gpu[~cand])), "non-candidates must score -inf"
    if not cand.any():
        return 0.0
    a, o = s_gpu[cand], s_o[cand]
    tol = SCORE_RTOL * np.abs(o) + floor * np.abs(o).max()
    err = np.abs(a - o)
    bad = np.nonzero(err > tol)[0]
    assert len(bad) == 0, f"{len(bad)} scores out of tolerance, worst {err.max():.3e}"
    # error relative to the score, with scores near zero measured against 1e-3 of the largest
    return float((err / np.maximum(np.abs(o), 1e-3 * np.abs(o).max())).max())


def band_positions(s_o, tau_o, cand):
    if not math.isfinite(tau_o):
        return np.zeros_like(cand)
    return cand & (np.abs(s_o - tau_o) <= BAND * abs(tau_o))


def check_keep(keep_gpu, n_keep_gpu, keep_o, n_keep_o, s_o, tau_o, cand):
    keep_gpu = np.asarray(keep_gpu).astype(bool)
    assert n_keep_gpu == n_keep_o, f"kept count {n_keep_gpu} != {n_keep_o}"
    assert int(keep_gpu.sum()) == n_keep_o
    band = band_positions(s_o, tau_o, cand)
    diff = keep_gpu != keep_o
    outside = diff & ~band
    assert not outside.any(), f"{int(outside.sum())} kept-set differences outside the band"
    return int(diff.sum())


def bf16_half_ulp(x):
    ax = np.abs(np.asarray(x, np.float64))
    e = np.floor(np.log2(np.where(ax > 0, ax, 1.0)))
    return np.where(ax > 0, np.exp2(e - 8), 0.0)


def check_attention(o_gpu, o_o, bf16: bool):
    o_gpu = np.asarray(o_gpu, np.float64)
    tol = ATTN_ATOL + (bf16_half_ulp(o_o) if bf16 else 0.0)
    err = np.abs(o_gpu - o_o)
    assert np.all(err <= tol), f"attention error {err.max():.3e} above tolerance"
    return float(err.max())


def oracle_scores_pair(k_pool, S, st, M, Hkv, R, blob, qpos, dead):
    """Oracle scores with the residual head, with and without its cross-attention (the
    '- x-attn' ablation of Sec. 3.3), from one rule-score pass: the oracle's own steps
    (rule, key means, memory mean, residual) composed as oracle.scores composes them."""
    import oracle
    S = np.asarray(S)
    N = len(S)
    full = np.full(N, -np.inf)
    nox = full.copy()
    idx = np.nonzero(st["cand"])[0]
    if st["skip"] or len(idx) == 0:
        return full, nox
    D = k_pool.shape[-1]
    rule = oracle.rule_scores(k_pool, S, st["cand"], M, Hkv, R)
    qpos = np.asarray(qpos, np.int64)
    qlive = qpos[S[qpos] != dead] if len(qpos) else qpos
    kb, kq, mb = oracle.kbar(k_pool, S, idx), oracle.kbar(k_pool, S, qlive), oracle.mbar(M)
    full[idx] = oracle.residual_scores(rule[idx], kb, mb, kq, blob, D, xattn=True)
    nox[idx] = oracle.residual_scores(rule[idx], kb, mb, kq, blob, D, xattn=False)
    return full, nox


def check_xattn_visible(full, nox, st, factor=10.0, floor=RESID_MFMA_FLOOR):
    """The cross-attention term of Eq. 6 must matter at this size: dropping it moves some
    score by more than `factor` times the score tolerance (the one the scores are checked
    with) and changes the kept set. A kernel that dropped or garbled the term would then
    fail the score comparison."""
    import oracle
    c = st["cand"]
    a, b = full[c], nox[c]
    tol = SCORE_RTOL * np.abs(a) + floor * np.abs(a).max()
    ratio = float((np.abs(a - b) / tol).max())
    assert ratio > factor, f"cross-attention moves scores by only {ratio:.1f}x the tolerance"
    k1 = oracle.select_budget(full, st)[0]
    k2 = oracle.select_budget(nox, st)[0]
    nd = int((k1 != k2).sum())
    assert nd >= 1, "cross-attention changes no kept position"
    return ratio, nd


def check_decode_on(o_gpu, q, k_pool, v_pool, live, bf16: bool):
    """Decode output against the oracle's attention over the given live slot list (the
    GPU's own, which is a valid answer whenever the kept set is)."""
    import oracle
    return check_attention(o_gpu, oracle.decode(q, k_pool, v_pool, live), bf16)
