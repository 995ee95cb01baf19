"""A multi-turn agent session on the Qwen3-8B shape (8 turns, 4096 -> 49,152 positions),
driven turn by turn through the five calls and, in lockstep, through the oracle.

Each turn appends a tool output and a query (their K/V rows written at slots taken
first from the slots freed so far, oldest first, then from unused ones), updates the
QueryMemory from the query span (R = G = 4 memory rows per KV head, lambda = 0.5,
starting from zero), and when N > C scores (residual head on), selects and redirects
with the system prefix of 64 positions radix-protected; then it decodes over the live
slots. After every turn the GPU's kept set must match the oracle's outside the
selection band; both sides then continue from the GPU's decision, so the slot maps,
freed and live lists are compared exactly turn after turn. The residual head's weights
make its cross-attention move every turn's scores and kept set visibly (checked on the
oracle), so a kernel that dropped or garbled it would fail the comparison."""
from collections import deque

import numpy as np
import pytest

import oracle
import synth
from paper_2606_09916_amd import ikv
from parity import (RESID_MFMA_FLOOR, check_attention, check_keep, check_scores, check_xattn_visible,
                    oracle_scores_pair)

pytestmark = pytest.mark.gpu
DEAD = synth.DEAD_SLOT
SEED = 4


def _t(a, dev, torch):
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
    return torch.from_numpy(a).to(dev)


def test_multi_turn_session(dev):
    import torch
    shape = synth.qwen3_8b_shape()
    L, Hq, Hkv, D = shape.L, shape.Hq, shape.Hkv, shape.D
    R = Hq // Hkv
    C, pi = 8192, 64
    plan = synth.multi_turn_plan(SEED)
    total = sum(a + q for a, q in plan)
    num_slots = 1 + total
    k_host = np.zeros((L, num_slots, Hkv, D), np.uint16)
    v_host = np.zeros((L, num_slots, Hkv, D), np.uint16)
    k_dev = torch.zeros((L, num_slots, Hkv, D), dtype=torch.bfloat16, device=dev)
    v_dev = torch.zeros_like(k_dev)
    pool = ikv.make_pool(k_dev, v_dev, L, Hq, Hkv, D, num_slots, DEAD)
    ikv.init_dead_slot(pool)
    blob = synth.residual_blob(D, seed=24, variant="scaled", units=L * Hkv, out_std=5e-3)
    blob_dev = torch.from_numpy(blob).to(dev)
    ws = ikv.Workspace(dev)
    M_dev = torch.zeros(L * Hkv * R * D, dtype=torch.float32, device=dev)
    M_o = np.zeros((L, Hkv * R, D))
    S = np.zeros(0, np.int32)
    free, fresh = deque(), 1
    compressed = 0
    for t, (n_tool, n_q) in enumerate(plan):
        N0 = len(S)
        N = N0 + n_tool + n_q
        new = []
        for _ in range(N - N0):
            if free:
                new.append(free.popleft())
            else:
                new.append(fresh)
                fresh += 1
        new = np.asarray(new, np.int64)
        k_rows, v_rows = synth.turn_kv_rows(SEED, t, N0, N - N0, shape)
        k_host[:, new] = k_rows
        v_host[:, new] = v_rows
        idx = torch.from_numpy(new).to(dev)
        k_dev[:, idx] = _t(k_rows, dev, torch)
        v_dev[:, idx] = _t(v_rows, dev, torch)
        S = np.concatenate([S, new.astype(np.int32)])
        qpos = np.arange(N - n_q, N, dtype=np.int32)
        sess = ikv.Sessions([dict(slot_off=0, mem_off=0, qspan_off=0, qpos_off=0, N=N, pi=pi, qs=N - n_q, qe=N,
                                  C=C, radix_prefix=pi, R=R, nq=n_q)], dev)

        # QueryMemory update from the span
        span = synth.turn_span_rows(SEED, t, qpos, shape, R)
        ikv.qm_update(pool, sess, M_dev, _t(span, dev, torch), 0.5)
        M_o = oracle.qm_update(M_o, synth.widen(span), 0.5)
        np.testing.assert_allclose(M_dev.cpu().numpy().reshape(M_o.shape), M_o, atol=1e-5, rtol=0)

        S_dev = torch.from_numpy(S).to(dev)
        sets = oracle.sets(S, pi, N - n_q, N, C, DEAD)
        if not sets["skip"]:
            compressed += 1
            scores = torch.empty(N, dtype=torch.float32, device=dev)
            keep = torch.empty(N, dtype=torch.uint8, device=dev)
            n_keep = torch.empty(1, dtype=torch.int32, device=dev)
            tau = torch.empty(1, dtype=torch.float32, device=dev)
            ikv.score_history(pool, sess, S_dev, M_dev, scores, ws, qpos=torch.from_numpy(qpos).to(dev),
                              residual=blob_dev, flags=ikv.IKV_RESIDUAL)
            ikv.select_budget(sess, S_dev, DEAD, scores, keep, n_keep, tau, ws)
            want, nox = oracle_scores_pair(k_host, S, sets, M_o, Hkv, R, blob, qpos, DEAD)
            ratio, nd = check_xattn_visible(want, nox, sets)
            check_scores(scores.cpu().numpy(), want, sets["cand"], floor=RESID_MFMA_FLOOR)
            keep_o, n_o, tau_o = oracle.select_budget(want, sets)
            keep_g = keep.cpu().numpy().astype(bool)
            ndiff = check_keep(keep_g, int(n_keep.item()), keep_o, n_o, want, tau_o, sets["cand"])
            print(f"turn {t}: N = {N}, live = {int(sets['live'].sum())}, kept = {n_o}, band differences = {ndiff}, "
                  f"cross-attention {ratio:.0f}x tolerance / {nd} kept positions")

            # redirect from the GPU's kept set, on both sides
            freed = torch.empty(N, dtype=torch.int32, device=dev)
            live = torch.empty(N, dtype=torch.int32, device=dev)
            n_freed = torch.empty(1, dtype=torch.int32, device=dev)
            n_live = torch.empty(1, dtype=torch.int32, device=dev)
            ikv.redirect_slots(sess, num_slots, S_dev, DEAD, keep, freed, n_freed, live, n_live, ws)
            S_o, freed_o, live_o = oracle.redirect(S, keep_g, DEAD, pi)
            S_g = S_dev.cpu().numpy()
            assert np.array_equal(S_g, S_o)
            nf, nl = int(n_freed.item()), int(n_live.item())
            assert np.array_equal(freed.cpu().numpy()[:nf], freed_o)
            assert np.array_equal(live.cpu().numpy()[:nl], live_o)
            assert np.all(S_g[:pi] == S[:pi])                     # the radix prefix is never dropped
            S = S_g
            free.extend(int(u) for u in freed_o)
        else:
            live_o = S[S != DEAD]
            live = torch.from_numpy(live_o.astype(np.int32)).to(dev)
            n_live = torch.tensor([len(live_o)], dtype=torch.int32, device=dev)
            print(f"turn {t}: N = {N} <= C, nothing evicted")

        # decode over the live slots
        q = synth.turn_decode_query(SEED, t, N, shape)
        out = torch.empty((1, L, Hq, D), dtype=torch.bfloat16, device=dev)
        ikv.decode_attend_slotmap(pool, sess, _t(q[None], dev, torch), live, n_live, out, ws)
        o_g = synth.widen(out.view(torch.int16).cpu().numpy().view(np.uint16)[0])
        o_o = oracle.decode(synth.widen(q), k_host, v_host, live_o)
        check_attention(o_g, o_o, bf16=True)
    assert compressed == len(plan) - 1                            # every turn after the first compresses
    assert len(S) == total
