"""Mutation check of the oracle pins.

Each plant is a plausible mistake in the float64 oracle (a dropped term, a wrong sign
or index, a transposed operand): one textual edit of the oracle's source, executed
as a fresh module whose functions replace the oracle's while the pins of
tests/test_oracle_pins.py run. Every plant must make at least one pin fail, and
without a plant every pin passes. Plants live here, on the CPU, and touch nothing
outside the oracle.
"""
import inspect
import itertools
import types

import pytest

import oracle
import oracle.ikv_oracle as ko
import test_oracle_pins as pins

# (name, text in the oracle's source, replacement); the text must occur exactly once.
PLANTS = [
    # ---- residual head, Eqs. 4-6
    ("drop b_Q", 'Qc = phi @ W["W_Q"].T + W["b_Q"]', 'Qc = phi @ W["W_Q"].T'),
    ("drop b_V", 'Vp = kq @ W["W_V"].T + W["b_V"]', 'Vp = kq @ W["W_V"].T'),
    ("drop b_1", 'W["W_1"].T + W["b_1"])', 'W["W_1"].T)'),
    ("drop b_2", 'y = hidden @ W["w_2"] + W["b_2"][0]', 'y = hidden @ W["w_2"]'),
    ("scale W_Q phi", "c = cross_attention(Qc, kq, W) if xattn", "c = cross_attention(0.5 * Qc, kq, W) if xattn"),
    ("mis-slice W_Q phi", 'Qc = phi @ W["W_Q"].T', 'Qc = np.roll(phi, 1, axis=1) @ W["W_Q"].T'),
    ("swap W_K and W_V", 'Kp = kq @ W["W_K"].T + W["b_K"]\n    Vp = kq @ W["W_V"].T + W["b_V"]',
     'Kp = kq @ W["W_V"].T + W["b_K"]\n    Vp = kq @ W["W_K"].T + W["b_V"]'),
    ("cross-attention scale 1/sqrt(D_C)", "X = Qc[:, sl] @ Kp[:, sl].T / math.sqrt(dh)",
     "X = Qc[:, sl] @ Kp[:, sl].T / math.sqrt(D_C)"),
    ("cross-attention softmax over the candidates", "P = P / P.sum(axis=1, keepdims=True)\n        c[:, sl]",
     "P = P / P.sum(axis=0, keepdims=True)\n        c[:, sl]"),
    ("dead query positions read", "qlive = qpos[np.asarray(S)[qpos] != dead] if len(qpos) else qpos",
     "qlive = qpos"),
    ("no alpha clip", "alpha = min(max(W[\"alpha\"][0], -ALPHA_CLIP), ALPHA_CLIP)", "alpha = W[\"alpha\"][0]"),
    ("tanh GELU", "return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))",
     "return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x ** 3)))"),
    ("[c ; phi] order", "np.concatenate([phi, c], axis=1)", "np.concatenate([c, phi], axis=1)"),
    ("phi without the product", "kb * mb[None, :], rule[:, None]", "kb, rule[:, None]"),
    ("k-bar a sum", "return acc / (L * Hkv)", "return acc / L"),
    ("m-bar over channels", "return M.reshape(-1, M.shape[-1]).mean(axis=0)",
     "return M.reshape(-1, M.shape[-1]).mean(axis=1)[:M.shape[-1]]"),
    # ---- rule score, Eq. 3
    ("rule without 1/sqrt(D)", "X = M[l, h * R:(h + 1) * R] @ Kl[:, h, :].T / math.sqrt(D)   # [R][|A|]",
     "X = M[l, h * R:(h + 1) * R] @ Kl[:, h, :].T   # [R][|A|]"),
    ("rule rows interleaved", "X = M[l, h * R:(h + 1) * R] @ Kl[:, h, :].T / math.sqrt(D)   # [R][|A|]",
     "X = M[l, h::Hkv] @ Kl[:, h, :].T / math.sqrt(D)   # [R][|A|]"),
    ("rule softmax over positions of every row", "P = P / P.sum(axis=1, keepdims=True)\n            rule",
     "P = P / P.sum()\n            rule"),
    ("forced positions are candidates", "cand = live & ~forced", "cand = live"),
    # ---- QueryMemory, Eq. 2
    ("no unit-norm projection", "return M / np.maximum(norm, NORM_EPS)", "return M"),
    ("decay on Enc", "M = decay * M_prev + enc", "M = M_prev + decay * enc"),
    ("Enc a sum", "enc = q.mean(axis=-2)", "enc = q.sum(axis=-2)"),
    # ---- selection, Eq. 1
    ("ties to the higher position", "order = np.lexsort((idx, -key))", "order = np.lexsort((-idx, -key))"),
    ("budget ignores the forced set", '"Cstar": max(0, C - int(forced.sum()))', '"Cstar": C'),
    ("NaN ranked first", "key = np.where(np.isnan(key), -np.inf, key)", "key = np.where(np.isnan(key), np.inf, key)"),
    ("gate on the live count", '"skip": N <= C', '"skip": int(live.sum()) <= C'),
    # ---- redirect and free, Eq. 7 and Sec. 3.4
    ("aliased slots freed", "if j >= radix_prefix and u != dead and u not in kept_slots:",
     "if j >= radix_prefix and u != dead:"),
    ("radix prefix off by one", "if j >= radix_prefix and u != dead and u not in kept_slots:",
     "if j > radix_prefix and u != dead and u not in kept_slots:"),
    ("live list in slot order", "live_list = S_new[S_new != dead]", "live_list = np.sort(S_new[S_new != dead])"),
    # ---- decode
    ("decode GQA head mapping", "            g = h // G\n            x = Kl", "            g = h % Hkv\n            x = Kl"),
    ("decode without 1/sqrt(D)", "x = Kl[:, g, :] @ q[l, h] / math.sqrt(D)", "x = Kl[:, g, :] @ q[l, h]"),
    # ---- baseline scorers on the substrate (Sec. 4.1)
    ("attention mass GQA head mapping", "            g = h // G\n            X = q[l, h]",
     "            g = h % Hkv\n            X = q[l, h]"),
    ("attention mass without 1/sqrt(D)", "X = q[l, h] @ Kl[:, g, :].T / math.sqrt(D)", "X = q[l, h] @ Kl[:, g, :].T"),
    ("SnapKV pooling after the unit sum", "out = max_pool(v, kernel).sum(axis=(0, 1))",
     "out = max_pool(v.sum(axis=(0, 1)), kernel)"),
    ("pool window one too wide", "    r = kernel // 2\n", "    r = kernel // 2 + 1\n"),
    ("recent window rounded down", "w = min(N, int(math.ceil(recent_ratio * C)))", "w = min(N, int(recent_ratio * C))"),
    # ---- compact apply path (Sec. 3.4, Table 7)
    ("re-rotation sign", "Kn[:, t] = rope_rotate(widen(k_pool[:, S[j]]), t - int(j), base, D)",
     "Kn[:, t] = rope_rotate(widen(k_pool[:, S[j]]), int(j) - t, base, D)"),
    ("rotation frequencies over D/2", "ang = float(delta) * base ** (-2.0 * np.arange(h) / D)",
     "ang = float(delta) * base ** (-2.0 * np.arange(h) / h)"),
    ("prefill not causal", "slots = np.concatenate([hist, span[:t + 1]])", "slots = np.concatenate([hist, span])"),
    ("prefill excludes its own key", "slots = np.concatenate([hist, span[:t + 1]])",
     "slots = np.concatenate([hist, span[:t]])"),
    ("rotate-half pairing", "return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)\n\n\ndef compact",
     "return np.concatenate([x1 * c + x2 * s, x2 * c - x1 * s], axis=-1)\n\n\ndef compact"),
]


def _pin_cases():
    """Every pin of test_oracle_pins.py as (name, zero-argument callable), with the
    parametrized ones expanded."""
    cases = []
    for name, fn in inspect.getmembers(pins, inspect.isfunction):
        if not name.startswith("test_") or fn.__module__ != pins.__name__:
            continue
        marks = [m for m in getattr(fn, "pytestmark", []) if m.name == "parametrize"]
        if not marks:
            cases.append((name, fn))
            continue
        grids = []
        for m in marks:
            argnames = [a.strip() for a in m.args[0].split(",")] if isinstance(m.args[0], str) else list(m.args[0])
            rows = [v if len(argnames) > 1 else (v,) for v in m.args[1]]
            grids.append([dict(zip(argnames, r)) for r in rows])
        for combo in itertools.product(*grids):
            kw = {k: v for d in combo for k, v in d.items()}
            cases.append((f"{name}{kw}", lambda fn=fn, kw=kw: fn(**kw)))
    return cases


def _failing_pins():
    failed = []
    for name, run in _pin_cases():
        try:
            run()
        except Exception:                        # an assertion, or a mistake that breaks the arithmetic
            failed.append(name)
    return failed


def _swap_in(monkeypatch, src):
    mod = types.ModuleType("ikv_oracle_planted")
    mod.__dict__["__name__"] = "ikv_oracle_planted"
    exec(compile(src, ko.__file__, "exec"), mod.__dict__)
    for name, obj in mod.__dict__.items():
        if inspect.isfunction(obj):
            monkeypatch.setattr(ko, name, obj)
            if hasattr(oracle, name):
                monkeypatch.setattr(oracle, name, obj)


def test_pins_pass_without_a_plant():
    assert _failing_pins() == []


@pytest.mark.parametrize("name,old,new", PLANTS, ids=[p[0] for p in PLANTS])
def test_every_plant_fails_a_pin(monkeypatch, name, old, new):
    src = inspect.getsource(ko)
    assert src.count(old) == 1, f"plant '{name}': its text occurs {src.count(old)} times in the oracle"
    _swap_in(monkeypatch, src.replace(old, new))
    failed = _failing_pins()
    assert failed, f"plant '{name}' passed every pin"
