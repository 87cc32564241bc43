"""The oracle pins catch plausible mistakes.

Each case plants one mistake in a private copy of the oracle source (on the
CPU, never on a device), reruns every pin in ``test_oracle_pins`` against the
mutant and requires at least one pin to fail.
"""

import inspect
import os
import types

import pytest

import tests.test_oracle_pins as pins
from oracle import exfold_oracle

SRC = inspect.getsource(exfold_oracle)

MUTANTS = {
    "silu sign": ("z / (1.0 + np.exp(-z))", "z / (1.0 + np.exp(z))"),
    "gate/up swapped": ("return (silu(gate) * up)", "return (silu(up) * gate)"),
    "router bias dropped": ("r = r + _f64(bias)[None, :]", "r = r"),
    "top-k ties to higher id": ("order = np.lexsort((ids, -logits[i]", "order = np.lexsort((-ids, -logits[i]"),
    "softmax over all experts": ("z.sum(axis=1, keepdims=True))", "np.exp(_f64(logits) - r.max(axis=1, keepdims=True)).sum(axis=1, keepdims=True))"),
    "prefill score ignores h": ("score = [ww[i, j] * hh[ids[i, j]]", "score = [ww[i, j]"),
    "prefill ties to later route": ("key=lambda j: (-score[j], j))", "key=lambda j: (-score[j], -j))"),
    "min-loss keeps last minimum": ("if loss_row[t] < loss_row[best]:", "if loss_row[t] <= loss_row[best]:"),
    "min-loss takes maximum": ("if loss_row[t] < loss_row[best]:", "if loss_row[t] > loss_row[best]:"),
    "scale table transposed": ("ww[i, j] * float(S[s, t_exp])", "ww[i, j] * float(S[t_exp, s])"),
    "fold renormalises": ("out_w[i, c] = np.float32(acc[j])", "out_w[i, c] = np.float32(acc[j] / sum(acc.values()))"),
    "decode score ignores h": ("score = {e: float(acc[e]) * hh[e]", "score = {e: float(acc[e])"),
    "decode pool ties to higher id": ("order = sorted(cand, key=lambda e: (-score[e], e))", "order = sorted(cand, key=lambda e: (-score[e], -e))"),
    "decode scale not applied": ("scl[s] = S[s, t]", "scl[s] = 1.0"),
    "pool members remapped": ("        if s in in_pool:\n            continue\n        t = min_loss_target", "        t = min_loss_target"),
    "permutation not stable": ("for j, e in enumerate(flat):\n        row_slot[cursor[e]] = j",
                               "for j, e in reversed(list(enumerate(flat))):\n        row_slot[cursor[e]] = j"),
    "shared expert dropped": ("y += expert_forward(x, layer.ws_gate_up, layer.ws_down)\n    return y\n\n\ndef folded",
                              "pass\n    return y\n\n\ndef folded"),
    "calibration weight is target norm": ("wi = math.sqrt(float(u @ u))", "wi = math.sqrt(float(U[[t for t in ev if t != s][0]] @ U[[t for t in ev if t != s][0]]))"),
    "ridge term in numerator": ("sc = A[s, t] / den", "sc = (A[s, t] + lam) / den"),
    "loss uses unclipped scalar": ("resid = C[s, t] - 2.0 * sc * A[s, t] + sc * sc * V[s, t]",
                                   "u_sc = A[s, t] / den\n            resid = C[s, t] - 2.0 * u_sc * A[s, t] + u_sc * u_sc * V[s, t]"),
    "loss sign error": ("- 2.0 * sc * A[s, t]", "+ 2.0 * sc * A[s, t]"),
    "unobserved loss zero": ("Lo = np.full((nn, nn), UNOBSERVED_LOSS)", "Lo = np.full((nn, nn), 0.0)"),
    "self scalar zero": ("S[s, t], Lo[s, t] = 1.0, 0.0", "S[s, t], Lo[s, t] = 0.0, 0.0"),
    "h is max norm": ("h[observed] = norm_sum[observed] / norm_cnt[observed]", "h[observed] = norm_sum[observed]"),
    "storage counts one table": ("return n_layers * n_experts * n_experts * 4 * 2", "return n_layers * n_experts * n_experts * 4"),
    "loss cap exclusive": ("float(L[s, ids[i, q]]) <= loss_cap]", "float(L[s, ids[i, q]]) < loss_cap]"),
    "capped route spread instead of dropped": ("                continue                                    # no admissible target: dropped",
                                              "                cands = ret"),
    "confidence not clipped": ("c = min(1.0, max(0.0, 1.0 - float(L[s, ids[i, q_t]])))", "c = 1.0 - float(L[s, ids[i, q_t]])"),
    "confidence spread uniform": ("acc[q] = acc[q] + rest * (ww[i, q] / w_ret)", "acc[q] = acc[q] + rest / len(ret)"),
    "confidence remainder to target": ("acc[q] = acc[q] + rest * (ww[i, q] / w_ret)", "acc[q_t] = acc[q_t] + rest * (ww[i, q] / w_ret)"),
    "diagonal numerator uses target energy": ("A[s, t] += wi * (v * u)", "A[s, t] += wi * (v * v)"),
    "diagonal ridge dropped": ("            den = V[s, t] + lam\n            dv =", "            den = V[s, t]\n            dv ="),
    "diagonal loss sign": ("resid = C[s, t] - 2.0 * float(dv @ A[s, t])", "resid = C[s, t] + 2.0 * float(dv @ A[s, t])"),
    "diagonal weight is target norm": ("            u = outputs[s][i]\n            wi = math.sqrt(float(u @ u))",
                                       "            u = outputs[s][i]\n            wi = math.sqrt(float(outputs[ev[-1]][i] @ outputs[ev[-1]][i]))"),
    "diagonal output ignores folds": ("coef = coef + ws * Dg[s, e]", "coef = coef"),
    "diagonal map of the source expert": ("coef = coef + ws * Dg[s, e]", "coef = coef + ws * Dg[e, s]"),
    "renorm to retained router sum": ("            for j in range(k):\n                w_all += ww[i, j]", "            for j in ret:\n                w_all += ww[i, j]"),
}


def _pin_functions():
    fns = []
    for name, fn in inspect.getmembers(pins, inspect.isfunction):
        if not name.startswith("test_"):
            continue
        marks = getattr(fn, "pytestmark", [])
        params = [m for m in marks if m.name == "parametrize"]
        if params:
            argname, values = params[0].args
            for v in values:
                fns.append((f"{name}[{v}]", lambda fn=fn, a=argname, v=v: fn(**{a: v})))
        else:
            fns.append((name, fn))
    return fns


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_pins_catch_mutant(mutant, monkeypatch):
    old, new = MUTANTS[mutant]
    assert SRC.count(old) >= 1, f"mutation site not found: {old!r}"
    mod = types.ModuleType("oracle_mutant")
    mod.__file__ = exfold_oracle.__file__
    exec(compile(SRC.replace(old, new, 1), "oracle_mutant", "exec"), mod.__dict__)
    monkeypatch.setattr(pins, "O", mod)
    caught = []
    for name, fn in _pin_functions():
        try:
            fn()
        except Exception:           # assertion, shape or value error: the mutant is caught
            caught.append(name)
    assert caught, f"no pin fails for mutant '{mutant}'"
