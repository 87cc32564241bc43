"""Plain CPU oracle for the ExFold folded mixture-of-experts layer.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code, header,
helper, table or constant generator with the HIP library, and it imports
nothing from the package.

Every function follows one passage of the paper (arXiv 2608.24938, "ExFold:
Unified Expert Folding for Training-Free MoE Prefill-Decode Acceleration"),
cited by section and equation label.  The code is written to be checked by
eye, not to be fast.

Conventions
-----------
* Floating point arithmetic is float64.  Inputs arrive as float32 arrays
  (bf16 data is widened to float32 first, which is exact) and are widened
  exactly to float64.
* Route metadata (Top-K ids, gate weights, folded ids and weights, the decode
  target/scale tables) uses the metadata format of the layer: int32 ids and
  float32 weights.  Each metadata weight is rounded once, round-to-nearest-
  even, from its float64 value.  Every discrete decision (Top-K, retained
  set, pool, minimum-loss target) is taken on those stored float32 values,
  with exact float64 products, so it is the same decision the device takes.
* Readings of the paper where it is silent are listed in ``READINGS`` below;
  each is applied here and by the device library alike.

Parity pins
-----------
Every function is pinned by ``tests/test_oracle_pins.py`` against something
other than itself (closed forms, brute force on tiny inputs, special cases
that reduce to textbook operations, invariants the paper states, and the
storage figure that the projector ablation table prints).  No function here
is "parity unpinned".
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

# Readings of passages the paper leaves open (applied by both sides).
READINGS = {
    "R1": "Router: softmax over the Top-K logits (Sec. 2.1, Eq. topk_gate) for every layer; "
          "an optional per-expert bias is added to the logits before Top-K.",
    "R2": "Top-K order: logit descending, expert id ascending on equal logits.",
    "R3": "h_e: mean of ||E_e(x)||_2 over the calibration tokens on which E_e was evaluated; "
          "an expert never evaluated gets the mean of the observed h.",
    "R4": "Prefill score w*h is the exact float64 product of two float32 values; "
          "ties keep the smaller route position.",
    "R5": "Retained prefill routes keep their original route order.",
    "R6": "Decode pool score: W_e = sum over slots of rint(w * 2^40) (exact integer), "
          "score_e = fl64(W_e * h_e).",
    "R7": "Pool candidates are experts with >= 1 routed slot; ties to the lower id; "
          "pool order is (score desc, id asc); |pool| = min(D, |candidates|).",
    "R8": "Minimum-loss target: first minimum in canonical order (route order in prefill, "
          "pool order in decode), strict '<'.",
    "R9": "Scalar of an unobserved pair is 0 (Eq. scalar_projector with empty sums).",
    "R10": "The loss of a pair uses the clipped scalar.",
    "R11": "epsilon in the normalised loss is 1e-12.",
    "R12": "Calibration weight w_i = ||u_i||_2 (source output norm), per (token, source).",
    "R13": "Decode keeps the [B,K] layout; duplicate ids after remapping are executed twice.",
    "R14": "Decode remapped weight: one float32 multiply w*S (retained slots copied).",
    "R15": "Shared expert: weight 1, added to every token, never selected or folded.",
    "R22": "Loss-cap safeguard: pairs with L > cap are not candidate targets; an omitted "
           "route without a candidate is dropped.",
    "R23": "Confidence split: c_s = clip(1 - min L[s, t], 0, 1) with L as the source-relative "
           "residual; the remainder w_s (1 - c_s) goes to the retained routes in proportion "
           "to their router weights.",
    "R24": "Renormalisation: retained weights scaled by (sum of the K router weights) / "
           "(sum of the folded weights) when that sum is positive.",
    "R26": "Diagonal projectors: no clipping; unobserved pair d = 0, loss 1e30; self pair d = 1, "
           "loss 0; a zero denominator gives d_n = 0.",
}

FIXED_POINT_BITS = 40       # R6
UNOBSERVED_LOSS = 1e30      # Appendix A, calibration protocol
DEFAULT_LAMBDA = 1e-3       # Sec. 5.1 hyperparameters; Appendix A
DEFAULT_CLIP = 4.0          # Appendix A: scalars clipped to [-4, 4]
EPSILON = 1e-12             # R11


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


def _meta_w(a) -> np.ndarray:
    """Round float64 gate weights to the float32 metadata format (RNE)."""
    return np.asarray(a, dtype=np.float64).astype(np.float32)


# ---------------------------------------------------------------------------
# Experts and router  (Sec. 2.1, Eq. gated_expert, Eq. topk_gate, Eq. moe_output)
# ---------------------------------------------------------------------------

def silu(z: np.ndarray) -> np.ndarray:
    """phi(z) = z / (1 + exp(-z)), the SiLU named after Eq. gated_expert."""
    z = _f64(z)
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def expert_forward(x, w_gate_up, w_down) -> np.ndarray:
    """E_e(x) = W_down (phi(W_gate x) * W_up x)   (Sec. 2.1, Eq. gated_expert).

    x: [T, d].  w_gate_up: [2I, d], rows 0..I-1 are W_gate, rows I..2I-1 are
    W_up.  w_down: [d, I].  Returns float64 [T, d].
    """
    x = _f64(x)
    wgu = _f64(w_gate_up)
    inter = wgu.shape[0] // 2
    gate = x @ wgu[:inter].T
    up = x @ wgu[inter:].T
    return (silu(gate) * up) @ _f64(w_down).T


def router_logits(x, w_router, bias=None) -> np.ndarray:
    """r(x) = W_r x (+ per-expert bias, reading R1)   (Sec. 2.1, before Eq. topk_gate)."""
    r = _f64(x) @ _f64(w_router).T
    if bias is not None:
        r = r + _f64(bias)[None, :]
    return r


def topk_ids(logits, top_k: int) -> np.ndarray:
    """S_K(x): the K largest logits, ordered (logit desc, id asc)   (Eq. topk_gate, R2).

    The comparison is made on the logits exactly as given (float32 logits from
    the device are compared as float32 values).
    """
    logits = np.asarray(logits)
    t, n = logits.shape
    out = np.empty((t, top_k), dtype=np.int32)
    ids = np.arange(n)
    for i in range(t):
        # lexsort: last key is primary -> descending logit, then ascending id
        order = np.lexsort((ids, -logits[i].astype(np.float64)))
        out[i] = order[:top_k]
    return out


def topk_softmax(logits, ids) -> np.ndarray:
    """alpha_e = exp(r_e) / sum_{j in S_K} exp(r_j) for e in S_K   (Eq. topk_gate).

    Evaluated in float64 with the maximum subtracted; returned in the float32
    metadata format.
    """
    r = np.take_along_axis(_f64(np.asarray(logits)), ids.astype(np.int64), axis=1)
    z = np.exp(r - r.max(axis=1, keepdims=True))
    return _meta_w(z / z.sum(axis=1, keepdims=True))


def route(logits, top_k: int):
    """Top-K routes and renormalised gate weights from router logits."""
    ids = topk_ids(logits, top_k)
    return ids, topk_softmax(logits, ids)


# ---------------------------------------------------------------------------
# Phase-specific selection  (Sec. 4.3 step 1; Appendix B.1, Eq. A6-A8)
# ---------------------------------------------------------------------------

def select_prefill(ids, w, h, k_pre: int) -> np.ndarray:
    """B_pre(x_i) = TopK_{e in S_K(x_i)}(w_{i,e} h_e, K_pre)   (Eq. prefill_budget).

    Returns keep[T, K] (bool): True for retained routes.  Scores are exact
    float64 products (R4); equal scores keep the smaller route position.
    K_pre >= K retains every route.
    """
    ids = np.asarray(ids)
    t, k = ids.shape
    keep = np.zeros((t, k), dtype=bool)
    if k_pre >= k:
        keep[:] = True
        return keep
    hh = _f64(h)
    ww = _f64(w)
    for i in range(t):
        score = [ww[i, j] * hh[ids[i, j]] for j in range(k)]
        order = sorted(range(k), key=lambda j: (-score[j], j))
        for j in order[:k_pre]:
            keep[i, j] = True
    return keep


def select_decode_pool(ids, w, h, n_experts: int, budget_d: int):
    """B_dec(X_q) = TopK_{e in union S_K}(sum_i w_{i,e} h_e, D)   (Eq. decode_budget).

    Reading R6: sum_i w_{i,e} is accumulated exactly as the integer
    W_e = sum rint(w * 2^40); score_e = fl64(W_e * h_e).  Candidates are the
    experts with at least one routed slot (R7).  Returns the pool (list of
    expert ids in (score desc, id asc) order, length min(D, |candidates|))
    and the candidate list.
    """
    ids = np.asarray(ids).reshape(-1)
    ww = _f64(w).reshape(-1)
    acc = [0] * n_experts
    cnt = [0] * n_experts
    scale = float(2 ** FIXED_POINT_BITS)
    for e, wv in zip(ids.tolist(), ww.tolist()):
        acc[e] += int(np.rint(wv * scale))
        cnt[e] += 1
    cand = [e for e in range(n_experts) if cnt[e] > 0]
    hh = [float(v) for v in _f64(h)]
    score = {e: float(acc[e]) * hh[e] for e in cand}
    order = sorted(cand, key=lambda e: (-score[e], e))
    return order[: min(budget_d, len(cand))], cand


def select_static_pool(h, budget_d: int):
    """B_dec^static = TopK_{e in 1..E}(h_e, D)   (Appendix B.1, Eq. A8); ties to the lower id."""
    hh = _f64(h)
    order = sorted(range(len(hh)), key=lambda e: (-hh[e], e))
    return order[: min(budget_d, len(hh))]


# ---------------------------------------------------------------------------
# Minimum-loss transfer and folding  (Sec. 4.3 steps 2-3; Eq. A9-A11)
# ---------------------------------------------------------------------------

def min_loss_target(loss_row, retained) -> int:
    """pi(s | B) = argmin_{t in B} l_{s->t}   (Eq. minimum_loss_assignment, R8).

    ``retained`` is the candidate set in canonical order; the first minimum
    wins (strict '<').
    """
    best = retained[0]
    for t in retained[1:]:
        if loss_row[t] < loss_row[best]:
            best = t
    return best


def fold_prefill(ids, w, keep, S, L):
    """Prefill fold: retained routes first, omitted routes coalesced   (Eq. prefill_fold, Eq. A10).

    w~_{i,t} = w_{i,t} + sum_{s omitted, pi(s)=t} w_{i,s} S_{s->t}, for t in B_pre.
    Omitted routes are visited in route order; the sum is float64 (each
    product of two float32 values is exact) and rounded once to float32.
    Returns (out_ids [T, K_out] int32, out_w [T, K_out] float32) with the
    retained routes in route order (R5); K_out = number retained per token.
    """
    ids = np.asarray(ids)
    t, k = ids.shape
    k_out = int(np.asarray(keep)[0].sum()) if t else 0
    out_ids = np.zeros((t, k_out), dtype=np.int32)
    out_w = np.zeros((t, k_out), dtype=np.float32)
    S = np.asarray(S, dtype=np.float32)
    L = np.asarray(L, dtype=np.float32)
    ww = _f64(w)
    for i in range(t):
        ret = [j for j in range(k) if keep[i, j]]
        assert len(ret) == k_out
        acc = {j: ww[i, j] for j in ret}
        ret_experts = [int(ids[i, j]) for j in ret]
        for j in range(k):
            if keep[i, j]:
                continue
            s = int(ids[i, j])
            t_exp = min_loss_target(L[s], ret_experts)
            j_t = ret[ret_experts.index(t_exp)]
            acc[j_t] = acc[j_t] + ww[i, j] * float(S[s, t_exp])
        for c, j in enumerate(ret):
            out_ids[i, c] = ids[i, j]
            out_w[i, c] = np.float32(acc[j])
    return out_ids, out_w


def fold_prefill_safeguarded(ids, w, keep, S, L, loss_cap=None, renorm: bool = False,
                             confidence: bool = False):
    """Prefill fold with the safeguards of the cross-model and DeepSeek-V4
    configurations (Appendix C; Appendix F, Eq. dsv4_confidence).

    * loss_cap: a directed pair (s, t) with L[s, t] > loss_cap is not a
      candidate target; an omitted route with no candidate is dropped (R22).
    * confidence: c_s = clip(1 - min over candidates of L[s, t], 0, 1); the
      minimum-loss target t* receives w_s c_s S[s, t*] and the remainder
      w_s (1 - c_s) is spread over the retained routes in proportion to their
      router weights, w_t / sum of retained w (R23; L is the source-relative
      residual of Eq. dsv4_confidence).
    * renorm: after folding, the retained weights are scaled by
      (sum of all K router weights) / (sum of the folded weights), when that
      sum is positive (R24).

    Arithmetic is float64 in this order, every product and sum rounded once
    (no fused multiply-add): for each retained route t (route order),
    acc_t = w_t, then for each omitted route s (route order) acc_t += (w_s c_s)
    S[s, t] if t is its target, then acc_t += (w_s (1 - c_s)) (w_t / W_ret);
    finally acc_t * (W_all / sum acc) when renormalising; one rounding to float32.
    Without safeguards the result equals ``fold_prefill``.
    """
    ids = np.asarray(ids)
    t, k = ids.shape
    k_out = int(np.asarray(keep)[0].sum()) if t else 0
    out_ids = np.zeros((t, k_out), dtype=np.int32)
    out_w = np.zeros((t, k_out), dtype=np.float32)
    S = np.asarray(S, dtype=np.float32)
    L = np.asarray(L, dtype=np.float32)
    ww = _f64(w)
    for i in range(t):
        ret = [j for j in range(k) if keep[i, j]]
        assert len(ret) == k_out
        acc = {j: ww[i, j] for j in ret}
        w_ret = 0.0
        for j in ret:
            w_ret += ww[i, j]
        for j in range(k):
            if keep[i, j]:
                continue
            s = int(ids[i, j])
            cands = [q for q in ret if loss_cap is None or float(L[s, ids[i, q]]) <= loss_cap]
            if not cands:
                continue                                    # no admissible target: dropped
            q_t = cands[0]
            for q in cands[1:]:                             # first minimum in route order
                if L[s, ids[i, q]] < L[s, ids[i, q_t]]:
                    q_t = q
            c = 1.0
            if confidence:
                c = min(1.0, max(0.0, 1.0 - float(L[s, ids[i, q_t]])))
            acc[q_t] = acc[q_t] + (ww[i, j] * c) * float(S[s, ids[i, q_t]])
            if confidence:
                rest = ww[i, j] * (1.0 - c)
                for q in ret:
                    acc[q] = acc[q] + rest * (ww[i, q] / w_ret)
        if renorm:
            w_all = 0.0
            for j in range(k):
                w_all += ww[i, j]
            tot = 0.0
            for j in ret:
                tot += acc[j]
            if tot > 0.0:
                f = w_all / tot
                for j in ret:
                    acc[j] = acc[j] * f
        for c_, j in enumerate(ret):
            out_ids[i, c_] = ids[i, j]
            out_w[i, c_] = np.float32(acc[j])
    return out_ids, out_w


def decode_tables(pool, S, L, n_experts: int):
    """Per-source target and scale for a decode pool   (Eq. A9; Appendix B.1 decode kernels).

    For s in the pool: target s, scale 1.  Otherwise target
    pi(s | B_dec) (first minimum over pool order) and scale S_{s->pi(s)}.
    """
    S = np.asarray(S, dtype=np.float32)
    L = np.asarray(L, dtype=np.float32)
    tgt = np.arange(n_experts, dtype=np.int32)
    scl = np.ones(n_experts, dtype=np.float32)
    in_pool = set(int(p) for p in pool)
    if not pool:
        return tgt, scl
    for s in range(n_experts):
        if s in in_pool:
            continue
        t = min_loss_target(L[s], [int(p) for p in pool])
        tgt[s] = t
        scl[s] = S[s, t]
    return tgt, scl


def fold_decode(ids, w, pool, S, L, n_experts: int):
    """Decode in-place remap (E_s, w_s) -> (E_pi(s), w_s S_{s->pi(s)})   (Eq. decode_remap, Eq. A11).

    The [B, K] layout is kept (R13).  Retained slots are copied unchanged; a
    remapped weight is the float64 product of two float32 values rounded once
    to float32, i.e. one float32 multiply (R14).
    Returns (ids' [B,K] int32, w' [B,K] float32, tgt [N], scl [N]).
    """
    ids = np.asarray(ids).astype(np.int32)
    w = np.asarray(w, dtype=np.float32)
    tgt, scl = decode_tables(pool, S, L, n_experts)
    in_pool = np.zeros(n_experts, dtype=bool)
    in_pool[[int(p) for p in pool]] = True
    new_ids = tgt[ids]
    prod = (_f64(w) * _f64(scl[ids])).astype(np.float32)
    new_w = np.where(in_pool[ids], w, prod).astype(np.float32)
    return new_ids.astype(np.int32), new_w, tgt, scl


# ---------------------------------------------------------------------------
# Token permutation  (routes grouped per expert before expert computation, Sec. 4.1)
# ---------------------------------------------------------------------------

def permute_routes(route_ids, n_experts: int):
    """Counting sort of the flat route slots j = i*K_out + k by expert id, stable in j.

    Returns (counts [N], offsets [N+1], row_slot [R]); row r of expert e's
    group (offsets[e] <= r < offsets[e+1]) executes slot row_slot[r].
    """
    flat = [int(e) for e in np.asarray(route_ids).reshape(-1)]
    counts = [0] * n_experts
    for e in flat:
        counts[e] += 1
    offsets = [0] * (n_experts + 1)
    for e in range(n_experts):
        offsets[e + 1] = offsets[e] + counts[e]
    cursor = offsets[:-1].copy()
    row_slot = [0] * len(flat)
    for j, e in enumerate(flat):
        row_slot[cursor[e]] = j
        cursor[e] += 1
    return (np.array(counts, dtype=np.int32), np.array(offsets, dtype=np.int32),
            np.array(row_slot, dtype=np.int32))


# ---------------------------------------------------------------------------
# Layer output  (Eq. moe_output with Eq. gated_expert; shared expert R15)
# ---------------------------------------------------------------------------

@dataclass
class Layer:
    """Weights of one MoE layer as float32 arrays (bf16 data widened exactly)."""
    w_router: np.ndarray          # [N, d]
    w_gate_up: np.ndarray         # [N, 2I, d]  (or a callable e -> [2I, d])
    w_down: np.ndarray            # [N, d, I]   (or a callable e -> [d, I])
    router_bias: np.ndarray | None = None   # [N]
    ws_gate_up: np.ndarray | None = None    # [2I_s, d] shared expert
    ws_down: np.ndarray | None = None       # [d, I_s]

    @property
    def n_experts(self) -> int:
        return self.w_router.shape[0]

    def expert(self, e: int):
        gu = self.w_gate_up(e) if callable(self.w_gate_up) else self.w_gate_up[e]
        dn = self.w_down(e) if callable(self.w_down) else self.w_down[e]
        return gu, dn


def moe_output(layer: Layer, x, route_ids, route_w, experts=None) -> np.ndarray:
    """y_i = sum over route slots (e, w) of w E_e(x_i), plus the shared expert   (Eq. moe_output).

    Works for any route layout [T, K_out], duplicates included (R13).  The
    shared expert, if present, is added with weight 1 (R15).  ``experts``
    restricts the evaluation to a subset of experts (used to sample outputs
    of large layers); None evaluates all.
    """
    x = _f64(x)
    ids = np.asarray(route_ids)
    ww = _f64(route_w)
    t = x.shape[0]
    y = np.zeros((t, x.shape[1]), dtype=np.float64)
    for e in (range(layer.n_experts) if experts is None else experts):
        tok, slot = np.nonzero(ids == e)
        if tok.size == 0:
            continue
        gu, dn = layer.expert(e)
        out = expert_forward(x[tok], gu, dn)
        np.add.at(y, tok, ww[tok, slot][:, None] * out)
    if layer.ws_gate_up is not None:
        y += expert_forward(x, layer.ws_gate_up, layer.ws_down)
    return y


def folded_output_by_definition(layer: Layer, x, ids, w, retained_sets, S, L) -> np.ndarray:
    """Eq. folded_moe evaluated term by term from every expert's output.

    y^_i = sum_{t in S_K cap B} alpha_t E_t(x_i) + sum_{s in O} alpha_s S_{s->t_s} E_{t_s}(x_i)
    with t_s = pi(s | B).  ``retained_sets[i]`` lists B for token i in
    canonical order.  Used only to pin fold-then-execute (Eq. prefill_fold and
    Eq. decode_remap) against the definition.
    """
    x = _f64(x)
    ids = np.asarray(ids)
    ww = _f64(w)
    n = layer.n_experts
    all_out = np.stack([expert_forward(x, *layer.expert(e)) for e in range(n)])  # [N, T, d]
    y = np.zeros((x.shape[0], x.shape[1]))
    S = np.asarray(S, dtype=np.float32)
    L = np.asarray(L, dtype=np.float32)
    for i in range(x.shape[0]):
        B = [int(b) for b in retained_sets[i]]
        for j in range(ids.shape[1]):
            e = int(ids[i, j])
            if e in B:
                y[i] += ww[i, j] * all_out[e, i]
            else:
                t = min_loss_target(L[e], B)
                y[i] += ww[i, j] * float(S[e, t]) * all_out[t, i]
    if layer.ws_gate_up is not None:
        y += expert_forward(x, layer.ws_gate_up, layer.ws_down)
    return y


def moe_forward(layer: Layer, x, top_k: int, phase: str, budget: int, S=None, L=None, h=None,
                logits=None):
    """Full folded layer: route, select, fold, execute   (Sec. 4.3).

    phase: 'dense' (unfolded, Eq. moe_output), 'prefill' (Eq. prefill_budget +
    prefill_fold), 'decode' (Eq. decode_budget + decode_remap) or
    'decode_static' (Eq. A8 + decode_remap).  ``logits`` overrides the router
    (so that discrete decisions can be taken on the device's float32 logits).
    Returns (y [T, d] float64, info dict of intermediates).
    """
    if logits is None:
        logits = router_logits(x, layer.w_router, layer.router_bias)
    ids, w = route(logits, top_k)
    info = {"logits": logits, "topk_ids": ids, "topk_w": w}
    n = layer.n_experts
    if phase == "dense":
        out_ids, out_w = ids, w
    elif phase == "prefill":
        keep = select_prefill(ids, w, h, budget)
        out_ids, out_w = fold_prefill(ids, w, keep, S, L)
        info["keep"] = keep
    elif phase in ("decode", "decode_static"):
        if phase == "decode":
            pool, cand = select_decode_pool(ids, w, h, n, budget)
            info["candidates"] = cand
        else:
            pool = select_static_pool(h, budget)
        out_ids, out_w, tgt, scl = fold_decode(ids, w, pool, S, L, n)
        info.update(pool=pool, tgt=tgt, scl=scl)
    else:
        raise ValueError(phase)
    info["fold_ids"], info["fold_w"] = out_ids, out_w
    y = moe_output(layer, x, out_ids, out_w)
    return y, info


# ---------------------------------------------------------------------------
# Projector calibration  (Sec. 4.2, Eq. calibration_outputs .. projection_loss;
# Appendix A calibration protocol; Appendix B, Eq. A1-A2)
# ---------------------------------------------------------------------------

def finalize_tables(A, V, C, n, lam: float, clip: float, eps: float = EPSILON):
    """Scalar projector and loss from the per-pair sufficient statistics.

    s*_{s->t} = A / (V + lambda)                    (Eq. scalar_projector, Eq. A1)
    clipped to [-clip, clip] when clip > 0           (Appendix A)
    l_{s->t} = (C - 2 s A + s^2 V) / (C + eps)       (Eq. A2 expanded; R10, R11)
    unobserved pairs: s = 0 (R9), l = 1e30; self pairs: s = 1, l = 0 (Appendix A).
    A = sum w <u, v>, V = sum w ||v||^2, C = sum w ||u||^2 (w = ||u||, R12).
    Returns float64 (S, L).
    """
    A, V, C = _f64(A), _f64(V), _f64(C)
    n = np.asarray(n)
    nn = A.shape[0]
    S = np.zeros((nn, nn))
    Lo = np.full((nn, nn), UNOBSERVED_LOSS)
    for s in range(nn):
        for t in range(nn):
            if s == t:
                S[s, t], Lo[s, t] = 1.0, 0.0
                continue
            if n[s, t] == 0:
                continue
            den = V[s, t] + lam
            sc = A[s, t] / den if den != 0.0 else 0.0
            if clip > 0:
                sc = min(max(sc, -clip), clip)
            S[s, t] = sc
            resid = C[s, t] - 2.0 * sc * A[s, t] + sc * sc * V[s, t]
            Lo[s, t] = max(0.0, resid) / (C[s, t] + eps)
    return S, Lo


def calibrate(layer: Layer, x_cal, top_k: int, lam: float = DEFAULT_LAMBDA,
              clip: float = DEFAULT_CLIP, mode: str = "corouted", logits=None):
    """Offline projector calibration   (Sec. 4.2; Appendix A; Appendix B Eq. A1-A2).

    1. Route the m calibration tokens (Eq. topk_gate).
    2. u_{i,e} = E_e(x_i) for e in S_K(x_i) ('corouted', Eq. calibration_outputs)
       or for every e ('common', the common-input capture of Appendix F).
    3. For every token and ordered pair s != t of evaluated experts, with
       w = ||u_{i,s}||: A += w <u_s, u_t>, V += w ||u_t||^2, C += w ||u_s||^2, n += 1.
    4. finalize_tables -> S, L; h_e = mean ||u_{i,e}|| (R3).
    Returns (S, L, h) as float32 plus a dict with A, V, C, n and the float64 tables.
    """
    x = _f64(x_cal)
    nn = layer.n_experts
    if logits is None:
        logits = router_logits(x, layer.w_router, layer.router_bias)
    ids = topk_ids(logits, top_k)
    m = x.shape[0]
    if mode == "corouted":
        evaluated = [list(map(int, ids[i])) for i in range(m)]
    elif mode == "common":
        evaluated = [list(range(nn)) for _ in range(m)]
    else:
        raise ValueError(mode)
    # expert outputs, one expert at a time
    outputs = {}
    for e in range(nn):
        tok = [i for i in range(m) if e in evaluated[i]]
        if tok:
            gu, dn = layer.expert(e)
            outputs[e] = dict(zip(tok, expert_forward(x[tok], gu, dn)))
    A = np.zeros((nn, nn))
    V = np.zeros((nn, nn))
    C = np.zeros((nn, nn))
    n = np.zeros((nn, nn), dtype=np.int64)
    norm_sum = np.zeros(nn)
    norm_cnt = np.zeros(nn, dtype=np.int64)
    for i in range(m):
        ev = evaluated[i]
        U = {e: outputs[e][i] for e in ev}
        for s in ev:
            u = U[s]
            wi = math.sqrt(float(u @ u))
            norm_sum[s] += wi
            norm_cnt[s] += 1
            for t in ev:
                if t == s:
                    continue
                v = U[t]
                A[s, t] += wi * float(u @ v)
                V[s, t] += wi * float(v @ v)
                C[s, t] += wi * float(u @ u)
                n[s, t] += 1
    S, Lo = finalize_tables(A, V, C, n, lam, clip)
    observed = norm_cnt > 0
    h = np.zeros(nn)
    h[observed] = norm_sum[observed] / norm_cnt[observed]
    if observed.any():
        h[~observed] = h[observed].mean()
    stats = dict(A=A, V=V, C=C, n=n, S64=S, L64=Lo, h64=h)
    return S.astype(np.float32), Lo.astype(np.float32), h.astype(np.float32), stats


# ---------------------------------------------------------------------------
# Diagonal projector family  (Appendix B, Eq. appendix_diagonal_projector; the
# unfused reconstruction path of the projector ablation)
# ---------------------------------------------------------------------------

def calibrate_diagonal(layer: Layer, x_cal, top_k: int, lam: float = DEFAULT_LAMBDA,
                       mode: str = "corouted", logits=None):
    """Per-dimension projectors d_{s->t} = sum_i w_i (v_i . u_i) / (sum_i w_i (v_i . v_i) + lambda)
    (element-wise, Eq. appendix_diagonal_projector) with w_i = ||u_i||, and their
    normalised reconstruction loss sum_i w_i ||u_i - d . v_i||^2 / (sum_i w_i ||u_i||^2 + eps)
    (Eq. appendix_projection_loss with the diagonal map; R26: no clipping; an
    unobserved pair has d = 0 and loss 1e30; d_{s->s} = 1, loss 0).

    Returns (Dg [N, N, d] float32, Ld [N, N] float32, stats dict with float64 A, V
    [N, N, d], C, n)."""
    x = _f64(x_cal)
    nn = layer.n_experts
    dd = x.shape[1]
    if logits is None:
        logits = router_logits(x, layer.w_router, layer.router_bias)
    ids = topk_ids(logits, top_k)
    m = x.shape[0]
    if mode == "corouted":
        evaluated = [list(map(int, ids[i])) for i in range(m)]
    elif mode == "common":
        evaluated = [list(range(nn)) for _ in range(m)]
    else:
        raise ValueError(mode)
    outputs = {}
    for e in range(nn):
        tok = [i for i in range(m) if e in evaluated[i]]
        if tok:
            gu, dn = layer.expert(e)
            outputs[e] = dict(zip(tok, expert_forward(x[tok], gu, dn)))
    A = np.zeros((nn, nn, dd))
    V = np.zeros((nn, nn, dd))
    C = np.zeros((nn, nn))
    n = np.zeros((nn, nn), dtype=np.int64)
    for i in range(m):
        ev = evaluated[i]
        for s in ev:
            u = outputs[s][i]
            wi = math.sqrt(float(u @ u))
            for t in ev:
                if t == s:
                    continue
                v = outputs[t][i]
                A[s, t] += wi * (v * u)
                V[s, t] += wi * (v * v)
                C[s, t] += wi * float(u @ u)
                n[s, t] += 1
    Dg = np.zeros((nn, nn, dd))
    Ld = np.full((nn, nn), UNOBSERVED_LOSS)
    for s in range(nn):
        for t in range(nn):
            if s == t:
                Dg[s, t], Ld[s, t] = 1.0, 0.0
                continue
            if n[s, t] == 0:
                continue
            den = V[s, t] + lam
            dv = np.where(den != 0.0, A[s, t] / np.where(den != 0.0, den, 1.0), 0.0)
            Dg[s, t] = dv
            resid = C[s, t] - 2.0 * float(dv @ A[s, t]) + float((dv * dv) @ V[s, t])
            Ld[s, t] = max(0.0, resid) / (C[s, t] + EPSILON)
    return Dg.astype(np.float32), Ld.astype(np.float32), dict(A=A, V=V, C=C, n=n, D64=Dg, L64=Ld)


def fold_prefill_diagonal(ids, w, keep, Ld):
    """Prefill selection with diagonal projectors: the retained routes keep their
    router weights, and each omitted route s (route order) is assigned to the
    first minimum of Ld[s, t] over the retained routes (Eq.
    appendix_minimum_loss_assignment with the diagonal family's loss).

    Returns (out_ids [T, K'] int32, out_w [T, K'] float32: the retained routes in
    route order, and fold [T] lists of (source expert, weight, retained position))."""
    ids = np.asarray(ids)
    t, k = ids.shape
    k_out = int(np.asarray(keep)[0].sum()) if t else 0
    out_ids = np.zeros((t, k_out), dtype=np.int32)
    out_w = np.zeros((t, k_out), dtype=np.float32)
    Ld = np.asarray(Ld, dtype=np.float32)
    folds = []
    for i in range(t):
        ret = [j for j in range(k) if keep[i, j]]
        ret_experts = [int(ids[i, j]) for j in ret]
        fl = []
        for j in range(k):
            if keep[i, j]:
                continue
            s = int(ids[i, j])
            tgt = min_loss_target(Ld[s], ret_experts)
            fl.append((s, float(np.float32(w[i, j])), ret_experts.index(tgt)))
        for c, j in enumerate(ret):
            out_ids[i, c] = ids[i, j]
            out_w[i, c] = w[i, j]
        folds.append(fl)
    return out_ids, out_w, folds


def diagonal_output(layer: Layer, x, out_ids, out_w, folds, Dg) -> np.ndarray:
    """y_i = sum over retained routes t of (w_t 1 + sum of w_s d_{s->t} over the
    omitted s folded onto t) . E_t(x_i), plus the shared expert (Eq. folded_moe
    with the diagonal map acting on the target's output)."""
    x = _f64(x)
    Dg = _f64(Dg)
    t = x.shape[0]
    y = np.zeros_like(x)
    for e in range(layer.n_experts):
        tok, slot = np.nonzero(np.asarray(out_ids) == e)
        if tok.size == 0:
            continue
        gu, dn = layer.expert(e)
        out = expert_forward(x[tok], gu, dn)
        for r, (i, q) in enumerate(zip(tok, slot)):
            coef = np.full(x.shape[1], float(out_w[i, q]))
            for s, ws, qq in folds[i]:
                if qq == q:
                    coef = coef + ws * Dg[s, e]
            y[i] += coef * out[r]
    if layer.ws_gate_up is not None:
        y += expert_forward(x, layer.ws_gate_up, layer.ws_down)
    return y


def table_storage_bytes(n_layers: int, n_experts: int, family: str) -> int:
    """Bytes of float32 projector state per model, as the projector ablation table counts it.

    'pair': one directed scalar table S and one loss table L of [N, N] per layer;
    'layer': one scalar per layer; 'global': one scalar per model.
    """
    if family == "pair":
        return n_layers * n_experts * n_experts * 4 * 2
    if family == "layer":
        return n_layers * 4
    if family == "global":
        return 4
    raise ValueError(family)
