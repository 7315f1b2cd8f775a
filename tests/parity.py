"""Helpers comparing the device path with the oracle (test infrastructure).

Selections: the oracle's unit order and float64 prefix masses decide which cut points K
are acceptable for each selection problem.  K must equal the oracle's K unless the
prefix mass is within BAND of gamma at the cut (the device accumulates masses in a
different order and precision); the device's K is read from its diagnostics and only
accepted if it is one of those cuts.  The expected block mask for that cut is then
rebuilt with the oracle's own functions and must match the device's lists exactly.
Pattern decisions must match unless |D_JS - tau| <= BAND, in which case the oracle is
re-run with the device's pattern forced.  At the cut, units whose scores are equal within
NEAR_TIE (relative) may be exchanged one for one (the device ranks float32 scores, the
oracle float64 ones); such exchanges are counted and the exchanged mask is again rebuilt
with the oracle's functions and compared exactly.  Query-aware rows that the minimum-budget
top-up, the per-row cap or a per-row cut shaped may differ from the oracle's by blocks whose
pooled scores tie within the float32 error bound of qa_score_error_bound (an "order tie");
these are counted too.  Every relaxation count has a stated maximum per call
(assert_relaxations_bounded): a count above it is a bug signal, not noise.
"""
from __future__ import annotations

import math
import sys
import time

import numpy as np

import oracle
from oracle import flexprefill as ofp

BAND = 1e-4          # cumulative-mass / JS-distance band around gamma / tau
NEAR_TIE = 2.0 ** -20   # relative score gap of a near-tie exchange at a cut
O_MAX_ABS = 2e-2     # bf16 output tolerance (max abs error)
O_MEAN_ABS = 2e-3    # bf16 output tolerance (mean abs error)
# stated maxima of the relaxation counts of one compare_selection call
MAX_BOUNDARY_PER_PROBLEM = 1 / 64    # cuts taken inside the gamma band, per selection problem
MAX_ORDER_TIES_PER_QA_ROW = 1 / 256  # order-tie rows, per query-aware row checked
MAX_NEAR_TIE_SWAPS = 2               # exchanges at a flattened cut


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def to_device(layer):
    import torch
    q = torch.from_numpy(layer.q).to(torch.bfloat16).cuda()
    k = torch.from_numpy(layer.k).to(torch.bfloat16).cuda()
    v = torch.from_numpy(layer.v).to(torch.bfloat16).cuda()
    return q, k, v


def allowed_cuts(sel: ofp.Selection, gamma: float, band: float = BAND):
    """Cut points k (number of units taken) acceptable under the mass band."""
    if gamma >= 1.0:
        return {sel.scores.size}
    incl = sel.prefix
    excl = incl - sel.scores[sel.order]
    ks = {sel.k}
    n = sel.scores.size
    ok = np.nonzero((excl < gamma + band) & (incl >= gamma - band))[0]
    ks.update(int(i) + 1 for i in ok)
    if incl[-1] < gamma + band:
        ks.add(n)
    return ks


def expected_mask_for_cuts(q_seq, k_seq, block, gamma, min_budget, scale, pattern, detail, cuts,
                           n, max_budget=0, vs_granularity=0):
    """Rebuild the oracle's block mask for the given cut points (oracle functions only)."""
    nb = -(-n // block)
    if pattern == oracle.PATTERN_QA:
        sel = detail["qa"]
        units = detail["unit_ids"][sel.order[:cuts[0]]]
        mask = oracle.tiles_from_query_aware(units, nb)
        mask = oracle.add_forced_and_min_budget(mask, oracle.PATTERN_QA, min_budget,
                                                detail["a_map"])
        return oracle.apply_max_budget(mask, oracle.PATTERN_QA, max_budget, detail["a_map"])
    sv, ss = detail["v"], detail["s"]
    vl, sl = sv.order[:cuts[0]], ss.order[:cuts[1]]
    if vs_granularity == 1:
        vl, sl = oracle.lines_of_blocks(vl, n, block), oracle.lines_of_blocks(sl, n, block)
    mask = oracle.tiles_from_vertical_slash(vl, sl, n, block)
    mask = oracle.add_forced_and_min_budget(mask, oracle.PATTERN_VS, min_budget)
    return oracle.apply_max_budget(mask, oracle.PATTERN_VS, max_budget)


def qa_row_for_cut(a_map, I, sel_row, k, min_budget, max_budget):
    """Row I of a per-query-block query-aware mask when that row's selection is cut after
    k units (oracle functions only)."""
    nb = a_map.shape[0]
    m = np.zeros((nb, nb), dtype=bool)
    m[I, sel_row.order[:k]] = True
    m = oracle.add_forced_and_min_budget(m, oracle.PATTERN_QA, min_budget, a_map)
    return oracle.apply_max_budget(m, oracle.PATTERN_QA, max_budget, a_map)[I]


U_F32 = 2.0 ** -24   # unit roundoff of float32 (round to nearest)


def qa_score_error_bound(q_seq, k_seq, block, scale):
    """Relative error bound eps[I, J] of a float32 evaluation of the pooled query-aware
    scores A_bar[I, J] = softmax_J(scale * Qbar_I . Kbar_J) (Algorithm 4, first two steps),
    excluding factors common to a whole row (the row sum), which do not change the order
    of a row's blocks.  First order in u = 2^-24, valid for any summation order
    (|fl(x_1 + ... + x_n) - sum x| <= (n - 1) u sum |x|):
      block means over c tokens: |dQbar_d| <= c u mean|q_d|, |dKbar_d| <= c u mean|k_d|;
      the d-term dot product: d u sum_d |Qbar_d Kbar_d|, plus u |L| for the scale;
      softmax: u |L - max_J L| for the shift, 4 u for exp, u for the normalising product.
    An error dL in the logit L changes the score by the factor exp(dL), i.e. relatively by
    dL.  Returns float64 [nb, nb] (zero above the diagonal)."""
    n, d = q_seq.shape
    nb = -(-n // block)
    q = np.asarray(q_seq, dtype=np.float64)
    k = np.asarray(k_seq, dtype=np.float64)
    cnt = np.array([min(block, n - J * block) for J in range(nb)], dtype=np.float64)

    def pooled(x):
        return (np.stack([x[J * block:(J + 1) * block].mean(axis=0) for J in range(nb)]),
                np.stack([np.abs(x[J * block:(J + 1) * block]).mean(axis=0) for J in range(nb)]))

    qb, qa = pooled(q)
    kb, ka = pooled(k)
    logit = scale * (qb @ kb.T)
    d_logit = scale * U_F32 * (d * (np.abs(qb) @ np.abs(kb).T)
                               + cnt[:, None] * (qa @ np.abs(kb).T)
                               + cnt[None, :] * (np.abs(qb) @ ka.T)) + U_F32 * np.abs(logit)
    causal = np.tril(np.ones((nb, nb), dtype=bool))
    mx = np.max(np.where(causal, logit, -np.inf), axis=1, keepdims=True)
    eps = d_logit + U_F32 * np.abs(logit - mx) + 5 * U_F32
    return np.where(causal, eps, 0.0)


def order_tie_ok(dev_row, exp_row, a_row, eps_row, I, required=None, pool=None):
    """True when query-block row I of the device differs from the oracle's only by blocks
    exchanged between scores that tie within their float32 error bounds: both rows keep the
    same number of blocks, both hold blocks 0 and I and every block of `required`, the
    device keeps only blocks of `pool` (when given), and every block kept by one row only
    lies within eps_row[J] + eps_row[K] (relative) of every block kept by the other row only.
    That is the only way in which ranking float32 instead of float64 pooled scores can change
    a minimum-budget top-up, a per-row cap or a per-row cut (the device ranks float32
    scores, the oracle float64 ones).  a_row: float64 A_bar[I, :]; eps_row: the bounds of
    qa_score_error_bound for that row."""
    dev_row = np.asarray(dev_row, dtype=bool)
    exp_row = np.asarray(exp_row, dtype=bool)
    if dev_row.sum() != exp_row.sum() or not (dev_row[0] and dev_row[I]):
        return False
    if required is not None and np.any(np.asarray(required, dtype=bool) & ~dev_row):
        return False
    if pool is not None and np.any(dev_row & ~np.asarray(pool, dtype=bool)):
        return False
    ins = np.nonzero(dev_row & ~exp_row)[0]
    outs = np.nonzero(exp_row & ~dev_row)[0]
    for J in ins:
        for K in outs:
            if abs(a_row[J] - a_row[K]) > (eps_row[J] + eps_row[K]) * max(a_row[J], a_row[K]):
                return False
    return True


def flat_row_tie_ok(dev_row, exp_row, base_row, a_row, eps_row, I, min_budget, max_budget):
    """order_tie_ok for row I of a flattened query-aware mask (Algorithm 4): only a row that
    the minimum-budget top-up or the per-row cap changed can hold an order tie.  base_row:
    the blocks of the row chosen by the flattened cut plus the forced blocks 0 and I.  With
    a top-up every base block stays and the added blocks may tie; with a cap the row keeps
    a subset of the base, whose dropped blocks may tie; otherwise nothing may differ."""
    base_row = np.asarray(base_row, dtype=bool)
    have = int(base_row[:I + 1].sum())
    if have < min(int(min_budget), I + 1):
        return order_tie_ok(dev_row, exp_row, a_row, eps_row, I, required=base_row)
    if max_budget > 0 and have > max_budget:
        forced = np.zeros_like(base_row)
        forced[[0, I]] = True
        return order_tie_ok(dev_row, exp_row, a_row, eps_row, I, required=forced, pool=base_row)
    return False


def qa_near_tie_mask(gm, detail, k, nb, min_budget, max_budget=0, rel=NEAR_TIE):
    """The flattened query-aware mask when the device, cutting after k units, exchanged units
    whose scores equal the score at the cut within `rel` (the device ranks float32 scores,
    the oracle float64 ones; with tens of millions of units the scores at the cut are that
    close).  Rebuilt with the oracle's functions from the oracle's selection with the
    exchange applied; None when the device mask is no such exchange."""
    sel = detail["qa"]
    cut = sel.scores[sel.order[k - 1]]
    near = np.abs(sel.scores - cut) <= rel * cut            # by flat causal position
    chosen = np.zeros(sel.scores.size, dtype=bool)
    chosen[sel.order[:k]] = True
    ti, tj = np.tril_indices(nb)                             # flat position -> tile
    dev = gm[ti, tj]
    swap_in = near & ~chosen & dev
    swap_out = near & chosen & ~dev
    if not swap_in.any() or swap_in.sum() != swap_out.sum():
        return None
    chosen[swap_in] = True
    chosen[swap_out] = False
    mask = oracle.tiles_from_query_aware(detail["unit_ids"][chosen], nb)
    mask = oracle.add_forced_and_min_budget(mask, oracle.PATTERN_QA, min_budget, detail["a_map"])
    return oracle.apply_max_budget(mask, oracle.PATTERN_QA, max_budget, detail["a_map"])


def compare_selection(layer, gpu, gamma, tau, min_budget, heads=None, scale=None,
                      max_budget=0, qa_mode=0, vs_granularity=0):
    """gpu: dict with 'masks' {(s,h): bool[nb,nb]}, 'pattern' [B*Hq], 'js' [B*Hq],
    'units' [B*Hq*2] (host arrays).  Returns statistics; raises AssertionError on a
    mismatch that the bands do not explain.  With qa_mode 1 every query-aware row is its
    own selection problem, checked row by row."""
    spec = layer.spec
    hq, hkv, d = layer.q.shape[1], layer.k.shape[1], layer.q.shape[2]
    G = hq // hkv
    scale = 1.0 / math.sqrt(d) if not scale else scale
    cu = layer.cu_seqlens
    stats = dict(heads=0, pattern_boundary=0, boundary_problems=0, exact_heads=0,
                 js_max_err=0.0, tiles=0, density=0.0, order_ties=0, near_tie_swaps=0,
                 qa_rows=0, qa_rows_differing=0, problems=0)
    sel_total = 0
    tiles_total = 0
    for s in range(len(cu) - 1):
        t0, t1 = int(cu[s]), int(cu[s + 1])
        n = t1 - t0
        for h in range(hq):
            if heads is not None and h not in heads:
                continue
            qs, ks = layer.q[t0:t1, h], layer.k[t0:t1, h // G]
            o = oracle.select_head(qs, ks, spec.block, gamma, tau, min_budget, scale, -1, True,
                                   max_budget, qa_mode, vs_granularity)
            gp = int(gpu["pattern"][s * hq + h])
            gm = gpu["masks"][(s, h)]
            stats["heads"] += 1
            if gamma >= 1.0:
                assert gp == oracle.PATTERN_DENSE, (s, h, gp)
                np.testing.assert_array_equal(gm, o["mask"], err_msg=f"dense mask s={s} h={h}")
                continue
            gjs = float(gpu["js"][s * hq + h])
            stats["js_max_err"] = max(stats["js_max_err"], abs(gjs - o["js"]))
            assert abs(gjs - o["js"]) <= 1e-3, (s, h, gjs, o["js"])
            if abs(o["js"] - tau) <= BAND:
                stats["pattern_boundary"] += 1
                if gp != o["pattern"]:
                    o = oracle.select_head(qs, ks, spec.block, gamma, tau, min_budget, scale, gp,
                                           True, max_budget, qa_mode, vs_granularity)
            assert gp == o["pattern"], f"pattern s={s} h={h}: gpu {gp} oracle {o['pattern']} " \
                                       f"js {o['js']:.6f} tau {tau}"
            det = o["detail"]
            gu = gpu["units"][(s * hq + h) * 2:(s * hq + h) * 2 + 2]
            nb_h = -(-n // spec.block)
            if gp == oracle.PATTERN_QA:
                stats["qa_rows"] += nb_h
                stats["problems"] += nb_h if qa_mode == 1 else 1
            else:
                stats["problems"] += 2
            eps = None            # float32 error bounds of the pooled scores, when needed

            def score_bounds():
                nonlocal eps
                if eps is None:
                    eps = qa_score_error_bound(qs, ks, spec.block, scale)
                return eps

            if gp == oracle.PATTERN_QA and qa_mode == 1:
                a_map = det["a_map"]
                exact = True
                for I, sel_row in enumerate(det["qa_rows"]):
                    exp_row = o["mask"][I]
                    if np.array_equal(gm[I], exp_row):
                        continue
                    exact = False
                    ok = any(np.array_equal(gm[I], qa_row_for_cut(a_map, I, sel_row, k,
                                                                  min_budget, max_budget))
                             for k in allowed_cuts(sel_row, gamma) if k != sel_row.k)
                    stats["qa_rows_differing"] += 1
                    if ok:
                        stats["boundary_problems"] += 1
                    elif order_tie_ok(gm[I], exp_row, a_map[I], score_bounds()[I], I):
                        stats["order_ties"] += 1
                    else:
                        raise AssertionError(
                            f"per-row query-aware s={s} h={h} I={I}: device "
                            f"{np.nonzero(gm[I])[0][:12].tolist()} oracle "
                            f"{np.nonzero(exp_row)[0][:12].tolist()}")
                stats["exact_heads"] += int(exact)
                sel_total += int(gm.sum())
                nb = gm.shape[0]
                tiles_total += nb * (nb + 1) // 2
                continue
            if gp == oracle.PATTERN_QA:
                allowed = [allowed_cuts(det["qa"], gamma)]
                cuts = (int(gu[0]),)
                oracle_cuts = (det["qa"].k,)
            else:
                allowed = [allowed_cuts(det["v"], gamma), allowed_cuts(det["s"], gamma)]
                cuts = (int(gu[0]), int(gu[1]))
                oracle_cuts = (det["v"].k, det["s"].k)
            for c, al in zip(cuts, allowed):
                assert c in al, f"s={s} h={h}: device K={c} not in allowed {sorted(al)[:8]}"
            if cuts != oracle_cuts:
                stats["boundary_problems"] += sum(int(a != b) for a, b in zip(cuts, oracle_cuts))
                exp = expected_mask_for_cuts(qs, ks, spec.block, gamma, min_budget, scale, gp, det,
                                             cuts, n, max_budget, vs_granularity)
            else:
                exp = o["mask"]
                stats["exact_heads"] += 1
            if not np.array_equal(gm, exp):
                rows = np.nonzero(np.any(gm != exp, axis=1))[0]
                alt = (qa_near_tie_mask(gm, det, cuts[0], gm.shape[0], min_budget, max_budget)
                       if gp == oracle.PATTERN_QA else None)
                base = None
                if gp == oracle.PATTERN_QA and (alt is None or not np.array_equal(gm, alt)):
                    nb_ = gm.shape[0]
                    base = oracle.tiles_from_query_aware(
                        det["unit_ids"][det["qa"].order[:cuts[0]]], nb_)
                    base[np.arange(nb_), 0] = True
                    base[np.arange(nb_), np.arange(nb_)] = True
                if alt is not None and np.array_equal(gm, alt):
                    stats["near_tie_swaps"] += 1
                elif base is not None and all(
                        flat_row_tie_ok(gm[I], exp[I], base[I], det["a_map"][I],
                                        score_bounds()[I], I, min_budget, max_budget)
                        for I in rows):
                    stats["order_ties"] += len(rows)
                else:
                    diff = np.argwhere(gm != exp)
                    raise AssertionError(f"block mask s={s} h={h} pattern {gp}: {len(diff)} "
                                         f"tiles differ, first {diff[:6].tolist()}")
            sel_total += int(gm.sum())
            nb = gm.shape[0]
            tiles_total += nb * (nb + 1) // 2
    stats["tiles"] = sel_total
    stats["density"] = sel_total / max(tiles_total, 1)
    return stats


def assert_relaxations_bounded(st):
    """Every relaxation of exact block-set equality stays under its stated maximum."""
    lim_b = max(2, int(st["problems"] * MAX_BOUNDARY_PER_PROBLEM))
    lim_o = max(2, int(st["qa_rows"] * MAX_ORDER_TIES_PER_QA_ROW))
    log(f"  relaxations: boundary cuts {st['boundary_problems']} (max {lim_b}), order ties "
        f"{st['order_ties']} (max {lim_o}), near-tie swaps {st['near_tie_swaps']} "
        f"(max {MAX_NEAR_TIE_SWAPS}), boundary patterns {st['pattern_boundary']}")
    assert st["boundary_problems"] <= lim_b, st
    assert st["order_ties"] <= lim_o, st
    assert st["near_tie_swaps"] <= MAX_NEAR_TIE_SWAPS, st


def compare_outputs(layer, o_gpu, masks, heads=None, row_blocks=None, scale=None, rng=None,
                    rows_per_head=None):
    """Oracle A(Q, K, V, S) on the given (oracle-side) masks vs the device output, on every
    query block, the blocks `row_blocks`, or (rows_per_head) the first and last block of
    every (sequence, head) plus rows_per_head - 2 distinct seeded random ones.
    Returns (max_abs, mean_abs)."""
    hq, hkv, d = layer.q.shape[1], layer.k.shape[1], layer.q.shape[2]
    G = hq // hkv
    block = layer.spec.block
    scale = 1.0 / math.sqrt(d) if not scale else scale
    cu = layer.cu_seqlens
    max_abs, sum_abs, cnt = 0.0, 0.0, 0
    for s in range(len(cu) - 1):
        t0, t1 = int(cu[s]), int(cu[s + 1])
        n = t1 - t0
        nb = -(-n // block)
        for h in range(hq):
            if heads is not None and h not in heads:
                continue
            rb = row_blocks
            if rows_per_head is not None:
                r = rng if rng is not None else np.random.default_rng(s * 1000 + h)
                inner = np.arange(1, nb - 1)
                take = min(max(rows_per_head - 2, 0), inner.size)
                pick = {0, nb - 1} | set(r.choice(inner, size=take, replace=False).tolist())
                rb = sorted(pick)
            ref = oracle.sparse_attention_rows(layer.q[t0:t1, h], layer.k[t0:t1, h // G],
                                               layer.v[t0:t1, h // G], masks[(s, h)], block,
                                               scale, rb)
            for I, rows in ref.items():
                got = o_gpu[t0 + I * block:t0 + I * block + rows.shape[0], h].astype(np.float64)
                err = np.abs(got - rows)
                max_abs = max(max_abs, float(err.max()))
                sum_abs += float(err.sum())
                cnt += err.size
    return max_abs, sum_abs / max(cnt, 1)


class Timer:
    def __init__(self, what):
        self.what = what

    def __enter__(self):
        self.t = time.time()
        return self

    def __exit__(self, *a):
        log(f"  [{self.what}: {time.time() - self.t:.2f}s]")
