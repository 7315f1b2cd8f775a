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
with the oracle's functions and compared exactly.
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


def order_tie_ok(dev_row, exp_row, a_map, I, rel=1e-5):
    """True when a query-aware row differs from the oracle's only by blocks whose pooled
    scores tie (within `rel`) with the last block the top-up or cap kept: the device
    ranks float32 scores, the oracle float64 ones."""
    if dev_row.sum() != exp_row.sum():
        return False
    diff = np.nonzero(dev_row != exp_row)[0]
    kept = [J for J in np.nonzero(exp_row)[0] if J not in (0, I)]
    if not kept:
        return False
    cut = min(a_map[I, J] for J in kept)
    return all(abs(a_map[I, J] - cut) <= rel * cut for J in diff)


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
                 js_max_err=0.0, tiles=0, density=0.0, order_ties=0, near_tie_swaps=0)
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
                    if ok:
                        stats["boundary_problems"] += 1
                    elif order_tie_ok(gm[I], exp_row, a_map, I):
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
                if alt is not None and np.array_equal(gm, alt):
                    stats["near_tie_swaps"] += 1
                elif gp == oracle.PATTERN_QA and all(order_tie_ok(gm[I], exp[I], det["a_map"], I)
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


def compare_outputs(layer, o_gpu, masks, heads=None, row_blocks=None, scale=None, rng=None,
                    rows_per_head=None):
    """Oracle A(Q, K, V, S) on the given (oracle-side) masks vs the device output.
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
                pick = {0, nb - 1} | set(r.integers(0, nb, size=max(rows_per_head - 2, 0)).tolist())
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
