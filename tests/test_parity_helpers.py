"""The comparison helpers relax exact block-set equality only in named, bounded ways; these
CPU tests check that each relaxation accepts what it is meant to and nothing else."""
import numpy as np

import oracle
import synth
from parity import NEAR_TIE, qa_near_tie_mask


def _qa_detail():
    spec = synth.SPECS["tiny"]
    layer = synth.make_layer(spec)
    n = spec.seqlens[0]
    o = oracle.select_head(layer.q[:n, 0], layer.k[:n, 0], spec.block, 0.9, 0.1, 1,
                           1.0 / np.sqrt(spec.d), oracle.PATTERN_QA, True)
    return o, spec.block, -(-n // spec.block)


def _tile(detail, rank, nb):
    u = int(detail["unit_ids"][detail["qa"].order[rank]])
    return divmod(u, nb)


def test_near_tie_exchange_at_the_cut_is_rebuilt_exactly():
    o, block, nb = _qa_detail()
    det, sel = o["detail"], o["detail"]["qa"]
    k = sel.k
    assert 0 < k < sel.scores.size
    (i_out, j_out), (i_in, j_in) = _tile(det, k - 1, nb), _tile(det, k, nb)
    # the seeded input puts two unforced tiles at the cut (a forced one would hide the exchange)
    assert not (i_out == j_out or j_out == 0 or i_in == j_in or j_in == 0)
    dev = o["mask"].copy()
    dev[i_out, j_out] = False
    dev[i_in, j_in] = True
    gap = abs(sel.scores[sel.order[k - 1]] - sel.scores[sel.order[k]]) / sel.scores[sel.order[k - 1]]
    # with a tolerance covering the two scores the exchange is recognised and rebuilt
    alt = qa_near_tie_mask(dev, det, k, nb, 1, rel=2 * gap + 1e-12)
    assert alt is not None and np.array_equal(alt, dev)
    # with one that does not (unless the scores really are equal), it is not
    if gap > 2 * NEAR_TIE:
        assert qa_near_tie_mask(dev, det, k, nb, 1) is None


def test_non_exchange_differences_are_not_accepted():
    o, block, nb = _qa_detail()
    det, sel = o["detail"], o["detail"]["qa"]
    k = sel.k
    # a selected unit far above the cut dropped: no near-tie partner
    i0, j0 = _tile(det, 0, nb)
    dev = o["mask"].copy()
    if i0 != j0 and j0 != 0:
        dev[i0, j0] = False
        alt = qa_near_tie_mask(dev, det, k, nb, 1, rel=1e-3)
        assert alt is None or not np.array_equal(alt, dev)
    # an extra tile with no unit dropped: counts do not balance
    dev = o["mask"].copy()
    i1, j1 = _tile(det, k, nb)
    dev[i1, j1] = True
    alt = qa_near_tie_mask(dev, det, k, nb, 1, rel=1.0)
    assert alt is None or not np.array_equal(alt, dev)


# ---------------------------------------------------------------- order ties (query-aware rows)

from parity import (U_F32, flat_row_tie_ok, order_tie_ok,  # noqa: E402
                    qa_score_error_bound)


def _row(nb, blocks):
    r = np.zeros(nb, dtype=bool)
    r[list(blocks)] = True
    return r


def test_order_tie_accepts_an_exchange_within_the_bound_only():
    nb, I = 12, 11
    a = np.linspace(1.0, 0.1, nb)            # distinct scores, block 0 highest
    a[5], a[7] = 0.40, 0.40 * (1 - 1.5e-4)   # 5 and 7 tie within 2 * 1e-4
    eps = np.full(nb, 1e-4)
    oracle_row = _row(nb, {0, I, 3, 5})
    device_row = _row(nb, {0, I, 3, 7})
    assert order_tie_ok(device_row, oracle_row, a, eps, I)
    # the same exchange with bounds too small to cover the gap
    assert not order_tie_ok(device_row, oracle_row, a, np.full(nb, 5e-5), I)
    # an exchange with a block whose score is far away (no tie)
    assert not order_tie_ok(_row(nb, {0, I, 3, 9}), oracle_row, a, eps, I)
    # different number of blocks
    assert not order_tie_ok(_row(nb, {0, I, 3, 5, 7}), oracle_row, a, eps, I)
    # the forced blocks must stay
    assert not order_tie_ok(_row(nb, {I, 3, 5, 7}), _row(nb, {0, I, 3, 5}), a, eps, I)


def test_order_tie_rejects_an_exchange_far_from_the_cut():
    """Two blocks leave and two enter: every entering block must tie with every leaving one,
    so dropping a block far above the cut is caught even when its partner ties."""
    nb, I = 12, 11
    a = np.linspace(1.0, 0.1, nb)
    a[5], a[7] = 0.40, 0.40 * (1 - 1e-5)
    a[2], a[8] = 0.80, 0.80 * (1 - 1e-5)     # a second tied pair, far from the first
    eps = np.full(nb, 1e-4)
    oracle_row = _row(nb, {0, I, 2, 5})
    assert order_tie_ok(_row(nb, {0, I, 8, 7}), oracle_row, a, eps, I) is False
    assert order_tie_ok(_row(nb, {0, I, 2, 7}), oracle_row, a, eps, I) is True


def test_flattened_rows_allow_ties_only_where_top_up_or_cap_acted():
    nb, I = 12, 11
    a = np.linspace(1.0, 0.1, nb)
    a[5], a[7] = 0.40, 0.40 * (1 - 1e-5)
    eps = np.full(nb, 1e-4)
    # top-up: the flattened cut chose {0, I, 3}; the minimum budget 4 added block 5
    base = _row(nb, {0, I, 3})
    oracle_row = _row(nb, {0, I, 3, 5})
    assert flat_row_tie_ok(_row(nb, {0, I, 3, 7}), oracle_row, base, a, eps, I, 4, 0)
    # a top-up may not drop a block the flattened cut chose
    assert not flat_row_tie_ok(_row(nb, {0, I, 5, 7}), oracle_row, base, a, eps, I, 4, 0)
    # no top-up (the cut already gave 4 blocks) and no cap: nothing may differ
    base4 = _row(nb, {0, I, 3, 5})
    assert not flat_row_tie_ok(_row(nb, {0, I, 3, 7}), oracle_row, base4, a, eps, I, 4, 0)
    # cap 3 over a base of 5 blocks: the kept blocks must come from the base
    base5 = _row(nb, {0, I, 4, 5, 7})
    capped = _row(nb, {0, I, 5})
    assert flat_row_tie_ok(_row(nb, {0, I, 7}), capped, base5, a, eps, I, 2, 3)
    assert not flat_row_tie_ok(_row(nb, {0, I, 6}), capped, base5, a, eps, I, 2, 3)


def test_score_error_bound_covers_a_float32_evaluation():
    """The bound holds for an independent float32 evaluation of A_bar (numpy float32 block
    means, float32 BLAS product, float32 exp): for every pair of blocks of a row, the ratio
    of their float32 scores is within eps_J + eps_K of the float64 ratio."""
    spec = synth.SPECS["llama32k"].with_seqlens((16384,), "bound-16k").with_params(
        hq=2, hkv=1, head_kinds=("qa", "qa"))
    layer = synth.make_layer(spec)
    b, scale = spec.block, 1.0 / np.sqrt(spec.d)
    q, k = layer.q[:, 0], layer.k[:, 0]
    eps = qa_score_error_bound(q, k, b, scale)
    a64 = oracle.query_aware_block_attention(q, k, b, scale)
    nb = a64.shape[0]
    q32 = np.stack([q[J * b:(J + 1) * b].astype(np.float32).mean(axis=0) for J in range(nb)])
    k32 = np.stack([k[J * b:(J + 1) * b].astype(np.float32).mean(axis=0) for J in range(nb)])
    logit = (q32 @ k32.T) * np.float32(scale)
    causal = np.tril(np.ones((nb, nb), dtype=bool))
    logit = np.where(causal, logit, np.float32(-np.inf))
    e = np.exp(logit - logit.max(axis=1, keepdims=True))
    a32 = (e / e.sum(axis=1, keepdims=True)).astype(np.float64)
    worst = 0.0
    for I in range(nb):
        ref = int(np.argmax(a64[I, :I + 1]))
        rel = (a32[I, :I + 1] / a64[I, :I + 1]) / (a32[I, ref] / a64[I, ref]) - 1.0
        lim = eps[I, :I + 1] + eps[I, ref]
        assert np.all(np.abs(rel) <= lim), (I, np.max(np.abs(rel) / lim))
        worst = max(worst, float(np.max(np.abs(rel) / lim)))
    assert eps.max() < 1e-2 and eps[causal].min() >= 5 * U_F32
    assert worst > 0.0          # the float32 evaluation does differ


def test_oracle_top_up_row_exchange_needs_a_tie():
    """On a real query-aware top-up row: exchanging the last block the top-up added with the
    next candidate is accepted only when the bounds cover the two scores' gap."""
    spec = synth.SPECS["tiny"]
    layer = synth.make_layer(spec)
    n, b, scale = spec.seqlens[0], spec.block, 1.0 / np.sqrt(spec.d)
    q, k = layer.q[:n, 0], layer.k[:n, 0]
    m = 8
    o = oracle.select_head(q, k, b, 0.5, 0.1, m, scale, oracle.PATTERN_QA, True)
    det = o["detail"]
    nb = o["mask"].shape[0]
    base = oracle.tiles_from_query_aware(det["unit_ids"][det["qa"].selected], nb)
    base[np.arange(nb), 0] = True
    base[np.arange(nb), np.arange(nb)] = True
    eps = qa_score_error_bound(q, k, b, scale)
    found = False
    for I in range(nb):
        if base[I, :I + 1].sum() >= min(m, I + 1) or I + 1 <= m:
            continue
        added = [int(J) for J in oracle.row_priority(I, oracle.PATTERN_QA, det["a_map"])
                 if o["mask"][I, J] and not base[I, J]]
        rest = [int(J) for J in oracle.row_priority(I, oracle.PATTERN_QA, det["a_map"])
                if not o["mask"][I, J]]
        if not added or not rest:
            continue
        out, inn = added[-1], rest[0]
        dev = o["mask"][I].copy()
        dev[out], dev[inn] = False, True
        a = det["a_map"][I]
        gap = abs(a[out] - a[inn]) / max(a[out], a[inn])
        ok = flat_row_tie_ok(dev, o["mask"][I], base[I], a, eps[I], I, m, 0)
        assert ok == (gap <= eps[I, out] + eps[I, inn])
        wide = np.full(nb, gap)           # bounds that cover the gap accept it
        assert flat_row_tie_ok(dev, o["mask"][I], base[I], a, wide, I, m, 0)
        found = True
        break
    assert found, "no top-up row in the seeded input"
