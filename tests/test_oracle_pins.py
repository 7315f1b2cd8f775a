"""Pins for the float64 oracle: closed forms, invariants, brute force and library special
cases, each chosen so a plausible slip (dropped term, wrong sign or index, transposed
operand, off-by-one causal limit) fails at least one of them."""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle.flexprefill import cumulative_select

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
RNG = np.random.default_rng(1234)


# ---------------------------------------------------------------- JS distance (Section 3, step 3)

def test_js_closed_forms_from_golden():
    with open(os.path.join(GOLDEN, "js_distance_closed_forms.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        got = oracle.js_distance(np.array(c["p"]), np.array(c["q"]))
        assert got == pytest.approx(c["d_js"], abs=1e-15), c["why"]


def test_js_matches_scipy_and_properties():
    from scipy.spatial.distance import jensenshannon
    for n in (2, 7, 64, 1024):
        for _ in range(5):
            p = RNG.random(n) ** 4
            q = RNG.random(n) ** 4
            p[RNG.random(n) < 0.2] = 0.0
            p /= p.sum()
            q /= q.sum()
            d = oracle.js_distance(p, q)
            assert d == pytest.approx(float(jensenshannon(p, q)), abs=1e-12)   # natural log
            assert d == pytest.approx(oracle.js_distance(q, p), abs=1e-15)     # symmetric
            assert 0.0 <= d <= math.sqrt(math.log(2)) + 1e-15
            assert oracle.js_distance(p, p) == 0.0


# ---------------------------------------------------------------- representative attention

def _uniform_closed_form(n, block):
    """Q = 0 makes every causal logit 0: P[r, j] = 1 / (i_r + 1) for j <= i_r.  Then
    a_v[j] = (1/b') sum_{r: i_r >= j} 1/(i_r+1), and a_s[o] takes the same form in o."""
    bp = min(block, n)
    rows = np.arange(n - bp, n)
    a = np.zeros(n)
    for i in rows:
        a[: i + 1] += 1.0 / (i + 1)
    return a / bp


@pytest.mark.parametrize("n,block", [(1, 8), (5, 8), (8, 8), (9, 8), (47, 8), (300, 128)])
def test_uniform_attention_closed_form(n, block):
    d = 16
    q = np.zeros((n, d))
    k = RNG.standard_normal((n, d))
    q_hat, rows = oracle.representative_queries(q, block)
    assert list(rows) == list(range(n - min(block, n), n))
    a_full = oracle.representative_attention(q_hat, rows, k, 0.25)
    a_v, a_s = oracle.vertical_slash_scores(a_full, rows)
    expect = _uniform_closed_form(n, block)
    np.testing.assert_allclose(a_v, expect, rtol=0, atol=1e-15)
    np.testing.assert_allclose(a_s, expect, rtol=0, atol=1e-15)
    nb = -(-n // block)
    blk = oracle.true_block_distribution(a_full, block)
    np.testing.assert_allclose(blk, [expect[J * block:(J + 1) * block].sum() for J in range(nb)],
                               atol=1e-15)


def test_sink_and_diagonal_lines():
    """A key with a dominant logit is a vertical line of mass ~1 and a set of b' slash lines
    at offsets i_r - j of mass 1/b' each; a dominant diagonal is the slash line o = 0."""
    n, block, d = 200, 16, 8
    k = RNG.standard_normal((n, d)) * 0.01
    q = RNG.standard_normal((n, d)) * 0.01
    k[37, 0] = 400.0
    q[:, 0] = 1.0
    q_hat, rows = oracle.representative_queries(q, block)
    a_full = oracle.representative_attention(q_hat, rows, k, 1.0)
    a_v, a_s = oracle.vertical_slash_scores(a_full, rows)
    assert a_v[37] == pytest.approx(1.0, abs=1e-12)
    np.testing.assert_allclose(a_s[rows - 37], 1.0 / block, atol=1e-12)
    # diagonal: each query's own key dominates
    k2 = RNG.standard_normal((n, 256))
    q2 = 80.0 * k2 / np.sum(k2 * k2, axis=1, keepdims=True)
    q_hat, rows = oracle.representative_queries(q2, block)
    a_full = oracle.representative_attention(q_hat, rows, k2, 1.0)
    a_v, a_s = oracle.vertical_slash_scores(a_full, rows)
    assert a_s[0] == pytest.approx(1.0, abs=1e-9)
    np.testing.assert_allclose(a_v[rows], 1.0 / block, atol=1e-9)


@pytest.mark.parametrize("n", [130, 256, 1000])
def test_score_invariants(n):
    block, d = 64, 32
    q = RNG.standard_normal((n, d))
    k = RNG.standard_normal((n, d))
    q_hat, rows = oracle.representative_queries(q, block)
    a_full = oracle.representative_attention(q_hat, rows, k, 1 / math.sqrt(d))
    a_v, a_s = oracle.vertical_slash_scores(a_full, rows)
    blk = oracle.true_block_distribution(a_full, block)
    a_bar = oracle.estimated_block_distribution(q_hat, k, block, 1 / math.sqrt(d))
    for x in (a_v, a_s, blk, a_bar):
        assert x.sum() == pytest.approx(1.0, abs=1e-12)
        assert np.all(x >= 0)
    nb = -(-n // block)
    np.testing.assert_allclose(blk, [a_v[J * block:(J + 1) * block].sum() for J in range(nb)],
                               atol=1e-14)
    # causal: keys after the last query row carry nothing (none exist), keys near the end
    # are only visible to the later rows
    assert a_full[0, rows[0] + 1:].sum() == 0.0


def test_estimated_distribution_block_constant_closed_form():
    """With every key of block J equal to c_J, avgpool(K) = c_J exactly and
    a_bar = softmax(scale * q_bar . c_J); also holds with a partial last block."""
    block, d, n = 16, 8, 16 * 5 + 3
    nb = -(-n // block)
    c = RNG.standard_normal((nb, d))
    k = np.repeat(c, block, axis=0)[:n]
    q = RNG.standard_normal((n, d))
    q_hat, _ = oracle.representative_queries(q, block)
    qbar = q[n - block:].mean(axis=0)
    logits = np.array([0.3 * qbar @ c[J] for J in range(nb)])
    expect = np.exp(logits - logits.max())
    expect /= expect.sum()
    got = oracle.estimated_block_distribution(q_hat, k, block, 0.3)
    np.testing.assert_allclose(got, expect, atol=1e-15)


def test_a_bar_equals_last_row_of_query_aware_map():
    block, d, n = 32, 16, 32 * 6
    q = RNG.standard_normal((n, d))
    k = RNG.standard_normal((n, d))
    q_hat, _ = oracle.representative_queries(q, block)
    a_bar = oracle.estimated_block_distribution(q_hat, k, block, 0.25)
    a_map = oracle.query_aware_block_attention(q, k, block, 0.25)
    np.testing.assert_allclose(a_map[-1], a_bar, atol=1e-15)
    np.testing.assert_allclose(a_map.sum(axis=1), 1.0, atol=1e-14)
    assert np.all(np.triu(a_map, 1) == 0.0)


def test_query_aware_map_block_constant_closed_form():
    block, d, n = 8, 4, 8 * 7
    nb = n // block
    cq = RNG.standard_normal((nb, d))
    ck = RNG.standard_normal((nb, d))
    q = np.repeat(cq, block, axis=0)
    k = np.repeat(ck, block, axis=0)
    got = oracle.query_aware_block_attention(q, k, block, 0.5)
    for I in range(nb):
        lg = np.array([0.5 * cq[I] @ ck[J] for J in range(I + 1)])
        e = np.exp(lg - lg.max())
        np.testing.assert_allclose(got[I, :I + 1], e / e.sum(), atol=1e-15)


# ---------------------------------------------------------------- selection (Appendix B optimum)

def _brute_min_subset(scores, gamma):
    n = len(scores)
    for size in range(1, n + 1):
        best = None
        for comb in itertools.combinations(range(n), size):
            m = sum(scores[c] for c in comb)
            if m >= gamma and (best is None or m > best[0] or (m == best[0] and comb < best[1])):
                best = (m, comb)
        if best is not None:
            return size, best[1]
    return n, tuple(range(n))


@pytest.mark.parametrize("trial", range(40))
def test_cumulative_select_brute_force(trial):
    rng = np.random.default_rng(trial)
    n = int(rng.integers(1, 12))
    if trial % 2:
        raw = rng.integers(0, 5, size=n).astype(np.float64)   # exact ties
        if raw.sum() == 0:
            raw[0] = 1.0
    else:
        raw = rng.random(n) ** 3
    scores = raw / raw.sum()
    gamma = float(rng.choice([0.3, 0.5, 0.75, 0.9, 0.999]))
    sel = cumulative_select(scores, gamma)
    size, comb = _brute_min_subset(list(scores), gamma)
    assert sel.k == size
    assert tuple(sorted(sel.selected.tolist())) == comb


def test_cumulative_select_special_cases():
    s = np.array([0.1, 0.6, 0.3])
    assert list(cumulative_select(s, 0.6).selected) == [1]
    assert cumulative_select(s, 0.55).k == 1
    assert cumulative_select(s, 0.61).k == 2
    assert cumulative_select(s, 2.0).k == 3            # never reached: everything
    t = np.array([0.25, 0.25, 0.25, 0.25])
    assert list(cumulative_select(t, 0.5).selected) == [0, 1]   # ties: lowest ids first
    assert cumulative_select(t, 0.5).k == 2                     # prefix >= gamma, not >


# ---------------------------------------------------------------- vertical-slash tile rule

def _token_mask_tiles(verticals, slashes, n, block):
    """Brute force: build the token-level mask of the extended lines (causal part only)
    and mark every tile holding a marked entry."""
    i = np.arange(n)[:, None]
    j = np.arange(n)[None, :]
    m = np.isin(j, np.asarray(verticals, dtype=np.int64)) | \
        np.isin(i - j, np.asarray(slashes, dtype=np.int64))
    m &= j <= i
    nb = -(-n // block)
    tiles = np.zeros((nb, nb), dtype=bool)
    ii, jj = np.nonzero(m)
    tiles[ii // block, jj // block] = True
    return tiles


@pytest.mark.parametrize("n,block", [(1, 8), (7, 8), (8, 8), (9, 8), (47, 8), (24, 8),
                                     (131, 16), (2048, 128)])
def test_vertical_slash_tiles_brute_force(n, block):
    rng = np.random.default_rng(n * 31 + block)
    for _ in range(6):
        nv = int(rng.integers(0, min(n, 6) + 1))
        ns = int(rng.integers(0, min(n, 12) + 1))
        verts = rng.choice(n, size=nv, replace=False)
        slashes = rng.choice(n, size=ns, replace=False)
        got = oracle.tiles_from_vertical_slash(verts, slashes, n, block)
        np.testing.assert_array_equal(got, _token_mask_tiles(verts, slashes, n, block))


def test_query_aware_tiles_mapping():
    nb = 5
    units = np.array([0 * nb + 0, 3 * nb + 1, 4 * nb + 4])
    m = oracle.tiles_from_query_aware(units, nb)
    assert m.sum() == 3 and m[0, 0] and m[3, 1] and m[4, 4]


def test_query_aware_index_flattening_order():
    """Flattened causal units are normalised by the total of the causal entries and ids
    follow u = I*nb + J."""
    nb = 4
    a_map = np.tril(RNG.random((nb, nb)) + 0.01)
    a_map /= a_map.sum(axis=1, keepdims=True)
    sel, ids = oracle.query_aware_index(a_map, 0.5)
    I, J = np.tril_indices(nb)
    assert list(ids) == list(I * nb + J)
    assert sel.scores.sum() == pytest.approx(1.0, abs=1e-15)
    np.testing.assert_allclose(sel.scores, a_map[I, J] / a_map[I, J].sum())


# ---------------------------------------------------------------- query-wise selection (R11)

@pytest.mark.parametrize("trial", range(12))
def test_query_aware_rows_brute_force(trial):
    """Every query block is its own minimal selection over its row of the pooled map:
    brute force over subsets of each row (normalised by the row's own sum)."""
    rng = np.random.default_rng(100 + trial)
    nb = int(rng.integers(1, 7))
    raw = np.tril(rng.random((nb, nb)) ** 2 + (trial % 3 == 0) * rng.integers(0, 3, (nb, nb)))
    raw[np.arange(nb), np.arange(nb)] += 1e-3            # no all-zero row
    gamma = float(rng.choice([0.3, 0.6, 0.9, 0.999]))
    sels = oracle.query_aware_index_rows(raw, gamma)
    assert len(sels) == nb
    for I, sel in enumerate(sels):
        row = raw[I, :I + 1] / raw[I, :I + 1].sum()
        size, comb = _brute_min_subset(list(row), gamma)
        assert sel.k == size, (I, sel.k, size)
        assert tuple(sorted(sel.selected.tolist())) == comb


def test_query_aware_rows_scale_invariance_and_coverage():
    """Row normalisation: scaling a row of the map does not change its selection, and the
    mask reaches gamma in every row while flatten selection does not have to."""
    nb, gamma = 6, 0.8
    a_map = np.tril(RNG.random((nb, nb)) + 0.05)
    a_map /= a_map.sum(axis=1, keepdims=True)
    base = oracle.tiles_from_query_aware_rows(oracle.query_aware_index_rows(a_map, gamma), nb)
    scaled = a_map * np.arange(1, nb + 1)[:, None] * 7.5
    again = oracle.tiles_from_query_aware_rows(oracle.query_aware_index_rows(scaled, gamma), nb)
    np.testing.assert_array_equal(base, again)
    for I in range(nb):
        got = a_map[I, base[I]].sum()
        assert got >= gamma - 1e-12
        # minimal: dropping the smallest selected block falls below gamma
        if base[I].sum() > 1:
            assert got - a_map[I, base[I]].min() < gamma
    # a peaked row and a flat row: flatten spends the budget on the peaked row first
    peaked = np.zeros((2, 2))
    peaked[0, 0] = 1.0
    peaked[1] = [0.5, 0.5]
    sel_flat, ids = oracle.query_aware_index(peaked, 0.6)
    flat_mask = oracle.tiles_from_query_aware(ids[sel_flat.selected], 2)
    row_mask = oracle.tiles_from_query_aware_rows(oracle.query_aware_index_rows(peaked, 0.6), 2)
    assert flat_mask.sum() == 2 and not flat_mask[1].all()
    assert row_mask[1].all() and row_mask[0, 0]


# ---------------------------------------------------------------- maximum budget (R12)

def test_max_budget_hand_examples():
    nb = 6
    full = np.tril(np.ones((nb, nb), dtype=bool))
    a_map = np.tril(np.full((nb, nb), 0.01))
    a_map[4, :5] = [0.05, 0.4, 0.1, 0.3, 0.15]
    qa = oracle.apply_max_budget(full, oracle.PATTERN_QA, 3, a_map)
    assert set(np.nonzero(qa[4])[0]) == {0, 1, 4}           # 0, I, then the largest score
    assert set(np.nonzero(qa[2])[0]) == {0, 1, 2}           # row already within the cap
    vs = oracle.apply_max_budget(full, oracle.PATTERN_VS, 3)
    assert set(np.nonzero(vs[5])[0]) == {0, 4, 5}           # nearest to the diagonal
    assert set(np.nonzero(vs[3])[0]) == {0, 2, 3}
    two = oracle.apply_max_budget(full, oracle.PATTERN_VS, 2)
    for I in range(nb):
        assert set(np.nonzero(two[I])[0]) == ({0, I} if I else {0})


@pytest.mark.parametrize("pattern", [0, 1])
def test_max_budget_properties(pattern):
    rng = np.random.default_rng(77 + pattern)
    nb = 20
    a_map = np.tril(rng.random((nb, nb)))
    mask = oracle.add_forced_and_min_budget(np.tril(rng.random((nb, nb)) < 0.5), pattern, 3,
                                            a_map)
    assert oracle.apply_max_budget(mask, pattern, 0, a_map) is mask       # no cap
    np.testing.assert_array_equal(oracle.apply_max_budget(mask, pattern, nb, a_map), mask)
    for M in (2, 4, 7):
        capped = oracle.apply_max_budget(mask, pattern, M, a_map)
        assert not np.any(capped & ~mask)                                  # only removes
        for I in range(nb):
            row = np.nonzero(capped[I])[0]
            assert len(row) == min(M, int(mask[I].sum()))
            assert 0 in row and I in row
            # what was dropped ranks below everything kept (other than 0 and I)
            pri = list(oracle.row_priority(I, pattern, a_map))
            kept = [pri.index(J) for J in row if J not in (0, I)]
            dropped = [pri.index(J) for J in np.nonzero(mask[I] & ~capped[I])[0]]
            if kept and dropped:
                assert max(kept) < min(dropped)


# ---------------------------------------------------------------- block-pooled lines (R13)

@pytest.mark.parametrize("n,block", [(1, 8), (7, 8), (8, 8), (9, 8), (47, 8), (130, 32)])
def test_pooled_vertical_slash_scores_and_tiles(n, block):
    """Pooled scores are block sums of the token-line scores (each family sums to 1), and
    the tiles of the selected blocks equal the token-line tiles of all their lines,
    checked against a brute-force token mask."""
    rng = np.random.default_rng(n * 31 + block)
    q = rng.standard_normal((n, 4))
    k = rng.standard_normal((n, 4))
    q_hat, rows = oracle.representative_queries(q, block)
    a_full = oracle.representative_attention(q_hat, rows, k, 0.5)
    a_v, a_s = oracle.vertical_slash_scores(a_full, rows)
    for gamma in (0.3, 0.7, 0.95):
        sv, ss, pv, ps = oracle.vertical_slash_index_pooled(a_full, rows, gamma, block)
        nb = -(-n // block)
        assert pv.shape == (nb,) and ps.shape == (nb,)
        assert pv.sum() == pytest.approx(1.0, abs=1e-12)
        assert ps.sum() == pytest.approx(1.0, abs=1e-12)
        for J in range(nb):
            assert pv[J] == pytest.approx(a_v[J * block:(J + 1) * block].sum(), abs=1e-15)
        vl = oracle.lines_of_blocks(sv.selected, n, block)
        sl = oracle.lines_of_blocks(ss.selected, n, block)
        assert len(vl) == sum(min((J + 1) * block, n) - J * block for J in sv.selected)
        got = oracle.tiles_from_vertical_slash(vl, sl, n, block)
        # brute force: token mask of the lines, tiles that hold a masked causal position
        tok = np.zeros((n, n), dtype=bool)
        for j in vl:
            tok[j:, j] = True
        for o in sl:
            i = np.arange(o, n)
            tok[i, i - o] = True
        want = np.zeros((nb, nb), dtype=bool)
        for I in range(nb):
            for J in range(I + 1):
                want[I, J] = tok[I * block:(I + 1) * block, J * block:(J + 1) * block].any()
        np.testing.assert_array_equal(got, want)


# ---------------------------------------------------------------- forced tiles and min budget

def test_forced_and_min_budget():
    nb = 12
    empty = np.zeros((nb, nb), dtype=bool)
    vs = oracle.add_forced_and_min_budget(empty, oracle.PATTERN_VS, 4)
    for I in range(nb):
        row = np.nonzero(vs[I])[0]
        assert 0 in row and I in row
        assert len(row) == min(4, I + 1)
        assert np.all(row <= I)
        if I >= 3:
            assert set(row) == {0, I, I - 1, I - 2}          # nearest diagonal first
    a_map = np.tril(RNG.random((nb, nb)))
    qa = oracle.add_forced_and_min_budget(empty, oracle.PATTERN_QA, 5, a_map)
    for I in range(5, nb):
        row = set(np.nonzero(qa[I])[0])
        cand = [J for J in range(1, I)]
        best = sorted(cand, key=lambda J: (-a_map[I, J], J))[:3]
        assert row == {0, I, *best}


# ---------------------------------------------------------------- A(Q, K, V, S)

def _random_mask(nb, rng, p=0.3):
    m = np.tril(rng.random((nb, nb)) < p)
    m[np.arange(nb), 0] = True
    m[np.arange(nb), np.arange(nb)] = True
    return m


@pytest.mark.parametrize("n,block", [(1, 8), (8, 8), (45, 8), (130, 32)])
def test_sparse_attention_two_formulations(n, block):
    rng = np.random.default_rng(n)
    d = 16
    q, k, v = (rng.standard_normal((n, d)) for _ in range(3))
    mask = _random_mask(-(-n // block), rng)
    rows = oracle.sparse_attention_rows(q, k, v, mask, block, 0.3)
    full = np.concatenate([rows[I] for I in sorted(rows)])
    dense_masked = oracle.sparse_attention_masked(q, k, v, mask, block, 0.3)
    np.testing.assert_allclose(full, dense_masked, atol=1e-12)


def test_dense_matches_torch_sdpa():
    import torch
    rng = np.random.default_rng(7)
    n, d, block = 200, 32, 16
    q, k, v = (rng.standard_normal((n, d)) for _ in range(3))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None, None], torch.from_numpy(k)[None, None],
        torch.from_numpy(v)[None, None], is_causal=True)[0, 0].numpy()
    scale = 1 / math.sqrt(d)
    np.testing.assert_allclose(oracle.dense_causal_attention(q, k, v, scale), ref, atol=1e-12)
    nb = -(-n // block)
    rows = oracle.sparse_attention_rows(q, k, v, np.tril(np.ones((nb, nb), bool)), block, scale)
    np.testing.assert_allclose(np.concatenate([rows[I] for I in sorted(rows)]), ref, atol=1e-12)


def test_error_bound_appendix_a():
    """|A - A_S| <= (1 - a_S) * sum_j |v_j| per query row and output dimension, with a_S
    the full-attention mass inside the selected set (Appendix A)."""
    rng = np.random.default_rng(11)
    n, d, block = 96, 8, 8
    q, k, v = (rng.standard_normal((n, d)) for _ in range(3))
    q *= 2.0
    mask = _random_mask(n // block, rng, 0.25)
    scale = 0.5
    full = oracle.dense_causal_attention(q, k, v, scale)
    rows = oracle.sparse_attention_rows(q, k, v, mask, block, scale)
    sparse = np.concatenate([rows[I] for I in sorted(rows)])
    logits = (q @ k.T) * scale
    for i in range(n):
        p = np.exp(logits[i, :i + 1] - logits[i, :i + 1].max())
        p /= p.sum()
        sel = mask[i // block, np.arange(i + 1) // block]
        a_s = p[sel].sum()
        bound = (1 - a_s) * np.abs(v[:i + 1]).sum(axis=0)
        assert np.all(np.abs(full[i] - sparse[i]) <= bound + 1e-12)


# ---------------------------------------------------------------- Algorithm 1 end to end

def test_gamma_one_is_dense_attention():
    rng = np.random.default_rng(3)
    n, d, block = 100, 16, 16
    q = rng.standard_normal((n, 2, d))
    k = rng.standard_normal((n, 1, d))
    v = rng.standard_normal((n, 1, d))
    res = oracle.select(q, k, np.array([0, n]), block, 1.0, 0.1, 1)
    nb = -(-n // block)
    for h in range(2):
        r = res[0][h]
        assert r["pattern"] == oracle.PATTERN_DENSE
        np.testing.assert_array_equal(r["mask"], np.tril(np.ones((nb, nb), bool)))
        rows = oracle.sparse_attention_rows(q[:, h], k[:, 0], v[:, 0], r["mask"], block, 0.25)
        np.testing.assert_allclose(np.concatenate([rows[I] for I in sorted(rows)]),
                                   oracle.dense_causal_attention(q[:, h], k[:, 0], v[:, 0], 0.25),
                                   atol=1e-12)


def test_pattern_decision_constructed_heads():
    """A sink-dominated head is vertical-slash (the pooled estimate misses the sink); a head
    whose keys and queries are constant per block is query-aware (pooling is exact)."""
    block, d, n = 32, 16, 32 * 16
    rng = np.random.default_rng(5)
    # sink head
    k = rng.standard_normal((n, d)) * 0.1
    q = rng.standard_normal((n, d)) * 0.1
    k[0, 0] = 60.0
    q[:, 0] = 1.0
    p, djs, *_ = oracle.sparse_pattern_search(q, k, block, 0.1, 1.0)
    assert p == oracle.PATTERN_VS and djs > 0.5
    # block-clustered head
    ck = rng.standard_normal((n // block, d))
    kq = np.repeat(ck, block, axis=0)
    qq = np.repeat(rng.standard_normal((n // block, d)), block, axis=0)
    p, djs, *_ = oracle.sparse_pattern_search(qq, kq, block, 0.1, 0.5)
    assert p == oracle.PATTERN_QA and djs < 0.05
    # tau = 0: no query-aware heads (strict comparison)
    p, djs, *_ = oracle.sparse_pattern_search(qq, kq, block, 0.0, 0.5)
    assert p == oracle.PATTERN_VS


def test_select_structure_on_synthetic_layer():
    import synth
    spec = synth.SPECS["tiny"]
    layer = synth.make_layer(spec)
    res = oracle.select(layer.q, layer.k, layer.cu_seqlens, spec.block, spec.gamma, spec.tau,
                        spec.min_budget)
    nb = -(-spec.seqlens[0] // spec.block)
    for r in res[0]:
        assert r["pattern"] == oracle.PATTERN_VS
        m = r["mask"]
        assert not np.any(np.triu(m, 1))
        assert np.all(m[np.arange(nb), 0]) and np.all(m[np.arange(nb), np.arange(nb)])
