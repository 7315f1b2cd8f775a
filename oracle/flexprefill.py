"""FlexPrefill reference implementation (float64, CPU) -- TEST INFRASTRUCTURE ONLY.

Per (sequence, query head h) with KV head g = h // (Hq/Hkv):

  Algorithm 1 (Sparse Attention): pattern <- Algorithm 2; index set S <- Algorithm 4
  (query-aware) or Algorithm 3 (vertical-slash); output A(Q, K, V, S).

Readings taken where the paper is silent (each is also listed in the design notes):

  R1  The representative set Q_hat is the last min(block, n) query rows; their positions
      are i_r = n - b' + r (Section 3, "Representative Query Selection"; Section 4.1).
  R2  Attention of Q_hat is token-causal (key j <= i_r), following the index sets of
      Section 2 (S_i contains only j <= i).  The pooled maps are block-causal with the
      diagonal block included.
  R3  a_hat = sumpool(softmax(Q_hat K^T / sqrt d)) is normalised to a distribution: the
      window sums are divided by the total mass of the map (= b').
  R4  The Jensen-Shannon divergence uses the natural logarithm, with 0 ln 0 = 0.
  R5  The head is query-aware iff D_JS < tau (strict), so tau = 0 gives no query-aware heads.
  R6  argsort ties are broken by unit id ascending (score descending first); prefix sums
      are float64; if the prefix never reaches gamma every unit is taken.
  R7  Vertical lines are key positions j; slash lines are offsets o = i - j.  A tile
      (I, J) of block_size x block_size is computed iff some selected line meets a
      causal position (i, j <= i) inside it.
  R8  The first and the diagonal key block of every query block are always kept
      (Section 4.1, implementation details), and every query-block row keeps at least
      min(m, I + 1) key blocks; missing blocks are added in the row's pooled-score order
      (query-aware) or nearest-to-diagonal first (vertical-slash).
  R9  gamma >= 1 means full attention: every causal tile (Appendix E labels gamma = 1 as
      full attention).
  R10 Pooling windows are aligned to token 0 of each sequence; a partial last window is
      averaged over its own tokens.
  R11 The query-wise alternative to the flatten step of Algorithm 4 (appendix "flatten
      ablation": the selected key blocks of each query block reach gamma): every query
      block I is its own selection problem over the key blocks J <= I, scored by
      A_bar[I, J] divided by the row's sum, with the rule of R6.
  R12 The maximum computational budget (appendix "maximum budget limit") is a cap of M
      key blocks per query-block row, applied after R8: a row with more than M blocks
      keeps blocks 0 and I and then its other blocks in the order R8 uses to add them
      (pooled score for query-aware heads, nearest to the diagonal for vertical-slash
      heads).  M = 0 means no cap.
  R13 Block-pooled vertical-slash lines (the alternative to Algorithm 3's token lines):
      a vertical unit is a key block J scored by the sum of a_v over its keys, a slash
      unit is an offset block [D*b, D*b + b) scored by the sum of a_s over its offsets;
      each family is selected by the rule of R6, and selecting a unit selects all of its
      lines, which then mark tiles as in R7.
"""
from __future__ import annotations

import math

import numpy as np

PATTERN_QA = 0      # query-specific ("query-aware") head
PATTERN_VS = 1      # vertical-slash head
PATTERN_DENSE = 2   # gamma >= 1: no search, every causal tile


def _softmax_rows(x: np.ndarray) -> np.ndarray:
    """Row softmax of a float64 matrix whose masked entries are -inf."""
    m = np.max(x, axis=-1, keepdims=True)
    m = np.where(np.isfinite(m), m, 0.0)
    e = np.exp(x - m)
    return e / np.sum(e, axis=-1, keepdims=True)


# ------------------------------------------------------------------ Algorithm 2 and its inputs

def representative_queries(q_seq: np.ndarray, block: int):
    """Q_hat = the last block_size query vectors (Section 3, step 1; R1).

    q_seq: [n, d] queries of one head of one sequence.  Returns (Q_hat [b', d] float64,
    rows [b'] absolute positions i_r).
    """
    n = q_seq.shape[0]
    bp = min(block, n)
    rows = np.arange(n - bp, n)
    return np.asarray(q_seq[n - bp:], dtype=np.float64), rows


def representative_attention(q_hat: np.ndarray, rows: np.ndarray, k_seq: np.ndarray,
                             scale: float) -> np.ndarray:
    """A_hat = softmax(Q_hat K^T / sqrt d) over the causal keys j <= i_r (Algorithm 3,
    first step; Section 3, step 2 second line; R2).  Returns [b', n] float64."""
    k64 = np.asarray(k_seq, dtype=np.float64)
    logits = (q_hat @ k64.T) * scale
    n = k64.shape[0]
    causal = np.arange(n)[None, :] <= rows[:, None]
    logits = np.where(causal, logits, -np.inf)
    return _softmax_rows(logits)


def vertical_slash_scores(a_hat: np.ndarray, rows: np.ndarray):
    """a_v = sum_vertical(A_hat) / sum(A_hat) and a_s = sum_slash(A_hat) / sum(A_hat)
    (Algorithm 3).  A vertical line is a key column j; a slash line is a diagonal of
    constant offset o = i - j >= 0 (R7).  Returns (a_v [n], a_s [n])."""
    bp, n = a_hat.shape
    total = float(np.sum(a_hat))
    a_v = np.sum(a_hat, axis=0) / total
    a_s = np.zeros(n, dtype=np.float64)
    for r in range(bp):
        i = int(rows[r])
        # offsets o = 0..i meet key j = i - o
        a_s[: i + 1] += a_hat[r, i::-1]
    a_s /= total
    return a_v, a_s


def true_block_distribution(a_hat: np.ndarray, block: int) -> np.ndarray:
    """a_hat_blocks = sumpool(softmax(Q_hat K^T / sqrt d)) with window block_size, as a
    distribution over key blocks (Section 3, step 2; Algorithm 2; R3)."""
    bp, n = a_hat.shape
    nb = -(-n // block)
    out = np.zeros(nb, dtype=np.float64)
    for J in range(nb):
        out[J] = np.sum(a_hat[:, J * block:min((J + 1) * block, n)])
    return out / np.sum(a_hat)


def _avgpool_rows(x: np.ndarray, block: int) -> np.ndarray:
    """Mean of each window of block_size rows, aligned at row 0 (R10)."""
    n = x.shape[0]
    nb = -(-n // block)
    x64 = np.asarray(x, dtype=np.float64)
    return np.stack([x64[J * block:min((J + 1) * block, n)].mean(axis=0) for J in range(nb)])


def estimated_block_distribution(q_hat: np.ndarray, k_seq: np.ndarray, block: int,
                                 scale: float) -> np.ndarray:
    """a_bar = softmax(avgpool(Q_hat) avgpool(K)^T / sqrt d) (Section 3, step 2).  Q_hat
    is a single window, so it pools to one vector; the last query block sees every key
    block (R2)."""
    q_bar = np.asarray(q_hat, dtype=np.float64).mean(axis=0)
    k_bar = _avgpool_rows(k_seq, block)
    return _softmax_rows((k_bar @ q_bar)[None, :] * scale)[0]


def js_distance(p: np.ndarray, q: np.ndarray) -> float:
    """D_JS(p, q) = sqrt(JSD(p || q)) = sqrt((KL(p || m) + KL(q || m)) / 2), m = (p + q)/2
    (equation for the JS distance, Section 3, step 3; R4)."""
    p = np.asarray(p, dtype=np.float64)
    q = np.asarray(q, dtype=np.float64)
    m = 0.5 * (p + q)

    def kl(a, b):
        nz = a > 0
        return float(np.sum(a[nz] * np.log(a[nz] / b[nz])))

    jsd = 0.5 * (kl(p, m) + kl(q, m))
    return math.sqrt(max(jsd, 0.0))


def sparse_pattern_search(q_seq: np.ndarray, k_seq: np.ndarray, block: int, tau: float,
                          scale: float):
    """Algorithm 2.  Returns (pattern, d_js, a_bar, a_hat_blocks, A_hat, rows)."""
    q_hat, rows = representative_queries(q_seq, block)
    a_bar = estimated_block_distribution(q_hat, k_seq, block, scale)
    a_full = representative_attention(q_hat, rows, k_seq, scale)
    a_blk = true_block_distribution(a_full, block)
    d_js = js_distance(a_bar, a_blk)
    pattern = PATTERN_QA if d_js < tau else PATTERN_VS     # R5
    return pattern, d_js, a_bar, a_blk, a_full, rows


# ------------------------------------------------------------------ cumulative-mass selection

class Selection:
    """Result of a cumulative-attention selection over a score vector.

    order   : unit ids sorted by (score desc, id asc)
    k       : K = min{k : sum of the first k scores >= gamma}, or all units
    prefix  : float64 inclusive prefix sums along `order`
    """

    def __init__(self, scores, order, k, prefix):
        self.scores = scores
        self.order = order
        self.k = k
        self.prefix = prefix

    @property
    def selected(self) -> np.ndarray:
        return self.order[: self.k]

    def boundary_units(self, gamma: float, band: float) -> np.ndarray:
        """Units whose exclusive prefix mass lies within `band` of gamma."""
        excl = self.prefix - self.scores[self.order]
        return self.order[np.abs(excl - gamma) <= band]


def cumulative_select(scores: np.ndarray, gamma: float) -> Selection:
    """argsort the scores descending and keep the shortest prefix whose mass reaches gamma
    (Algorithms 3 and 4, "minimum computational budget"; the objective equation of
    Section 3 with the greedy optimum of Appendix B; R6)."""
    scores = np.asarray(scores, dtype=np.float64)
    ids = np.arange(scores.size)
    order = np.lexsort((ids, -scores))
    prefix = np.cumsum(scores[order])
    hit = np.nonzero(prefix >= gamma)[0]
    k = int(hit[0]) + 1 if hit.size else int(scores.size)
    return Selection(scores, order, k, prefix)


# ------------------------------------------------------------------ Algorithm 3

def vertical_slash_index(a_hat: np.ndarray, rows: np.ndarray, gamma: float):
    """Algorithm 3: a_v, a_s; their argsorts; K_v, K_s; S_v and S_s (as two selections)."""
    a_v, a_s = vertical_slash_scores(a_hat, rows)
    return cumulative_select(a_v, gamma), cumulative_select(a_s, gamma), a_v, a_s


def vertical_slash_index_pooled(a_hat: np.ndarray, rows: np.ndarray, gamma: float,
                                block: int):
    """Block-pooled variant of Algorithm 3 (R13): a_v and a_s summed over blocks of `block`
    key positions / offsets, each selected by cumulative mass.  Returns the two selections
    (unit ids = block indices) and the pooled scores."""
    a_v, a_s = vertical_slash_scores(a_hat, rows)
    n = a_v.shape[0]
    nb = -(-n // block)
    pv = np.array([a_v[J * block:(J + 1) * block].sum() for J in range(nb)])
    ps = np.array([a_s[D * block:(D + 1) * block].sum() for D in range(nb)])
    return cumulative_select(pv, gamma), cumulative_select(ps, gamma), pv, ps


def lines_of_blocks(units, n: int, block: int) -> np.ndarray:
    """Every line (key position or offset) of the given blocks of lines (R13)."""
    out = [np.arange(u * block, min((u + 1) * block, n)) for u in np.asarray(units, dtype=int)]
    return np.concatenate(out) if out else np.zeros(0, dtype=np.int64)


def tiles_from_vertical_slash(verticals, slashes, n: int, block: int) -> np.ndarray:
    """Extend the selected lines to the whole attention matrix (Section 3, vertical-slash
    head, third item) and mark each block_size x block_size tile the lines meet (R7).

    Tile (I, J), J <= I, is marked iff a selected vertical j lies in key block J, or a
    selected slash o has a causal position in the tile: rows i in [I*b, e_I), keys
    j = i - o in [J*b, e_J), with e_X = min((X+1)*b, n).  Returns bool [nb, nb].
    """
    nb = -(-n // block)
    mask = np.zeros((nb, nb), dtype=bool)
    causal = np.tril(np.ones((nb, nb), dtype=bool))
    # a vertical line j runs down key column j for every row i >= j
    vert_blocks = np.zeros(nb, dtype=bool)
    for j in np.asarray(verticals, dtype=np.int64):
        vert_blocks[j // block] = True
    mask |= causal & vert_blocks[None, :]
    # a slash line o meets, over the rows [I*b, e_I) of query block I, the keys
    # [I*b - o, e_I - 1 - o] clipped to j >= 0; that interval is shorter than a block, so
    # it meets exactly the key blocks holding its two ends.
    I = np.arange(nb)
    i_lo = I * block
    i_hi = np.minimum((I + 1) * block, n) - 1
    for o in np.asarray(slashes, dtype=np.int64):
        hi = i_hi - o
        ok = hi >= 0
        lo = np.maximum(i_lo - o, 0)
        mask[I[ok], lo[ok] // block] = True
        mask[I[ok], hi[ok] // block] = True
    return mask & causal


# ------------------------------------------------------------------ Algorithm 4

def query_aware_block_attention(q_seq: np.ndarray, k_seq: np.ndarray, block: int,
                                scale: float) -> np.ndarray:
    """A_bar = softmax(avgpool(Q) avgpool(K)^T / sqrt d) with block-causal rows (Algorithm 4,
    first two steps; R2, R10).  Returns [nb, nb] float64, zero above the diagonal."""
    q_bar = _avgpool_rows(q_seq, block)
    k_bar = _avgpool_rows(k_seq, block)
    logits = (q_bar @ k_bar.T) * scale
    nb = logits.shape[0]
    causal = np.arange(nb)[None, :] <= np.arange(nb)[:, None]
    return _softmax_rows(np.where(causal, logits, -np.inf))


def query_aware_index(a_bar_map: np.ndarray, gamma: float):
    """Algorithm 4: flatten and normalise the causal entries of A_bar (unit id u = I*nb + J,
    row-major), argsort, keep the minimal prefix with mass >= gamma.  Returns
    (selection over the flat causal units, flat unit ids)."""
    nb = a_bar_map.shape[0]
    I, J = np.tril_indices(nb)
    flat = a_bar_map[I, J]
    flat = flat / np.sum(flat)
    sel = cumulative_select(flat, gamma)
    unit_ids = I * nb + J
    return sel, unit_ids


def query_aware_index_rows(a_bar_map: np.ndarray, gamma: float):
    """Query-wise variant of Algorithm 4 (R11): for each query block I, the key blocks
    J <= I scored by A_bar[I, J] / sum_J A_bar[I, J], argsorted, and the minimal prefix with
    mass >= gamma.  Returns one Selection per query block (unit id = J)."""
    nb = a_bar_map.shape[0]
    sels = []
    for I in range(nb):
        row = a_bar_map[I, :I + 1]
        sels.append(cumulative_select(row / np.sum(row), gamma))
    return sels


def tiles_from_query_aware_rows(sels, nb: int) -> np.ndarray:
    mask = np.zeros((nb, nb), dtype=bool)
    for I, sel in enumerate(sels):
        mask[I, sel.selected] = True
    return mask


def tiles_from_query_aware(selected_units: np.ndarray, nb: int) -> np.ndarray:
    mask = np.zeros((nb, nb), dtype=bool)
    su = np.asarray(selected_units, dtype=np.int64)
    mask[su // nb, su % nb] = True
    return mask


# ------------------------------------------------------------------ guards (R8)

def add_forced_and_min_budget(mask: np.ndarray, pattern: int, min_budget: int,
                              a_bar_map: np.ndarray | None = None) -> np.ndarray:
    """Keep the first and the diagonal key block of every query block, then top each row
    up to min(m, I + 1) key blocks (Section 4.1, implementation details; R8)."""
    mask = mask.copy()
    nb = mask.shape[0]
    for I in range(nb):
        mask[I, 0] = True
        mask[I, I] = True
        target = min(int(min_budget), I + 1)
        have = int(np.count_nonzero(mask[I, :I + 1]))
        if have >= target:
            continue
        if pattern == PATTERN_QA:
            cand = np.arange(I + 1)
            order = cand[np.lexsort((cand, -a_bar_map[I, :I + 1]))]
        else:
            order = np.arange(I - 1, -1, -1)
        for J in order:
            if have >= target:
                break
            if not mask[I, J]:
                mask[I, J] = True
                have += 1
    return mask


def row_priority(I: int, pattern: int, a_bar_map: np.ndarray | None = None) -> np.ndarray:
    """Key blocks of row I in the order R8 adds them and R12 keeps them: pooled score
    descending then J ascending (query-aware), or nearest to the diagonal first
    (vertical-slash)."""
    if pattern == PATTERN_QA:
        cand = np.arange(I + 1)
        return cand[np.lexsort((cand, -a_bar_map[I, :I + 1]))]
    return np.arange(I, -1, -1)


def apply_max_budget(mask: np.ndarray, pattern: int, max_budget: int,
                     a_bar_map: np.ndarray | None = None) -> np.ndarray:
    """Cap every row at max_budget key blocks (R12): blocks 0 and I first, then the row's
    other blocks in row_priority order.  max_budget <= 0 leaves the mask unchanged."""
    if max_budget <= 0:
        return mask
    mask = mask.copy()
    nb = mask.shape[0]
    for I in range(nb):
        if int(np.count_nonzero(mask[I, :I + 1])) <= max_budget:
            continue
        keep = {0, I}
        for J in row_priority(I, pattern, a_bar_map):
            if len(keep) >= max_budget:
                break
            if mask[I, J]:
                keep.add(int(J))
        mask[I, :] = False
        mask[I, sorted(keep)] = True
    return mask


# ------------------------------------------------------------------ Algorithm 1 selection part

def select_head(q_seq, k_seq, block, gamma, tau, min_budget, scale, force_pattern=-1,
                keep_detail=False, max_budget=0, qa_mode=0, vs_granularity=0):
    """Pattern search and index selection for one head of one sequence (Algorithm 1 up to
    the final attention).  qa_mode 0 selects query-aware units over the flattened map
    (Algorithm 4), 1 per query block (R11); max_budget caps the rows (R12);
    vs_granularity 0 selects token lines (Algorithm 3), 1 block-pooled lines (R13).
    Returns a dict with pattern, d_js, tile mask and counts."""
    n = q_seq.shape[0]
    nb = -(-n // block)
    if gamma >= 1.0:                                          # R9
        mask = np.tril(np.ones((nb, nb), dtype=bool))
        return dict(pattern=PATTERN_DENSE, js=float("nan"), mask=mask, units=(nb * (nb + 1) // 2,
                    0), detail=None)
    pattern, d_js, a_bar, a_blk, a_full, rows = sparse_pattern_search(q_seq, k_seq, block, tau,
                                                                      scale)
    if force_pattern in (PATTERN_QA, PATTERN_VS):
        pattern = force_pattern
    detail = dict(a_bar=a_bar, a_blk=a_blk) if keep_detail else None
    if pattern == PATTERN_QA:
        a_map = query_aware_block_attention(q_seq, k_seq, block, scale)
        if qa_mode == 1:
            row_sels = query_aware_index_rows(a_map, gamma)
            mask = tiles_from_query_aware_rows(row_sels, nb)
            units = (sum(sl.k for sl in row_sels), 0)
            if keep_detail:
                detail.update(qa_rows=row_sels, a_map=a_map)
        else:
            sel, unit_ids = query_aware_index(a_map, gamma)
            mask = tiles_from_query_aware(unit_ids[sel.selected], nb)
            units = (sel.k, 0)
            if keep_detail:
                detail.update(qa=sel, unit_ids=unit_ids, a_map=a_map)
        mask = add_forced_and_min_budget(mask, PATTERN_QA, min_budget, a_map)
        mask = apply_max_budget(mask, PATTERN_QA, max_budget, a_map)
    else:
        if vs_granularity == 1:
            sel_v, sel_s, a_v, a_s = vertical_slash_index_pooled(a_full, rows, gamma, block)
            mask = tiles_from_vertical_slash(lines_of_blocks(sel_v.selected, n, block),
                                             lines_of_blocks(sel_s.selected, n, block), n,
                                             block)
        else:
            sel_v, sel_s, a_v, a_s = vertical_slash_index(a_full, rows, gamma)
            mask = tiles_from_vertical_slash(sel_v.selected, sel_s.selected, n, block)
        mask = add_forced_and_min_budget(mask, PATTERN_VS, min_budget)
        mask = apply_max_budget(mask, PATTERN_VS, max_budget)
        units = (sel_v.k, sel_s.k)
        if keep_detail:
            detail.update(v=sel_v, s=sel_s, a_v=a_v, a_s=a_s)
    return dict(pattern=pattern, js=d_js, mask=mask, units=units, detail=detail)


def select(q, k, cu_seqlens, block, gamma, tau, min_budget, scale=None, force_pattern=None,
           heads=None, keep_detail=False, max_budget=0, qa_mode=0, vs_granularity=0):
    """Selection for a packed layer.  q: [T, Hq, d], k: [T, Hkv, d].  Returns a list over
    sequences of lists over heads (None for heads not requested) of select_head dicts.
    force_pattern: None, or an int (all heads), or a dict {(seq, head): pattern}."""
    hq, hkv, d = q.shape[1], k.shape[1], q.shape[2]
    group = hq // hkv
    scale = 1.0 / math.sqrt(d) if not scale else float(scale)
    out = []
    for s in range(len(cu_seqlens) - 1):
        t0, t1 = int(cu_seqlens[s]), int(cu_seqlens[s + 1])
        per_head = []
        for h in range(hq):
            if heads is not None and h not in heads:
                per_head.append(None)
                continue
            fp = -1
            if isinstance(force_pattern, dict):
                fp = force_pattern.get((s, h), -1)
            elif force_pattern is not None:
                fp = int(force_pattern)
            per_head.append(select_head(q[t0:t1, h], k[t0:t1, h // group], block, gamma, tau,
                                        min_budget, scale, fp, keep_detail, max_budget,
                                        qa_mode, vs_granularity))
        out.append(per_head)
    return out


# ------------------------------------------------------------------ A(Q, K, V, S)

def sparse_attention_rows(q_seq, k_seq, v_seq, mask, block, scale, row_blocks=None):
    """A(Q, K, V, S) (Section 2, sparse attention with mask M_S) computed by gathering, for
    each query block I, the keys of its marked tiles and applying the causal limit
    j <= i.  Returns {I: [rows of block I, d] float64}."""
    n = q_seq.shape[0]
    nb = -(-n // block)
    q64 = np.asarray(q_seq, dtype=np.float64)
    k64 = np.asarray(k_seq, dtype=np.float64)
    v64 = np.asarray(v_seq, dtype=np.float64)
    out = {}
    for I in (range(nb) if row_blocks is None else row_blocks):
        i_idx = np.arange(I * block, min((I + 1) * block, n))
        tiles = np.nonzero(mask[I, :I + 1])[0]
        j_idx = np.concatenate([np.arange(J * block, min((J + 1) * block, n)) for J in tiles]) \
            if tiles.size else np.zeros(0, dtype=np.int64)
        logits = (q64[i_idx] @ k64[j_idx].T) * scale
        logits = np.where(j_idx[None, :] <= i_idx[:, None], logits, -np.inf)
        p = _softmax_rows(logits)
        out[int(I)] = p @ v64[j_idx]
    return out


def sparse_attention_masked(q_seq, k_seq, v_seq, mask, block, scale):
    """Same result from the dense formulation: softmax((Q K^T + M_S) / sqrt d) V with
    M_S = 0 on S and -inf elsewhere (Section 2).  Small n only.  Returns [n, d]."""
    n = q_seq.shape[0]
    q64 = np.asarray(q_seq, dtype=np.float64)
    k64 = np.asarray(k_seq, dtype=np.float64)
    v64 = np.asarray(v_seq, dtype=np.float64)
    i = np.arange(n)[:, None]
    j = np.arange(n)[None, :]
    in_s = (j <= i) & mask[i // block, j // block]
    m_s = np.where(in_s, 0.0, -np.inf)
    return _softmax_rows((q64 @ k64.T + m_s) * scale) @ v64


def dense_causal_attention(q_seq, k_seq, v_seq, scale):
    """Full causal attention: every j <= i."""
    n = q_seq.shape[0]
    q64 = np.asarray(q_seq, dtype=np.float64)
    k64 = np.asarray(k_seq, dtype=np.float64)
    v64 = np.asarray(v_seq, dtype=np.float64)
    logits = (q64 @ k64.T) * scale
    logits = np.where(np.arange(n)[None, :] <= np.arange(n)[:, None], logits, -np.inf)
    return _softmax_rows(logits) @ v64
