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
