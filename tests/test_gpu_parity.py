"""Device path vs oracle on the same seeded inputs (needs an MI355X and the built library).

Every case goes through the C ABI (Python binding = argument marshalling only)."""
import math
import types

import numpy as np
import pytest

import oracle
import synth
from parity import (O_MAX_ABS, O_MEAN_ABS, Timer, assert_relaxations_bounded, compare_outputs,
                    compare_selection, log, to_device)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2502_20766_amd as fpx
    fpx.lib()          # fails loudly if the library is missing
    return fpx


def _fpx():
    import paper_2502_20766_amd as fpx
    return fpx


def run_gpu(layer, gamma, tau, min_budget, force_pattern=-1, max_budget=0, qa_mode=0,
            vs_granularity=0, softmax_scale=0.0):
    fpx = _fpx()
    q, k, v = to_device(layer)
    idx = fpx.select(q, k, layer.cu_seqlens, gamma, tau, min_budget, force_pattern=force_pattern,
                     max_budget=max_budget, qa_mode=qa_mode, vs_granularity=vs_granularity,
                     softmax_scale=softmax_scale)
    o = fpx.sparse_attn(q, k, v, idx)
    torch.cuda.synchronize()
    return dict(masks=fpx.masks_from_indices(idx), pattern=idx.pattern.cpu().numpy(),
                js=idx.js.cpu().numpy(), units=idx.units.cpu().numpy(),
                o=o.float().cpu().numpy(), idx=idx, q=q, k=k, v=v)


def check_lists_structure(idx, layer, min_budget):
    """Every row ascending, unique, inside [0, I], holds 0 and I, >= min(m, I+1) blocks."""
    fpx = _fpx()
    masks = fpx.masks_from_indices(idx)
    kb_idx = idx.kb_idx.cpu().numpy()
    kb_cnt = idx.kb_cnt.cpu().numpy()
    shape = idx.shape
    nbs = shape.nb()
    tri = np.concatenate([[0], np.cumsum(nbs * (nbs + 1) // 2)])
    nb_off = np.concatenate([[0], np.cumsum(nbs)])
    hq = shape.c.num_q_heads
    for s, nb in enumerate(nbs):
        for h in range(hq):
            for I in range(nb):
                c = kb_cnt[h * nb_off[-1] + nb_off[s] + I]
                base = h * tri[-1] + tri[s] + I * (I + 1) // 2
                row = kb_idx[base:base + c]
                assert c >= min(max(min_budget, 2 if I > 0 else 1), I + 1)
                assert np.all(np.diff(row) > 0) and row[0] == 0 and row[-1] == I
    return masks


# ---------------------------------------------------------------- attention on oracle masks

ATTN_CASES = [
    # (name, seqlens, hq, hkv, d, mask density, sampled query blocks per head or None = all)
    ("tiny-dense-d64", (2048,), 2, 2, 64, 1.0, None),
    ("ragged-varlen-d128", (300, 129, 1, 1000, 128), 4, 2, 128, 0.4, None),
    ("gqa8-d128-n4096", (4096,), 8, 2, 128, 0.3, None),
    ("d64-varlen", (257, 640), 4, 4, 64, 0.5, None),
    # KV head counts that do not divide the 8 XCDs, and more than 8 of them
    ("hkv3-varlen-d128", (1500, 700), 6, 3, 128, 0.4, None),
    ("hkv16-d64", (900,), 16, 16, 64, 0.5, None),
    # more than 16384 (head, query block) items per KV group: plain dispatch order
    ("plain-order-g128-d64", (16500, 300), 128, 1, 64, 0.1, 3),
]


@pytest.mark.parametrize("case", ATTN_CASES, ids=[c[0] for c in ATTN_CASES])
def test_sparse_attention_on_oracle_masks(case):
    name, seqlens, hq, hkv, d, dens, rows = case
    log(f"[attn-oracle-masks] {name}")
    fpx = _fpx()
    kinds = tuple("vs" if h % 2 == 0 else "qa" for h in range(hq))
    spec = synth.LayerSpec(name, seqlens, hq, hkv, d, 128, kinds, 8, 0.9, 0.1, 2, 777)
    layer = synth.make_layer(spec)
    rng = np.random.default_rng(99)
    masks = {}
    for s, n in enumerate(seqlens):
        nb = -(-n // 128)
        for h in range(hq):
            m = np.tril(rng.random((nb, nb)) < dens)
            m[np.arange(nb), 0] = True
            m[np.arange(nb), np.arange(nb)] = True
            masks[(s, h)] = m
    q, k, v = to_device(layer)
    shape = fpx.Shape(layer.cu_seqlens, hq, hkv, d)
    idx = fpx.indices_from_masks(shape, masks, q.device)
    o = fpx.sparse_attn(q, k, v, idx)
    torch.cuda.synchronize()
    mx, mean = compare_outputs(layer, o.float().cpu().numpy(), masks, rows_per_head=rows)
    log(f"  max_abs {mx:.3e} mean_abs {mean:.3e}")
    assert mx <= O_MAX_ABS and mean <= O_MEAN_ABS


def test_sparse_attention_empty_rows_and_out_of_range_blocks():
    """A row with no listed blocks yields zeros; listed blocks outside [0, I] are skipped."""
    fpx = _fpx()
    spec = synth.LayerSpec("edge", (384,), 2, 1, 128, 128, ("vs", "qa"), 4, 0.9, 0.1, 1, 5)
    layer = synth.make_layer(spec)
    q, k, v = to_device(layer)
    shape = fpx.Shape(layer.cu_seqlens, 2, 1, 128)
    masks = {(0, 0): np.tril(np.ones((3, 3), bool)), (0, 1): np.tril(np.ones((3, 3), bool))}
    idx = fpx.indices_from_masks(shape, masks, q.device)
    # head 1, row 1: no blocks; head 0 row 2: first entry replaced by an invalid block 7
    nb_total = 3
    idx.kb_cnt[1 * nb_total + 1] = 0
    tri_total = 6
    idx.kb_idx[0 * tri_total + 3] = 7       # row I=2 of head 0 starts at 3: [0,1,2] -> [7,1,2]
    o = fpx.sparse_attn(q, k, v, idx).float().cpu().numpy()
    assert np.all(o[128:256, 1] == 0.0)
    m = np.tril(np.ones((3, 3), bool))
    m[2, 0] = False
    ref = oracle.sparse_attention_rows(layer.q[:, 0], layer.k[:, 0], layer.v[:, 0], m, 128,
                                       1 / math.sqrt(128), [2])
    assert np.abs(o[256:384, 0] - ref[2]).max() <= O_MAX_ABS


@pytest.mark.parametrize("block", [128, 64])
def test_sparse_attention_rising_and_jumping_scores(block):
    """Scores that rise along a row's key blocks, by less than 8 (log2 units) per block on
    head 0 and with jumps of 20-40 on head 1, so that the running reference max of the
    online softmax is kept through small rises (weights above 1) and moved on large ones."""
    fpx = _fpx()
    n, d = 2048, 128
    nb = n // block
    rng = np.random.default_rng(4242)
    scale = 1.0 / math.sqrt(d)
    u = np.ones(d) / math.sqrt(d)
    alpha = 8.0
    per_unit = alpha * scale / math.log(2.0)     # log2-domain score per unit of beta
    rises = {0: 2.5 * np.arange(nb),
             1: np.repeat(np.array([0, 0, 30, 2, 5, 40, 41, 3, 60, 58, 61, 90, 20, 95, 96, 130.0]),
                          128 // block)}
    q = np.zeros((n, 2, d), np.float32)
    k = np.zeros((n, 1, d), np.float32)
    v = rng.standard_normal((n, 1, d)).astype(np.float32)
    for h in range(2):
        q[:, h] = alpha * u + 0.05 * rng.standard_normal((n, d))
    # one KV head: the two query heads see different rises through different Q directions
    w = rng.standard_normal(d)
    w -= (w @ u) * u
    w /= np.linalg.norm(w)
    q[:, 1] = alpha * w + 0.05 * rng.standard_normal((n, d))
    for J in range(nb):
        kb = slice(J * block, (J + 1) * block)
        k[kb, 0] = ((rises[0][J] / per_unit) * u + (rises[1][J] / per_unit) * w
                    + 0.3 * rng.standard_normal((block, d)))
    q, k, v = (synth.round_to_bf16(x) for x in (q, k, v))
    masks = {(0, 0): np.tril(np.ones((nb, nb), bool))}
    m1 = np.tril(rng.random((nb, nb)) < 0.5)
    m1[np.arange(nb), 0] = True
    m1[np.arange(nb), np.arange(nb)] = True
    masks[(0, 1)] = m1
    layer = types.SimpleNamespace(q=q, k=k, v=v, cu_seqlens=np.array([0, n], np.int32),
                                  spec=types.SimpleNamespace(block=block))
    qd, kd, vd = to_device(layer)
    shape = fpx.Shape(layer.cu_seqlens, 2, 1, d, block)
    idx = fpx.indices_from_masks(shape, masks, qd.device)
    o = fpx.sparse_attn(qd, kd, vd, idx)
    torch.cuda.synchronize()
    mx, mean = compare_outputs(layer, o.float().cpu().numpy(), masks)
    log(f"[attn-rising-scores] block {block} max_abs {mx:.3e} mean_abs {mean:.3e}")
    assert mx <= O_MAX_ABS and mean <= O_MEAN_ABS


# ---------------------------------------------------------------- full path vs oracle

# the largest packed batch the ABI takes (FP_MAX_BATCH = 64 sequences), lengths from 1 token
# to ~2200 around block multiples
MAX_BATCH_SEQLENS = (1, 2, 3, 64, 65, 127, 128, 129) + tuple(
    (37 * i * i + 11 * i) % 2200 + 1 for i in range(56))
MAX_BATCH = synth.SPECS["qwen_varlen"].with_seqlens(MAX_BATCH_SEQLENS, "max-batch-64").with_params(
    hq=8, hkv=2, head_kinds=("vs", "qa") * 4)

SELECT_CASES = [
    ("tiny", synth.SPECS["tiny"], None),
    ("mixed-8h-n8192", synth.SPECS["llama32k"].with_seqlens((8192,), "mixed-8h-n8192")
     .with_params(hq=8, hkv=2, head_kinds=("vs", "qa") * 4), None),
    ("ragged-varlen", synth.SPECS["qwen_varlen"].with_seqlens((300, 129, 1, 2000, 4096),
                                                              "ragged-varlen"), None),
    ("glm-gqa16-n8192", synth.SPECS["glm64k"].with_seqlens((8192,), "glm-gqa16-n8192"), None),
    ("max-batch-64", MAX_BATCH, None),
    # d 64 with four query heads per statistics workgroup (half of its threads take no part
    # in the tile copy): 64 / 16 heads at 32k
    ("d64-gqa4-n32768", synth.SPECS["llama32k"].with_params(
        hq=64, hkv=16, d=64, head_kinds=("vs", "qa") * 32), None),
]


@pytest.mark.parametrize("case", SELECT_CASES, ids=[c[0] for c in SELECT_CASES])
def test_select_and_attention_vs_oracle(case):
    name, spec, heads = case
    log(f"[select+attn] {name} seqlens={spec.seqlens} hq={spec.hq} hkv={spec.hkv} "
        f"gamma={spec.gamma} tau={spec.tau} m={spec.min_budget}")
    layer = synth.make_layer(spec)
    g = run_gpu(layer, spec.gamma, spec.tau, spec.min_budget)
    check_lists_structure(g["idx"], layer, spec.min_budget)
    with Timer("oracle selection"):
        st = compare_selection(layer, g, spec.gamma, spec.tau, spec.min_budget)
    log(f"  {st}")
    assert_relaxations_bounded(st)
    mx, mean = compare_outputs(layer, g["o"], g["masks"], rows_per_head=6)
    log(f"  output max_abs {mx:.3e} mean_abs {mean:.3e}")
    assert mx <= O_MAX_ABS and mean <= O_MEAN_ABS


@pytest.mark.parametrize("scale_factor", [0.6, 1.5])
def test_non_default_softmax_scale(scale_factor):
    """A softmax scale other than 1/sqrt(d): the selection (every kernel that scales
    logits) and the attention (which takes the scale fp_select recorded in the indices)
    against the oracle run with the same scale."""
    spec = SELECT_CASES[1][1]
    scale = scale_factor / math.sqrt(spec.d)
    log(f"[softmax scale {scale:.5f}] {spec.name}")
    layer = synth.make_layer(spec)
    g = run_gpu(layer, spec.gamma, spec.tau, spec.min_budget, softmax_scale=scale)
    assert abs(g["idx"].softmax_scale - scale) <= 1e-7 * scale
    with Timer("oracle selection"):
        st = compare_selection(layer, g, spec.gamma, spec.tau, spec.min_budget, scale=scale)
    log(f"  {st}")
    assert_relaxations_bounded(st)
    mx, mean = compare_outputs(layer, g["o"], g["masks"], rows_per_head=6, scale=scale)
    log(f"  output max_abs {mx:.3e} mean_abs {mean:.3e}")
    assert mx <= O_MAX_ABS and mean <= O_MEAN_ABS


@pytest.mark.parametrize("force", [0, 1])
def test_forced_patterns(force):
    spec = SELECT_CASES[1][1]
    log(f"[forced pattern {force}] {spec.name}")
    layer = synth.make_layer(spec)
    g = run_gpu(layer, spec.gamma, spec.tau, spec.min_budget, force_pattern=force)
    assert np.all(g["pattern"] == force)
    # compare against the oracle with the same forced pattern
    hq = spec.hq
    ores = oracle.select(layer.q, layer.k, layer.cu_seqlens, spec.block, spec.gamma, spec.tau,
                         spec.min_budget, force_pattern=force)
    for h in range(hq):
        np.testing.assert_array_equal(g["masks"][(0, h)], ores[0][h]["mask"],
                                      err_msg=f"head {h}")


@pytest.mark.parametrize("gamma", [1.0])
def test_gamma_one_is_dense(gamma):
    spec = synth.SPECS["tiny"]
    log(f"[gamma=1 dense] {spec.name}")
    layer = synth.make_layer(spec)
    g = run_gpu(layer, gamma, spec.tau, spec.min_budget)
    assert np.all(g["pattern"] == oracle.PATTERN_DENSE)
    n = spec.seqlens[0]
    for h in range(spec.hq):
        ref = oracle.dense_causal_attention(layer.q[:, h], layer.k[:, h], layer.v[:, h],
                                            1 / math.sqrt(spec.d))
        err = np.abs(g["o"][:n, h] - ref)
        log(f"  head {h} max_abs {err.max():.3e} mean_abs {err.mean():.3e}")
        assert err.max() <= O_MAX_ABS and err.mean() <= O_MEAN_ABS


def test_tau_zero_gives_only_vertical_slash():
    spec = SELECT_CASES[1][1]
    layer = synth.make_layer(spec)
    g = run_gpu(layer, spec.gamma, 0.0, spec.min_budget)
    assert np.all(g["pattern"] == oracle.PATTERN_VS)


def test_determinism_bitwise():
    spec = SELECT_CASES[1][1]
    log(f"[determinism] {spec.name}")
    layer = synth.make_layer(spec)
    a = run_gpu(layer, spec.gamma, spec.tau, spec.min_budget)
    b = run_gpu(layer, spec.gamma, spec.tau, spec.min_budget)
    for key in ("pattern", "js", "units"):
        np.testing.assert_array_equal(a[key], b[key])
    np.testing.assert_array_equal(a["idx"].kb_cnt.cpu().numpy(), b["idx"].kb_cnt.cpu().numpy())
    for key in a["masks"]:        # the listed blocks (entries past kb_cnt are unspecified)
        np.testing.assert_array_equal(a["masks"][key], b["masks"][key])
    np.testing.assert_array_equal(a["o"], b["o"])


# ---------------------------------------------------------------- selection variants

MIXED = synth.SPECS["llama32k"].with_seqlens((8192,), "mixed-8h-n8192").with_params(
    hq=8, hkv=2, head_kinds=("vs", "qa") * 4)
RAGGED = synth.SPECS["qwen_varlen"].with_seqlens((300, 129, 1, 2000, 4096), "ragged-varlen")
GLM = synth.SPECS["glm64k"].with_seqlens((8192,), "glm-gqa16-n8192")

VARIANT_CASES = [
    # (name, spec, qa_mode, max_budget, min_budget or None = the spec's, vs_granularity)
    ("rows-mixed-8h-n8192", MIXED, 1, 0, None, 0),
    ("rows-ragged-varlen", RAGGED, 1, 0, None, 0),
    ("rows-glm-gqa16-n8192", GLM, 1, 0, None, 0),
    ("cap16-mixed-8h-n8192", MIXED, 0, 16, None, 0),
    ("rows-cap12-mixed-8h-n8192", MIXED, 1, 12, None, 0),
    ("cap2-ragged-varlen", RAGGED, 0, 2, 1, 0),
    ("rows-cap9-glm-gqa16-n8192", GLM, 1, 9, None, 0),
    ("pooled-mixed-8h-n8192", MIXED, 0, 0, None, 1),
    ("pooled-ragged-varlen", RAGGED, 0, 0, None, 1),
    ("pooled-rows-cap10-mixed-8h-n8192", MIXED, 1, 10, None, 1),
    # the ends of the minimum budget's range: none, and FP_MAX_MIN_BUDGET blocks
    ("min0-mixed-8h-n8192", MIXED, 0, 0, 0, 0),
    ("min64-ragged-varlen", RAGGED, 0, 0, 64, 0),
    ("rows-min64-glm-gqa16-n8192", GLM, 1, 0, 64, 0),
]


@pytest.mark.parametrize("case", VARIANT_CASES, ids=[c[0] for c in VARIANT_CASES])
def test_query_wise_selection_and_max_budget_vs_oracle(case):
    """Per-query-block query-aware selection, the per-row cap and block-pooled
    vertical-slash lines, against the oracle."""
    name, spec, qa_mode, max_budget, mb, vsg = case
    min_budget = spec.min_budget if mb is None else mb
    log(f"[selection variant] {name} qa_mode={qa_mode} max_budget={max_budget} m={min_budget} "
        f"vs_granularity={vsg}")
    layer = synth.make_layer(spec)
    g = run_gpu(layer, spec.gamma, spec.tau, min_budget, max_budget=max_budget, qa_mode=qa_mode,
                vs_granularity=vsg)
    check_lists_structure(g["idx"], layer, min_budget)
    if max_budget:
        assert int(g["idx"].kb_cnt.max()) <= max_budget
    with Timer("oracle selection"):
        st = compare_selection(layer, g, spec.gamma, spec.tau, min_budget,
                               max_budget=max_budget, qa_mode=qa_mode, vs_granularity=vsg)
    log(f"  {st}")
    assert_relaxations_bounded(st)
    mx, mean = compare_outputs(layer, g["o"], g["masks"], rows_per_head=4)
    log(f"  output max_abs {mx:.3e} mean_abs {mean:.3e}")
    assert mx <= O_MAX_ABS and mean <= O_MEAN_ABS


# ---------------------------------------------------------------- block 64

B64_ATTN_CASES = [
    # (name, seqlens, hq, hkv, d, mask density)
    ("b64-ragged-varlen-d128", (300, 129, 1, 1000, 64, 65), 4, 2, 128, 0.4),
    ("b64-gqa4-d64-n2048", (2048,), 8, 2, 64, 0.5),
    ("b64-dense-d128-n1000", (1000,), 2, 1, 128, 1.0),
]


@pytest.mark.parametrize("case", B64_ATTN_CASES, ids=[c[0] for c in B64_ATTN_CASES])
def test_block64_attention_on_oracle_masks(case):
    name, seqlens, hq, hkv, d, dens = case
    log(f"[b64 attn-oracle-masks] {name}")
    fpx = _fpx()
    kinds = tuple("vs" if h % 2 == 0 else "qa" for h in range(hq))
    spec = synth.LayerSpec(name, seqlens, hq, hkv, d, 64, kinds, 8, 0.9, 0.1, 2, 4242)
    layer = synth.make_layer(spec)
    rng = np.random.default_rng(64)
    masks = {}
    for s_, n in enumerate(seqlens):
        nb = -(-n // 64)
        for h in range(hq):
            m = np.tril(rng.random((nb, nb)) < dens)
            m[np.arange(nb), 0] = True
            m[np.arange(nb), np.arange(nb)] = True
            masks[(s_, h)] = m
    q, k, v = to_device(layer)
    shape = fpx.Shape(layer.cu_seqlens, hq, hkv, d, 64)
    idx = fpx.indices_from_masks(shape, masks, q.device)
    o = fpx.sparse_attn(q, k, v, idx)
    torch.cuda.synchronize()
    mx, mean = compare_outputs(layer, o.float().cpu().numpy(), masks)
    log(f"  max_abs {mx:.3e} mean_abs {mean:.3e}")
    assert mx <= O_MAX_ABS and mean <= O_MEAN_ABS


def test_block64_edges():
    """Block 64: a query block with no listed blocks gets zeros beside neighbours that list
    many; an entry outside a query block's causal range (the next query block's diagonal
    block, a block past the sequence end) is skipped; the last block is partial."""
    fpx = _fpx()
    n, nb = 300, 5      # blocks of 64, the last holding 44 tokens
    log(f"[b64 edges] n={n}")
    spec = synth.LayerSpec("b64-edges", (n,), 2, 1, 128, 64, ("vs", "qa"), 4, 0.9, 0.1, 1, 11)
    layer = synth.make_layer(spec)
    q, k, v = to_device(layer)
    shape = fpx.Shape(layer.cu_seqlens, 2, 1, 128, 64)
    full = np.tril(np.ones((nb, nb), bool))
    idx = fpx.indices_from_masks(shape, {(0, 0): full, (0, 1): full}, q.device)
    tri = [I * (I + 1) // 2 for I in range(nb + 1)]
    # head 0: row 2 [0, 1, 2] -> [3, 1, 2]; row 4 [0, 1, 2, 3, 4] -> [0, 1, 9, 3, 4]
    idx.kb_idx[tri[2]] = 3
    idx.kb_idx[tri[4] + 2] = 9
    # head 1: rows 0 and 3 list nothing (rows 1 and 2 list every block)
    idx.kb_cnt[nb + 0] = 0
    idx.kb_cnt[nb + 3] = 0
    o = fpx.sparse_attn(q, k, v, idx).float().cpu().numpy()
    assert np.all(o[0:64, 1] == 0.0) and np.all(o[192:256, 1] == 0.0)
    m0 = full.copy()
    m0[2, 0] = False
    m0[4, 2] = False
    m1 = full.copy()
    m1[0, :] = False
    m1[3, :] = False
    for h, m in ((0, m0), (1, m1)):
        rows = [I for I in range(nb) if m[I].any()]
        ref = oracle.sparse_attention_rows(layer.q[:, h], layer.k[:, 0], layer.v[:, 0], m, 64,
                                           1 / math.sqrt(128), rows)
        for I in rows:
            err = np.abs(o[I * 64:min((I + 1) * 64, n), h] - ref[I]).max()
            assert err <= O_MAX_ABS, (h, I, err)


B64_SELECT_CASES = [
    ("b64-tiny", synth.SPECS["tiny"].with_params(block=64)),
    ("b64-mixed-8h-n8192", MIXED.with_params(block=64)),
    ("b64-ragged-varlen", RAGGED.with_params(block=64)),
    ("b64-glm-gqa16-n8192", GLM.with_params(block=64)),
    ("b64-max-batch-64", MAX_BATCH.with_params(block=64)),
]


@pytest.mark.parametrize("case", B64_SELECT_CASES, ids=[c[0] for c in B64_SELECT_CASES])
def test_block64_select_and_attention_vs_oracle(case):
    """The whole path at block size 64 (block sets exact up to the gamma band, outputs on
    the device's lists)."""
    fpx = _fpx()
    name, spec = case
    log(f"[b64 select+attn] {name} seqlens={spec.seqlens} hq={spec.hq} hkv={spec.hkv}")
    layer = synth.make_layer(spec)
    q, k, v = to_device(layer)
    idx = fpx.select(q, k, layer.cu_seqlens, spec.gamma, spec.tau, spec.min_budget, block=64)
    o = fpx.sparse_attn(q, k, v, idx)
    torch.cuda.synchronize()
    g = dict(masks=fpx.masks_from_indices(idx), pattern=idx.pattern.cpu().numpy(),
             js=idx.js.cpu().numpy(), units=idx.units.cpu().numpy(),
             o=o.float().cpu().numpy(), idx=idx)
    check_lists_structure(idx, layer, spec.min_budget)
    with Timer("oracle selection"):
        st = compare_selection(layer, g, spec.gamma, spec.tau, spec.min_budget)
    log(f"  {st}")
    assert_relaxations_bounded(st)
    mx, mean = compare_outputs(layer, g["o"], g["masks"], rows_per_head=6)
    log(f"  output max_abs {mx:.3e} mean_abs {mean:.3e}")
    assert mx <= O_MAX_ABS and mean <= O_MEAN_ABS
