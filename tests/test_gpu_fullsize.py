"""Device path vs oracle at the full workload sizes, in the launch configuration the benchmark
times (same library calls, same shapes).  Block sets are compared for every head and
sequence; outputs on sampled query blocks (first, last and 62 seeded random rows of every
head and sequence), which the oracle computes one block at a time.  Every relaxation count
(cuts inside the gamma band, order ties, near-tie exchanges) is asserted against its stated
maximum."""
import numpy as np
import pytest

import synth
from parity import (O_MAX_ABS, O_MEAN_ABS, Timer, assert_relaxations_bounded, compare_outputs,
                    compare_selection, log, to_device)

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2502_20766_amd as fpx
    fpx.lib()
    return fpx


CASES = [
    ("llama3-8b-n32768", "llama32k", None),
    ("llama3-8b-n131072", "llama128k", None),
    ("glm4-9b-n65536", "glm64k", None),
    ("qwen2-7b-varlen-gamma0.85", "qwen_varlen", 0.85),
    ("qwen2-7b-varlen-gamma0.9", "qwen_varlen", 0.9),
    ("qwen2-7b-varlen-gamma0.95", "qwen_varlen", 0.95),
]
ROWS_PER_HEAD = 64          # first, last and 62 seeded random query blocks


def _check_layer(name, spec, gamma, max_budget=0, qa_mode=0, vs_granularity=0):
    import paper_2502_20766_amd as fpx
    log(f"[fullsize] {name}: seqlens={spec.seqlens} hq={spec.hq} hkv={spec.hkv} gamma={gamma} "
        f"tau={spec.tau} m={spec.min_budget} max_budget={max_budget} qa_mode={qa_mode} "
        f"vs_granularity={vs_granularity}")
    with Timer("generate"):
        layer = synth.make_layer(spec)
    q, k, v = to_device(layer)
    with Timer("device select + attention"):
        idx = fpx.select(q, k, layer.cu_seqlens, gamma, spec.tau, spec.min_budget,
                         block=spec.block, max_budget=max_budget, qa_mode=qa_mode,
                         vs_granularity=vs_granularity)
        o = fpx.sparse_attn(q, k, v, idx)
        torch.cuda.synchronize()
    g = dict(masks=fpx.masks_from_indices(idx), pattern=idx.pattern.cpu().numpy(),
             js=idx.js.cpu().numpy(), units=idx.units.cpu().numpy())
    if max_budget:
        assert int(idx.kb_cnt.max()) <= max_budget
    o_host = o.float().cpu().numpy()
    del q, k, v, o
    with Timer("oracle selection, all heads"):
        st = compare_selection(layer, g, gamma, spec.tau, spec.min_budget,
                               max_budget=max_budget, qa_mode=qa_mode,
                               vs_granularity=vs_granularity)
    log(f"  {st}")
    assert_relaxations_bounded(st)
    with Timer("oracle sampled outputs"):
        mx, mean = compare_outputs(layer, o_host, g["masks"], rows_per_head=ROWS_PER_HEAD)
    log(f"  output max_abs {mx:.3e} mean_abs {mean:.3e}")
    assert mx <= O_MAX_ABS and mean <= O_MEAN_ABS


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_fullsize_selection_and_sampled_outputs(case):
    name, key, gamma = case
    spec = synth.SPECS[key]
    _check_layer(name, spec, spec.gamma if gamma is None else gamma)


def test_fullsize_block64():
    """The 128k Llama-shaped layer with key blocks of 64 tokens (up to 2048 blocks per row,
    twice the attention items of block 128): every block set against the oracle, outputs on
    sampled query blocks."""
    spec = synth.SPECS["llama128k"].with_params(block=64)
    _check_layer("llama3-8b-n131072-block64", spec, spec.gamma)


def test_fullsize_block_pooled_lines():
    """The 128k Llama-shaped layer with block-pooled vertical-slash lines (key blocks and
    offset blocks of lines as the selection units) at gamma 0.9."""
    spec = synth.SPECS["llama128k"]
    _check_layer("llama3-8b-n131072-pooled-lines", spec, 0.9, vs_granularity=1)


def test_maximum_sequence_length():
    """One sequence at the longest supported length: 8192 blocks of 128 tokens (1,048,576
    tokens), a vertical-slash and a query-aware head over one KV head.  Every block set is
    checked against the oracle, outputs on sampled query blocks.  The attention work order of
    this shape (2 heads x 8192 blocks in the KV group) is exactly the in-LDS sort's capacity."""
    from synth.layers import LayerSpec
    spec = LayerSpec("max-2h-n1048576", (1 << 20,), 2, 1, 128, 128, ("vs", "qa"), 16, 0.95,
                     0.1, 8, 20250228 + 9)
    _check_layer(spec.name, spec, spec.gamma)


@pytest.mark.parametrize("gamma", [0.85, 0.95])
def test_gamma_sweep_selection_reduced_varlen(gamma):
    """The gamma sweep of the varlen Qwen-shaped layer, on shortened sequences."""
    import paper_2502_20766_amd as fpx
    spec = synth.SPECS["qwen_varlen"].with_seqlens((2048, 4096, 8192, 16384), "qwen-varlen-short")
    log(f"[gamma sweep] {spec.name} gamma={gamma}")
    layer = synth.make_layer(spec)
    q, k, v = to_device(layer)
    idx = fpx.select(q, k, layer.cu_seqlens, gamma, spec.tau, spec.min_budget)
    o = fpx.sparse_attn(q, k, v, idx)
    torch.cuda.synchronize()
    g = dict(masks=fpx.masks_from_indices(idx), pattern=idx.pattern.cpu().numpy(),
             js=idx.js.cpu().numpy(), units=idx.units.cpu().numpy())
    st = compare_selection(layer, g, gamma, spec.tau, spec.min_budget)
    log(f"  {st}")
    assert_relaxations_bounded(st)
    mx, mean = compare_outputs(layer, o.float().cpu().numpy(), g["masks"], rows_per_head=3)
    log(f"  output max_abs {mx:.3e} mean_abs {mean:.3e}")
    assert mx <= O_MAX_ABS and mean <= O_MEAN_ABS


LONG_ROW_CASES = [
    # (log2 tokens, max_budget, qa_mode): 2048, 4096 and 8192 key blocks per row at most,
    # i.e. 8 and 16 sort slots per thread of 256, and 16 per thread of 512
    (18, 0, 1),
    (19, 24, 1),
    (20, 0, 1),
    (20, 40, 0),
]


@pytest.mark.parametrize("case", LONG_ROW_CASES, ids=[f"n2^{c[0]}-cap{c[1]}-qa{c[2]}"
                                                     for c in LONG_ROW_CASES])
def test_long_rows_per_query_block_and_capped(case):
    """Per-query-block selection and the per-row cap on rows of up to 8192 key blocks: a
    vertical-slash and a query-aware head over one KV head, every block set checked against
    the oracle, outputs on sampled query blocks."""
    from synth.layers import LayerSpec
    lg, max_budget, qa_mode = case
    spec = LayerSpec(f"rows-2h-n{1 << lg}", (1 << lg,), 2, 1, 128, 128, ("vs", "qa"), 16, 0.95,
                     0.1, 8, 20250228 + 11 + lg)
    _check_layer(spec.name, spec, spec.gamma, max_budget=max_budget, qa_mode=qa_mode)
