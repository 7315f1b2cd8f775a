"""The C ABI library: it loads on a machine without a GPU, exports every entry point the
header declares, and rejects every invalid argument on the host (fp_validate and the
size queries touch no device)."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2502_20766_amd as fpx

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "flexprefill.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(fpx.LIB_PATH):
        from paper_2502_20766_amd import _build
        _build.build()
    return fpx.lib()


def _declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fp_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    syms = _declared_symbols()
    assert {"fp_select", "fp_sparse_attn", "fp_validate", "fp_indices_size",
            "fp_select_workspace_size", "fp_attn_workspace_size", "fp_status_string",
            "fp_last_error"} <= set(syms)
    for s in syms:
        assert hasattr(lib, s), s


def test_status_strings(lib):
    for code in range(5):
        assert lib.fp_status_string(code)
    assert lib.fp_last_error() == b""


def _shape(cu=(0, 2048), hq=2, hkv=2, d=64, block=128):
    return fpx.Shape(np.array(cu, dtype=np.int32), hq, hkv, d, block)


def test_sizes(lib):
    sh = _shape(cu=(0, 300, 429, 1453), hq=4, hkv=2, d=128)
    n_idx, n_cnt = fpx.indices_size(sh)
    nbs = np.array([3, 2, 8])
    assert n_cnt == 4 * nbs.sum()
    assert n_idx == 4 * int((nbs * (nbs + 1) // 2).sum())
    p = fpx.params(0.9, 0.1, 8)
    ws = fpx.select_workspace_size(sh, p)
    assert ws > 0 and ws % 256 == 0
    assert fpx.select_workspace_size(sh, fpx.params(1.0, 0.1, 8)) == 0
    # attention: 16-byte work items per query head and block, 8 counters, one V^T copy, the
    # items' 8-byte sort keys and 16-byte unsorted records
    nb = int(nbs.sum())
    need = 16 * 4 * nb + 8 * 4 + 2 * 2 * nb * 128 * 128 + (8 + 16) * 4 * nb
    assert need <= fpx.attn_workspace_size(sh) <= need + 5 * 256
    # larger problems need no less workspace
    sh2 = _shape(cu=(0, 300, 429, 4000), hq=4, hkv=2, d=128)
    assert fpx.select_workspace_size(sh2, p) >= ws


@pytest.mark.parametrize("kw,status", [
    (dict(hq=3, hkv=2), fpx.FP_ERR_INVALID_ARG),
    (dict(hq=0), fpx.FP_ERR_INVALID_ARG),
    (dict(d=96), fpx.FP_ERR_UNSUPPORTED),
    (dict(block=32), fpx.FP_ERR_UNSUPPORTED),
    (dict(block=64), fpx.FP_OK),
    (dict(block=64, cu=(0, 8192 * 64 + 1)), fpx.FP_ERR_UNSUPPORTED),  # > 8192 blocks
    (dict(cu=(0, 100, 90)), fpx.FP_ERR_INVALID_ARG),      # non-monotone
    (dict(cu=(0, 100, 100)), fpx.FP_ERR_INVALID_ARG),     # empty sequence
    (dict(cu=(5, 100)), fpx.FP_ERR_INVALID_ARG),          # cu[0] != 0
    (dict(cu=tuple(range(0, 66 * 10, 10))), fpx.FP_ERR_UNSUPPORTED),   # batch > 64
    (dict(cu=(0, 8192 * 128 + 1)), fpx.FP_ERR_UNSUPPORTED),            # > 1M tokens
])
def test_validate_shape_errors(lib, kw, status):
    sh = _shape(**kw)
    assert fpx.validate(sh, fpx.params(0.9, 0.1, 1), 1 << 40) == status
    assert fpx.validate(sh, None, 1 << 40) == status


@pytest.mark.parametrize("p,status", [
    (dict(gamma=0.0, tau=0.1), fpx.FP_ERR_INVALID_ARG),
    (dict(gamma=-0.5, tau=0.1), fpx.FP_ERR_INVALID_ARG),
    (dict(gamma=1.5, tau=0.1), fpx.FP_ERR_INVALID_ARG),
    (dict(gamma=float("nan"), tau=0.1), fpx.FP_ERR_INVALID_ARG),
    (dict(gamma=0.9, tau=-0.1), fpx.FP_ERR_INVALID_ARG),
    (dict(gamma=0.9, tau=1.5), fpx.FP_ERR_INVALID_ARG),
    (dict(gamma=0.9, tau=0.1, min_budget=-1), fpx.FP_ERR_INVALID_ARG),
    (dict(gamma=0.9, tau=0.1, min_budget=65), fpx.FP_ERR_UNSUPPORTED),
    (dict(gamma=0.9, tau=0.1, softmax_scale=-1.0), fpx.FP_ERR_INVALID_ARG),
    (dict(gamma=0.9, tau=0.1, force_pattern=2), fpx.FP_ERR_INVALID_ARG),
    (dict(gamma=0.9, tau=0.1, max_budget=-1), fpx.FP_ERR_INVALID_ARG),
    (dict(gamma=0.9, tau=0.1, max_budget=1), fpx.FP_ERR_INVALID_ARG),     # cannot hold 0, I
    (dict(gamma=0.9, tau=0.1, min_budget=8, max_budget=4), fpx.FP_ERR_INVALID_ARG),
    (dict(gamma=0.9, tau=0.1, min_budget=8, max_budget=8), fpx.FP_OK),
    (dict(gamma=0.9, tau=0.1, min_budget=2, max_budget=2), fpx.FP_OK),
    (dict(gamma=0.9, tau=0.1, qa_mode=2), fpx.FP_ERR_INVALID_ARG),
    (dict(gamma=0.9, tau=0.1, qa_mode=1), fpx.FP_OK),
    (dict(gamma=0.9, tau=0.1, vs_granularity=-1), fpx.FP_ERR_INVALID_ARG),
    (dict(gamma=0.9, tau=0.1, vs_granularity=2), fpx.FP_ERR_INVALID_ARG),
    (dict(gamma=0.9, tau=0.1, vs_granularity=1), fpx.FP_OK),
    (dict(gamma=0.9, tau=0.1), fpx.FP_OK),
    (dict(gamma=1.0, tau=0.0, min_budget=64, force_pattern=1), fpx.FP_OK),
])
def test_validate_param_errors(lib, p, status):
    assert fpx.validate(_shape(), fpx.params(**p), 1 << 40) == status


def test_validate_workspace(lib):
    sh = _shape()
    p = fpx.params(0.9, 0.1, 1)
    need = fpx.select_workspace_size(sh, p)
    assert fpx.validate(sh, p, need) == fpx.FP_OK
    assert fpx.validate(sh, p, need - 1) == fpx.FP_ERR_WORKSPACE
    need_a = fpx.attn_workspace_size(sh)
    assert fpx.validate(sh, None, need_a) == fpx.FP_OK
    assert fpx.validate(sh, None, need_a - 1) == fpx.FP_ERR_WORKSPACE


def test_null_pointers_rejected_before_any_launch(lib):
    sh = _shape()
    p = fpx.params(0.9, 0.1, 1)
    assert lib.fp_validate(None, ctypes.byref(p), 0) == fpx.FP_ERR_INVALID_ARG
    bad = fpx.FpShape(1, None, 2, 2, 64, 128)
    assert lib.fp_validate(ctypes.byref(bad), ctypes.byref(p), 1 << 40) == fpx.FP_ERR_INVALID_ARG
    idx = fpx.FpIndices(None, None, None, None, None, 0.0)
    # null tensors: rejected on the host, nothing enqueued
    st = lib.fp_select(ctypes.byref(sh.c), None, None, ctypes.byref(p), ctypes.byref(idx), None,
                       1 << 30, None)
    assert st == fpx.FP_ERR_INVALID_ARG
    st = lib.fp_sparse_attn(ctypes.byref(sh.c), None, None, None, ctypes.byref(idx), None,
                            None, 1 << 30, None)
    assert st == fpx.FP_ERR_INVALID_ARG
    # workspace check comes first for a too-small size
    st = lib.fp_select(ctypes.byref(sh.c), None, None, ctypes.byref(p), ctypes.byref(idx), None,
                       0, None)
    assert st == fpx.FP_ERR_WORKSPACE


def test_product_path_has_no_oracle_dependency():
    """The binding and the native sources never reference the oracle package."""
    pkg = os.path.dirname(fpx.__file__)
    for root, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".cpp", ".h")):
                text = open(os.path.join(root, f)).read()
                assert "import oracle" not in text and "from oracle" not in text, f


@pytest.mark.parametrize("scale,status", [
    (-1.0, fpx.FP_ERR_INVALID_ARG), (float("nan"), fpx.FP_ERR_INVALID_ARG),
    (float("inf"), fpx.FP_ERR_INVALID_ARG)])
def test_attention_scale_comes_from_the_indices_and_is_checked(lib, scale, status):
    """fp_sparse_attn takes its softmax scale from fp_indices.softmax_scale (the scale
    fp_select used); an invalid one is rejected on the host before anything is enqueued.
    The pointers are never dereferenced: the check fails first."""
    sh = _shape()
    ws = fpx.attn_workspace_size(sh)
    fake = ctypes.c_void_p(16)
    idx = fpx.FpIndices(16, 16, 16, 16, 16, scale)
    st = lib.fp_sparse_attn(ctypes.byref(sh.c), fake, fake, fake, ctypes.byref(idx), fake, fake,
                            ws, None)
    assert st == status


def test_fp_indices_layout_matches_the_header():
    """The binding's ctypes mirror of fp_indices has the header's field order and offsets."""
    text = open(HEADER).read()
    body = re.search(r"typedef struct fp_indices \{(.*?)\} fp_indices;", text, re.S).group(1)
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    fields = re.findall(r"\b([a-z_]+);", body)
    assert fields == [f[0] for f in fpx.FpIndices._fields_]
    assert fpx.FpIndices.softmax_scale.offset == 5 * ctypes.sizeof(ctypes.c_void_p)


SH = dict(cu=(0, 300, 1000), hq=4, hkv=2, d=128)


@pytest.mark.parametrize("kw,ok", [
    (dict(q=(1000, 4, 128), k=(1000, 2, 128), v=(1000, 2, 128), o=(1000, 4, 128)), True),
    (dict(q=(999, 4, 128)), False),                 # T differs from cu_seqlens[-1]
    (dict(k=(1001, 2, 128)), False),
    (dict(q=(1000, 2, 128)), False),                # query heads
    (dict(k=(1000, 4, 128)), False),                # KV heads
    (dict(k=(1000, 2, 64)), False),                 # head dim
    (dict(v=(1000, 2, 64)), False),                 # v must match k
    (dict(o=(1000, 4, 64)), False),                 # out must match q
    (dict(o=(1000, 4)), False),
])
def test_check_shapes_tensors(lib, kw, ok):
    sh = _shape(**SH)
    if ok:
        fpx.check_shapes(sh, **kw)
    else:
        with pytest.raises(ValueError):
            fpx.check_shapes(sh, **kw)


def test_check_shapes_index_buffers(lib):
    sh = _shape(**SH)
    n_idx, n_cnt = fpx.indices_size(sh)
    b, hq = 2, 4
    fpx.check_shapes(sh, index_lens=(n_idx, n_cnt, b * hq, b * hq, b * hq * 2))
    for i, short in enumerate((n_idx - 1, n_cnt - 1, b * hq - 1, b * hq - 1, b * hq * 2 - 1)):
        lens = [n_idx, n_cnt, b * hq, b * hq, b * hq * 2]
        lens[i] = short
        with pytest.raises(ValueError):
            fpx.check_shapes(sh, index_lens=tuple(lens))
