"""fp_sparse_attn_noalloc (the entry point whose workspace is the library's fixed device
scratch array) against fp_sparse_attn on the same inputs and lists, through the C ABI:
two calls in a row, the second on a smaller problem, each compared with the workspace
entry point's output and with the oracle on sampled rows."""
import numpy as np
import pytest

import synth
from parity import O_MAX_ABS, O_MEAN_ABS, compare_outputs, log, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2502_20766_amd as fpx
    fpx.lib()
    return fpx


def _case(seqlens, hq, hkv, gamma):
    import paper_2502_20766_amd as fpx
    kinds = tuple("vs" if h % 2 == 0 else "qa" for h in range(hq))
    spec = synth.LayerSpec(f"noalloc-{sum(seqlens)}", seqlens, hq, hkv, 128, 128, kinds, 16,
                           gamma, 0.1, 8, 4711 + sum(seqlens))
    layer = synth.make_layer(spec)
    q, k, v = to_device(layer)
    idx = fpx.select(q, k, layer.cu_seqlens, gamma, spec.tau, spec.min_budget)
    ws_bytes = fpx.attn_workspace_size(idx.shape)
    assert ws_bytes <= fpx.NOALLOC_SCRATCH_BYTES
    return layer, q, k, v, idx


def test_noalloc_matches_workspace_entry_point_twice():
    import paper_2502_20766_amd as fpx
    cases = [((9000, 300, 4100), 8, 2, 0.9), ((2048, 1), 4, 2, 0.95)]   # the second is smaller
    for seqlens, hq, hkv, gamma in cases:
        log(f"[noalloc] seqlens={seqlens} hq={hq} hkv={hkv}")
        layer, q, k, v, idx = _case(seqlens, hq, hkv, gamma)
        o_ref = fpx.sparse_attn(q, k, v, idx)
        o_na = torch.full_like(q, float("nan"))
        fpx.sparse_attn_noalloc(q, k, v, idx, o_na)
        torch.cuda.synchronize()
        a, b = o_ref.float().cpu().numpy(), o_na.float().cpu().numpy()
        assert np.all(np.isfinite(b))
        diff = np.abs(a - b)
        log(f"  vs fp_sparse_attn: max_abs {diff.max():.3e}")
        assert diff.max() <= O_MAX_ABS and diff.mean() <= O_MEAN_ABS
        masks = fpx.masks_from_indices(idx)
        mx, mean = compare_outputs(layer, b, masks, rows_per_head=6)
        log(f"  vs oracle: max_abs {mx:.3e} mean_abs {mean:.3e}")
        assert mx <= O_MAX_ABS and mean <= O_MEAN_ABS


def test_noalloc_rejects_problems_beyond_the_scratch():
    import paper_2502_20766_amd as fpx
    shape = fpx.Shape(np.array([0, 131072], dtype=np.int32), 32, 8, 128)
    assert fpx.attn_workspace_size(shape) > fpx.NOALLOC_SCRATCH_BYTES
    q = torch.zeros((131072, 32, 128), dtype=torch.bfloat16, device="cuda")
    k = torch.zeros((131072, 8, 128), dtype=torch.bfloat16, device="cuda")
    idx = fpx.empty_indices(shape, q.device)
    with pytest.raises(fpx.FlexPrefillError) as e:
        fpx.sparse_attn_noalloc(q, k, k, idx, q)
    assert e.value.status == fpx.FP_ERR_WORKSPACE
