"""The layer (fp_select, then fp_sparse_attn or fp_sparse_attn_noalloc) captured into a HIP
graph and replayed.  Both calls enqueue kernel launches only (no memsets, no host
synchronisation, no allocation once their buffers are given), so a caller can capture them;
every replay, with eager work and synchronisations in between, must reproduce the eager
results bit for bit (selection and attention are deterministic)."""
import numpy as np
import pytest

import synth
from parity import log, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

REPLAYS = 4


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2502_20766_amd as fpx
    fpx.lib()
    return fpx


def _layer():
    kinds = ("vs", "qa", "vs", "qa", "qa", "vs", "vs", "qa")
    spec = synth.LayerSpec("graph-8h-n12k", (8192, 300, 3500), 8, 2, 128, 128, kinds, 16, 0.9,
                           0.1, 8, 20250228 + 77)
    layer = synth.make_layer(spec)
    return spec, layer


def _index_arrays(idx):
    return [x.cpu().numpy().copy() for x in (idx.kb_idx, idx.kb_cnt, idx.pattern, idx.js,
                                             idx.units)]


@pytest.mark.parametrize("noalloc", [False, True], ids=["workspace", "noalloc"])
def test_layer_graph_replays_match_eager(noalloc):
    import paper_2502_20766_amd as fpx
    spec, layer = _layer()
    q, k, v = to_device(layer)
    cu = layer.cu_seqlens
    shape = fpx.Shape(cu, spec.hq, spec.hkv, spec.d, spec.block)
    p = fpx.params(spec.gamma, spec.tau, spec.min_budget)
    ws_sel = torch.empty(max(fpx.select_workspace_size(shape, p), 1), dtype=torch.uint8,
                         device=q.device)
    ws_att = torch.empty(max(fpx.attn_workspace_size(shape), 1), dtype=torch.uint8,
                         device=q.device)
    idx = fpx.empty_indices(shape, q.device)
    o = torch.empty_like(q)

    def layer_step():
        fpx.select(q, k, cu, spec.gamma, spec.tau, spec.min_budget, out=idx, workspace=ws_sel)
        if noalloc:
            fpx.sparse_attn_noalloc(q, k, v, idx, o)
        else:
            fpx.sparse_attn(q, k, v, idx, out=o, workspace=ws_att)

    def clobber():
        # every output overwritten with a known pattern (entries past a row's list stay so)
        o.fill_(float("nan"))
        for x in (idx.kb_idx, idx.kb_cnt, idx.units):
            x.fill_(-7)
        idx.pattern.fill_(255)
        idx.js.fill_(float("nan"))

    # eager reference (this also resolves the no-allocation scratch address before capture)
    clobber()
    layer_step()
    torch.cuda.synchronize()
    ref_idx, ref_o = _index_arrays(idx), o.view(torch.int16).cpu().numpy().copy()
    assert np.all(np.isfinite(o.float().cpu().numpy()))

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):        # warm-up on the capture stream, as torch advises
        layer_step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        layer_step()
    torch.cuda.synchronize()

    junk = torch.randn(1 << 20, device=q.device)
    for r in range(REPLAYS):
        # eager work between the replays: overwrite every output, run an unrelated kernel
        clobber()
        junk.mul_(1.0001)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got_idx = _index_arrays(idx)
        for name, a, b in zip(("kb_idx", "kb_cnt", "pattern", "js", "units"), ref_idx, got_idx):
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), (r, name)
        assert np.array_equal(ref_o, o.view(torch.int16).cpu().numpy()), r
        log(f"[graph] {'noalloc' if noalloc else 'workspace'} replay {r}: identical to eager")
