"""The transfer calls captured in a HIP graph: every call is stream-ordered,
allocates nothing and clears what it needs with kernels, so a captured call
replays the same work.  The graph is replayed several times with eager work
and synchronizations between the replays, and every replay must reproduce the
eager result bit for bit, on the fused path, the staged path and
hf_transfer_kv_noalloc."""

import numpy as np
import pytest

from paper_2609_32259_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch
    assert torch.cuda.is_available(), "GPU test needs a GPU"
    from paper_2609_32259_amd import heterofold
    heterofold.lib()
    return torch


@pytest.mark.parametrize("variant", ["fused", "staged", "noalloc"])
def test_transfer_replays_in_a_graph(torch, variant):
    from paper_2609_32259_amd import heterofold as hf
    from paper_2609_32259_amd.path import TransferPath
    cfg = synth.LLAMA8B_14B_8K.with_(name=f"graph {variant}", T_s=300, L_r=4)
    wl = synth.make_workload(cfg, seed=50, device="cuda")
    print(f"[gpu-graph] {variant} T_r={list(wl.seg.r_len)}", flush=True)
    path = TransferPath(wl.seg, wl.S, wl.A, wl.bias, wl.rope, cfg.L_r, cfg.H_r,
                        staged=(variant == "staged"))
    path.build_alignment()
    lmap = path.build_layer_map()

    def call():
        if variant == "noalloc":
            hf.hf_transfer_kv_noalloc(wl.seg.s_len, wl.seg.r_len, path.alignment, lmap, wl.S,
                                      path.R, path.A_packed, wl.bias, path.rope)
        else:
            path.transfer()

    call()
    torch.cuda.synchronize()
    ref = path.R.clone()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):  # captures on torch's capture stream, which the binding uses
        call()
    torch.cuda.synchronize()
    for i in range(4):
        path.R.fill_(7.0)              # eager work between the replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(path.R.view(torch.int16), ref.view(torch.int16)), f"replay {i}"
    assert bool(torch.isfinite(ref.float()).all())
