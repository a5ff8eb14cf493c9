"""GPU: two transfers in flight at once on two streams.

Each call keeps its state in the caller's workspace (work counter, staging
records, slabs) and takes work items from a counter without waiting on other
workgroups, so two calls with their own workspaces may run concurrently.  A
fused interpolating-map transfer and a staged three-layer-map transfer are
launched alternately on two streams (default priority), twice each per round,
and after every round both receiver caches must equal their results from a
call run alone, bit for bit.  Inputs are seeded and synthetic
(``paper_2609_32259_amd.synth``)."""

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


def test_two_transfers_on_two_streams(torch):
    from paper_2609_32259_amd.path import TransferPath
    cfg_a = synth.LLAMA8B_14B_8K.with_(name="stream a", T_s=2000, L_r=6)
    cfg_b = synth.LLAMA8B_14B_8K.with_(name="stream b", T_s=1500, L_r=6, layer_map="neighbor3")
    wl_a = synth.make_workload(cfg_a, seed=70, device="cuda")
    wl_b = synth.make_workload(cfg_b, seed=71, device="cuda")
    p_a = TransferPath(wl_a.seg, wl_a.S, wl_a.A, wl_a.bias, wl_a.rope, cfg_a.L_r, cfg_a.H_r,
                       staged=False)
    p_b = TransferPath(wl_b.seg, wl_b.S, wl_b.A, wl_b.bias, wl_b.rope, cfg_b.L_r, cfg_b.H_r,
                       layer_map="neighbor3", staged=True)
    ref_a = p_a.step().clone()
    ref_b = p_b.step().clone()
    torch.cuda.synchronize()
    s_a, s_b = torch.cuda.Stream(), torch.cuda.Stream()
    for rnd in range(3):
        print(f"[gpu-streams] round {rnd}", flush=True)
        p_a.R.zero_()
        p_b.R.zero_()
        torch.cuda.synchronize()
        for _ in range(2):
            p_a.step(stream=s_a)
            p_b.step(stream=s_b)
        torch.cuda.synchronize()
        assert torch.equal(p_a.R.view(torch.int16), ref_a.view(torch.int16)), rnd
        assert torch.equal(p_b.R.view(torch.int16), ref_b.view(torch.int16)), rnd
