"""hf_transfer_kv_noalloc against hf_transfer_kv: the same kernels with the
workspace in the library's own device array.  Two calls in a row through the
C ABI, the second on a smaller batch, so the second reads an array that still
holds the first call's tables and records.  Results must be bit-identical to
hf_transfer_kv's on the same inputs, rows past each length untouched, and the
device's free memory unchanged by the call."""

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


def _batch(cfg, seed, lengths, pos0):
    rng = np.random.default_rng(seed)
    parts = []
    for n_s in lengths:
        sb, se = synth.segment_tokens(rng, n_s, *cfg.s_len)
        rb, re_ = synth.segment_chars(rng, int(se[-1]), *cfg.r_len)
        parts.append((sb, se, rb, re_))
    seg = synth.concat_segmentations(parts)
    S = synth.make_cache(cfg, seg, seed=seed, device="cuda")
    A, bias = synth.make_maps(cfg, seed=seed, device="cuda")
    rope = synth.rope_params(cfg, pos0_s=np.array(pos0[0], np.int32),
                             pos0_r=np.array(pos0[1], np.int32))
    return synth.Workload(cfg, seg, S, A, bias, rope)


def _both(torch, cfg, wl):
    from paper_2609_32259_amd import heterofold as hf
    from paper_2609_32259_amd.path import TransferPath
    print(f"[no-alloc] {cfg.name} B={wl.seg.batch} T_s={list(wl.seg.s_len)} "
          f"T_r={list(wl.seg.r_len)}", flush=True)
    T_cap = int(wl.seg.r_len.max()) + 9
    shape = (wl.seg.batch, cfg.L_r, 2, cfg.H_r, T_cap, cfg.d_h)
    R_ref = torch.full(shape, 5.0, dtype=torch.bfloat16, device="cuda")
    path = TransferPath(wl.seg, wl.S, wl.A, wl.bias, wl.rope, cfg.L_r, cfg.H_r, R=R_ref)
    path.build_alignment()
    lmap = path.build_layer_map()
    path.transfer()
    R_na = torch.full(shape, 5.0, dtype=torch.bfloat16, device="cuda")
    torch.cuda.synchronize()
    free0, _ = torch.cuda.mem_get_info()
    hf.hf_transfer_kv_noalloc(wl.seg.s_len, wl.seg.r_len, path.alignment, lmap, wl.S, R_na,
                              path.A_packed, wl.bias, path.rope)
    torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info()
    return R_ref, R_na, free0, free1


def test_noalloc_matches_transfer_kv_on_two_calls(torch):
    # First call: a batch of three 14B-shape sequences (RoPE offsets, ragged
    # tiles); second call: one shorter sequence.  Then the same pair on the
    # four-receiver-head kernel.
    for H_r in (8, 4):
        cfg = synth.LLAMA8B_14B_8K.with_(name=f"no-alloc H_r={H_r}", H_r=H_r, L_r=5)
        calls = [_batch(cfg, 50 + H_r, [1500, 37, 900], ([0, 11, 400], [3, 0, 90])),
                 _batch(cfg, 60 + H_r, [260], ([5], [0]))]
        for k, wl in enumerate(calls):
            R_ref, R_na, free0, free1 = _both(torch, cfg, wl)
            assert torch.equal(R_na.view(torch.int16), R_ref.view(torch.int16)), \
                f"H_r={H_r} call {k}: hf_transfer_kv_noalloc differs from hf_transfer_kv"
            for b in range(wl.seg.batch):
                T_r = int(wl.seg.r_len[b])
                assert bool((R_na[b, :, :, :, T_r:, :] == 5.0).all())
            assert bool((R_na[:, :, :, :, :1, :] != 5.0).any())
            if k > 0:  # the array was resolved by an earlier call: nothing new on the device
                assert free1 == free0, f"free device memory changed by {free0 - free1} bytes"


def test_noalloc_refuses_oversized_scratch(torch):
    from paper_2609_32259_amd import heterofold as hf
    from paper_2609_32259_amd.path import TransferPath
    cfg = synth.LLAMA8B_14B_8K.with_(name="no-alloc too large", L_r=2)
    wl = _batch(cfg, 70, [100], ([200_000], [0]))   # 100 MB of RoPE table rows: past the array
    path = TransferPath(wl.seg, wl.S, wl.A, wl.bias, wl.rope, cfg.L_r, cfg.H_r)
    path.build_alignment()
    lmap = path.build_layer_map()
    with pytest.raises(hf.HeteroFoldError) as ei:
        hf.hf_transfer_kv_noalloc(wl.seg.s_len, wl.seg.r_len, path.alignment, lmap, wl.S, path.R,
                                  path.A_packed, wl.bias, path.rope)
    assert ei.value.status == -6
