"""GPU parity of the paper-faithful options (the map on x / r, Eq. 3 / 9;
the receiver's key normalization before its RoPE, App. B.1) against the
fp64 oracle, through hf_transfer_kv and hf_transfer_kv_taps."""

import numpy as np
import pytest

from paper_2609_32259_amd import synth

from _compare import Case, windows

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch
    assert torch.cuda.is_available(), "GPU test needs a GPU"
    from paper_2609_32259_amd import heterofold
    heterofold.lib()
    return torch


def _compare(torch, cfg, wl, mode="overlap", staged=None):
    from paper_2609_32259_amd.path import TransferPath
    assert wl.opts is not None
    print(f"[gpu-opts] {cfg.name} map={cfg.layer_map} post-rope keys={cfg.sender_keys_post_rope} "
          f"B={wl.seg.batch} T_r={list(wl.seg.r_len)} staged={staged}", flush=True)
    path = TransferPath(wl.seg, wl.S, wl.A, wl.bias, wl.rope, cfg.L_r, cfg.H_r, mode=mode,
                        layer_map=cfg.layer_map, opts=wl.opts, staged=staged)
    R = path.step()
    torch.cuda.synchronize()
    Case(cfg, wl, R, mode, tag="gpu-opts",
         scale_product=path.staged and cfg.layer_map == "neighbor3").check_all()


def test_opts_fp32(torch):
    cfg = synth.TINY_F32.with_(name="tiny-f32 opts", paper_opts=True, rope=(1.0e4, 5.0e5))
    _compare(torch, cfg, synth.make_workload(cfg, seed=30, device="cuda"))


def test_opts_fp32_taps_pre_rope_keys(torch):
    cfg = synth.TINY_F32.with_(name="tiny-f32 paper", paper_opts=True, rope=(1.0e4, 5.0e5),
                               layer_map="neighbor3", L_s=10, sender_keys_post_rope=False)
    _compare(torch, cfg, synth.make_workload(cfg, seed=31, device="cuda"), "ta")


@pytest.mark.parametrize("H_r", [8, 4, 2])
def test_opts_bf16_receiver_heads(torch, H_r):
    cfg = synth.LLAMA8B_14B_8K.with_(name=f"14b opts H_r={H_r}", H_r=H_r, T_s=300, L_r=4,
                                     paper_opts=True)
    _compare(torch, cfg, synth.make_workload(cfg, seed=32, device="cuda"))


@pytest.mark.parametrize("staged", [False, True], ids=["fused", "staged"])
def test_opts_bf16_inv_r_only(torch, staged):
    # 1/r without the key norm: on the interpolating map the staged path serves it
    # (the build scales the layer weights by 1/r, as the fused build does).
    cfg = synth.LLAMA8B_14B_8K.with_(name="14b 1/r only", T_s=300, L_r=4, paper_opts=True)
    wl = synth.make_workload(cfg, seed=34, device="cuda")
    opts = dict(wl.opts)
    opts["k_norm"] = None
    _compare(torch, cfg, synth.Workload(cfg, wl.seg, wl.S, wl.A, wl.bias, wl.rope, opts),
             staged=staged)


@pytest.mark.parametrize("staged", [False, True], ids=["fused", "staged"])
def test_opts_bf16_taps_inv_r_only(torch, staged):
    # Concatenated taps with 1/r and no key norm: on the staged path the common
    # multiply kernel scales the product by 1/r.
    cfg = synth.LLAMA8B_14B_32K_PAPER.with_(name="paper taps 1/r only", T_s=330, L_r=5)
    wl = synth.make_workload(cfg, seed=36, device="cuda")
    opts = dict(wl.opts)
    opts["k_norm"] = None
    _compare(torch, cfg, synth.Workload(cfg, wl.seg, wl.S, wl.A, wl.bias, wl.rope, opts),
             staged=staged)


@pytest.mark.parametrize("H_r,staged", [(8, False), (8, True), (4, False)])
def test_opts_bf16_paper_construction(torch, H_r, staged):
    # With 8 receiver heads both paths: on the staged path the key norm runs in
    # the multiply's epilogue and 1/r scales the product (the slabs of
    # concatenated taps are shared by receiver layers with different r).
    cfg = synth.LLAMA8B_14B_32K_PAPER.with_(name=f"paper small H_r={H_r}", H_r=H_r, T_s=350,
                                            L_r=5)
    _compare(torch, cfg, synth.make_workload(cfg, seed=33, device="cuda"), staged=staged)


@pytest.mark.parametrize("staged", [False, True], ids=["fused", "staged"])
def test_opts_bf16_key_norm_interpolating(torch, staged):
    # The key norm and 1/r on the interpolating map (the staged build scales the
    # features by 1/r; the multiply's epilogue normalizes the keys).
    cfg = synth.LLAMA8B_14B_8K.with_(name="14b key norm", T_s=300, L_r=4, paper_opts=True)
    _compare(torch, cfg, synth.make_workload(cfg, seed=35, device="cuda"), staged=staged)


@pytest.mark.parametrize("staged", [False, True], ids=["fused", "staged"])
@pytest.mark.parametrize("n_taps", [1, 2])
def test_opts_bf16_other_tap_counts(torch, n_taps, staged):
    # The paper's construction with one or two concatenated taps per receiver
    # layer (explicit tap tables, far-apart and repeated sender layers).
    from paper_2609_32259_amd.path import TransferPath
    cfg = synth.LLAMA8B_14B_8K.with_(name=f"14b {n_taps} taps paper", T_s=200, L_r=4,
                                     layer_map="neighbor3", paper_opts=True,
                                     sender_keys_post_rope=False)
    seg = synth.make_segmentation(cfg, seed=36)
    S = synth.make_cache(cfg, seg, seed=36, device="cuda")
    g = torch.Generator(device="cuda").manual_seed(36)
    A = (torch.randn((cfg.L_r, 2, cfg.d_r, n_taps * cfg.d_in), generator=g, device="cuda")
         / np.sqrt(n_taps * cfg.d_in)).to(torch.bfloat16)
    _, bias = synth.make_maps(cfg, seed=36, device="cuda")
    taps = np.array([[0, 31, 7][:n_taps], [5, 5, 5][:n_taps], [31, 0, 16][:n_taps],
                     [12, 13, 14][:n_taps]], np.int32)
    wl = synth.Workload(cfg, seg, S, A, bias, synth.rope_params(cfg),
                        synth.make_opts(cfg, seed=36, device="cuda"))
    print(f"[gpu-opts] {cfg.name} T_r={list(wl.seg.r_len)} staged={staged}", flush=True)
    path = TransferPath(wl.seg, wl.S, wl.A, wl.bias, wl.rope, cfg.L_r, cfg.H_r,
                        layer_map="neighbor3", opts=wl.opts, staged=staged)
    path.build_alignment()
    path.layer_map = taps
    path.transfer()
    torch.cuda.synchronize()
    Case(cfg, wl, path.R, "overlap", layer_map=taps, tag="gpu-opts",
         scale_product=path.staged).check_all()


def _random_paper_case(seed, staged):
    """A seeded irregular batch through the paper's construction: three-layer
    map, 1/r and the receiver key norm, sender keys pre- or post-RoPE; 1-4
    sequences around the tile edges, irregular receiver tokenizations (or
    none), 3-8 sender and 2-5 receiver layers, 2/4/8 receiver heads (8 on the
    staged path), per-sequence RoPE offsets, either alignment mode."""
    rng = np.random.default_rng(8000 + seed)
    H_r = 8 if staged else (2, 4, 8, 4)[seed]
    cfg = synth.LLAMA8B_14B_8K.with_(name=f"random paper batch {seed}", H_r=H_r,
                                     layer_map="neighbor3", paper_opts=True,
                                     sender_keys_post_rope=bool(seed % 2),
                                     L_s=int(rng.integers(3, 9)), L_r=int(rng.integers(2, 6)))
    parts = []
    for _ in range(int(rng.integers(1, 5))):
        sb, se = synth.segment_tokens(rng, int(rng.choice([1, 63, 64, 65, 255, 257, 400])), 1, 7)
        if rng.random() < 0.15:
            rb = re_ = np.zeros(0, np.int32)
        else:
            rb, re_ = synth.segment_messy(rng, int(se[-1]), 1, int(rng.choice([2, 8, 20])),
                                          p_empty=0.1, p_gap=0.1, p_dup_end=0.1)
        parts.append((sb, se, rb, re_))
    seg = synth.concat_segmentations(parts)
    S = synth.make_cache(cfg, seg, seed=seed, device="cuda")
    A, bias = synth.make_maps(cfg, seed=seed, device="cuda")
    rope = synth.rope_params(cfg, pos0_s=rng.integers(0, 200, seg.batch).astype(np.int32),
                             pos0_r=rng.integers(0, 200, seg.batch).astype(np.int32))
    wl = synth.Workload(cfg, seg, S, A, bias, rope, synth.make_opts(cfg, seed=seed, device="cuda"))
    return cfg, wl, ("overlap" if seed < 2 else "ta")


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("staged", [False, True], ids=["fused", "staged"])
def test_opts_bf16_random_paper_batches(torch, seed, staged):
    cfg, wl, mode = _random_paper_case(seed, staged)
    _compare(torch, cfg, wl, mode, staged=staged)


@pytest.mark.parametrize("staged", [False, True], ids=["fused", "staged"])
def test_full_14b_shape_32k_paper_construction(torch, staged):
    """The benchmark's paper-construction workload: every layer and role, on
    windows of rows, on both paths."""
    from paper_2609_32259_amd.path import TransferPath
    cfg = synth.LLAMA8B_14B_32K_PAPER
    wl = synth.make_workload(cfg, seed=0, device="cuda")
    print(f"[gpu-opts] full-size {cfg.name} T_r={list(wl.seg.r_len)} staged={staged}", flush=True)
    path = TransferPath(wl.seg, wl.S, wl.A, wl.bias, wl.rope, cfg.L_r, cfg.H_r,
                        layer_map=cfg.layer_map, opts=wl.opts, staged=staged)
    R = path.step()
    torch.cuda.synchronize()
    rng = np.random.default_rng(97)
    Case(cfg, wl, R, tag="gpu-opts-32k", scale_product=path.staged).check_all(
        windows_of=lambda b, T_r: windows(T_r, 64, rng, n_mid=2, width=384))
