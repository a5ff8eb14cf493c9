"""GPU parity of the concatenated-tap transfer (the paper's three-layer
neighbourhood map, Sec. 3.1 Eq. 1-2): hf_transfer_kv_taps against the fp64
oracle (``features_taps`` + ``map_features``, as ``transfer_taps``).  Small
cases element by element over every layer, role and row; the full-size 32K
workload on every layer and role, over windows of rows (head, tail, across
row-tile edges), in the launch configuration the benchmark times.  Gates:
tests/_parity.py."""

import numpy as np
import pytest

from oracle import layer_map as lm
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


def _run(torch, cfg, wl, mode, taps, R=None, staged=None):
    from paper_2609_32259_amd.path import TransferPath
    path = TransferPath(wl.seg, wl.S, wl.A, wl.bias, wl.rope, cfg.L_r, cfg.H_r, mode=mode, R=R,
                        layer_map="neighbor3", staged=staged)
    path.build_alignment()
    if taps is None:
        path.build_layer_map()
    else:
        path.layer_map = np.asarray(taps, np.int32)
    path.transfer()
    torch.cuda.synchronize()
    return path


def _compare_full(torch, cfg, wl, mode="overlap", taps=None, staged=None):
    taps_np = lm.neighbor3(cfg.L_s, cfg.L_r) if taps is None else np.asarray(taps)
    print(f"[gpu-taps] {cfg.name} mode={mode} B={wl.seg.batch} T_r={list(wl.seg.r_len)} "
          f"n_taps={taps_np.shape[1]} rope={wl.rope is not None} staged={staged}", flush=True)
    path = _run(torch, cfg, wl, mode, taps, staged=staged)
    Case(cfg, wl, path.R, mode, layer_map=taps_np, tag="gpu-taps").check_all()


@pytest.mark.parametrize("mode", ["overlap", "ta"])
def test_taps_fp32(torch, mode):
    cfg = synth.TINY_F32.with_(name="tiny-f32 neighbor3", layer_map="neighbor3", L_s=11)
    wl = synth.make_workload(cfg, seed=20, device="cuda")
    _compare_full(torch, cfg, wl, mode)


# The staged path (aligned features of each sender layer written to the
# workspace, then a separate multiply) serves bf16 with 8 sender and 8 receiver
# heads and is the default there; tests of that shape run both paths.
BOTH_PATHS = pytest.mark.parametrize("staged", [False, True], ids=["fused", "staged"])


@BOTH_PATHS
def test_taps_bf16_14b_shape_small(torch, staged):
    cfg = synth.LLAMA8B_14B_8K.with_(name="14b n3 small", layer_map="neighbor3", T_s=300, L_r=6)
    wl = synth.make_workload(cfg, seed=21, device="cuda")
    _compare_full(torch, cfg, wl, "overlap", staged=staged)
    _compare_full(torch, cfg, wl, "ta", staged=staged)


def test_taps_bf16_four_receiver_heads_outlier_keys(torch):
    cfg = synth.LLAMA8B_QWEN7B_4K.with_(name="qwen7b n3 small", layer_map="neighbor3", T_s=400,
                                        L_r=5)
    wl = synth.make_workload(cfg, seed=22, device="cuda")
    _compare_full(torch, cfg, wl, "overlap")


def test_taps_bf16_two_receiver_heads(torch):
    cfg = synth.LLAMA8B_14B_8K.with_(name="8->2 heads n3", layer_map="neighbor3", H_r=2, L_r=3,
                                     T_s=500)
    wl = synth.make_workload(cfg, seed=23, device="cuda")
    _compare_full(torch, cfg, wl, "overlap")


def test_taps_bf16_reverse_batched(torch):
    cfg = synth.QWEN7B_LLAMA8B_B4.with_(name="reverse n3", layer_map="neighbor3", L_r=5)
    parts = []
    rng = np.random.default_rng(24)
    for T in (70, 1, 260):
        sb, se = synth.segment_tokens(rng, T, *cfg.s_len)
        rb, re_ = synth.segment_chars(rng, int(se[-1]), *cfg.r_len)
        parts.append((sb, se, rb, re_))
    seg = synth.concat_segmentations(parts)
    S = synth.make_cache(cfg, seg, seed=24, device="cuda")
    A, bias = synth.make_maps(cfg, seed=24, device="cuda")
    rope = synth.rope_params(cfg, pos0_s=np.array([4, 0, 90], np.int32),
                             pos0_r=np.array([0, 2, 17], np.int32))
    _compare_full(torch, cfg, synth.Workload(cfg, seg, S, A, bias, rope), "overlap")


@BOTH_PATHS
@pytest.mark.parametrize("n_taps", [1, 2])
def test_taps_bf16_other_tap_counts(torch, n_taps, staged):
    base = synth.LLAMA8B_14B_8K.with_(name=f"14b {n_taps} taps", T_s=200, L_r=4)
    cfg = base.with_(layer_map="neighbor3")
    seg = synth.make_segmentation(cfg, seed=25)
    S = synth.make_cache(cfg, seg, seed=25, device="cuda")
    g = torch.Generator(device="cuda").manual_seed(25)
    A = (torch.randn((cfg.L_r, 2, cfg.d_r, n_taps * cfg.d_in), generator=g, device="cuda")
         / np.sqrt(n_taps * cfg.d_in)).to(torch.bfloat16)
    _, bias = synth.make_maps(cfg, seed=25, device="cuda")
    taps = np.array([[0, 31, 7][:n_taps], [5, 5, 5][:n_taps], [31, 0, 16][:n_taps],
                     [12, 13, 14][:n_taps]], np.int32)
    _compare_full(torch, cfg, synth.Workload(cfg, seg, S, A, bias, synth.rope_params(cfg)),
                  "overlap", taps=taps, staged=staged)


def test_taps_bf16_beyond_staging_capacity(torch):
    cfg = synth.LLAMA8B_14B_8K.with_(name="n3 unstaged", layer_map="neighbor3", L_r=3)
    rng = np.random.default_rng(26)
    sb1, se1 = synth.segment_tokens(rng, 150, 1, 7)
    sb2, se2 = synth.segment_tokens(rng, 800, 1, 2)
    sb = np.concatenate([sb1, sb2 + se1[-1]]).astype(np.int32)
    se = np.concatenate([se1, se2 + se1[-1]]).astype(np.int32)
    rb1, re1 = synth.segment_chars(rng, int(se1[-1]), 1, 8)
    rl = rng.integers(8, 17, 400)
    re2 = (np.cumsum(rl) + se1[-1]).astype(np.int32)
    re2 = re2[re2 <= se[-1]]
    rb2 = np.concatenate([[se1[-1]], re2[:-1]]).astype(np.int32)
    seg = synth.concat_segmentations([(sb, se, np.concatenate([rb1, rb2]).astype(np.int32),
                                       np.concatenate([re1, re2]).astype(np.int32))])
    S = synth.make_cache(cfg, seg, seed=26, device="cuda")
    A, bias = synth.make_maps(cfg, seed=26, device="cuda")
    _compare_full(torch, cfg, synth.Workload(cfg, seg, S, A, bias, synth.rope_params(cfg)),
                  "overlap")


@BOTH_PATHS
def test_taps_bf16_identity_first_block_is_bit_exact(torch, staged):
    cfg = synth.LLAMA8B_14B_8K.with_(name="n3 identity", layer_map="neighbor3", L_s=9, L_r=9,
                                     T_s=150, rope=None)
    wl = synth.make_workload(cfg, seed=27, device="cuda")
    seg = synth.concat_segmentations([(wl.seg.s_beg, wl.seg.s_end, wl.seg.s_beg, wl.seg.s_end)])
    A = torch.zeros((cfg.L_r, 2, cfg.d_r, 3 * cfg.d_in), dtype=torch.bfloat16, device="cuda")
    A[..., :cfg.d_in] = torch.eye(cfg.d_r, dtype=torch.bfloat16, device="cuda")
    wl = synth.Workload(cfg, seg, wl.S, A, None, None)
    taps = lm.neighbor3(cfg.L_s, cfg.L_r)
    for mode in ("overlap", "ta"):
        R = _run(torch, cfg, wl, mode, None, staged=staged).R
        for l in range(cfg.L_r):
            assert torch.equal(R[0, l, :, :, :150, :].view(torch.int16),
                               wl.S[0, int(taps[l, 0]), :, :, :150, :].view(torch.int16))


def test_full_14b_shape_32k_neighbor3(torch):
    """The benchmark's neighbourhood-map workload on both paths (the staged
    path is the benchmark's): every layer and role, on windows of rows, each
    window's oracle result checking both."""
    cfg = synth.LLAMA8B_14B_32K_N3
    wl = synth.make_workload(cfg, seed=0, device="cuda")
    print(f"[gpu-taps] full-size {cfg.name} T_r={list(wl.seg.r_len)}, both paths", flush=True)
    R = {"fused": _run(torch, cfg, wl, "overlap", None, staged=False).R,
         "staged": _run(torch, cfg, wl, "overlap", None, staged=True).R}
    rng = np.random.default_rng(98)
    Case(cfg, wl, R, tag="gpu-taps-32k").check_all(
        windows_of=lambda b, T_r: windows(T_r, 64, rng, n_mid=2, width=384))
