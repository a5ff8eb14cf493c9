"""GPU transfer parity: hf_transfer_kv against the fp64 oracle.

Small cases are compared element by element over every layer, role and row
(several row tiles with a ragged tail).  At full size every layer, role and
sequence is compared, in the launch configuration the benchmark times: the
headline 32K workload on every row, the others on windows of rows (the head,
the tail, and windows across row-tile edges).  Gates: tests/_parity.py.
Inputs are seeded and synthetic (``paper_2609_32259_amd.synth``)."""

import numpy as np
import pytest

from oracle import alignment as al
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


def _path(cfg, wl, mode="overlap", rope=None, R=None, staged=None):
    from paper_2609_32259_amd.path import TransferPath
    return TransferPath(wl.seg, wl.S, wl.A, wl.bias, wl.rope if rope is None else rope,
                        cfg.L_r, cfg.H_r, mode=mode, R=R, staged=staged)


def _np64(t):
    return t.float().cpu().numpy().astype(np.float64)


def _compare_full(torch, cfg, wl, mode="overlap", rope="cfg", R=None, staged=None):
    """Every element of every layer, role and sequence."""
    if rope != "cfg":
        wl = synth.Workload(cfg, wl.seg, wl.S, wl.A, wl.bias, rope, wl.opts)
    print(f"[gpu-transfer] {cfg.name} mode={mode} B={wl.seg.batch} T_s={list(wl.seg.s_len)} "
          f"T_r={list(wl.seg.r_len)} rope={wl.rope is not None} staged={staged}", flush=True)
    path = _path(cfg, wl, mode, R=R, staged=staged)
    R = path.step()
    torch.cuda.synchronize()
    Case(cfg, wl, R, mode, tag="gpu-transfer").check_all()
    return path


# --- fp32 -------------------------------------------------------------------

@pytest.mark.parametrize("mode", ["overlap", "ta"])
def test_tiny_fp32(torch, mode):
    cfg = synth.TINY_F32
    wl = synth.make_workload(cfg, seed=0, device="cuda")
    _compare_full(torch, cfg, wl, mode)


def test_fp32_rope_batched_offsets(torch):
    cfg = synth.TINY_F32.with_(name="fp32 rope", L_s=3, L_r=5, H_s=2, H_r=3, d_h=64,
                               n_chars=900, rope=(1.0e4, 5.0e5), batch=3)
    wl = synth.make_workload(cfg, seed=1, device="cuda")
    rope = synth.rope_params(cfg, pos0_s=np.array([0, 7, 1000], np.int32),
                             pos0_r=np.array([5, 0, 333], np.int32))
    _compare_full(torch, cfg, wl, "overlap", rope=rope)


# Unusual fp32 shapes: head sizes from 4 to 256 channels, 1-6 heads on either
# side, odd layer counts, RoPE on or off, batches of 1-3 sequences.
FP32_SHAPES = [(4, 1, 5, 2, 1), (12, 3, 1, 3, 4), (20, 5, 3, 4, 6), (96, 2, 6, 5, 2),
               (256, 1, 2, 2, 3), (64, 4, 3, 6, 5)]  # d_h, H_s, H_r, L_s, L_r


@pytest.mark.parametrize("i", range(len(FP32_SHAPES)))
def test_fp32_unusual_shapes(torch, i):
    d_h, H_s, H_r, L_s, L_r = FP32_SHAPES[i]
    rope = (1.0e4, 5.0e5) if i % 2 == 0 else None
    cfg = synth.TINY_F32.with_(name=f"fp32 d_h={d_h} {H_s}->{H_r} heads", d_h=d_h, H_s=H_s,
                               H_r=H_r, L_s=L_s, L_r=L_r, n_chars=500, rope=rope, batch=1 + i % 3)
    wl = synth.make_workload(cfg, seed=90 + i, device="cuda")
    if rope is not None:
        rng = np.random.default_rng(90 + i)
        wl = synth.Workload(cfg, wl.seg, wl.S, wl.A, wl.bias,
                            synth.rope_params(cfg, pos0_s=rng.integers(0, 99, cfg.batch),
                                              pos0_r=rng.integers(0, 99, cfg.batch)))
    _compare_full(torch, cfg, wl, "overlap" if i < 3 else "ta")


# --- bf16, small sizes, every element ----------------------------------------

# The staged path (aligned features written to the workspace, then a separate
# multiply) serves bf16 with 8 sender and 8 receiver heads; tests of that shape
# run both paths.
BOTH_PATHS = pytest.mark.parametrize("staged", [False, True], ids=["fused", "staged"])


@BOTH_PATHS
@pytest.mark.parametrize("mode", ["overlap", "ta"])
def test_bf16_14b_shape_small(torch, mode, staged):
    cfg = synth.LLAMA8B_14B_8K.with_(T_s=300)          # 5 row tiles of 64, ragged tail
    wl = synth.make_workload(cfg, seed=2, device="cuda")
    _compare_full(torch, cfg, wl, mode, staged=staged)


def test_bf16_qwen7b_shape_small(torch):
    cfg = synth.LLAMA8B_QWEN7B_4K.with_(T_s=500)        # 4 receiver heads: 64-row tiles
    wl = synth.make_workload(cfg, seed=3, device="cuda")
    _compare_full(torch, cfg, wl, "overlap")


def test_bf16_reverse_batched_ragged(torch):
    cfg = synth.QWEN7B_LLAMA8B_B4
    parts = []
    rng = np.random.default_rng(4)
    for T in (1, 100, 333, 65):
        sb, se = synth.segment_tokens(rng, T, *cfg.s_len)
        rb, re_ = synth.segment_chars(rng, int(se[-1]), *cfg.r_len)
        parts.append((sb, se, rb, re_))
    seg = synth.concat_segmentations(parts)
    S = synth.make_cache(cfg, seg, seed=4, device="cuda")
    A, bias = synth.make_maps(cfg, seed=4, device="cuda")
    rope = synth.rope_params(cfg, pos0_s=np.array([0, 3, 50, 9], np.int32),
                             pos0_r=np.array([2, 0, 11, 70], np.int32))
    wl = synth.Workload(cfg, seg, S, A, bias, rope)
    _compare_full(torch, cfg, wl, "overlap")


@pytest.mark.parametrize("H_r,staged", [(8, False), (8, True), (4, False)])
def test_bf16_batch_with_empty_sequences(torch, H_r, staged):
    # A sequence with no tokens and one with sender tokens but no receiver
    # tokens own no row tiles (and no staging records); the sequences around
    # them still map correctly, and no receiver row outside the lengths changes.
    cfg = synth.LLAMA8B_14B_8K.with_(name=f"empty sequences H_r={H_r}", H_r=H_r, L_r=3)
    rng = np.random.default_rng(12)
    parts = []
    for n_s, with_r in ((0, False), (150, True), (40, False), (90, True)):
        sb, se = synth.segment_tokens(rng, n_s, 1, 7)
        n_chars = int(se[-1]) if n_s and with_r else 0
        rb, re_ = synth.segment_chars(rng, n_chars, 1, 8)
        parts.append((sb, se, rb, re_))
    seg = synth.concat_segmentations(parts)
    assert list(seg.r_len == 0) == [True, False, True, False]
    S = synth.make_cache(cfg, seg, seed=12, device="cuda")
    A, bias = synth.make_maps(cfg, seed=12, device="cuda")
    rope = synth.rope_params(cfg, pos0_s=np.array([0, 5, 9, 300], np.int32),
                             pos0_r=np.array([0, 2, 0, 40], np.int32))
    wl = synth.Workload(cfg, seg, S, A, bias, rope)
    T_cap = int(seg.r_len.max()) + 21
    R = torch.full((4, cfg.L_r, 2, cfg.H_r, T_cap, cfg.d_h), 3.0, dtype=torch.bfloat16,
                   device="cuda")
    _compare_full(torch, cfg, wl, "overlap", R=R, staged=staged)
    for b in range(4):
        T_r = int(seg.r_len[b])
        assert bool((R[b, :, :, :, T_r:, :] == 3.0).all()), f"sequence {b}: rows past {T_r} changed"


@pytest.mark.parametrize("H_r", [8, 4])
def test_bf16_tiles_beyond_staging_capacity(torch, H_r):
    # Long receiver tokens over short sender tokens make some 64-row tiles read
    # more sender rows than the LDS staging holds; those tiles take the
    # global-memory build.  Mixed with ordinary tiles in one launch.
    cfg = synth.LLAMA8B_14B_8K.with_(name=f"unstaged H_r={H_r}", H_r=H_r, L_r=3)
    rng = np.random.default_rng(11)
    sb1, se1 = synth.segment_tokens(rng, 200, 1, 7)
    sb2, se2 = synth.segment_tokens(rng, 900, 1, 2)
    sb = np.concatenate([sb1, sb2 + se1[-1]]).astype(np.int32)
    se = np.concatenate([se1, se2 + se1[-1]]).astype(np.int32)
    rb1, re1 = synth.segment_chars(rng, int(se1[-1]), 1, 8)
    rl = rng.integers(8, 17, 400)
    re2 = (np.cumsum(rl) + se1[-1]).astype(np.int32)
    re2 = re2[re2 <= se[-1]]
    rb2 = np.concatenate([[se1[-1]], re2[:-1]]).astype(np.int32)
    seg = synth.concat_segmentations([(sb, se, np.concatenate([rb1, rb2]).astype(np.int32),
                                       np.concatenate([re1, re2]).astype(np.int32))])
    S = synth.make_cache(cfg, seg, seed=11, device="cuda")
    A, bias = synth.make_maps(cfg, seed=11, device="cuda")
    wl = synth.Workload(cfg, seg, S, A, bias, synth.rope_params(cfg))
    _compare_full(torch, cfg, wl, "overlap")


@pytest.mark.parametrize("H_r,staged", [(8, False), (8, True), (4, False)])
def test_bf16_full_batch_of_short_sequences(torch, H_r, staged):
    # 64 sequences (the batch limit) of 0 to 200 sender tokens: many tiles with
    # ragged tails, sequences without tiles, and fewer work items than compute
    # units at L_r = 1, so the work decoding and the per-sequence tile starts are
    # exercised together.
    cfg = synth.LLAMA8B_14B_8K.with_(name=f"64 short sequences H_r={H_r}", H_r=H_r, L_r=1)
    rng = np.random.default_rng(14)
    parts = []
    for n_s in rng.integers(0, 201, 64):
        sb, se = synth.segment_tokens(rng, int(n_s), 1, 7)
        rb, re_ = synth.segment_chars(rng, int(se[-1]) if n_s else 0, 1, 8)
        parts.append((sb, se, rb, re_))
    seg = synth.concat_segmentations(parts)
    S = synth.make_cache(cfg, seg, seed=14, device="cuda")
    A, bias = synth.make_maps(cfg, seed=14, device="cuda")
    rope = synth.rope_params(cfg, pos0_s=rng.integers(0, 50, 64).astype(np.int32),
                             pos0_r=rng.integers(0, 50, 64).astype(np.int32))
    wl = synth.Workload(cfg, seg, S, A, bias, rope)
    T_cap = int(seg.r_len.max()) + 5
    R = torch.full((64, cfg.L_r, 2, cfg.H_r, T_cap, cfg.d_h), 3.0, dtype=torch.bfloat16,
                   device="cuda")
    _compare_full(torch, cfg, wl, "overlap", R=R, staged=staged)
    for b in range(64):
        T_r = int(seg.r_len[b])
        assert bool((R[b, :, :, :, T_r:, :] == 3.0).all()), f"sequence {b}: rows past {T_r} changed"


@pytest.mark.parametrize("H_r", [8, 4])
def test_bf16_sender_slab_beyond_32_bit_offsets(torch, H_r):
    # A sender cache with a token capacity of 1.2M: one (layer, role) slab spans
    # 7 head strides of 1.2M x 128 bf16 (2.4 GB), past what a 32-bit buffer
    # offset reaches, so the build reads the rows with 64-bit addresses instead.
    cfg = synth.LLAMA8B_14B_8K.with_(name=f"1.2M-token sender capacity H_r={H_r}", H_r=H_r,
                                     L_s=2, L_r=3)
    rng = np.random.default_rng(15)
    sb, se = synth.segment_tokens(rng, 300, 1, 7)
    rb, re_ = synth.segment_chars(rng, int(se[-1]), 1, 8)
    seg = synth.concat_segmentations([(sb, se, rb, re_)])
    S_small = synth.make_cache(cfg, seg, seed=15, device="cuda")
    T_cap = 1_200_000
    assert (cfg.H_s - 1) * T_cap * cfg.d_h * 2 >= 1 << 31
    S = torch.zeros((1, cfg.L_s, 2, cfg.H_s, T_cap, cfg.d_h), dtype=torch.bfloat16, device="cuda")
    S[:, :, :, :, :300, :] = S_small
    del S_small
    A, bias = synth.make_maps(cfg, seed=15, device="cuda")
    rope = synth.rope_params(cfg, pos0_s=np.array([7], np.int32), pos0_r=np.array([3], np.int32))
    wl = synth.Workload(cfg, seg, S, A, bias, rope)
    _compare_full(torch, cfg, wl, "overlap")
    del wl, S
    torch.cuda.empty_cache()


@pytest.mark.parametrize("H_r", [8, 4])
def test_bf16_runs_too_wide_for_the_rotation_table(torch, H_r):
    # One-character sender tokens under 4-6 character receiver tokens: about 5
    # entries per row, so a tile stays within the staged entry count, but a run
    # of rows spans more sender positions than the in-LDS rotation table holds.
    # Key tiles then build from global memory while value tiles stay staged.
    cfg = synth.LLAMA8B_14B_8K.with_(name=f"wide runs H_r={H_r}", H_r=H_r, L_r=3)
    rng = np.random.default_rng(13)
    sb, se = synth.segment_tokens(rng, 1500, 1, 1)
    rb, re_ = synth.segment_chars(rng, int(se[-1]), 4, 6)
    seg = synth.concat_segmentations([(sb, se, rb, re_)])
    row_ptr, col, _, _ = al.build_alignment(sb, se, rb, re_, "overlap")
    assert np.diff(row_ptr[::64]).max() <= 512          # every tile's entries are staged
    assert col[row_ptr[8]] - col[0] >= 16               # a run of 8 rows spans 16+ tokens
    S = synth.make_cache(cfg, seg, seed=13, device="cuda")
    A, bias = synth.make_maps(cfg, seed=13, device="cuda")
    wl = synth.Workload(cfg, seg, S, A, bias, synth.rope_params(cfg, pos0_s=np.array([3], np.int32)))
    _compare_full(torch, cfg, wl, "overlap")


def test_bf16_two_receiver_heads(torch):
    cfg = synth.LLAMA8B_14B_8K.with_(name="8->2 heads", H_r=2, L_r=3, T_s=700)   # 256-row tiles
    wl = synth.make_workload(cfg, seed=5, device="cuda")
    _compare_full(torch, cfg, wl, "overlap")


def test_bf16_identity_is_bit_exact(torch):
    cfg = synth.LLAMA8B_14B_8K.with_(name="identity", L_s=3, L_r=3, T_s=200, rope=None)
    wl = synth.make_workload(cfg, seed=6, device="cuda")
    seg = synth.concat_segmentations([(wl.seg.s_beg, wl.seg.s_end, wl.seg.s_beg, wl.seg.s_end)])
    eye = torch.eye(cfg.d_r, dtype=torch.bfloat16, device="cuda")
    A = eye.expand(cfg.L_r, 2, cfg.d_r, cfg.d_in).contiguous()
    wl = synth.Workload(cfg, seg, wl.S, A, None, None)
    for mode in ("overlap", "ta"):
        path = _path(cfg, wl, mode)
        R = path.step()
        torch.cuda.synchronize()
        assert torch.equal(R[:, :, :, :, :200, :].view(torch.int16),
                           wl.S[:, :, :, :, :200, :].view(torch.int16))


def test_bf16_equal_rope_round_trip(torch):
    # Same theta and positions on both sides with identity maps: un-rotation
    # then rotation returns the keys to within one bf16 rounding.
    cfg = synth.LLAMA8B_14B_8K.with_(name="rope round trip", L_s=2, L_r=2, T_s=150,
                                     rope=(5.0e5, 5.0e5))
    wl = synth.make_workload(cfg, seed=7, device="cuda")
    seg = synth.concat_segmentations([(wl.seg.s_beg, wl.seg.s_end, wl.seg.s_beg, wl.seg.s_end)])
    A = torch.eye(cfg.d_r, dtype=torch.bfloat16, device="cuda").expand(2, 2, cfg.d_r, cfg.d_in).contiguous()
    wl = synth.Workload(cfg, seg, wl.S, A, None, synth.rope_params(cfg))
    R = _path(cfg, wl).step()
    torch.cuda.synchronize()
    got, ref = _np64(R[0, :, 0, :, :150, :]), _np64(wl.S[0, :, 0, :, :150, :])
    # each rounding (of the un-rotated key, then of the output) is at most a
    # half-ulp of the rotated pair's magnitude
    pair = np.sqrt(ref[..., :64] ** 2 + ref[..., 64:] ** 2)
    pair = np.concatenate([pair, pair], axis=-1)
    assert np.all(np.abs(got - ref) <= 2.0 ** -7 * pair)
    assert torch.equal(R[0, :, 1, :, :150, :].view(torch.int16), wl.S[0, :, 1, :, :150, :].view(torch.int16))


@BOTH_PATHS
def test_bf16_tile_multiple_lengths(torch, staged):
    # Identical tokenizations in TA mode give T_r = T_s exactly: sequences of
    # 512 and 256 rows fill whole 256-row multiply tiles, 257 and 65 rows leave
    # one row in the last tile, and a 1-row sequence is a tile of its own.
    cfg = synth.LLAMA8B_14B_8K.with_(name="tile-multiple lengths", L_r=3)
    rng = np.random.default_rng(15)
    parts = []
    for n in (512, 256, 257, 65, 1):
        sb, se = synth.segment_tokens(rng, n, 1, 7)
        parts.append((sb, se, sb.copy(), se.copy()))
    seg = synth.concat_segmentations(parts)
    assert list(seg.r_len) == [512, 256, 257, 65, 1]
    S = synth.make_cache(cfg, seg, seed=15, device="cuda")
    A, bias = synth.make_maps(cfg, seed=15, device="cuda")
    rope = synth.rope_params(cfg, pos0_s=np.array([0, 9, 3, 100, 7], np.int32),
                             pos0_r=np.array([4, 0, 31, 32, 5], np.int32))
    _compare_full(torch, cfg, synth.Workload(cfg, seg, S, A, bias, rope), "ta", staged=staged)


@BOTH_PATHS
def test_bf16_batch_of_long_ragged_sequences(torch, staged):
    # Three sequences of several 256-row multiply tiles each, with ragged ends
    # and per-sequence RoPE offsets: the staged path's per-sequence tile starts
    # and slab rows well past the first tile.
    cfg = synth.LLAMA8B_14B_8K.with_(name="three long sequences", L_r=3)
    rng = np.random.default_rng(16)
    parts = []
    for n_s in (1500, 1111, 1337):
        sb, se = synth.segment_tokens(rng, n_s, 1, 7)
        rb, re_ = synth.segment_chars(rng, int(se[-1]), 1, 8)
        parts.append((sb, se, rb, re_))
    seg = synth.concat_segmentations(parts)
    S = synth.make_cache(cfg, seg, seed=16, device="cuda")
    A, bias = synth.make_maps(cfg, seed=16, device="cuda")
    rope = synth.rope_params(cfg, pos0_s=np.array([0, 40, 7], np.int32),
                             pos0_r=np.array([3, 0, 250], np.int32))
    _compare_full(torch, cfg, synth.Workload(cfg, seg, S, A, bias, rope), "overlap", staged=staged)


def _random_case(seed, staged):
    """A seeded irregular batch: 1-5 sequences of 1-513 sender tokens (around
    the 64- and 256-row tile edges), receiver tokenizations with empty tokens,
    gaps and split ends over the same text (sometimes none at all), 3-6 sender
    and 2-5 receiver layers, 2/4/8 receiver heads (8 on the staged path), per-
    sequence RoPE offsets and either alignment mode."""
    rng = np.random.default_rng(7000 + seed)
    H_r = 8 if staged else int(rng.choice([2, 4, 8]))
    cfg = synth.LLAMA8B_14B_8K.with_(name=f"random batch {seed}", H_r=H_r,
                                     L_s=int(rng.integers(3, 7)), L_r=int(rng.integers(2, 6)))
    parts = []
    for _ in range(int(rng.integers(1, 6))):
        n_s = int(rng.choice([1, 7, 63, 64, 65, 255, 256, 300, 513]))
        sb, se = synth.segment_tokens(rng, n_s, 1, 7)
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
    mode = "overlap" if seed % 2 == 0 else "ta"
    return cfg, synth.Workload(cfg, seg, S, A, bias, rope), mode


@pytest.mark.parametrize("seed", range(6))
@BOTH_PATHS
def test_bf16_random_batches(torch, seed, staged):
    cfg, wl, mode = _random_case(seed, staged)
    _compare_full(torch, cfg, wl, mode, staged=staged)


@BOTH_PATHS
def test_bf16_rows_past_length_untouched_and_deterministic(torch, staged):
    cfg = synth.LLAMA8B_14B_8K.with_(T_s=260, L_r=4)
    wl = synth.make_workload(cfg, seed=8, device="cuda")
    T_r = int(wl.seg.r_len[0])
    R = torch.full((1, cfg.L_r, 2, cfg.H_r, T_r + 37, cfg.d_h), 7.0, dtype=torch.bfloat16,
                   device="cuda")
    path = _path(cfg, wl, R=R, staged=staged)
    out1 = path.step().clone()
    out2 = path.step().clone()
    torch.cuda.synchronize()
    assert torch.equal(out1.view(torch.int16), out2.view(torch.int16))
    assert bool((out1[:, :, :, :, T_r:, :] == 7.0).all())


# --- bf16, other sender head counts ------------------------------------------

@pytest.mark.parametrize("H_s,H_r", [(1, 8), (2, 8), (2, 4), (16, 8), (16, 4)])
def test_bf16_sender_head_counts(torch, H_s, H_r):
    # 1 and 2 sender heads: the tiled kernel with 8 and 4 waves per sender head;
    # 16 sender heads: more than the tiled kernel's LDS tile holds, so the
    # direct kernel runs.  Several row tiles with a ragged tail, RoPE on keys.
    cfg = synth.LLAMA8B_14B_8K.with_(name=f"{H_s}->{H_r} heads", H_s=H_s, H_r=H_r, L_s=5,
                                     L_r=4, T_s=333)
    wl = synth.make_workload(cfg, seed=40 + H_s, device="cuda")
    _compare_full(torch, cfg, wl, "overlap")


# --- bf16, full sizes ----------------------------------------------------------

def _run_full(torch, cfg, seed=0, staged=None):
    wl = synth.make_workload(cfg, seed=seed, device="cuda")
    print(f"[gpu-transfer] full-size {cfg.name} B={wl.seg.batch} T_s={list(wl.seg.s_len)} "
          f"T_r={list(wl.seg.r_len)} staged={staged}", flush=True)
    R = _path(cfg, wl, staged=staged).step()
    torch.cuda.synchronize()
    return wl, R


def _compare_windows(torch, cfg, seed=0, width=512, n_mid=3):
    """All layers, roles and sequences, on windows of rows: the head, the
    tail and windows starting 3 rows before a random 64-row tile edge."""
    wl, R = _run_full(torch, cfg, seed)
    rng = np.random.default_rng(99)
    return Case(cfg, wl, R, tag="gpu-transfer").check_all(
        windows_of=lambda b, T_r: windows(T_r, 64, rng, n_mid=n_mid, width=width))


def test_full_qwen7b_shape_4k(torch):
    _compare_windows(torch, synth.LLAMA8B_QWEN7B_4K, width=1024)


def test_full_14b_shape_8k(torch):
    _compare_windows(torch, synth.LLAMA8B_14B_8K, width=1024)


@pytest.mark.parametrize("T", [1024, 4096, 16384, 32768])
def test_full_reverse_batch4(torch, T):
    _compare_windows(torch, synth.QWEN7B_LLAMA8B_B4.with_(T_s=T), width=384, n_mid=2)


@pytest.fixture(scope="module")
def full_32k(torch):
    """The headline workload on both paths, each in the benchmark's launch
    configuration (the fused path is the benchmark's), from the same inputs, so
    that one oracle computation per layer and role checks both results."""
    cfg = synth.LLAMA8B_14B_32K
    wl, R_fused = _run_full(torch, cfg, staged=False)
    R_staged = _path(cfg, wl, staged=True).step()
    torch.cuda.synchronize()
    yield Case(cfg, wl, {"fused": R_fused, "staged": R_staged}, tag="gpu-transfer-32k")
    del wl, R_fused, R_staged
    torch.cuda.empty_cache()


@pytest.mark.parametrize("group", range(8))
def test_full_14b_shape_32k_every_row(full_32k, group):
    """Every row of layers 5 group .. 5 group + 4, K and V, against the oracle,
    on both paths."""
    full_32k.check_all(layers=range(5 * group, 5 * group + 5), verbose=True)
