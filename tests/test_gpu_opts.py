"""GPU parity of the paper-faithful options (the map on x / r, Eq. 3 / 9;
the receiver's key normalization before its RoPE, App. B.1) against the
fp64 oracle, through hf_transfer_kv and hf_transfer_kv_taps."""

import numpy as np
import pytest

from oracle import alignment as al
from oracle import layer_map as lm
from oracle import transfer as tr
from paper_2609_32259_amd import synth

from _parity import check_layer, rounding_bound_normed

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch
    assert torch.cuda.is_available(), "GPU test needs a GPU"
    from paper_2609_32259_amd import heterofold
    heterofold.lib()
    return torch


def _np64(t):
    return t.float().cpu().numpy().astype(np.float64)


def _opts64(opts):
    return dict(inv_r=_np64(opts["inv_r"]), k_norm=_np64(opts["k_norm"]),
                k_norm_eps=opts["k_norm_eps"])


def _compare(torch, cfg, wl, mode="overlap"):
    from paper_2609_32259_amd.path import TransferPath
    assert wl.opts is not None
    print(f"[gpu-opts] {cfg.name} map={cfg.layer_map} post-rope keys={cfg.sender_keys_post_rope} "
          f"B={wl.seg.batch} T_r={list(wl.seg.r_len)}", flush=True)
    path = TransferPath(wl.seg, wl.S, wl.A, wl.bias, wl.rope, cfg.L_r, cfg.H_r, mode=mode,
                        layer_map=cfg.layer_map, opts=wl.opts)
    R = path.step()
    torch.cuda.synchronize()
    o64 = _opts64(wl.opts)
    worst = (0.0, 0.0)
    for b in range(wl.seg.batch):
        T_r = int(wl.seg.r_len[b])
        if T_r == 0:
            continue
        csr = al.build_alignment(*wl.seg.seq(b), mode)
        T_s = int(wl.seg.s_len[b])
        S = _np64(wl.S[b, :, :, :, :T_s, :])
        rp = None
        if wl.rope is not None:
            rp = dict(wl.rope)
            for k in ("pos0_s", "pos0_r"):
                rp[k] = 0 if wl.rope.get(k) is None else int(np.asarray(wl.rope[k])[b])
        if cfg.layer_map == "neighbor3":
            ref = tr.transfer_taps(S, lm.neighbor3(cfg.L_s, cfg.L_r), csr, _np64(wl.A),
                                   _np64(wl.bias), rp, H_r=cfg.H_r, opts=o64)
        else:
            ref = tr.transfer(S, lm.interp2(cfg.L_s, cfg.L_r), csr, _np64(wl.A), _np64(wl.bias),
                              rp, H_r=cfg.H_r, opts=o64)
        got = _np64(R[b, :, :, :, :T_r, :])
        for l in range(cfg.L_r):
            for c in range(2):
                bound = None
                if c == 0 and cfg.dtype == "bf16":   # normed keys: quantization-limited gate
                    if cfg.layer_map == "neighbor3":
                        x = tr.features_taps(S, lm.neighbor3(cfg.L_s, cfg.L_r), csr, rp, l, c)
                    else:
                        x = tr.features(S, lm.interp2(cfg.L_s, cfg.L_r), csr, rp, l, c)
                    x = x * o64["inv_r"][l, c]
                    bound = rounding_bound_normed(ref[l, c], x, _np64(wl.A[l, c]),
                                                  _np64(wl.bias[l, c]), o64["k_norm"][l],
                                                  o64["k_norm_eps"], rp is not None)
                rel, mx = check_layer(got[l, c], ref[l, c], f"{cfg.name} b={b} l={l} c={c}",
                                      dtype=cfg.dtype, quantization_limited=bound is not None,
                                      bound=bound)
                worst = (max(worst[0], rel), max(worst[1], mx))
    print(f"[gpu-opts]   worst rel-Fro {worst[0]:.3e}, max|err| {worst[1]:.3e}", flush=True)


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


@pytest.mark.parametrize("H_r", [8, 4])
def test_opts_bf16_paper_construction(torch, H_r):
    cfg = synth.LLAMA8B_14B_32K_PAPER.with_(name=f"paper small H_r={H_r}", H_r=H_r, T_s=350,
                                            L_r=5)
    _compare(torch, cfg, synth.make_workload(cfg, seed=33, device="cuda"))


def test_full_14b_shape_32k_paper_construction(torch):
    """The benchmark's paper-construction workload, sampled rows."""
    from paper_2609_32259_amd.path import TransferPath
    cfg = synth.LLAMA8B_14B_32K_PAPER
    wl = synth.make_workload(cfg, seed=0, device="cuda")
    print(f"[gpu-opts] full-size {cfg.name} T_r={list(wl.seg.r_len)}", flush=True)
    path = TransferPath(wl.seg, wl.S, wl.A, wl.bias, wl.rope, cfg.L_r, cfg.H_r,
                        layer_map=cfg.layer_map, opts=wl.opts)
    R = path.step()
    torch.cuda.synchronize()
    taps = lm.neighbor3(cfg.L_s, cfg.L_r)
    T_r = int(wl.seg.r_len[0])
    rng = np.random.default_rng(97)
    rows = sorted({0, 63, 64, T_r // 3, T_r - 1, *rng.integers(0, T_r, 16).tolist()})
    csr = al.build_alignment(*wl.seg.seq(0), "overlap")
    rp = dict(wl.rope, pos0_s=0, pos0_r=0)
    o64 = _opts64(wl.opts)
    get = lambda l, c, idx: _np64(wl.S[0, l, c][:, torch.as_tensor(idx, device="cuda"), :])  # noqa: E731
    for l in (0, 17, 39):
        for c in (0, 1):
            ref, x = tr.transfer_rows_taps(get, taps, csr, _np64(wl.A[l, c]),
                                           _np64(wl.bias[l, c]), rp, cfg.d_h, l, c, rows,
                                           return_features=True, opts=o64)
            got = _np64(R[0, l, c][:, torch.as_tensor(rows, device="cuda"), :])
            bound = None
            if c == 0:
                bound = rounding_bound_normed(ref, x, _np64(wl.A[l, c]), _np64(wl.bias[l, c]),
                                              o64["k_norm"][l], o64["k_norm_eps"], True)
            check_layer(got, ref, f"{cfg.name} l={l} c={c} rows={len(rows)}",
                        quantization_limited=bound is not None, bound=bound)
