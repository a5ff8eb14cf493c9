"""GPU: caches in other memory layouts than [B, L, 2, H, T_cap, d_h] packed.

The cache descriptors carry a stride per dimension (channels contiguous), so a
caller may pass token-major caches ([B, L, 2, T_cap, H, d_h] storage viewed
head-major) or rows padded past d_h.  The kernels address the caches only
through those strides, so the receiver cache must come out bit-identical to
the packed layout's, on both maps and both paths, with the padding columns of
a padded receiver untouched; one token-major case is also checked against the
fp64 oracle.  Inputs are seeded and synthetic (``paper_2609_32259_amd.synth``).
"""

import numpy as np
import pytest

from paper_2609_32259_amd import synth

from _compare import Case

pytestmark = pytest.mark.gpu

CFG = synth.LLAMA8B_14B_8K.with_(name="layouts", T_s=600, L_s=5, L_r=6, batch=2)
PAD = 8  # bf16 elements past d_h in a padded row (16 bytes)


@pytest.fixture(scope="module")
def torch():
    import torch
    assert torch.cuda.is_available(), "GPU test needs a GPU"
    from paper_2609_32259_amd import heterofold
    heterofold.lib()
    return torch


def _token_major(torch, shape, dtype):
    """A zeroed head-major view [B, L, 2, H, T, d] of token-major storage."""
    B, L, two, H, T, d = shape
    st = torch.zeros((B, L, two, T, H, d), dtype=dtype, device="cuda")
    return st.permute(0, 1, 2, 4, 3, 5), st


def _padded(torch, shape, dtype, pad_fill=0.0):
    """A zeroed view of rows padded by PAD elements, the padding set to pad_fill."""
    st = torch.zeros(tuple(shape[:-1]) + (shape[-1] + PAD,), dtype=dtype, device="cuda")
    st[..., shape[-1]:] = pad_fill
    return st[..., : shape[-1]], st


def _sender(torch, S, kind):
    if kind == "packed":
        return S
    make = _token_major if kind == "token-major" else _padded
    view = make(torch, S.shape, S.dtype)[0]
    view.copy_(S)
    return view


def _receiver(torch, shape, kind, dtype=None):
    dtype = torch.bfloat16 if dtype is None else dtype
    if kind == "packed":
        return torch.zeros(shape, dtype=dtype, device="cuda"), None
    if kind == "token-major":
        return _token_major(torch, shape, dtype)
    return _padded(torch, shape, dtype, pad_fill=7.0)


def _run(torch, wl, S, R, layer_map, staged, cfg=CFG):
    from paper_2609_32259_amd.path import TransferPath
    path = TransferPath(wl.seg, S, wl.A, wl.bias, wl.rope, cfg.L_r, cfg.H_r, R=R,
                        layer_map=layer_map, staged=staged)
    out = path.step()
    torch.cuda.synchronize()
    assert path.staged == staged
    return out


def _workload(torch, layer_map):
    cfg = CFG.with_(layer_map=layer_map)
    wl = synth.make_workload(cfg, seed=61, device="cuda")
    rope = synth.rope_params(cfg, pos0_s=np.array([0, 37]), pos0_r=np.array([5, 0]))
    return cfg, synth.Workload(cfg, wl.seg, wl.S, wl.A, wl.bias, rope)


COMBOS = [("packed", "token-major"), ("token-major", "packed"), ("padded", "padded"),
          ("token-major", "token-major")]


@pytest.mark.parametrize("layer_map", ["interp2", "neighbor3"])
@pytest.mark.parametrize("staged", [False, True], ids=["fused", "staged"])
def test_layouts_match_the_packed_result(torch, layer_map, staged):
    cfg, wl = _workload(torch, layer_map)
    T_cap = int(wl.seg.r_len.max()) + 3
    shape = (wl.seg.batch, CFG.L_r, 2, CFG.H_r, T_cap, CFG.d_h)
    R0, _ = _receiver(torch, shape, "packed")
    ref = _run(torch, wl, wl.S, R0, layer_map, staged).clone()
    for s_kind, r_kind in COMBOS:
        S = _sender(torch, wl.S, s_kind)
        R, storage = _receiver(torch, shape, r_kind)
        print(f"[gpu-layouts] {layer_map} staged={staged} sender {s_kind} receiver {r_kind} "
              f"strides S {tuple(S.stride())} R {tuple(R.stride())}", flush=True)
        got = _run(torch, wl, S, R, layer_map, staged)
        assert torch.equal(got.view(torch.int16), ref.view(torch.int16)), (s_kind, r_kind)
        if r_kind == "padded":  # the columns past d_h keep their fill
            assert bool((storage[..., CFG.d_h:] == 7.0).all())


@pytest.mark.parametrize("staged", [False, True], ids=["fused", "staged"])
def test_token_major_against_the_oracle(torch, staged):
    cfg, wl = _workload(torch, "neighbor3")
    S = _sender(torch, wl.S, "token-major")
    shape = (wl.seg.batch, CFG.L_r, 2, CFG.H_r, int(wl.seg.r_len.max()), CFG.d_h)
    R, _ = _receiver(torch, shape, "token-major")
    R = _run(torch, wl, S, R, "neighbor3", staged)
    wl_tm = synth.Workload(cfg, wl.seg, S, wl.A, wl.bias, wl.rope)
    Case(cfg, wl_tm, R, tag="gpu-layouts").check_all()


def test_fp32_layouts(torch):
    """The fp32 kernel (any even d_h; here 64) through the same strides."""
    cfg = synth.TINY_F32.with_(name="fp32 layouts", batch=2)
    wl = synth.make_workload(cfg, seed=62, device="cuda")
    T_cap = int(wl.seg.r_len.max()) + 2
    shape = (wl.seg.batch, cfg.L_r, 2, cfg.H_r, T_cap, cfg.d_h)
    ref = _run(torch, wl, wl.S, _receiver(torch, shape, "packed", torch.float32)[0], "interp2",
               False, cfg).clone()
    for s_kind, r_kind in COMBOS:
        S = _sender(torch, wl.S, s_kind)
        R, storage = _receiver(torch, shape, r_kind, torch.float32)
        print(f"[gpu-layouts] fp32 sender {s_kind} receiver {r_kind} strides S {tuple(S.stride())} "
              f"R {tuple(R.stride())}", flush=True)
        got = _run(torch, wl, S, R, "interp2", False, cfg)
        assert torch.equal(got, ref), (s_kind, r_kind)
        if r_kind == "padded":
            assert bool((storage[..., cfg.d_h:] == 7.0).all())
        if (s_kind, r_kind) == ("token-major", "token-major"):
            Case(cfg, synth.Workload(cfg, wl.seg, S, wl.A, wl.bias, wl.rope), got,
                 tag="gpu-layouts").check_all()
