"""The GPU tests' comparison helper (tests/_compare.py) on the CPU.

A batch of four sequences with per-sequence RoPE offsets goes through the CPU
emulation of the bf16 path's arithmetic (test_parity_bound._emulate) to give a
receiver cache R.  Case must accept R checked whole and on row windows (their
rows mapped and gated together), accept it in a dict next to a second copy,
and reject a planted error in a row a window covers while ignoring one in a
row no window covers.  The planted error is in the emulated cache, on the CPU.
"""

import numpy as np
import pytest
import torch

from _compare import Case, seq_rope, windows
from oracle import alignment as al
from oracle import layer_map as lm
from oracle import transfer as tr
from paper_2609_32259_amd import synth
from test_parity_bound import _emulate

CFG = synth.QWEN7B_LLAMA8B_B4.with_(name="compare windows", T_s=640, L_s=3, L_r=4)


@pytest.fixture(scope="module")
def case_inputs():
    wl = synth.make_workload(CFG, seed=12, device="cpu")
    rope = synth.rope_params(CFG, pos0_s=np.array([0, 5, 130, 7]), pos0_r=np.array([0, 9, 3, 200]))
    wl = synth.Workload(CFG, wl.seg, wl.S, wl.A, wl.bias, rope)
    lt = lm.interp2(CFG.L_s, CFG.L_r)
    T_cap = int(max(wl.seg.r_len)) + 5
    R = torch.zeros((wl.seg.batch, CFG.L_r, 2, CFG.H_r, T_cap, CFG.d_h), dtype=torch.bfloat16)
    A = wl.A.float().numpy().astype(np.float64)
    bias = wl.bias.float().numpy().astype(np.float64)
    for b in range(wl.seg.batch):
        S = wl.S[b].float().numpy().astype(np.float64)
        csr = al.build_alignment(*wl.seg.seq(b), "overlap")
        rp = seq_rope(rope, b)
        T_r = int(wl.seg.r_len[b])
        for l in range(CFG.L_r):
            for c in (0, 1):
                x = tr.features(S, lt, csr, rp, l, c)
                y = _emulate(x, A[l, c], bias[l, c], c, l, rp, None, np.arange(T_r),
                             rope_shift=rp["pos0_r"])
                R[b, l, c, :, :T_r, :] = torch.from_numpy(y).to(torch.bfloat16)
    return wl, R


def _windows(b, T_r):
    return windows(T_r, 64, np.random.default_rng(b), n_mid=2, width=96)


def test_whole_and_windowed_checks_pass(case_inputs):
    wl, R = case_inputs
    assert min(int(t) for t in wl.seg.r_len) > 2 * 96 + 64  # every sequence gets mid windows
    w_all = Case(CFG, wl, R, tag="cpu-compare").check_all()
    w_win = Case(CFG, wl, {"a": R, "b": R.clone()}, tag="cpu-compare").check_all(windows_of=_windows)
    assert w_all.gate <= 1.0 and w_win.gate <= 1.0


def test_planted_error_in_a_window_fails(case_inputs):
    wl, R = case_inputs
    b, l, c, h, e = 2, 1, 0, 5, 17
    r0, r1 = _windows(b, int(wl.seg.r_len[b]))[1]
    Rp = R.clone()
    Rp[b, l, c, h, r0 + 40, e] += 0.25
    with pytest.raises(AssertionError, match="kernel-arithmetic gate|2e-2"):
        Case(CFG, wl, {"good": R, "planted": Rp}, tag="cpu-compare").check_all(windows_of=_windows)
    # the same error in a row outside every window is not looked at
    covered = np.zeros(int(wl.seg.r_len[b]), bool)
    for q0, q1 in _windows(b, int(wl.seg.r_len[b])):
        covered[q0:q1] = True
    outside = int(np.nonzero(~covered)[0][0])
    Rq = R.clone()
    Rq[b, l, c, h, outside, e] += 0.25
    Case(CFG, wl, Rq, tag="cpu-compare").check_all(windows_of=_windows)
    with pytest.raises(AssertionError):
        Case(CFG, wl, Rq, tag="cpu-compare").check_all()
