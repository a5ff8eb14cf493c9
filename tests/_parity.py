"""Tolerance checks shared by the GPU parity tests.

bf16 outputs: per (layer, role), relative Frobenius error <= 5e-3 and max
elementwise |error| <= 2e-2 against the fp64 oracle.

One workload draws log-normal(0, 1) per-channel key scales, so a few feature
channels reach |x| ~ 1e2.  There the bf16 representation itself forbids the
literal max-abs gate: the mapped features are bf16 (half-ulp 0.5 at
|x| in [128, 256)) and so are the outputs (half-ulp 1/32 at |y| in [8, 16)).
For that case ("quantization-limited") every element must satisfy
|error| <= 2e-2, or else lie within the worst-case first-order error of the
two roundings the arithmetic performs,
    half_ulp(y) + sum_k |A_nk| half_ulp(x_k)   (+ an fp32 accumulation term),
which a wrong index, sign or dropped term would exceed.
Keys that go through the receiver's key normalization (RMSNorm per head,
then RoPE) have |y| of several units, where the output's own half-ulp
(1/64 at |y| in [4, 8)) again leaves little room under 2e-2.  They are
gated the same way with the first-order bound carried through the norm and
the rotation (``rounding_bound_normed``).
fp32 outputs: the same gates, plus relative Frobenius error <= 1e-5.
"""

import numpy as np

REL_FRO = 5e-3
MAX_ABS = 2e-2


def bf16_half_ulp(y):
    a = np.abs(np.asarray(y, dtype=np.float64))
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -126)))
    return 2.0 ** (e - 8)


def err_stats(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    d = got - ref
    nref = np.linalg.norm(ref)
    rel = np.linalg.norm(d) / nref if nref > 0 else np.linalg.norm(d)
    return rel, (float(np.max(np.abs(d))) if d.size else 0.0), d


def rounding_bound(ref, x, A):
    """Per-element first-order bound of bf16-rounding x and y.
    ref [H_r, T, d_h] oracle outputs; x [T, d_S] oracle features; A [d_R, d_S]."""
    H_r, T, d_h = ref.shape
    Aa = np.abs(np.asarray(A, dtype=np.float64))
    bx = bf16_half_ulp(x) @ Aa.T                         # [T, d_R]
    acc = 1e-5 * (np.abs(x) @ Aa.T)                      # fp32 accumulation, generous
    b = (bx + acc).reshape(T, H_r, d_h).transpose(1, 0, 2)
    return bf16_half_ulp(np.abs(ref) * (1 + 2.0 ** -7) + b) + b


def rounding_bound_normed(ref, x, A, b, g, eps, rotated):
    """First-order bound for keys y = R(q) norm(A x + b) with x and y rounded
    to bf16.  ref [H_r, T, d_h] oracle outputs; x [T, d_S] oracle features
    (as the map sees them, 1/r applied); A [d_R, d_S]; b [d_R] or None;
    g [d_h] norm weights; eps; rotated: whether the receiver RoPE follows."""
    H_r, T, d_h = ref.shape
    Aa = np.abs(np.asarray(A, dtype=np.float64))
    x = np.asarray(x, dtype=np.float64)
    y = x @ np.asarray(A, dtype=np.float64).T
    if b is not None:
        y = y + np.asarray(b, dtype=np.float64)[None, :]
    e = bf16_half_ulp(x) @ Aa.T + 1e-5 * (np.abs(x) @ Aa.T)          # error before the norm
    y = y.reshape(T, H_r, d_h)
    e = e.reshape(T, H_r, d_h)
    rho = np.sqrt(np.mean(y * y, axis=-1, keepdims=True) + float(eps))
    en = np.linalg.norm(e, axis=-1, keepdims=True)
    gg = np.abs(np.asarray(g, dtype=np.float64))
    e = gg * (e / rho + np.abs(y) * en / (np.sqrt(d_h) * rho * rho))  # through the RMSNorm
    e = e + 1e-6 * gg * np.abs(y) / rho
    if rotated:                                                       # pair mixing by RoPE
        h = d_h // 2
        e = np.concatenate([e[..., :h] + e[..., h:], e[..., :h] + e[..., h:]], axis=-1)
    e = e.transpose(1, 0, 2)
    return bf16_half_ulp(np.abs(ref) * (1 + 2.0 ** -7) + e) + e


def check_layer(got, ref, where, dtype="bf16", quantization_limited=False, x=None, A=None,
                bound=None):
    rel, mx, d = err_stats(got, ref)
    assert np.all(np.isfinite(got)), f"{where}: non-finite output"
    assert rel <= REL_FRO, f"{where}: rel Frobenius {rel:.3e} > {REL_FRO}"
    if dtype == "f32":
        assert rel <= 1e-5, f"{where}: fp32 rel Frobenius {rel:.3e} > 1e-5"
    if quantization_limited:
        if bound is None:
            assert x is not None and A is not None, "quantization-limited gate needs x and A"
            bound = rounding_bound(ref, x, A)
        bad = (np.abs(d) > MAX_ABS) & (np.abs(d) > bound)
        assert not bad.any(), (f"{where}: {int(bad.sum())} elements beyond both 2e-2 and the "
                               f"rounding bound; worst |err| {mx:.3e}")
    else:
        assert mx <= MAX_ABS, f"{where}: max |err| {mx:.3e} > {MAX_ABS}"
    return rel, mx
