"""Tolerance checks shared by the GPU parity tests.

bf16 outputs: per (layer, role), relative Frobenius error <= 5e-3 and max
elementwise |error| <= 2e-2 against the fp64 oracle.  Where the receiver
values are large enough that bf16 cannot represent them to 2e-2 at all
(|y| >= 8 gives a half-ulp of 1/32), the max-abs gate is taken on the error
beyond the output's own half-ulp ("quantization-limited"); that relaxation is
only used for the configuration with log-normal outlier key channels.
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


def check_layer(got, ref, where, dtype="bf16", quantization_limited=False):
    rel, mx, d = err_stats(got, ref)
    assert np.all(np.isfinite(got)), f"{where}: non-finite output"
    assert rel <= REL_FRO, f"{where}: rel Frobenius {rel:.3e} > {REL_FRO}"
    if dtype == "f32":
        assert rel <= 1e-5, f"{where}: fp32 rel Frobenius {rel:.3e} > 1e-5"
    if quantization_limited:
        excess = np.abs(d) - bf16_half_ulp(ref)
        assert float(np.max(excess, initial=0.0)) <= MAX_ABS, \
            f"{where}: max |err| beyond half-ulp {np.max(excess):.3e} > {MAX_ABS}"
    else:
        assert mx <= MAX_ABS, f"{where}: max |err| {mx:.3e} > {MAX_ABS}"
    return rel, mx
