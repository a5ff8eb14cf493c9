"""C-ABI checks that need no GPU: the library loads and exports every
declared symbol, host-only entry points, and host-side argument validation
(every call below fails before touching the HIP runtime)."""

import ctypes as C
import os
import re

import numpy as np
import pytest

from oracle import layer_map as lm
from paper_2609_32259_amd import heterofold as hf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(hf.LIB_PATH):
        from paper_2609_32259_amd import build
        build.build()
    return hf.lib()


def _declared():
    src = open(os.path.join(ROOT, "include", "heterofold.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(hf_[a-z0-9_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported(L):
    decl = _declared()
    assert len(decl) >= 14
    for name in decl:
        assert hasattr(L, name), name
    assert sorted(hf.exported_symbols()) == decl


def test_version(L):
    assert hf.hf_version() == 2


@pytest.mark.parametrize("L_s,L_r", [(4, 6), (32, 40), (32, 28), (28, 32), (1, 3), (5, 1), (7, 7)])
def test_layer_map_matches_oracle(L, L_s, L_r):
    got = hf.hf_build_layer_map(L_s, L_r)
    exp = lm.interp2(L_s, L_r)
    for g, e in zip(got, exp):
        assert np.array_equal(g, e)


def test_layer_map_errors(L):
    with pytest.raises(hf.HeteroFoldError) as ei:
        hf.hf_build_layer_map(0, 3)
    assert ei.value.status == -2
    with pytest.raises(hf.HeteroFoldError) as ei:
        hf.hf_build_layer_map(3, 3, mode=7)
    assert ei.value.status == -4


def test_validate_offsets_host(L):
    hf.hf_validate_offsets_host([0, 3, 3, 5], [3, 3, 5, 9])
    hf.hf_validate_offsets_host([], [])
    for beg, end in (([0, 2], [3, 5]), ([2], [1]), ([-1], [0]), ([3, 0], [4, 1])):
        with pytest.raises(hf.HeteroFoldError) as ei:
            hf.hf_validate_offsets_host(beg, end)
        assert ei.value.status == -3


def test_nnz_capacity(L):
    assert hf.hf_alignment_nnz_capacity([10, 15], [8, 12]) == 25 + 40
    assert hf.hf_alignment_nnz_capacity([10, 15], [8, 12], "ta") == 20
    assert hf.hf_alignment_nnz_capacity([0], [0]) == 0
    with pytest.raises(hf.HeteroFoldError) as ei:
        hf.hf_alignment_nnz_capacity([-1, 10], [0, 8])
    assert ei.value.status == -2
    with pytest.raises(hf.HeteroFoldError) as ei:
        hf.hf_alignment_nnz_capacity([1], [1], 7)
    assert ei.value.status == -4
    s, r = np.array([3], np.int32), np.array([2], np.int32)
    assert L.hf_alignment_nnz_capacity(0, _p(s), _p(r), 0) == -1
    assert L.hf_alignment_nnz_capacity(1, None, _p(r), 0) == -1


def _p(a):
    return a.ctypes.data_as(C.POINTER(C.c_int32))


def test_alignment_host_validation(L):
    s_cu = np.array([0, 10], np.int32)
    r_cu = np.array([0, 9], np.int32)
    fake = C.c_void_p(0x1000)
    args = lambda **kw: dict(dict(B=1, s_cu=_p(s_cu), r_cu=_p(r_cu), sb=fake, se=fake, rb=fake, re=fake,  # noqa: E731
                                  mode=0, rp=fake, col=fake, num=fake, den=fake, cap=28, ws=fake,
                                  wsb=1 << 20, st=None), **kw)

    def call(a):
        return L.hf_build_alignment(a["B"], a["s_cu"], a["r_cu"], a["sb"], a["se"], a["rb"],
                                    a["re"], a["mode"], a["rp"], a["col"], a["num"], a["den"],
                                    a["cap"], a["ws"], a["wsb"], a["st"])

    assert call(args(B=0)) == -2
    assert call(args(mode=5)) == -4
    assert call(args(rp=None)) == -1
    assert call(args(col=None)) == -1
    assert call(args(cap=27)) == -6           # overlap needs T_s + 2 T_r = 28
    assert call(args(cap=8, mode=1)) == -6    # TA needs T_r = 9
    assert call(args(ws=None)) == -1
    assert call(args(wsb=1)) == -6
    bad = np.array([0, 0], np.int32)
    assert call(args(s_cu=_p(bad))) == -2   # receiver tokens but no sender tokens
    assert L.hf_last_error().decode()


def _desc(ptr=0x1000, dtype=1, L_=4, H=8, d=128, T=64):
    st_t = d
    st_h = T * d
    st_c = H * st_h
    st_l = 2 * st_c
    st_b = L_ * st_l
    return hf.hf_kv_desc(C.c_void_p(ptr), dtype, L_, H, d, T, st_b, st_l, st_c, st_h, st_t)


def test_transfer_host_validation(L):
    s_len = np.array([64], np.int32)
    r_len = np.array([60], np.int32)
    lt = [np.ascontiguousarray(x, dtype=np.int32) for x in lm.interp2(4, 6)]
    fake = C.c_void_p(0x1000)

    def call(sd=None, rd=None, B=1, sl=s_len, rl=r_len, table=lt, A=fake, Ab=None, rope=None,
             ws=None, wsb=0, rp=fake, opts=None):
        sd = sd or _desc()
        rd = rd or _desc(L_=6)
        if Ab is None:
            Ab = L.hf_packed_maps_bytes(rd.L, rd.H * rd.d_h, sd.H * sd.d_h, sd.dtype)
        return L.hf_transfer_kv(B, _p(sl), _p(rl), rp, fake, fake, fake, *[_p(t) for t in table],
                                C.byref(sd), C.byref(rd), A, Ab, None,
                                C.byref(rope) if rope is not None else None,
                                C.byref(opts) if opts is not None else None, ws, wsb, None)

    assert call(B=0) == -2
    assert call(rp=None) == -1
    assert call(A=None) == -1
    unpacked = 6 * 2 * 1024 * 1024 * 2                         # A [L_r][2][d_r][d_in], bf16
    assert call(Ab=unpacked) == -2                             # an unpacked map is refused
    assert "hf_pack_maps" in L.hf_last_error().decode()
    assert call(Ab=unpacked + 256 + 2) == -2
    assert call(sd=_desc(ptr=0)) == -1
    assert call(sd=_desc(dtype=0)) == -5                       # dtypes differ
    assert call(sd=_desc(dtype=9)) == -5
    assert call(sd=_desc(d=64), rd=_desc(L_=6, d=64)) == -8    # bf16 needs d_h = 128
    assert call(rd=_desc(L_=6, H=3)) == -8                     # receiver heads
    assert call(sd=_desc(ptr=0x1008)) == -2                    # misaligned
    assert call(rl=np.array([65], np.int32)) == -2             # longer than T_cap
    bad = [t.copy() for t in lt]
    bad[0][2] = 4
    assert call(table=bad) == -2                               # sender layer out of range
    bad = [t.copy() for t in lt]
    bad[2][1] = bad[3][1]
    assert call(table=bad) == -2                               # rem >= den
    r, keep = hf.make_rope(5e5, 1e9)
    assert call(rope=r) == -1                                  # RoPE needs a workspace
    r2, keep2 = hf.make_rope(-1.0, 1e9)
    assert call(rope=r2, ws=fake, wsb=1 << 30) == -2
    assert call(opts=hf.hf_transfer_opts(None, C.c_void_p(0x1000), -1.0)) == -2      # eps < 0
    assert call(opts=hf.hf_transfer_opts(None, C.c_void_p(0x1000), float("nan"))) == -2
    assert call(opts=hf.hf_transfer_opts(C.c_void_p(0x1002), None, 0.0)) == -2      # misaligned
    assert call(sd=_desc(dtype=0, d=96), rd=_desc(L_=6, dtype=0, d=96),
                opts=hf.hf_transfer_opts(None, C.c_void_p(0x1000), 1e-6)) == -8   # fp32 norm d_h
    # cos/sin tables: 64 sender + 60 receiver positions x 64 pairs x 8 bytes, then
    # one 8 KB staging record per 64-row receiver tile and 256 bytes of work counter
    assert L.hf_transfer_workspace_bytes(1, _p(s_len), _p(r_len), C.byref(_desc()),
                                         C.byref(_desc(L_=6)), C.byref(r)) == 64 * 512 + 60 * 512 + 8192 + 256


def test_transfer_workspace_records(L):
    s_len = np.array([64, 64, 64], np.int32)
    r_len = np.array([60, 0, 64], np.int32)
    lt = [np.ascontiguousarray(x, dtype=np.int32) for x in lm.interp2(4, 6)]
    fake = C.c_void_p(0x1000)

    def wsb(sd, rd):
        return L.hf_transfer_workspace_bytes(3, _p(s_len), _p(r_len), C.byref(sd), C.byref(rd), None)

    # bf16 with 8 or 4 receiver heads: one record per non-empty 64-row tile, and
    # the work counter
    assert wsb(_desc(), _desc(L_=6)) == 2 * 8192 + 256
    assert wsb(_desc(H=4), _desc(L_=6, H=4)) == 2 * 8192 + 256
    r130 = np.array([130], np.int32)
    assert L.hf_transfer_workspace_bytes(1, _p(np.array([200], np.int32)), _p(r130),
                                         C.byref(_desc(T=256)), C.byref(_desc(L_=6, T=256)),
                                         None) == 3 * 8192 + 256
    # kernels that keep no records: 2 receiver heads, more than 8 sender heads, fp32
    assert wsb(_desc(), _desc(L_=6, H=2)) == 0
    assert wsb(_desc(H=16), _desc(L_=6)) == 0
    assert wsb(_desc(dtype=0), _desc(L_=6, dtype=0)) == 0

    def call(ws, n):
        sd, rd = _desc(), _desc(L_=6)
        Ab = L.hf_packed_maps_bytes(6, 1024, 1024, 1)
        return L.hf_transfer_kv(3, _p(s_len), _p(r_len), fake, fake, fake, fake,
                                *[_p(t) for t in lt], C.byref(sd), C.byref(rd), fake, Ab, None,
                                None, None, ws, n, None)

    assert call(None, 0) == -1                       # records need a workspace
    assert call(C.c_void_p(0x100000), 8192) == -6    # too small
    assert call(C.c_void_p(0x100000 + 16), 1 << 20) == -2   # not 256-byte aligned


def test_transfer_staged_workspace_bytes(L):
    # The staged path's size: the fused path's workspace, a 16 KB table, and one
    # slab per (role, receiver layer) -- interpolating map -- or per (role, sender
    # layer) -- concatenated taps -- of 2 bytes x 1024 features x 256 rows per
    # 256-row tile of each sequence.
    s_len = np.array([64, 64, 700], np.int32)
    r_len = np.array([60, 0, 513], np.int32)     # 1 + 0 + 3 row tiles of 256
    sd, rd = _desc(L_=4, T=1024), _desc(L_=6, T=1024)

    def st(n_taps, sd=sd, rd=rd, B=3):
        return L.hf_transfer_staged_workspace_bytes(B, _p(s_len), _p(r_len), C.byref(sd),
                                                    C.byref(rd), None, n_taps)

    base = L.hf_transfer_workspace_bytes(3, _p(s_len), _p(r_len), C.byref(sd), C.byref(rd), None)
    slab = 4 * 256 * 1024 * 2
    assert st(0) == base + 16384 + 2 * 6 * slab          # receiver layers
    for n_taps in (1, 2, 3):
        assert st(n_taps) == base + 16384 + 2 * 4 * slab  # sender layers
    # shapes and arguments the staged path does not serve
    assert st(4) == 0 and st(-1) == 0 and st(0, B=0) == 0
    assert st(0, rd=_desc(L_=6, H=4, T=1024)) == 0            # 4 receiver heads
    assert st(0, sd=_desc(L_=4, H=16, T=1024)) == 0           # 16 sender heads
    assert st(0, sd=_desc(L_=4, dtype=0, T=1024), rd=_desc(L_=6, dtype=0, T=1024)) == 0  # fp32
    assert st(0, sd=_desc(L_=4, d=64, T=1024), rd=_desc(L_=6, d=64, T=1024)) == 0     # d_h 64


def test_pack_host_validation(L):
    fake = C.c_void_p(0x1000)
    assert L.hf_pack_maps(2, 100, 1024, 1, fake, C.c_void_p(0x100000), None) == -2   # d_r % 32
    assert L.hf_pack_maps(2, 128, 1024, 3, fake, C.c_void_p(0x100000), None) == -5
    assert L.hf_pack_maps(2, 128, 1024, 1, None, C.c_void_p(0x100000), None) == -1
    assert L.hf_pack_maps(2, 128, 128, 1, fake, C.c_void_p(0x1000 + 64), None) == -2  # overlap
    assert hf.hf_packed_maps_bytes(40, 1024, 1024, 1) == 256 + 40 * 2 * 1024 * 1024 * 2
    assert hf.hf_packed_maps_bytes(40, 1024, 1024, 0) == 256 + 40 * 2 * 1024 * 1024 * 4
    assert hf.hf_packed_maps_bytes(40, 1024, 1024, 5) == 0


def test_profiler_host_calls(L):
    hf.hf_profiler_enable(False)
    hf.hf_profiler_reset()
    assert hf.hf_profiler_query(hf.HF_KERNEL_TRANSFER) == (0.0, 0)
    with pytest.raises(hf.HeteroFoldError):
        hf.hf_profiler_query(99)
    assert hf.hf_profiler_samples(hf.HF_KERNEL_TRANSFER).size == 0
    with pytest.raises(hf.HeteroFoldError):
        hf.hf_profiler_samples(-1)


@pytest.mark.parametrize("L_s,L_r", [(32, 40), (32, 28), (28, 32), (36, 32), (40, 36), (4, 6),
                                     (9, 9), (1, 3), (5, 1), (3, 20), (64, 7)])
def test_layer_taps_match_oracle(L, L_s, L_r):
    """hf_build_layer_taps against the oracle's Eq. 1 table (itself pinned by
    the worked rows and the App. B.4 parameter counts)."""
    assert np.array_equal(hf.hf_build_layer_taps(L_s, L_r), lm.neighbor3(L_s, L_r))


def test_layer_taps_errors(L):
    with pytest.raises(hf.HeteroFoldError) as ei:
        hf.hf_build_layer_taps(0, 3)
    assert ei.value.status == -2
    assert L.hf_build_layer_taps(3, 3, None) == -1


def test_transfer_taps_host_validation(L):
    s_len = np.array([64], np.int32)
    r_len = np.array([60], np.int32)
    taps = np.ascontiguousarray(lm.neighbor3(4, 6), dtype=np.int32)
    fake = C.c_void_p(0x1000)

    def call(n=3, tp=taps, sd=None, rd=None):
        sd = sd or _desc()
        rd = rd or _desc(L_=6)
        Ab = L.hf_packed_maps_bytes(rd.L, rd.H * rd.d_h, max(n, 1) * sd.H * sd.d_h, sd.dtype)
        return L.hf_transfer_kv_taps(1, _p(s_len), _p(r_len), fake, fake, fake, fake, n,
                                     _p(tp) if tp is not None else None, C.byref(sd),
                                     C.byref(rd), fake, Ab, None, None, None, None, 0, None)

    assert call(tp=None) == -1
    assert call(n=0) == -2
    assert call(n=4) == -2
    bad = taps.copy()
    bad[5, 2] = 4
    assert call(tp=bad) == -2                                  # sender layer out of range
    bad = taps.copy()
    bad[1, 0] = -1
    assert call(tp=bad) == -2
    assert call(sd=_desc(d=64), rd=_desc(L_=6, d=64)) == -8    # bf16 needs d_h = 128


def test_recolor_host_validation(L):
    fake = C.c_void_p(0x10000)
    ws = C.c_void_p(0x100000)
    big = 1 << 40
    # moments: n, sizes, dtype, NULLs, leading dimensions, workspace
    args = lambda **k: dict(dict(n=100, p=8, q=4, dtype=0, x=fake, ldx=8, y=fake, ldy=4, w=None,
                                 r=C.c_void_p(0x20000), mu=C.c_void_p(0x30000),
                                 cov=C.c_void_p(0x40000), ws=ws, wsb=big), **k)
    def mom(a):
        return L.hf_recolor_moments(a["n"], a["p"], a["q"], a["dtype"], a["x"], a["ldx"], a["y"],
                                    a["ldy"], a["w"], a["r"], a["mu"], a["cov"], a["ws"],
                                    a["wsb"], None)
    assert mom(args(n=0)) == -2
    assert mom(args(p=0)) == -2
    assert mom(args(p=40000, q=40000)) == -2
    assert mom(args(dtype=7)) == -5
    assert mom(args(x=None)) == -1
    assert mom(args(ldx=7)) == -2
    assert mom(args(mu=C.c_void_p(0x40000 + 8))) == -2      # inside cov
    assert mom(args(ws=None)) == -1
    assert mom(args(ws=C.c_void_p(0x100000 + 16))) == -2    # not 256-B aligned
    assert mom(args(wsb=16)) == -6
    assert hf.hf_recolor_moments_workspace_bytes(1 << 20, 3072, 1024) > 0
    assert L.hf_recolor_moments_workspace_bytes(0, 3, 3) == 0
    # solve
    def sol(p=8, q=4, mu=C.c_void_p(0x30000), cov=C.c_void_p(0x40000), ridge=0.0,
            A=C.c_void_p(0x80000), b=C.c_void_p(0x90000), ws=ws, wsb=big):
        return L.hf_recolor_solve(p, q, mu, cov, ridge, A, b, None, ws, wsb, None)
    assert sol(p=0) == -2
    assert sol(ridge=-1.0) == -2
    assert sol(ridge=float("nan")) == -2
    assert sol(ridge=float("inf")) == -2
    assert sol(A=None) == -1
    assert sol(A=C.c_void_p(0x40000)) == -2                 # output over the input
    assert sol(b=C.c_void_p(0x80000 + 8)) == -2             # b inside A
    assert sol(wsb=8) == -6
    assert sol(A=C.c_void_p(0x80004)) == -2                 # misaligned
    assert hf.hf_recolor_solve_workspace_bytes(3072, 1024) > 5 * 3072 * 3072 * 8
    # fold
    def fold(p=8, q=4, rank=2, A=C.c_void_p(0x80000), b=C.c_void_p(0x90000),
             B=C.c_void_p(0xA0000), G=C.c_void_p(0xB0000), Ao=C.c_void_p(0xC0000),
             bo=C.c_void_p(0xD0000), wsb=big):
        return L.hf_fold_map(p, q, rank, A, b, B, G, Ao, bo, ws, wsb, None)
    assert fold(rank=0) == -2
    assert fold(G=None) == -1
    assert fold(Ao=C.c_void_p(0x80000 + 8)) == -2          # partial overlap with A
    assert fold(Ao=C.c_void_p(0xA0000)) == -2              # over B
    assert fold(wsb=0) == -6
    assert hf.hf_fold_workspace_bytes(3072, 16) >= 16 * 3072 * 8
    # product
    def gemm(m=4, n=4, k=4, A=fake, lda=4, ak=0, B=fake, ldb=4, bk=1, D=C.c_void_p(0x50000),
             ldd=4, beta=0.0, Cp=None, ldc=0):
        return L.hf_gemm_f64(m, n, k, A, lda, ak, B, ldb, bk, D, ldd, 1.0, beta, Cp, ldc, 0.0,
                             None)
    assert gemm(m=0) == -2
    assert gemm(m=65535 * 64 + 1) == -2
    assert gemm(k=-1) == -2
    assert gemm(D=None) == -1
    assert gemm(beta=1.0) == -1
    assert gemm(lda=3) == -2
    assert gemm(ak=1, lda=3) == -2
    assert gemm(ldd=3) == -2
    assert gemm(beta=1.0, Cp=fake, ldc=3) == -2


def test_transfer_noalloc_host_validation(L):
    # Host checks run before any HIP call; a transfer whose scratch exceeds the
    # library's array is refused with HF_ERR_CAPACITY.
    s_len = np.array([64], np.int32)
    r_len = np.array([60], np.int32)
    lt = [np.ascontiguousarray(x, dtype=np.int32) for x in lm.interp2(4, 6)]
    fake = C.c_void_p(0x1000)
    sd, rd = _desc(), _desc(L_=6)
    Ab = L.hf_packed_maps_bytes(6, 1024, 1024, 1)

    def call(rope=None, Ab=Ab, sd=sd, rp=fake):
        return L.hf_transfer_kv_noalloc(1, _p(s_len), _p(r_len), rp, fake, fake, fake,
                                        *[_p(t) for t in lt], C.byref(sd), C.byref(rd), fake, Ab,
                                        None, C.byref(rope) if rope is not None else None, None,
                                        None)

    assert call(rp=None) == -1
    assert call(Ab=Ab - 256) == -2                              # unpacked map
    assert call(sd=_desc(d=64)) == -2                           # d_h differs
    far = np.array([100_000_000], np.int32)                     # RoPE tables past 64 MiB
    r, keep = hf.make_rope(5e5, 1e9, pos0_s=far)
    assert call(rope=r) == -6
    assert "hf_transfer_kv_noalloc" in L.hf_last_error().decode()
    r0, keep0 = hf.make_rope(5e5, 1e9)
    assert 0 < L.hf_transfer_workspace_bytes(1, _p(s_len), _p(r_len), C.byref(sd), C.byref(rd),
                                             C.byref(r0)) < 64 << 20
