"""Seeded synthetic workloads for the transfer path.

This module only draws random inputs; it holds none of the method's
arithmetic.  Tests, the benchmark and the smoke check all take their inputs
from here, and then hand the same values to the HIP path and to the CPU
oracle.

A workload is one or more sequences of shared raw text, segmented twice (once
per tokenizer) into character spans, plus a sender KV cache shaped like a
real model's, and one affine map and bias per receiver layer and role.  The
real models, tokenizers and long-document datasets the paper evaluates on are
not used: random character segmentations stand in for the two tokenizers, and
normal / log-normal values stand in for cache activations.

Seeding: ``numpy.random.SeedSequence(seed).spawn(4)`` gives the streams for
(sender segmentation, receiver segmentation, cache values, maps); each batch
entry spawns its own children.  "N(0, v)" means variance v.

Keys that the sender stores after its own RoPE are drawn directly as the
stored values: a rotation of an i.i.d. N(0, 1) pair is again i.i.d. N(0, 1),
so drawing the stored post-RoPE key gives the distribution of rotating a
drawn pre-RoPE key, without any rotation here.
"""

from __future__ import annotations

import dataclasses
from dataclasses import dataclass
from typing import Optional, Tuple

import numpy as np


@dataclass(frozen=True)
class Config:
    name: str
    dtype: str                      # "f32" or "bf16": storage of caches and maps
    L_s: int
    L_r: int
    H_s: int
    H_r: int
    d_h: int
    T_s: Optional[int] = None       # sender tokens per sequence (None: use n_chars)
    n_chars: Optional[int] = None   # shared text length (when T_s is None)
    s_len: Tuple[int, int] = (1, 7)  # sender token length U{lo..hi}
    r_len: Tuple[int, int] = (1, 8)  # receiver token length U{lo..hi}
    k_scale_sigma: Optional[float] = None   # log-normal(0, s) per-channel K scales
    v_scale_sigma: Optional[float] = None   # log-normal(0, s) per-channel V scales
    scale_per_role_layer: bool = True       # scales drawn per (layer, role, channel)
    bias_var: float = 0.05
    rope: Optional[Tuple[float, float]] = None   # (theta_s, theta_r): keys stored post-RoPE
    batch: int = 1
    layer_map: str = "interp2"      # "interp2" or "neighbor3" (three concatenated sender layers)
    sender_keys_post_rope: bool = True   # False: the payload's keys are pre-RoPE (no un-rotation)
    paper_opts: bool = False        # draw 1/r per (layer, role) and receiver key-norm weights

    @property
    def d_in(self) -> int:
        return self.H_s * self.d_h

    @property
    def n_taps(self) -> int:
        return 3 if self.layer_map == "neighbor3" else 1

    @property
    def d_map_in(self) -> int:
        """Input size of each map: the concatenated features of n_taps layers."""
        return self.n_taps * self.d_in

    @property
    def d_r(self) -> int:
        return self.H_r * self.d_h

    def with_(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


# Tiny CPU-scale fp32 transfer: 1,200 characters, 4 -> 6 layers, 2 KV heads of 64.
TINY_F32 = Config("tiny-f32 1200ch 4->6L 2x64", "f32", L_s=4, L_r=6, H_s=2, H_r=2, d_h=64,
                  n_chars=1200, s_len=(1, 6), r_len=(1, 8), k_scale_sigma=0.5,
                  v_scale_sigma=0.5, bias_var=0.1)
# Llama-8B -> Qwen-7B shape, 4,096 sender tokens, no RoPE, outlier K channels.
LLAMA8B_QWEN7B_4K = Config("llama8b->qwen7b-shape T_s=4096", "bf16", L_s=32, L_r=28, H_s=8,
                           H_r=4, d_h=128, T_s=4096, k_scale_sigma=1.0,
                           scale_per_role_layer=True, bias_var=0.05)
# Llama-8B -> 14B shape with post-RoPE sender keys, theta 5e5 -> 1e9.
LLAMA8B_14B_8K = Config("llama8b->14b-shape T_s=8192 rope", "bf16", L_s=32, L_r=40, H_s=8,
                        H_r=8, d_h=128, T_s=8192, bias_var=0.05, rope=(5.0e5, 1.0e9))
LLAMA8B_14B_32K = LLAMA8B_14B_8K.with_(name="llama8b->14b-shape T_s=32768 rope", T_s=32768)
# The same shape with the paper's three-layer neighbourhood map (A is d_r x 3 d_in).
LLAMA8B_14B_32K_N3 = LLAMA8B_14B_32K.with_(name="llama8b->14b-shape T_s=32768 rope neighbor3",
                                           layer_map="neighbor3")
# The paper's cache construction at that shape: three-layer map, pre-RoPE
# sender keys, the map on x / r, the receiver's key norm, then its RoPE.
LLAMA8B_14B_32K_PAPER = LLAMA8B_14B_32K_N3.with_(
    name="llama8b->14b-shape T_s=32768 neighbor3 pre-rope 1/r knorm",
    sender_keys_post_rope=False, paper_opts=True)
# Qwen-7B -> Llama-8B shape (layer upsampling), batch of 4, theta 1e6 -> 5e5.
QWEN7B_LLAMA8B_B4 = Config("qwen7b->llama8b-shape B=4 rope", "bf16", L_s=28, L_r=32, H_s=4,
                           H_r=8, d_h=128, T_s=4096, bias_var=0.05, rope=(1.0e6, 5.0e5),
                           batch=4)

CONFIGS = {
    "tiny": TINY_F32,
    "qwen7b-4k": LLAMA8B_QWEN7B_4K,
    "14b-8k": LLAMA8B_14B_8K,
    "14b-32k": LLAMA8B_14B_32K,
    "14b-32k-n3": LLAMA8B_14B_32K_N3,
    "14b-32k-paper": LLAMA8B_14B_32K_PAPER,
    "reverse-b4": QWEN7B_LLAMA8B_B4,
}


# ----------------------------------------------------------------------------
# Segmentations (character spans [beg, end) per token)
# ----------------------------------------------------------------------------

def segment_tokens(rng: np.random.Generator, n_tokens: int, lo: int, hi: int):
    """n_tokens back-to-back tokens with lengths U{lo..hi}."""
    lens = rng.integers(lo, hi + 1, size=n_tokens, dtype=np.int64)
    end = np.cumsum(lens)
    return (end - lens).astype(np.int32), end.astype(np.int32)


def segment_chars(rng: np.random.Generator, n_chars: int, lo: int, hi: int):
    """Back-to-back tokens with lengths U{lo..hi} covering exactly n_chars
    characters; the last token is cut to end at n_chars."""
    if n_chars <= 0:
        return np.zeros(0, np.int32), np.zeros(0, np.int32)
    lens = rng.integers(lo, hi + 1, size=n_chars, dtype=np.int64)  # enough: lo >= 1
    end = np.cumsum(lens)
    n = int(np.searchsorted(end, n_chars, side="left")) + 1
    end = end[:n].copy()
    end[-1] = n_chars
    beg = np.concatenate([[0], end[:-1]])
    return beg.astype(np.int32), end.astype(np.int32)


def segment_messy(rng: np.random.Generator, n_chars: int, lo: int, hi: int,
                  p_empty: float = 0.05, p_gap: float = 0.05, max_gap: int = 3,
                  p_dup_end: float = 0.03):
    """A segmentation with the irregularities real tokenizer offsets show:
    empty tokens (beg == end), skipped characters (gaps between tokens), and
    split tokens that end at the same character as their neighbour
    (a zero-length tail token).  Spans stay sorted and non-overlapping."""
    beg, end = [], []
    pos = 0
    while pos < n_chars:
        if rng.random() < p_gap:
            pos = min(n_chars, pos + int(rng.integers(1, max_gap + 1)))
            if pos >= n_chars:
                break
        if rng.random() < p_empty:
            beg.append(pos)
            end.append(pos)
        ln = int(rng.integers(lo, hi + 1))
        e = min(n_chars, pos + ln)
        beg.append(pos)
        end.append(e)
        if rng.random() < p_dup_end:
            beg.append(e)
            end.append(e)
        pos = e
    return np.asarray(beg, np.int32), np.asarray(end, np.int32)


def _child_seeds(seed: int, n: int):
    return np.random.SeedSequence(seed).spawn(n)


@dataclass
class Segmentation:
    s_beg: np.ndarray   # int32 [sum T_s], concatenated over the batch
    s_end: np.ndarray
    r_beg: np.ndarray   # int32 [sum T_r]
    r_end: np.ndarray
    s_cu: np.ndarray    # int32 [B+1] prefix sums of T_s
    r_cu: np.ndarray    # int32 [B+1] prefix sums of T_r

    @property
    def s_len(self):
        return np.diff(self.s_cu).astype(np.int32)

    @property
    def r_len(self):
        return np.diff(self.r_cu).astype(np.int32)

    @property
    def batch(self):
        return self.s_cu.size - 1

    def seq(self, b):
        """Spans of sequence b: (s_beg, s_end, r_beg, r_end)."""
        s0, s1, r0, r1 = self.s_cu[b], self.s_cu[b + 1], self.r_cu[b], self.r_cu[b + 1]
        return self.s_beg[s0:s1], self.s_end[s0:s1], self.r_beg[r0:r1], self.r_end[r0:r1]


def concat_segmentations(parts):
    """parts: list of (s_beg, s_end, r_beg, r_end) per sequence."""
    s_cu = np.concatenate([[0], np.cumsum([p[0].size for p in parts])]).astype(np.int32)
    r_cu = np.concatenate([[0], np.cumsum([p[2].size for p in parts])]).astype(np.int32)
    cat = lambda k: (np.concatenate([p[k] for p in parts]).astype(np.int32)  # noqa: E731
                     if parts else np.zeros(0, np.int32))
    return Segmentation(cat(0), cat(1), cat(2), cat(3), s_cu, r_cu)


def make_segmentation(cfg: Config, seed: int = 0, T_s: Optional[int] = None,
                      batch: Optional[int] = None) -> Segmentation:
    B = cfg.batch if batch is None else batch
    T_s = cfg.T_s if T_s is None else T_s
    seg_seq, rseg_seq, _, _ = _child_seeds(seed, 4)
    s_children, r_children = seg_seq.spawn(B), rseg_seq.spawn(B)
    parts = []
    for b in range(B):
        rs, rr = np.random.default_rng(s_children[b]), np.random.default_rng(r_children[b])
        if T_s is not None:
            s_beg, s_end = segment_tokens(rs, T_s, *cfg.s_len)
            n_chars = int(s_end[-1]) if T_s > 0 else 0
        else:
            n_chars = cfg.n_chars
            s_beg, s_end = segment_chars(rs, n_chars, *cfg.s_len)
        r_beg, r_end = segment_chars(rr, n_chars, *cfg.r_len)
        parts.append((s_beg, s_end, r_beg, r_end))
    return concat_segmentations(parts)


# ----------------------------------------------------------------------------
# Caches and maps (torch tensors, drawn on the requested device)
# ----------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _torch_gen(seed_seq, device):
    torch = _torch()
    g = torch.Generator(device=device)
    g.manual_seed(int(seed_seq.generate_state(1, dtype=np.uint64)[0] & ((1 << 63) - 1)))
    return g


def storage_dtype(cfg: Config):
    torch = _torch()
    return torch.float32 if cfg.dtype == "f32" else torch.bfloat16


@dataclass
class Workload:
    cfg: Config
    seg: Segmentation
    S: "object"          # torch [B, L_s, 2, H_s, T_cap, d_h], storage dtype
    A: "object"          # torch [L_r, 2, d_r, d_in], storage dtype
    bias: "object"       # torch fp32 [L_r, 2, d_r]
    rope: Optional[dict]
    opts: Optional[dict] = None   # inv_r, k_norm, k_norm_eps (make_opts)

    @property
    def T_cap_s(self):
        return int(self.S.shape[4])


def make_cache(cfg: Config, seg: Segmentation, seed: int = 0, device="cpu"):
    """Sender cache [B, L_s, 2, H_s, T_cap, d_h]; rows past a sequence's length
    are zero.  Values N(0,1), optionally times per-channel log-normal scales."""
    torch = _torch()
    _, _, val_seq, _ = _child_seeds(seed, 4)
    B = seg.batch
    T_cap = max(1, int(seg.s_len.max()) if B else 1)
    dt = storage_dtype(cfg)
    S = torch.zeros((B, cfg.L_s, 2, cfg.H_s, T_cap, cfg.d_h), dtype=dt, device=device)
    scale_seq, *b_seqs = val_seq.spawn(B + 1)
    rs = np.random.default_rng(scale_seq)
    scales = np.ones((cfg.L_s, 2, cfg.H_s, 1, cfg.d_h), dtype=np.float64)
    for role, sig in ((0, cfg.k_scale_sigma), (1, cfg.v_scale_sigma)):
        if sig is not None:
            if cfg.scale_per_role_layer:
                scales[:, role] = rs.lognormal(0.0, sig, size=(cfg.L_s, cfg.H_s, 1, cfg.d_h))
            else:
                scales[:, role] = rs.lognormal(0.0, sig, size=(1, cfg.H_s, 1, cfg.d_h))
    sc = torch.as_tensor(scales, dtype=torch.float32, device=device)
    for b in range(B):
        g = _torch_gen(b_seqs[b], device)
        T = int(seg.s_len[b])
        for l in range(cfg.L_s):
            z = torch.randn((2, cfg.H_s, T, cfg.d_h), generator=g, dtype=torch.float32,
                            device=device)
            S[b, l, :, :, :T, :] = (z * sc[l]).to(dt)
    return S


def make_maps(cfg: Config, seed: int = 0, device="cpu"):
    """A [L_r, 2, d_r, n] ~ N(0, 1/n) with n = cfg.d_map_in, in the storage
    dtype, and bias [L_r, 2, d_r] ~ N(0, bias_var) in fp32."""
    torch = _torch()
    _, _, _, map_seq = _child_seeds(seed, 4)
    g = _torch_gen(map_seq, device)
    n = cfg.d_map_in
    A = torch.randn((cfg.L_r, 2, cfg.d_r, n), generator=g, dtype=torch.float32,
                    device=device) * (1.0 / np.sqrt(n))
    bias = torch.randn((cfg.L_r, 2, cfg.d_r), generator=g, dtype=torch.float32,
                       device=device) * float(np.sqrt(cfg.bias_var))
    return A.to(storage_dtype(cfg)), bias


def rope_params(cfg: Config, pos0_s=None, pos0_r=None):
    if cfg.rope is None:
        return None
    return dict(theta_s=float(cfg.rope[0]), theta_r=float(cfg.rope[1]),
                unrotate_sender_k=bool(cfg.sender_keys_post_rope), rotate_receiver_k=True,
                pos0_s=pos0_s, pos0_r=pos0_r)


def make_opts(cfg: Config, seed: int = 0, device="cpu", eps: float = 1e-6):
    """The paper-faithful options, or None: inv_r [L_r, 2] ~ 1 / U(0.8, 1.25)
    and receiver key-norm weights [L_r, d_h] ~ U(0.5, 1.5), fp32, drawn from
    the map stream after the maps."""
    if not cfg.paper_opts:
        return None
    torch = _torch()
    _, _, _, map_seq = _child_seeds(seed, 4)
    g = _torch_gen(map_seq.spawn(1)[0], device)
    r = 0.8 + 0.45 * torch.rand((cfg.L_r, 2), generator=g, dtype=torch.float32, device=device)
    k_norm = 0.5 + torch.rand((cfg.L_r, cfg.d_h), generator=g, dtype=torch.float32, device=device)
    return dict(inv_r=(1.0 / r).contiguous(), k_norm=k_norm, k_norm_eps=float(eps))


def make_workload(cfg: Config, seed: int = 0, device="cpu", T_s: Optional[int] = None,
                  batch: Optional[int] = None) -> Workload:
    seg = make_segmentation(cfg, seed, T_s=T_s, batch=batch)
    S = make_cache(cfg, seg, seed, device)
    A, bias = make_maps(cfg, seed, device)
    return Workload(cfg, seg, S, A, bias, rope_params(cfg), make_opts(cfg, seed, device))


# ----------------------------------------------------------------------------
# Calibration samples for the offline map construction
# ----------------------------------------------------------------------------

@dataclass(frozen=True)
class CalibConfig:
    """Paired calibration features for one receiver layer and role.

    n aligned tokens split over two corpora (``corpus_split`` of them in the
    first), sender features of size p (the concatenated taps), receiver
    features of size q."""
    name: str
    n: int
    p: int
    q: int
    dtype: str = "f32"
    corpus_split: float = 0.6
    noise: float = 0.5
    dup_block: int = 0      # >0: columns [dup_block, 2 dup_block) repeat [0, dup_block)


CALIB_SMALL = CalibConfig("calibration 3000 tokens 100->37", n=3000, p=100, q=37)
CALIB_14B = CalibConfig("calibration llama8b->14b-shape 2^20 tokens 3x1024->1024", n=1 << 20,
                        p=3072, q=1024)
CALIB_CONFIGS = {"calib-small": CALIB_SMALL, "calib-14b": CALIB_14B}


def make_calibration(cfg: CalibConfig, seed: int = 0, device="cpu"):
    """Seeded samples (x [n, p], y [n, q], w [n]).

    x: independent N(0, (1 + k)^-1) channels k = 0..p-1 (a decaying spectrum),
    mixed by two random Householder reflections, times per-channel log-normal
    scales (sigma 0.5), plus per-channel offsets N(0, 0.25).  y: x times a
    N(0, 1/p) matrix, plus N(0, noise^2) noise and offsets N(0, 0.25).  Weights
    give the two corpora equal total weight (1/2 each, uniform inside a
    corpus).  x and y are stored in cfg.dtype; w is fp32."""
    torch = _torch()
    seqs = np.random.SeedSequence(seed).spawn(3)
    g = _torch_gen(seqs[0], device)
    f32 = torch.float32
    n, p, q = cfg.n, cfg.p, cfg.q
    var = 1.0 / torch.sqrt(1.0 + torch.arange(p, dtype=f32, device=device))
    x = torch.randn((n, p), generator=g, dtype=f32, device=device) * var
    for _ in range(2):
        v = torch.randn(p, generator=g, dtype=f32, device=device)
        v = v / torch.linalg.vector_norm(v)
        x -= 2.0 * (x @ v)[:, None] * v[None, :]
    x *= torch.exp(0.5 * torch.randn(p, generator=g, dtype=f32, device=device))
    x += 0.5 * torch.randn(p, generator=g, dtype=f32, device=device)
    if cfg.dup_block:
        x[:, cfg.dup_block:2 * cfg.dup_block] = x[:, :cfg.dup_block]
    g2 = _torch_gen(seqs[1], device)
    Cm = torch.randn((p, q), generator=g2, dtype=f32, device=device) / float(np.sqrt(p))
    y = x @ Cm
    y += cfg.noise * torch.randn((n, q), generator=g2, dtype=f32, device=device)
    y += 0.5 * torch.randn(q, generator=g2, dtype=f32, device=device)
    n_a = max(1, min(n - 1, int(round(cfg.corpus_split * n)))) if n > 1 else n
    w = torch.empty(n, dtype=f32, device=device)
    w[:n_a] = 0.5 / n_a
    if n > n_a:
        w[n_a:] = 0.5 / (n - n_a)
    dt = f32 if cfg.dtype == "f32" else torch.bfloat16
    return x.to(dt), y.to(dt), w
