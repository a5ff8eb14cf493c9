"""GPU-vs-oracle comparison shared by the GPU parity tests.

For one sequence of a batch, a window of receiver rows [r0, r1) (the whole
sequence by default) and a set of receiver layers, the oracle's features are
formed from the sender tokens the window reads (oracle.transfer.features /
features_taps on the sliced sender cache, with the sender RoPE positions
shifted to match), then mapped (oracle.transfer.map_features), and every
element of the GPU result in the window is checked by _parity.check_layer.
Windows keep full-size checks affordable: the oracle's cost grows with the
windows, not with the sequence.  The windows of a sequence are mapped, gated
and compared together, so a per-layer figure such as rel-Fro covers all of
them.
"""

import numpy as np

from _parity import Worst, check_layer, kernel_gate
from oracle import alignment as al
from oracle import layer_map as lm
from oracle import transfer as tr


def np64(t):
    return t.float().cpu().numpy().astype(np.float64)


def opts64(opts):
    if opts is None:
        return None
    return dict(inv_r=None if opts.get("inv_r") is None else np64(opts["inv_r"]),
                k_norm=None if opts.get("k_norm") is None else np64(opts["k_norm"]),
                k_norm_eps=opts.get("k_norm_eps", 1e-6))


def seq_rope(rope, b):
    if rope is None:
        return None
    rp = dict(rope)
    for k in ("pos0_s", "pos0_r"):
        rp[k] = 0 if rope.get(k) is None else int(np.asarray(rope[k])[b])
    return rp


def csr_window(csr, r0, r1):
    """Rows [r0, r1) of a CSR table, with sender columns shifted to start at
    the smallest one they read: (csr_w, c0, c1) with columns in [c0, c1)."""
    row_ptr, col, num, den = (np.asarray(t, dtype=np.int64) for t in csr)
    e0, e1 = int(row_ptr[r0]), int(row_ptr[r1])
    c0, c1 = int(col[e0:e1].min()), int(col[e0:e1].max()) + 1
    return (row_ptr[r0:r1 + 1] - e0, col[e0:e1] - c0, num[e0:e1], den[r0:r1]), c0, c1


def windows(T_r, tile, rng, n_mid=2, width=256):
    """Receiver-row windows for a sampled check: the head, the tail, and
    n_mid windows starting just before a row-tile edge at random."""
    out = [(0, min(width, T_r))]
    for _ in range(n_mid):
        if T_r > 2 * width + tile:
            t = int(rng.integers(1, (T_r - width) // tile)) * tile
            out.append((t - 3, min(T_r, t - 3 + width)))
    out.append((max(0, T_r - width), T_r))
    return out


class Case:
    """GPU results to check: cfg, workload, the receiver cache R a path wrote
    (or a dict {label: R} of several paths' caches for the same inputs, each
    checked against one oracle computation), the alignment mode and the layer
    map ("interp2", "neighbor3" or an explicit [L_r][n] tap table).
    scale_product: the path applied 1/r to the product A x_j instead of to x_j
    before its bf16 rounding (the staged path with concatenated taps); the
    kernel-arithmetic gate then rounds x_j unscaled and maps it with A / r."""

    def __init__(self, cfg, wl, R, mode="overlap", layer_map=None, tag="gpu",
                 scale_product=False):
        self.cfg, self.wl, self.mode, self.tag = cfg, wl, mode, tag
        self.results = dict(R) if isinstance(R, dict) else {"": R}
        self.scale_product = scale_product
        lmap = cfg.layer_map if layer_map is None else layer_map
        if isinstance(lmap, str) and lmap == "interp2":
            self.lt, self.taps = lm.interp2(cfg.L_s, cfg.L_r), None
        elif isinstance(lmap, str):
            self.lt, self.taps = None, lm.neighbor3(cfg.L_s, cfg.L_r)
        else:
            self.lt, self.taps = None, np.asarray(lmap)
        self.opts = opts64(wl.opts)
        self._csr = {}

    def csr(self, b):
        if b not in self._csr:
            self._csr[b] = al.build_alignment(*self.wl.seg.seq(b), self.mode)
        return self._csr[b]

    def qlimited(self, c):
        """Keys with log-normal outlier channels, or after the key norm."""
        cfg = self.cfg
        return c == 0 and cfg.dtype == "bf16" and (bool(cfg.k_scale_sigma) or
                                                   self.opts is not None)

    def check(self, b, layers, spans=None, roles=(0, 1), worst=None, verbose=False):
        """Sequence b, the given receiver layers and roles, on the row windows
        spans [(r0, r1), ...] (the whole sequence by default).  Each window's
        features are formed from the sender tokens it reads; the windows' rows
        are then mapped, gated and compared together, one oracle map and one
        gate per (layer, role), with rel-Fro over all of them."""
        cfg, wl = self.cfg, self.wl
        T_r = int(wl.seg.r_len[b])
        spans = [(0, T_r)] if spans is None else spans
        spans = [(r0, min(r1, T_r)) for r0, r1 in spans if min(r1, T_r) > r0]
        worst = Worst() if worst is None else worst
        if not spans:
            return worst
        rope = seq_rope(wl.rope, b)
        win = []  # (r0, r1, csr_w, c0, c1, rope_w) per window
        for r0, r1 in spans:
            csr_w, c0, c1 = csr_window(self.csr(b), r0, r1)
            win.append((r0, r1, csr_w, c0, c1,
                        None if rope is None else dict(rope, pos0_s=rope["pos0_s"] + c0)))
        rows = np.concatenate([np.arange(r0, r1) for r0, r1 in spans])
        span_txt = ",".join(f"[{r0},{r1})" for r0, r1 in spans)
        A_all, b_all = wl.A, wl.bias
        for l in layers:
            if self.taps is None:
                lo, hi, rem, den = (int(t[l]) for t in self.lt)
                need = [lo] if rem == 0 else [lo, hi]
                sub = (np.array([0]), np.array([len(need) - 1]), np.array([rem]), np.array([den]))
            else:
                need = sorted(set(int(t) for t in self.taps[l]))
                sub = np.array([[need.index(int(t)) for t in self.taps[l]]])
            # the windows' sender columns only, both roles
            S_w = [np64(wl.S[b][:, :, :, c0:c1, :][need]) for _, _, _, c0, c1, _ in win]
            for c in roles:
                parts = []
                for S, (_, _, csr_w, _, _, rope_w) in zip(S_w, win):
                    if self.taps is None:
                        parts.append(tr.features(S, sub, csr_w, rope_w, 0, c))
                    else:
                        parts.append(tr.features_taps(S, sub, csr_w, rope_w, 0, c))
                x = np.concatenate(parts, axis=0)
                xs = tr.scaled_features(x, l, c, self.opts)
                A = np64(A_all[l, c])
                bias = None if b_all is None else np64(b_all[l, c])
                ref = tr.map_features(xs, A, bias, c, cfg.d_h, l, rope, self.opts, rows)
                gate = None
                if cfg.dtype == "bf16":
                    inv_r = None if self.opts is None else self.opts.get("inv_r")
                    if self.scale_product and inv_r is not None:
                        o = dict(self.opts, inv_r=None)
                        gate = kernel_gate(np.asarray(x, np.float64), A * float(inv_r[l, c]), bias, c,
                                           cfg.d_h, l, rope, o, rows)
                    else:
                        gate = kernel_gate(xs, A, bias, c, cfg.d_h, l, rope, self.opts, rows)
                for label, R in self.results.items():
                    got = np.concatenate([np64(R[b, l, c, :, r0:r1, :]) for r0, r1 in spans], axis=1)
                    where = f"{cfg.name}{' ' + label if label else ''} b={b} l={l} c={c} rows={span_txt}"
                    s = check_layer(got, ref, where, dtype=cfg.dtype,
                                    max_abs="report" if self.qlimited(c) else "ulp", gate=gate)
                    worst.add(s)
                    if verbose:
                        print(f"[{self.tag}] {where}: rel-Fro {s['rel']:.3e} max|err| {s['max']:.3e} "
                              f"#>2e-2 {s['n_over']} #>2e-2+ulp {s['n_over_ulp']} "
                              f"gate {s['gate']:.2f}", flush=True)
        return worst

    def check_all(self, layers=None, windows_of=None, verbose=False):
        """Every sequence of the batch, all layers by default, whole
        sequences or the windows windows_of(b, T_r) gives."""
        worst = Worst()
        layers = range(self.cfg.L_r) if layers is None else layers
        for b in range(self.wl.seg.batch):
            T_r = int(self.wl.seg.r_len[b])
            spans = None if windows_of is None else windows_of(b, T_r)
            self.check(b, layers, spans, worst=worst, verbose=verbose)
        print(f"[{self.tag}] {self.cfg.name}: {worst}", flush=True)
        return worst
