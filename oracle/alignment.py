"""Cross-tokenizer alignment oracle (test infrastructure; see package docstring).

Inputs are the character spans of the tokens of ONE sequence, as produced by
the two tokenizers over the same raw text: token t covers characters
[beg[t], end[t]).  A token with beg == end is empty.

Two alignments are defined, both returned as a CSR span table
(row_ptr[T_r+1], col[nnz], num[nnz], den[T_r]) where receiver row j reads the
sender tokens col[row_ptr[j]:row_ptr[j+1]] with weights num/den[j]:

* Token Alignment (TA), Sec. 3.1 paragraph "Token Alignment" and App. B.1:
  nonempty sender and receiver tokens are paired when they end at the same
  character.  A receiver token without such a partner takes the sender token
  of the latest preceding shared boundary; before the first shared boundary it
  takes the first sender token.  Sender states are never averaged, so every
  row holds one entry with weight 1.
  Readings where the paper is silent: when several nonempty sender tokens end
  at the same character, the one with the largest index is the partner (it is
  the latest causal state at that boundary, matching "the same causal prefix
  endpoint" of the worked example); empty receiver tokens take no partner of
  their own and are forward-filled; with no nonempty sender token at all the
  "first sender token" is index 0.

* Overlap-weighted span alignment: receiver token j reads every sender token i
  whose character span overlaps its own, weighted by the number of shared
  characters o_ji = max(0, min(e_i, e_j) - max(b_i, b_j)); den_j = sum_i o_ji.
  A receiver token that overlaps no sender token (an empty token, a gap, or a
  token past the sender's text) falls back to its TA entry with weight 1.
"""

from __future__ import annotations

import numpy as np


def _as_int(a):
    return np.asarray(a, dtype=np.int64)


def first_nonempty(beg, end) -> int:
    """Index of the first nonempty token; 0 when every token is empty."""
    beg, end = _as_int(beg), _as_int(end)
    idx = np.nonzero(beg < end)[0]
    return int(idx[0]) if idx.size else 0


def ta_alignment(s_beg, s_end, r_beg, r_end) -> np.ndarray:
    """TA map a(j) for every receiver token j (int64 [T_r]).

    Sec. 3.1 "Token Alignment"; App. B.1 (definition of a(j)).
    """
    s_beg, s_end, r_beg, r_end = map(_as_int, (s_beg, s_end, r_beg, r_end))
    # Character end -> largest nonempty sender index ending there.
    partner = {}
    for i in range(s_end.size):
        if s_beg[i] < s_end[i]:
            partner[int(s_end[i])] = i  # later (larger) indices overwrite
    a = np.empty(r_end.size, dtype=np.int64)
    last = None
    fallback = first_nonempty(s_beg, s_end)
    for j in range(r_end.size):
        if r_beg[j] < r_end[j] and int(r_end[j]) in partner:
            last = partner[int(r_end[j])]
        a[j] = fallback if last is None else last
    return a


def ta_csr(s_beg, s_end, r_beg, r_end):
    """TA as a CSR table: one entry per row, num = den = 1."""
    a = ta_alignment(s_beg, s_end, r_beg, r_end)
    n = a.size
    return (np.arange(n + 1, dtype=np.int64), a.copy(),
            np.ones(n, dtype=np.int64), np.ones(n, dtype=np.int64))


def overlap_csr(s_beg, s_end, r_beg, r_end):
    """Overlap-weighted span alignment as a CSR table.

    Row j lists, in ascending order, every sender token i with o_ji > 0,
    storing col = i and num = o_ji; den_j = sum of the row's num.  Rows with no
    overlap hold the single TA entry (col = a(j), num = den = 1).
    """
    s_beg, s_end, r_beg, r_end = map(_as_int, (s_beg, s_end, r_beg, r_end))
    a_ta = ta_alignment(s_beg, s_end, r_beg, r_end)
    row_ptr = [0]
    col, num, den = [], [], []
    for j in range(r_end.size):
        o = np.minimum(s_end, r_end[j]) - np.maximum(s_beg, r_beg[j])
        idx = np.nonzero(o > 0)[0]
        if idx.size == 0:
            col.append(int(a_ta[j]))
            num.append(1)
            den.append(1)
        else:
            col.extend(int(i) for i in idx)
            num.extend(int(v) for v in o[idx])
            den.append(int(o[idx].sum()))
        row_ptr.append(len(col))
    return (np.asarray(row_ptr, dtype=np.int64), np.asarray(col, dtype=np.int64),
            np.asarray(num, dtype=np.int64), np.asarray(den, dtype=np.int64))


MODES = {"overlap": overlap_csr, "ta": ta_csr}


def build_alignment(s_beg, s_end, r_beg, r_end, mode: str = "overlap"):
    """One sequence: CSR table in the requested mode ("overlap" or "ta")."""
    return MODES[mode](s_beg, s_end, r_beg, r_end)


def build_alignment_batched(s_cu, r_cu, s_beg, s_end, r_beg, r_end,
                            mode: str = "overlap"):
    """Several independent sequences concatenated.

    s_cu / r_cu are [B+1] prefix sums of the per-sequence token counts.  Rows
    of sequence b follow those of sequence b-1; col stays local to the
    sequence (0-based within sequence b); row_ptr is global.
    """
    s_cu, r_cu = _as_int(s_cu), _as_int(r_cu)
    rp_all, col_all, num_all, den_all = [np.zeros(1, dtype=np.int64)], [], [], []
    base = 0
    for b in range(s_cu.size - 1):
        ss, se = s_cu[b], s_cu[b + 1]
        rs, re_ = r_cu[b], r_cu[b + 1]
        rp, col, num, den = build_alignment(s_beg[ss:se], s_end[ss:se],
                                            r_beg[rs:re_], r_end[rs:re_], mode)
        rp_all.append(rp[1:] + base)
        base += int(rp[-1])
        col_all.append(col)
        num_all.append(num)
        den_all.append(den)
    cat = lambda xs: (np.concatenate(xs) if xs else np.zeros(0, dtype=np.int64))  # noqa: E731
    return cat(rp_all), cat(col_all), cat(num_all), cat(den_all)


def same_index_alignment(s_beg, s_end, r_beg, r_end) -> np.ndarray:
    """Same-index pairing, the baseline the token-position mismatch of App. B.1
    is compared against: counting nonempty tokens from one, the k-th nonempty
    receiver token takes the min(k, n_S)-th nonempty sender token, so receiver
    positions past the sender sequence reuse its last token.  Returned as
    0-based indices into the full sender token list (int64 [T_r]); an empty
    receiver token takes the entry of the nonempty token before it (or the
    first one), which the mismatch never reads.  With no nonempty sender
    token every entry is 0."""
    s_beg, s_end, r_beg, r_end = map(_as_int, (s_beg, s_end, r_beg, r_end))
    s_ne = np.nonzero(s_beg < s_end)[0]
    a = np.zeros(r_end.size, dtype=np.int64)
    if s_ne.size == 0:
        return a
    k = 0  # nonempty receiver tokens seen so far
    cur = int(s_ne[0])
    for j in range(r_end.size):
        if r_beg[j] < r_end[j]:
            k += 1
            cur = int(s_ne[min(k, s_ne.size) - 1])
        a[j] = cur
    return a


def position_mismatch(s_beg, s_end, r_beg, r_end, a) -> float:
    """Token-position mismatch m_d of App. B.1, in characters: the mean over
    the nonempty receiver tokens j of |e^S_a(j) - e^R_j|, where e are the
    character end offsets and a(j) the sender index assigned to receiver token
    j (ta_alignment or same_index_alignment).  0 when no receiver token is
    nonempty.  A diagnostic of the alignment; the transfer never uses it."""
    s_beg, s_end, r_beg, r_end, a = map(_as_int, (s_beg, s_end, r_beg, r_end, a))
    J = np.nonzero(r_beg < r_end)[0]
    if J.size == 0:
        return 0.0
    return float(np.mean(np.abs(s_end[a[J]] - r_end[J])))
