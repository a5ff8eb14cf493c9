"""Pins for the alignment oracle: the paper's worked example, brute force at
character level, a closed form and invariants.  CPU only."""

import json
import os

import numpy as np
import pytest

from oracle import alignment as al
from paper_2609_32259_amd import synth


def _spans_from_ends(ends):
    ends = np.asarray(ends, dtype=np.int64)
    return np.concatenate([[0], ends[:-1]]), ends


@pytest.fixture(scope="module")
def example(golden_dir):
    with open(os.path.join(golden_dir, "ta_worked_example.json")) as f:
        return json.load(f)


def _sides(example, src, dst):
    sb, se = _spans_from_ends(example[src]["end"])
    rb, re_ = _spans_from_ends(example[dst]["end"])
    return sb, se, rb, re_


def test_worked_example_token_texts(example):
    # The end offsets printed in the paper are those of the printed tokens.
    for side in ("qwen3", "ministral3"):
        toks = example[side]["tokens"]
        assert "".join(toks) == example["text"]
        assert list(np.cumsum([len(t) for t in toks])) == example[side]["end"]


@pytest.mark.parametrize("src,dst,key", [("qwen3", "ministral3", "qwen3_to_ministral3"),
                                         ("ministral3", "qwen3", "ministral3_to_qwen3")])
def test_ta_worked_example(example, src, dst, key):
    a = al.ta_alignment(*_sides(example, src, dst))
    assert a.tolist() == example["expected_ta"][key]


def test_ta_worked_example_stated_outcomes(example):
    # Qwen3 -> Ministral-3: receiver ends 9 and 12 reuse the sender state ending at 3.
    sb, se, rb, re_ = _sides(example, "qwen3", "ministral3")
    a = al.ta_alignment(sb, se, rb, re_)
    for j, e in enumerate(re_):
        if e in (9, 12):
            assert se[a[j]] == 3
    # Ministral-3 -> Qwen3: the receiver token ending at 16 uses the sender state ending at 16.
    sb, se, rb, re_ = _sides(example, "ministral3", "qwen3")
    a = al.ta_alignment(sb, se, rb, re_)
    j16 = int(np.nonzero(re_ == 16)[0][0])
    assert se[a[j16]] == 16


@pytest.mark.parametrize("src,dst,key", [("qwen3", "ministral3", "qwen3_to_ministral3"),
                                         ("ministral3", "qwen3", "ministral3_to_qwen3")])
def test_overlap_worked_example(example, src, dst, key):
    rp, col, num, den = al.overlap_csr(*_sides(example, src, dst))
    exp = example["expected_overlap"][key]
    assert rp.tolist() == exp["row_ptr"]
    assert col.tolist() == exp["col"]
    assert num.tolist() == exp["num"]
    assert den.tolist() == exp["den"]


# --- brute force ------------------------------------------------------------

def brute_overlap(s_beg, s_end, r_beg, r_end):
    """Character-level membership: count, for every character of receiver
    token j, which nonempty sender tokens contain it."""
    a_ta = brute_ta(s_beg, s_end, r_beg, r_end)
    rows = []
    for j in range(len(r_beg)):
        counts = {}
        for ch in range(int(r_beg[j]), int(r_end[j])):
            for i in range(len(s_beg)):
                if int(s_beg[i]) <= ch < int(s_end[i]):
                    counts[i] = counts.get(i, 0) + 1
        if counts:
            rows.append(sorted(counts.items()))
        else:
            rows.append([(int(a_ta[j]), 1)])
    rp = [0]
    col, num, den = [], [], []
    for r in rows:
        col += [i for i, _ in r]
        num += [n for _, n in r]
        den.append(sum(n for _, n in r))
        rp.append(len(col))
    return rp, col, num, den


def brute_ta(s_beg, s_end, r_beg, r_end):
    """Backward search per receiver token for the latest receiver token at or
    before it whose end is a shared nonempty boundary."""
    s_ends = [(i, int(e)) for i, (b, e) in enumerate(zip(s_beg, s_end)) if b < e]
    first = s_ends[0][0] if s_ends else 0
    out = []
    for j in range(len(r_beg)):
        pick = None
        for jj in range(j, -1, -1):
            if r_beg[jj] < r_end[jj]:
                cands = [i for i, e in s_ends if e == int(r_end[jj])]
                if cands:
                    pick = max(cands)
                    break
        out.append(first if pick is None else pick)
    return out


def _small_cases():
    cases = []
    for seed in range(6):
        rng = np.random.default_rng(seed)
        n = int(rng.integers(1, 60))
        cases.append(("clean", synth.segment_chars(rng, n, 1, 6) + synth.segment_chars(rng, n, 1, 8)))
        m = int(rng.integers(1, 60))
        cases.append(("messy", synth.segment_messy(rng, n, 1, 5, p_empty=0.2, p_gap=0.2)
                      + synth.segment_messy(rng, m, 1, 7, p_empty=0.2, p_gap=0.2, p_dup_end=0.2)))
    return cases


@pytest.mark.parametrize("kind,case", _small_cases())
def test_overlap_matches_brute_force(kind, case):
    s_beg, s_end, r_beg, r_end = case
    rp, col, num, den = al.overlap_csr(s_beg, s_end, r_beg, r_end)
    brp, bcol, bnum, bden = brute_overlap(s_beg, s_end, r_beg, r_end)
    assert rp.tolist() == brp and col.tolist() == bcol
    assert num.tolist() == bnum and den.tolist() == bden


@pytest.mark.parametrize("kind,case", _small_cases())
def test_ta_matches_brute_force(kind, case):
    s_beg, s_end, r_beg, r_end = case
    assert al.ta_alignment(s_beg, s_end, r_beg, r_end).tolist() == brute_ta(s_beg, s_end, r_beg, r_end)


def test_identical_tokenizations_give_identity():
    rng = np.random.default_rng(3)
    b, e = synth.segment_chars(rng, 500, 1, 7)
    assert al.ta_alignment(b, e, b, e).tolist() == list(range(b.size))
    rp, col, num, den = al.overlap_csr(b, e, b, e)
    assert rp.tolist() == list(range(b.size + 1))
    assert col.tolist() == list(range(b.size))
    assert np.array_equal(num, den) and np.array_equal(den, e - b)


@pytest.mark.parametrize("seed", range(4))
def test_overlap_closed_form_and_invariants(seed):
    """Two tilings of the same character range: the number of entries equals
    the number of distinct token boundaries; every row's weights sum to the
    receiver token's length; spans tile the range (every sender token is read);
    rows are contiguous, ascending, and consecutive rows share at most one
    sender token."""
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(200, 2000))
    sb, se = synth.segment_chars(rng, n, 1, 7)
    rb, re_ = synth.segment_chars(rng, n, 1, 8)
    rp, col, num, den = al.overlap_csr(sb, se, rb, re_)
    assert col.size == len(set(se.tolist()) | set(re_.tolist()))
    assert np.array_equal(np.add.reduceat(num, rp[:-1]), den)
    assert np.array_equal(den, re_ - rb)
    assert set(col.tolist()) == set(range(sb.size))
    for j in range(rb.size):
        c = col[rp[j]:rp[j + 1]]
        assert np.all(np.diff(c) == 1)
        if j:
            prev = col[rp[j - 1]:rp[j]]
            assert c[0] >= prev[-1] and len(set(c) & set(prev)) <= 1


def test_overlap_fallback_rows():
    # Receiver tokens beyond the sender's text and empty receiver tokens fall
    # back to their TA entry with weight 1.
    sb, se = np.array([0, 3]), np.array([3, 5])
    rb, re_ = np.array([0, 2, 5, 6, 6]), np.array([2, 5, 6, 6, 9])
    rp, col, num, den = al.overlap_csr(sb, se, rb, re_)
    assert rp.tolist() == [0, 1, 3, 4, 5, 6]
    assert col.tolist() == [0, 0, 1, 1, 1, 1]
    assert num.tolist() == [2, 1, 2, 1, 1, 1]
    assert den.tolist() == [2, 3, 1, 1, 1]


def test_ta_all_empty_sender_and_leading_rows():
    sb, se = np.array([0, 0, 1]), np.array([0, 1, 3])
    rb, re_ = np.array([0, 2]), np.array([2, 3])
    # first nonempty sender token is 1; no shared end at 2; end 3 matches sender 2
    assert al.ta_alignment(sb, se, rb, re_).tolist() == [1, 2]
    assert al.ta_alignment(np.array([1, 2]), np.array([1, 2]), rb, re_).tolist() == [0, 0]


def test_batched_matches_per_sequence():
    cfg = synth.TINY_F32
    seg = synth.make_segmentation(cfg, seed=5, batch=3)
    for mode in ("overlap", "ta"):
        rp, col, num, den = al.build_alignment_batched(seg.s_cu, seg.r_cu, seg.s_beg, seg.s_end,
                                                       seg.r_beg, seg.r_end, mode)
        for b in range(3):
            r0, r1 = seg.r_cu[b], seg.r_cu[b + 1]
            prp, pcol, pnum, pden = al.build_alignment(*seg.seq(b), mode)
            assert np.array_equal(rp[r0:r1 + 1] - rp[r0], prp)
            assert np.array_equal(col[rp[r0]:rp[r1]], pcol)
            assert np.array_equal(num[rp[r0]:rp[r1]], pnum)
            assert np.array_equal(den[r0:r1], pden)


# --- token-position mismatch (App. B.1) ---------------------------------------
# Hand-worked on the Sec. 3.1 example.  Qwen3 ends {3, 16, 23, 24}, Ministral-3
# ends {3, 9, 12, 16, 23, 24}.
#   Qwen3 -> Ministral-3, TA a = [0, 0, 0, 1, 2, 3]: sender ends [3, 3, 3, 16, 23, 24]
#     against [3, 9, 12, 16, 23, 24] -> |diffs| [0, 6, 9, 0, 0, 0] -> 15 / 6 = 2.5.
#   Same-index a = [0, 1, 2, 3, 3, 3]: ends [3, 16, 23, 24, 24, 24] -> [0, 7, 11, 8, 1, 0]
#     -> 27 / 6 = 4.5.
#   Ministral-3 -> Qwen3, TA a = [0, 3, 4, 5]: ends [3, 16, 23, 24] -> 0.
#   Same-index a = [0, 1, 2, 3]: ends [3, 9, 12, 16] against [3, 16, 23, 24] -> 26 / 4 = 6.5.
@pytest.mark.parametrize("src,dst,ta_m,same_a,same_m", [
    ("qwen3", "ministral3", 2.5, [0, 1, 2, 3, 3, 3], 4.5),
    ("ministral3", "qwen3", 0.0, [0, 1, 2, 3], 6.5)])
def test_position_mismatch_worked_example(example, src, dst, ta_m, same_a, same_m):
    sb, se, rb, re_ = _sides(example, src, dst)
    a_ta = al.ta_alignment(sb, se, rb, re_)
    assert al.position_mismatch(sb, se, rb, re_, a_ta) == ta_m
    a_si = al.same_index_alignment(sb, se, rb, re_)
    assert a_si.tolist() == same_a
    assert al.position_mismatch(sb, se, rb, re_, a_si) == same_m


def test_position_mismatch_skips_empty_receiver_tokens(example):
    # An empty receiver token inserted at character 9 is not in J_d: the mean is
    # still over the six nonempty tokens, and same-index counting skips it.
    sb, se, rb, re_ = _sides(example, "qwen3", "ministral3")
    rb2 = np.insert(rb, 2, 9)
    re2 = np.insert(re_, 2, 9)
    a_ta = al.ta_alignment(sb, se, rb2, re2)
    assert al.position_mismatch(sb, se, rb2, re2, a_ta) == 2.5
    a_si = al.same_index_alignment(sb, se, rb2, re2)
    assert a_si.tolist() == [0, 1, 1, 2, 3, 3, 3]
    assert al.position_mismatch(sb, se, rb2, re2, a_si) == 4.5


def test_position_mismatch_identical_tokenizations_is_zero():
    rng = np.random.default_rng(3)
    sb, se = synth.segment_tokens(rng, 200, 1, 7)
    for a in (al.ta_alignment(sb, se, sb, se), al.same_index_alignment(sb, se, sb, se)):
        assert a.tolist() == list(range(200))
        assert al.position_mismatch(sb, se, sb, se, a) == 0.0


def test_position_mismatch_brute_force():
    # Against a direct loop over nonempty receiver tokens with 1-based counting.
    rng = np.random.default_rng(4)
    for _ in range(20):
        n = 300
        sb, se = synth.segment_messy(rng, n, 1, 6)
        rb, re_ = synth.segment_chars(rng, n, 1, 8)
        s_ne = [i for i in range(len(sb)) if sb[i] < se[i]]
        tot, cnt, k = 0, 0, 0
        for j in range(len(rb)):
            if rb[j] < re_[j]:
                k += 1
                i = s_ne[min(k, len(s_ne)) - 1] if s_ne else 0
                tot += abs(int(se[i]) - int(re_[j]))
                cnt += 1
        a = al.same_index_alignment(sb, se, rb, re_)
        assert al.position_mismatch(sb, se, rb, re_, a) == (tot / cnt if cnt else 0.0)
