"""Pins of the oracle's transition-table estimation (Sec. 3.3, Q derived from
the corpus): pair counts against a plain dictionary count, hand-worked
tables, the orientation (row = previous token), the invariants of the
counts and of the smoothed table, and consistency with the chain the corpus
was drawn from."""
import collections

import numpy as np
import pytest

from oracle.qestimate import bigram_counts, log_q
from paper_2410_13839_amd.workloads import CORPORA, EOS_ID, VOCAB, CorpusSpec, make_corpus, make_logq


def _dict_counts(tokens, offsets, V, eos, count_eos):
    c = collections.Counter()
    bad_pairs = bad_seqs = 0
    n = len(tokens)
    for u in range(len(offsets) - 1):
        s, e = int(offsets[u]), int(offsets[u + 1])
        if not (0 <= s <= e <= n):
            bad_seqs += 1
            continue
        seq = [int(t) for t in tokens[s:e]] + ([eos] if count_eos and e > s else [])
        for a, b in zip(seq, seq[1:]):
            if 0 <= a < V and 0 <= b < V:
                c[(a, b)] += 1
            else:
                bad_pairs += 1
    return c, bad_pairs, bad_seqs


def _ragged(rng, n_seqs, V, bad=False):
    lens = rng.integers(0, 12, size=n_seqs)
    lens[:3] = [0, 1, 2]
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    toks = rng.integers(0, V, size=int(offs[-1])).astype(np.int32)
    if bad:
        toks[rng.integers(0, len(toks), size=5)] = rng.choice([-3, V, V + 7], size=5)
        offs = offs.copy()
        offs[4] = offs[5] + 1                        # one decreasing pair of offsets
    return toks, offs


@pytest.mark.parametrize("count_eos", [False, True])
@pytest.mark.parametrize("bad", [False, True])
def test_counts_match_a_dictionary_count(count_eos, bad):
    rng = np.random.default_rng(3 + count_eos + 2 * bad)
    V = 17
    toks, offs = _ragged(rng, 60, V - 1, bad)
    C, bp, bs = bigram_counts(toks, offs, V, V - 1, count_eos)
    ref, rbp, rbs = _dict_counts(toks, offs, V, V - 1, count_eos)
    dense = np.zeros((V, V), np.uint32)
    for (a, b), n in ref.items():
        dense[a, b] = n
    assert np.array_equal(C, dense)
    assert (bp, bs) == (rbp, rbs)
    if bad:
        assert bp > 0 and bs > 0


def test_hand_worked_alternation():
    """One utterance 0 1 0 1 0 over V = 4: C(0,1) = C(1,0) = 2; with
    alpha = 1, Q(0,1) = 3/6, Q(0,0) = 1/6, Q(1,0) = 3/6; row 2 is uniform."""
    toks = np.array([0, 1, 0, 1, 0], np.int32)
    C, _, _ = bigram_counts(toks, np.array([0, 5]), 4, 3, False)
    assert C[0, 1] == 2 and C[1, 0] == 2 and C.sum() == 4
    lq = log_q(C, 1.0).astype(np.float64)
    assert np.allclose(np.exp(lq[0]), [1 / 6, 3 / 6, 1 / 6, 1 / 6], rtol=1e-6)
    assert np.allclose(np.exp(lq[1]), [3 / 6, 1 / 6, 1 / 6, 1 / 6], rtol=1e-6)
    assert np.allclose(np.exp(lq[2]), 0.25, rtol=1e-6)
    C2, _, _ = bigram_counts(toks, np.array([0, 5]), 4, 3, True)       # + (0, EOS)
    assert C2[0, 3] == 1 and C2.sum() == 5


def test_orientation_is_previous_to_next():
    C, _, _ = bigram_counts(np.array([5, 7], np.int32), np.array([0, 2]), 9, 8, False)
    assert C[5, 7] == 1 and C[7, 5] == 0 and C.sum() == 1


def test_no_pair_spans_two_utterances():
    toks = np.array([1, 2, 3, 4], np.int32)
    C, _, _ = bigram_counts(toks, np.array([0, 2, 2, 4]), 6, 5, False)
    assert C[1, 2] == 1 and C[3, 4] == 1 and C[2, 3] == 0 and C.sum() == 2


def test_count_invariants_on_the_small_corpus():
    cp = make_corpus(CORPORA["small"])
    lens = np.diff(cp.offsets)
    for count_eos in (False, True):
        C, bp, bs = bigram_counts(cp.tokens, cp.offsets, VOCAB, EOS_ID, count_eos)
        assert bp == 0 and bs == 0
        assert int(C.sum(dtype=np.int64)) == int(np.maximum(lens - 1, 0).sum()) + (int((lens > 0).sum()) if count_eos else 0)
        # row sums: how often a token is followed by anything
        follows = np.zeros(VOCAB, np.int64)
        for u in range(len(lens)):
            s, e = cp.offsets[u], cp.offsets[u + 1]
            np.add.at(follows, cp.tokens[s:e] if count_eos else cp.tokens[s:e - 1], 1)
        assert np.array_equal(C.sum(axis=1, dtype=np.int64), follows)
        assert C[:, EOS_ID].sum() == (int((lens > 0).sum()) if count_eos else 0)
        assert C[EOS_ID].sum() == 0


def test_smoothed_table_is_row_stochastic():
    cp = make_corpus(CORPORA["small"])
    C, _, _ = bigram_counts(cp.tokens, cp.offsets, VOCAB, EOS_ID, True)
    for alpha in (1.0, 0.25):
        lq = log_q(C, alpha)
        assert lq.dtype == np.float32 and np.all(np.isfinite(lq))
        assert np.allclose(np.exp(lq.astype(np.float64)).sum(axis=1), 1.0, atol=1e-5)
    lq0 = log_q(C, 0.0)
    assert np.array_equal(np.isneginf(lq0[C.sum(axis=1) > 0]), C[C.sum(axis=1) > 0] == 0)
    assert np.all(lq0[EOS_ID] == np.float32(-np.log(VOCAB)))       # empty row: uniform


def test_estimate_recovers_the_chain():
    """Counts of long chains drawn from a synthetic 32-code Q estimate Q:
    every row is within total variation 0.05 of the true row, while the
    transposed table is not (Q is far from symmetric)."""
    spec = CorpusSpec("lln", 64, 6000.0, 6000, 6000, seed=7)
    lq_true = make_logq(v=33, eos_id=32)
    cp = make_corpus(spec, lq_true, chains=64, n_codes=32)
    C, bp, _ = bigram_counts(cp.tokens, cp.offsets, 33, 32, False)
    assert bp == 0 and C.sum() == 64 * 5999
    q = np.exp(lq_true[:32, :32].astype(np.float64))
    q /= q.sum(axis=1, keepdims=True)
    est = np.exp(log_q(C, 0.0).astype(np.float64))[:32, :32]
    tv = 0.5 * np.abs(est - q).sum(axis=1)
    tv_t = 0.5 * np.abs(est - q.T / q.T.sum(axis=1, keepdims=True)).sum(axis=1)
    assert tv.max() < 0.05, tv.max()
    assert tv_t.min() > 0.2, tv_t.min()
