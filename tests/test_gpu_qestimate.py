"""GPU parity of the transition-table estimation (Sec. 3.3: Q derived from
the corpus).  Bigram counts and the input-error tallies must equal the
oracle's exactly; log Q is evaluated in double on both sides and rounded to
float32, so it must agree to within one float32 ulp (the two libraries' double
logarithms may differ in the last bit) with identical -inf entries."""
import numpy as np
import pytest

from gpu_common import log
from oracle.qestimate import bigram_counts, log_q
from paper_2410_13839_amd.workloads import CORPORA, EOS_ID, VOCAB, make_corpus

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _gpu(tokens, offsets, V, eos, count_eos, alpha):
    from paper_2410_13839_amd.binding import estimate_logq
    t = torch.from_numpy(np.ascontiguousarray(tokens, np.int32)).cuda()
    o = torch.from_numpy(np.ascontiguousarray(offsets, np.int64)).cuda()
    counts, lq, status = estimate_logq(t, o, V, eos, count_eos, alpha)
    torch.cuda.synchronize()
    return counts.cpu().numpy().view(np.uint32), lq.cpu().numpy(), status.cpu().numpy()


def _ulp_distance(a, b):
    ia = a.view(np.int32).astype(np.int64)
    ib = b.view(np.int32).astype(np.int64)
    ia = np.where(ia < 0, -(ia & 0x7FFFFFFF), ia)
    ib = np.where(ib < 0, -(ib & 0x7FFFFFFF), ib)
    return np.abs(ia - ib)


def _check(tokens, offsets, V, eos, count_eos, alpha):
    C, lq, status = _gpu(tokens, offsets, V, eos, count_eos, alpha)
    rC, bp, bs = bigram_counts(tokens, offsets, V, eos, count_eos)
    assert np.array_equal(C, rC)
    assert status.tolist() == [bp, bs, 0]
    rlq = log_q(rC, alpha)
    inf = np.isneginf(rlq)
    assert np.array_equal(np.isneginf(lq), inf)
    d = _ulp_distance(lq[~inf], rlq[~inf])
    assert d.max(initial=0) <= 1, d.max()
    return C, lq, status


def _ragged(rng, n_seqs, V, max_len, bad):
    lens = rng.integers(0, max_len, size=n_seqs)
    lens[:4] = [0, 1, 2, 0]
    lens[-1] = 50        # skipped when `bad`: frees more tokens than the 3 that utterance 5 then overlaps
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    toks = rng.integers(0, V, size=int(offs[-1])).astype(np.int32)
    if bad:
        toks[rng.integers(0, len(toks), size=7)] = rng.choice([-1, V, 1 << 20], size=7)
        offs[6] = offs[7] + 3                     # utterance 5 decreasing, 6 also
        offs[-1] = offs[-1] + 5                   # the last one runs past the tokens
    return toks, offs


@pytest.mark.parametrize("count_eos", [False, True])
@pytest.mark.parametrize("bad", [False, True])
@pytest.mark.parametrize("V,alpha", [(33, 0.0), (33, 1.0), (VOCAB, 0.5)])
def test_ragged_corpora_exact(count_eos, bad, V, alpha):
    rng = np.random.default_rng(10 * V + 2 * count_eos + bad)
    toks, offs = _ragged(rng, 700, V - 1, 90, bad)
    _, _, status = _check(toks, offs, V, V - 1, count_eos, alpha)
    if bad:
        assert status[0] > 0 and status[1] >= 2


@pytest.mark.parametrize("case", ["wide_vocab", "long_utterances", "many_utterances"])
def test_every_counting_path(case):
    """The count paths: a vocabulary with more than 64 key buckets (keys
    written one by one), utterance ranges whose spans exceed the LDS bitmap
    (per-utterance walk), and more than a million utterances (offsets read
    from memory)."""
    rng = np.random.default_rng({"wide_vocab": 1, "long_utterances": 2, "many_utterances": 3}[case])
    if case == "wide_vocab":
        V = 2000
        lens = rng.integers(0, 300, size=900)
    elif case == "long_utterances":
        V = VOCAB
        lens = np.array([70000, 3, 0, 90001, 5, 66000])
    else:
        V = 64
        lens = rng.integers(0, 3, size=1_050_000)
    offs = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    toks = rng.integers(0, V - 1, size=int(offs[-1])).astype(np.int32)
    for count_eos in (False, True):
        _check(toks, offs, V, V - 1, count_eos, 1.0)


def test_empty_corpora():
    for toks, offs in ((np.zeros(0, np.int32), np.zeros(1, np.int64)),
                       (np.zeros(0, np.int32), np.zeros(4, np.int64)),
                       (np.array([3], np.int32), np.array([0, 0, 1, 1]))):
        for count_eos in (False, True):
            C, lq, status = _check(toks, offs, 9, 8, count_eos, 1.0)
            assert C.sum() == (1 if (count_eos and len(toks)) else 0)


def test_counts_accumulate_across_calls():
    """Two calls over the two halves of a corpus add up to one call over all of it."""
    from paper_2410_13839_amd.binding import MTP_Q_COUNT_EOS, mtp_q_count, mtp_q_workspace_size
    cp = make_corpus(CORPORA["small"])
    h = len(cp.offsets) // 2
    t = torch.from_numpy(cp.tokens).cuda()
    counts = torch.zeros((VOCAB, VOCAB), dtype=torch.int32, device="cuda")
    status = torch.zeros(3, dtype=torch.int64, device="cuda")
    nb = mtp_q_workspace_size(t.numel(), len(cp.offsets), VOCAB)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    st = torch.cuda.current_stream()
    for part in (cp.offsets[:h + 1], cp.offsets[h:]):
        o = torch.from_numpy(np.ascontiguousarray(part)).cuda()
        mtp_q_count(t.data_ptr(), t.numel(), o.data_ptr(), o.numel() - 1, VOCAB, EOS_ID, MTP_Q_COUNT_EOS,
                    counts.data_ptr(), status.data_ptr(), ws.data_ptr(), nb, st.cuda_stream)
    torch.cuda.synchronize()
    rC, _, _ = bigram_counts(cp.tokens, cp.offsets, VOCAB, EOS_ID, True)
    assert np.array_equal(counts.cpu().numpy().view(np.uint32), rC)
    assert status.cpu().tolist() == [0, 0, 0]


def test_overlapping_utterances_beyond_the_token_count_are_refused():
    """offsets [0, 8, 0, 8] over 8 tokens: utterances 0 and 2 are the same
    range (16 pairs with the EOS pairs, more than the 8 tokens), utterance 1
    runs backwards.  Nothing is counted; status = [0, 1, 1]."""
    toks = np.arange(8, dtype=np.int32)
    C, lq, status = _gpu(toks, np.array([0, 8, 0, 8], np.int64), 9, 8, True, 1.0)
    assert status.tolist() == [0, 1, 1]
    assert C.sum() == 0
    assert np.all(lq == np.float32(-np.log(9.0)))


def test_libritts_scale_corpus_exact():
    """The 354,780-utterance, ~105 M-token corpus (the benchmark's input):
    every count exact, log Q within one ulp."""
    log("q estimation: generating the corpus")
    cp = make_corpus(CORPORA["libritts_train"])
    log(f"q estimation: {cp.tokens.size} tokens, running")
    C, lq, status = _check(cp.tokens, cp.offsets, VOCAB, EOS_ID, True, 1.0)
    assert status.tolist() == [0, 0, 0]
    assert int(C.sum(dtype=np.int64)) == cp.tokens.size
