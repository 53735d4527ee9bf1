"""mtp_q_count_noalloc (the bigram count on the library's fixed scratch, for
callers that cannot allocate) against mtp_q_count with a caller workspace:
the counts and input-error tallies must be identical, on two calls in a row
with the second corpus smaller than the first, and sizes beyond the fixed
scratch are refused before anything is launched."""
import numpy as np
import pytest

from gpu_common import log
from paper_2410_13839_amd.workloads import CORPORA, EOS_ID, VOCAB, CorpusSpec, make_corpus

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _both(tokens, offsets, V, eos, flags):
    from paper_2410_13839_amd.binding import mtp_q_count, mtp_q_count_noalloc, mtp_q_workspace_size
    st = torch.cuda.current_stream()
    t = torch.from_numpy(np.ascontiguousarray(tokens, np.int32)).cuda()
    o = torch.from_numpy(np.ascontiguousarray(offsets, np.int64)).cuda()
    n_tok, n_seq = int(t.numel()), int(o.numel() - 1)
    out = []
    for noalloc in (False, True):
        counts = torch.zeros((V, V), dtype=torch.int32, device="cuda")
        status = torch.zeros(3, dtype=torch.int64, device="cuda")
        if noalloc:
            mtp_q_count_noalloc(t.data_ptr(), n_tok, o.data_ptr(), n_seq, V, eos, flags, counts.data_ptr(),
                                status.data_ptr(), st.cuda_stream)
        else:
            ws_bytes = mtp_q_workspace_size(n_tok, n_seq, V)
            ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
            mtp_q_count(t.data_ptr(), n_tok, o.data_ptr(), n_seq, V, eos, flags, counts.data_ptr(),
                        status.data_ptr(), ws.data_ptr(), ws_bytes, st.cuda_stream)
        torch.cuda.synchronize()
        out.append((counts.cpu().numpy().view(np.uint32), status.cpu().numpy()))
    return out


def test_noalloc_count_equals_workspace_count_twice_second_smaller():
    from paper_2410_13839_amd.binding import MTP_Q_COUNT_EOS
    big = make_corpus(CorpusSpec("noalloc_big", 20000, 297.0, 13, 1750, seed=71))     # ~5.9 M tokens
    small = make_corpus(CORPORA["small"])
    for name, cp, V, eos, flags in (("big", big, VOCAB, EOS_ID, MTP_Q_COUNT_EOS), ("small", small, VOCAB, EOS_ID, 0)):
        log(f"noalloc: {name} corpus, {cp.tokens.size} tokens, {cp.offsets.size - 1} utterances")
        (c_ws, s_ws), (c_na, s_na) = _both(cp.tokens, cp.offsets, V, eos, flags)
        assert np.array_equal(c_ws, c_na), name
        assert np.array_equal(s_ws, s_na), name
        assert int(c_na.sum(dtype=np.uint64)) > 0


def test_noalloc_count_refuses_sizes_beyond_its_scratch():
    from paper_2410_13839_amd.binding import (MTP_ENOMEM, MTP_Q_NOALLOC_SCRATCH_BYTES, MTPError,
                                              mtp_q_count_noalloc, mtp_q_workspace_size)
    n_tok = 12_000_000
    assert mtp_q_workspace_size(n_tok, n_tok // 300, VOCAB) > MTP_Q_NOALLOC_SCRATCH_BYTES
    # valid device pointers of the right sizes: only the scratch limit refuses the call
    t = torch.zeros(n_tok, dtype=torch.int32, device="cuda")
    o = torch.zeros(n_tok // 300 + 1, dtype=torch.int64, device="cuda")
    counts = torch.zeros((VOCAB, VOCAB), dtype=torch.int32, device="cuda")
    status = torch.zeros(3, dtype=torch.int64, device="cuda")
    with pytest.raises(MTPError) as e:
        mtp_q_count_noalloc(t.data_ptr(), n_tok, o.data_ptr(), n_tok // 300, VOCAB, EOS_ID, 0, counts.data_ptr(),
                            status.data_ptr(), torch.cuda.current_stream().cuda_stream)
    assert e.value.code == MTP_ENOMEM
    torch.cuda.synchronize()
    assert int(counts.abs().sum()) == 0 and status.cpu().tolist() == [0, 0, 0]
