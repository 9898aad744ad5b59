"""Coded shuffling on the GPU (coded_shuffle_encode / coded_shuffle_decode)
against the oracle: the multicast rows and every worker's decoded rows are
fp32 sums and differences in a fixed order, so they compare bit for bit;
with integer-valued rows every decoded row is the data row exactly."""
import numpy as np
import pytest

import synth
from oracle import shuffle as sh
from tests.gpu_helpers import torch_mod

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    t = torch_mod()
    if not t.cuda.is_available():
        pytest.skip("no GPU")
    return t


def run_iteration(lib, torch, st, dA, r):
    coded_rows, terms = st.plan()
    tb = st.tables()
    dev = {k: torch.from_numpy(tb[k]).cuda() for k in ("enc_off", "enc_rows", "term_msg")}
    M = torch.full((max(coded_rows, 1), r), float("nan"), dtype=torch.float32, device="cuda")[:coded_rows]
    out = torch.full((max(terms, 1), r), float("nan"), dtype=torch.float32, device="cuda")[:terms]
    lib.coded_shuffle_encode(dA, dev["enc_off"], dev["enc_rows"], M)
    lib.coded_shuffle_decode(dA, M, dev["enc_off"], dev["enc_rows"], dev["term_msg"], out)
    torch.cuda.synchronize()
    return tb, M.cpu().numpy(), out.cpu().numpy()


@pytest.mark.parametrize("n,q,cache,r", [(8, 4000, 1000, 64), (5, 200, 70, 37), (16, 3200, 400, 256),
                                         (3, 18, 6, 5), (50, 5000, 500, 128)])
def test_shuffle_kernels_bit_exact(lib, torch, n, q, cache, r):
    A = synth.gaussian((q, r), 51, synth.STREAM_A)
    dA = torch.from_numpy(A).cuda()
    st = lib.Shuffle(n, q, cache, 9)
    ref = sh.initial_state(n, q, cache, 9)
    for _ in range(3):
        tb, M, out = run_iteration(lib, torch, st, dA, r)
        p = sh.plan(ref)
        assert np.array_equal(tb["enc_rows"], p.enc_rows)
        M_ref = sh.encode(A, p)
        assert np.array_equal(M, M_ref)
        assert np.array_equal(out, sh.decode(A, M_ref, p))
        st.commit()
        ref = sh.commit(ref, p)


def test_shuffle_integer_rows_decode_exactly(lib, torch):
    n, q, cache, r = 10, 2000, 400, 96
    A = synth.integers((q, r), 52, synth.STREAM_A, lo=-100, hi=100).astype(np.float32)
    dA = torch.from_numpy(A).cuda()
    st = lib.Shuffle(n, q, cache, 4)
    for _ in range(3):
        tb, M, out = run_iteration(lib, torch, st, dA, r)
        assert np.array_equal(out, A[tb["enc_rows"]])
        # every worker now holds its whole new set: cached rows plus decoded rows
        t, assign, sig = st.state()
        for i in range(n):
            have = set(np.nonzero((sig >> np.uint64(i)) & np.uint64(1))[0]) | set(tb["enc_rows"][tb["term_worker"] == i])
            assert set(np.nonzero(tb["next_assign"] == i)[0]) <= have
        st.commit()


def test_shuffle_bad_table_entries_give_nan_rows(lib, torch):
    """An entry out of range is caught before any load: its message and the terms
    decoded from it come out NaN, everything else is unaffected."""
    n, q, cache, r = 6, 600, 200, 32
    A = synth.gaussian((q, r), 53, synth.STREAM_A)
    dA = torch.from_numpy(A).cuda()
    st = lib.Shuffle(n, q, cache, 5)
    coded_rows, terms = st.plan()
    tb = st.tables()
    p = sh.plan(sh.initial_state(n, q, cache, 5))
    bad = int(np.argmax(np.diff(tb["enc_off"]) >= 2))      # a message with at least two terms
    rows = tb["enc_rows"].copy()
    rows[tb["enc_off"][bad]] = q + 5
    dev_off, dev_rows, dev_msg = (torch.from_numpy(x).cuda() for x in (tb["enc_off"], rows, tb["term_msg"]))
    M = torch.empty((coded_rows, r), dtype=torch.float32, device="cuda")
    out = torch.empty((terms, r), dtype=torch.float32, device="cuda")
    lib.coded_shuffle_encode(dA, dev_off, dev_rows, M)
    lib.coded_shuffle_decode(dA, M, dev_off, dev_rows, dev_msg, out)
    torch.cuda.synchronize()
    Mh, oh = M.cpu().numpy(), out.cpu().numpy()
    M_ref = sh.encode(A, p)
    assert np.all(np.isnan(Mh[bad]))
    keep = np.arange(coded_rows) != bad
    assert np.array_equal(Mh[keep], M_ref[keep])
    in_bad = tb["term_msg"] == bad
    assert np.all(np.isnan(oh[in_bad]))
    assert np.array_equal(oh[~in_bad], sh.decode(A, M_ref, p)[~in_bad])


def test_shuffle_nothing_to_send(lib, torch):
    """Caches holding every row: the plan has no messages and no terms (as the
    oracle's), both kernels accept the empty tables and enqueue nothing, and
    the next iteration plans the same way."""
    n, q, r = 4, 100, 64
    A = synth.gaussian((q, r), 52, synth.STREAM_A)
    dA = torch.from_numpy(A).cuda()
    st = lib.Shuffle(n, q, q, 3)
    ref = sh.initial_state(n, q, q, 3)
    for _ in range(2):
        tb, M, out = run_iteration(lib, torch, st, dA, r)
        p = sh.plan(ref)
        assert p.coded_rows == 0 and p.uncoded_rows == 0
        assert M.shape == (0, r) and out.shape == (0, r)
        assert np.array_equal(tb["enc_off"], p.enc_off) and np.array_equal(tb["next_assign"], p.new_assign)
        st.commit()
        ref = sh.commit(ref, p)
