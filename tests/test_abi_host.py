"""Host-side checks of the C-ABI library that need no GPU: it loads, exports
every function the header declares, and its host logic (the survivor draw)
agrees bit for bit with the oracle."""
import ctypes
import os

import numpy as np
import pytest

from oracle import coded as oc


def test_library_exports_every_header_function(lib):
    names = lib.header_functions()
    assert len(names) >= 14
    h = lib.lib()
    for name in names:
        assert hasattr(h, name), name
    assert "gfx950" in lib.version()


def test_status_strings(lib):
    for code, name in [(lib.CODED_OK, "CODED_OK"), (lib.CODED_ERR_ARG, "CODED_ERR_ARG"),
                       (lib.CODED_ERR_TOO_FEW, "CODED_ERR_TOO_FEW"), (lib.CODED_ERR_HIP, "CODED_ERR_HIP"),
                       (lib.CODED_ERR_UNSUPPORTED, "CODED_ERR_UNSUPPORTED")]:
        assert lib.status_string(code) == name


@pytest.mark.parametrize("n,k,seed", [(4, 2, 0), (4, 2, 17), (16, 12, 2), (32, 24, 3), (64, 48, 4), (20, 16, 5),
                                      (128, 100, 9), (5, 5, 1), (7, 1, 8)])
def test_survivor_draw_matches_oracle_bit_exact(lib, n, k, seed):
    for d in list(range(60)) + [2 ** 39 + 5, 123456789]:
        got, t = lib.coded_draw_survivors(n, k, seed, d)
        want, t_ref = oc.draw_survivors(n, k, seed, d)
        assert np.array_equal(got, want), (d, got, want)
        assert t == pytest.approx(t_ref, rel=1e-15)


def test_survivor_draw_shift_rate(lib):
    for d in range(20):
        got, t = lib.coded_draw_survivors(10, 5, 7, d, 2.0, 0.5)
        want, t_ref = oc.draw_survivors(10, 5, 7, d, 2.0, 0.5)
        assert np.array_equal(got, want)
        assert t == pytest.approx(t_ref, rel=1e-15)


def test_survivor_sets_match_oracle(lib):
    got, nxt = lib.coded_draw_survivor_sets(64, 48, 4, 500, min_parity=8)
    want, nxt_ref = oc.draw_survivor_sets(64, 48, 4, 500, min_parity=8)
    assert np.array_equal(got, want) and nxt == nxt_ref
    got, nxt = lib.coded_draw_survivor_sets(4, 2, 0, 6, min_parity=0)
    want, nxt_ref = oc.draw_survivor_sets(4, 2, 0, 6, min_parity=0)     # all C(4,2) sets
    assert np.array_equal(got, want) and nxt == nxt_ref
    got, nxt = lib.coded_draw_survivor_sets(6, 3, 5, 10, min_parity=2)  # all 9 + 1 qualifying sets
    want, nxt_ref = oc.draw_survivor_sets(6, 3, 5, 10, min_parity=2)
    assert np.array_equal(got, want) and nxt == nxt_ref


def test_survivor_set_batch_beyond_the_qualifying_sets_is_refused(lib):
    """More sets than exist fail at once (no endless drawing): C(4,2) = 6 sets,
    10 sets of (6,3) with at least 2 parity workers, 4 of (5,4) with its parity worker."""
    for n, k, batch, m_min in [(4, 2, 7, 0), (6, 3, 11, 2), (5, 4, 5, 1)]:
        with pytest.raises(lib.CodedError) as e:
            lib.coded_draw_survivor_sets(n, k, 0, batch, min_parity=m_min)
        assert e.value.status == lib.CODED_ERR_ARG
    # one set with all 16 parity workers exists, and it is found
    got, _ = lib.coded_draw_survivor_sets(20, 16, 0, 1, min_parity=4)
    assert np.sum(got[0] >= 16) == 4


def test_host_argument_errors(lib):
    with pytest.raises(lib.CodedError) as e:
        lib.coded_draw_survivors(4, 5, 0, 0)
    assert e.value.status == lib.CODED_ERR_ARG
    with pytest.raises(lib.CodedError):
        lib.coded_draw_survivors(4, 2, 0, 0, 1.0, 0.0)          # rate must be > 0
    with pytest.raises(lib.CodedError):
        lib.coded_draw_survivors(4, 2, 0, 2 ** 40)              # draw field is 40 bits
    with pytest.raises(lib.CodedError):
        lib.coded_draw_survivor_sets(8, 6, 0, 3, min_parity=3)  # at most n-k parity survivors
    h = lib.lib()
    # NULL pointers are rejected, not dereferenced
    assert h.coded_draw_survivors(4, 2, 0, 0, 1.0, 1.0, None, None) == lib.CODED_ERR_ARG
    assert h.coded_code_create(4, 2, None, 2, None, 0, ctypes.byref(ctypes.c_void_p())) == lib.CODED_ERR_ARG
    G = np.vstack([np.eye(2), np.ones((2, 2))])
    G[0, 1] = 0.5                                               # not systematic
    assert h.coded_code_create(4, 2, G.ctypes.data, 2, None, 0, ctypes.byref(ctypes.c_void_p())) == \
        lib.CODED_ERR_UNSUPPORTED
    assert h.coded_code_create(4, 2, np.eye(4, 2).ctypes.data, 3, None, 0, ctypes.byref(ctypes.c_void_p())) == \
        lib.CODED_ERR_ARG
    assert h.coded_encode(None, 0, None, 0, 0, 1, None, None) == lib.CODED_ERR_ARG
    assert h.coded_encode_worker_mm(None, 1, None, 0, 0, 1, None, None, 0, 1, None, 0, None, None) == \
        lib.CODED_ERR_ARG
    assert h.coded_decode(None, None, 0, None, 2, 0, 0, None, 1, None, None) == lib.CODED_ERR_ARG
    assert h.coded_straggler_matmul(None, 0, None, 0, 0, 1, None, None, 1, 1, 0, 0, 1.0, 1.0, 1.0, 0, None, 2, None,
                                    None, 1, None, None, None, None, None) == lib.CODED_ERR_ARG


@pytest.mark.parametrize("n,mu", [(10, 1.0), (100, 0.5), (1000, 1.0), (64, 2.0), (7, 0.1)])
def test_optimal_k_matches_oracle(lib, n, mu):
    from oracle import runtime as rt
    ks, ts, kb = lib.coded_optimal_k(n, mu)
    ks_ref, ts_ref, _ = rt.optimal_mds(n, mu)
    assert ks == pytest.approx(ks_ref, rel=1e-12) and ts == pytest.approx(ts_ref, rel=1e-12)
    assert kb == rt.best_integer_k(n, mu)


@pytest.mark.parametrize("n,q,cache,seed", [(2, 4, 2, 0), (5, 200, 70, 3), (8, 4000, 1000, 11), (3, 18, 6, 1),
                                            (16, 1600, 100, 7), (64, 640, 64, 2)])
def test_shuffle_planner_matches_oracle_bit_exact(lib, n, q, cache, seed):
    """The library's host planner (partition, caches, messages, cache rule) against
    the oracle's, over three iterations."""
    from oracle import shuffle as sh
    st = lib.Shuffle(n, q, cache, seed)
    ref = sh.initial_state(n, q, cache, seed)
    for _ in range(3):
        t, assign, sig = st.state()
        assert t == ref.t
        assert np.array_equal(assign, ref.assign)
        assert np.array_equal(sig, sh.signatures(ref.cached))
        coded_rows, terms = st.plan()
        p = sh.plan(ref)
        assert (coded_rows, terms) == (p.coded_rows, p.uncoded_rows)
        tb = st.tables()
        assert np.array_equal(tb["next_assign"], p.new_assign)
        for key in ("enc_off", "enc_rows", "term_worker", "term_msg"):
            assert np.array_equal(tb[key], getattr(p, key)), key
        st.commit()
        ref = sh.commit(ref, p)


def test_shuffle_argument_errors(lib):
    h = lib.lib()
    out = ctypes.c_void_p()
    assert h.coded_shuffle_create(0, 10, 5, 0, ctypes.byref(out)) == lib.CODED_ERR_ARG
    assert h.coded_shuffle_create(65, 650, 50, 0, ctypes.byref(out)) == lib.CODED_ERR_ARG
    assert h.coded_shuffle_create(3, 10, 5, 0, ctypes.byref(out)) == lib.CODED_ERR_SHAPE      # 3 does not divide 10
    assert h.coded_shuffle_create(2, 10, 4, 0, ctypes.byref(out)) == lib.CODED_ERR_ARG        # cache < q/n
    st = lib.Shuffle(2, 10, 6, 0)
    with pytest.raises(lib.CodedError):
        st.commit()                                          # nothing planned
    assert h.coded_shuffle_tables(st.handle, None, None, None, None, None) == lib.CODED_ERR_ARG
    assert h.coded_shuffle_plan(None, None, None) == lib.CODED_ERR_ARG


def test_noalloc_scratch_size_matches_header(lib):
    """The binding's copy of CODED_NOALLOC_SCRATCH_BYTES equals the header's definition."""
    import re
    text = open(lib.HEADER).read()
    m = re.search(r"#define\s+CODED_NOALLOC_SCRATCH_BYTES\s+\((\d+)u\s*<<\s*(\d+)\)", text)
    assert m, "CODED_NOALLOC_SCRATCH_BYTES not found in the header"
    assert lib.CODED_NOALLOC_SCRATCH_BYTES == int(m.group(1)) << int(m.group(2))


def test_planes_constant_matches_header(lib):
    import re
    m = re.search(r"#define\s+CODED_PLANES_LO_BF16\s+(\d+)", open(lib.HEADER).read())
    assert m and lib.CODED_PLANES_LO_BF16 == int(m.group(1))


def test_code_device_buffer_is_the_callers(lib):
    """coded_code_bytes sizes the caller's buffer (G in fp64, then P in fp32, each
    256-byte aligned); coded_code_create refuses a missing or short buffer before
    touching the device."""
    assert lib.coded_code_bytes(4, 2) == 256 + 256
    assert lib.coded_code_bytes(4, 4) == 256
    assert lib.coded_code_bytes(64, 48) == 64 * 48 * 8 + 16 * 48 * 4
    assert lib.coded_code_bytes(20, 16) == 2560 + 256
    assert lib.coded_code_bytes(5, 3) == 256 + 256                 # 120 B of G, 24 B of P
    h = lib.lib()
    G = np.vstack([np.eye(2), np.ones((2, 2))])
    out = ctypes.c_void_p()
    assert h.coded_code_create(4, 2, G.ctypes.data, 2, None, 512, ctypes.byref(out)) == lib.CODED_ERR_ARG
    assert "device_buf" in lib.last_error()
    with pytest.raises(lib.CodedError):
        lib.coded_code_bytes(2, 3)


def test_calibration_library_exports_its_probes():
    """The device-ceiling probes (calib/ceilings.hip) build into their own library with five entry points."""
    from paper_1512_02673_amd import build as _build
    if not os.path.exists(_build.CALIB_PATH):
        _build.build_calib()
    h = ctypes.CDLL(_build.CALIB_PATH)
    for name in ("calib_read", "calib_write", "calib_read_rows", "calib_rate", "calib_tile_pattern"):
        assert hasattr(h, name), name
