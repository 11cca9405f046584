"""CPU checks of the C ABI boundary: the library loads, exports every function the public
header declares, and rejects bad arguments with the documented status codes before making
any HIP call (so none of these touch a GPU)."""
import ctypes
import math
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rlcs.h")


@pytest.fixture(scope="module")
def lib():
    from paper_2608_17641_amd import _native
    from paper_2608_17641_amd.build import build
    build(force=False)
    return _native.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rlcs_[a-z_]+)\s*\(", text)))


def test_header_declares_the_expected_entry_points():
    names = declared_functions()
    for n in ("rlcs_gae", "rlcs_vtrace", "rlcs_retrace", "rlcs_td_lambda", "rlcs_discounted",
              "rlcs_elig_trace", "rlcs_episodic_prefix", "rlcs_affine_scan",
              "rlcs_workspace_size", "rlcs_status_string", "rlcs_version"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    from paper_2608_17641_amd import _native
    for name in declared_functions():
        assert hasattr(lib, name), f"librlcs.so does not export {name}"
        assert name in _native.PROTOTYPES, f"binding has no prototype for {name}"


def test_status_strings_and_version(lib):
    for code in range(5):
        assert lib.rlcs_status_string(code)
    assert b"unknown" in lib.rlcs_status_string(99)
    assert lib.rlcs_version() >= 100


def test_workspace_size(lib):
    fixed = 64 + 1024 * 64  # header, draw slots (one per row or column block)
    assert lib.rlcs_workspace_size(0, 5) == fixed
    # one 16-byte record per 1024-step tile of every row (the shortest split tile, float32)
    assert lib.rlcs_workspace_size(64, 4096) == fixed + 16 * 64 * 4
    assert lib.rlcs_workspace_size(1, 4097) == fixed + 16 * 5
    assert lib.rlcs_workspace_size(5000, 3) == fixed + 16 * 5000
    assert lib.rlcs_workspace_size(-1, 5) == fixed
    assert lib.rlcs_workspace_size(2 ** 40, 2 ** 23) == 0  # overflows


FAKE = ctypes.c_void_p(0x10000)       # never dereferenced: every call below fails validation
FAKE2 = ctypes.c_void_p(0x20000)
MISALIGNED = ctypes.c_void_p(0x10001)


def gae(lib, **kw):
    a = dict(r=FAKE, v=FAKE, term=None, trunc=None, bv=None, boot=None, adv=FAKE2, ret=None,
             N=4, T=8, gamma=0.99, lam=0.95, dtype=0, ws=None, ws_bytes=0, stream=None)
    a.update(kw)
    return lib.rlcs_gae(*a.values())


def test_gae_validation(lib):
    from paper_2608_17641_amd import _native as n
    assert gae(lib, N=-1) == n.RLCS_ERR_INVALID_ARG
    assert gae(lib, T=-3) == n.RLCS_ERR_INVALID_ARG
    assert gae(lib, dtype=7) == n.RLCS_ERR_DTYPE
    assert gae(lib, r=None) == n.RLCS_ERR_INVALID_ARG
    assert gae(lib, adv=None) == n.RLCS_ERR_INVALID_ARG
    assert gae(lib, trunc=FAKE) == n.RLCS_ERR_INVALID_ARG  # trunc without bv
    for bad in (-0.1, 1.5, math.nan):
        assert gae(lib, gamma=bad) == n.RLCS_ERR_INVALID_ARG
        assert gae(lib, lam=bad) == n.RLCS_ERR_INVALID_ARG
    assert gae(lib, r=MISALIGNED) == n.RLCS_ERR_INVALID_ARG
    assert gae(lib, N=2**40, T=2**30) == n.RLCS_ERR_INVALID_ARG  # N*T overflows
    assert gae(lib, N=1, T=2**30 + 1) == n.RLCS_ERR_INVALID_ARG  # row longer than supported
    # empty problems are no-ops, even with null pointers
    assert gae(lib, N=0, r=None, v=None, adv=None) == n.RLCS_OK
    assert gae(lib, T=0, r=None, v=None, adv=None) == n.RLCS_OK


def test_other_entry_points_validation(lib):
    from paper_2608_17641_amd import _native as n
    P = None
    # vtrace: clip thresholds must be > 0 (inf allowed), NaN rejected
    def vt(**kw):
        a = dict(r=FAKE, v=FAKE, lr=FAKE, term=P, trunc=P, bv=P, boot=P, vs=FAKE2, pg=P, N=2,
                 T=3, gamma=0.9, rho_bar=1.0, c_bar=1.0, dtype=0, ws=P, wsb=0, s=P)
        a.update(kw)
        return lib.rlcs_vtrace(*a.values())
    assert vt(rho_bar=0.0) == n.RLCS_ERR_INVALID_ARG
    assert vt(c_bar=-1.0) == n.RLCS_ERR_INVALID_ARG
    assert vt(c_bar=math.nan) == n.RLCS_ERR_INVALID_ARG
    assert vt(lr=None) == n.RLCS_ERR_INVALID_ARG
    assert vt(N=0, rho_bar=math.inf, c_bar=math.inf) == n.RLCS_OK
    assert lib.rlcs_retrace(FAKE, FAKE, None, FAKE, P, P, P, P, FAKE2, P, 2, 3, 0.9, 0.9, 1.0,
                            0, P, 0, P) == n.RLCS_ERR_INVALID_ARG  # eq missing
    assert lib.rlcs_td_lambda(FAKE, FAKE, P, FAKE, P, P, FAKE2, 2, 3, 0.9, 0.9, 0, P, 0, P) \
        == n.RLCS_ERR_INVALID_ARG  # trunc without bv
    assert lib.rlcs_discounted(FAKE, P, P, P, P, FAKE2, 2, 3, 1.01, 0, P, 0, P) \
        == n.RLCS_ERR_INVALID_ARG
    assert lib.rlcs_elig_trace(FAKE, P, P, None, 2, 3, 0.9, 0.9, 0, P, 0, P) \
        == n.RLCS_ERR_INVALID_ARG
    assert lib.rlcs_episodic_prefix(FAKE, P, P, FAKE2, 2, 3, 5, 0, P, 0, P) \
        == n.RLCS_ERR_INVALID_ARG  # bad boundary enum
    assert lib.rlcs_episodic_prefix(FAKE, P, P, FAKE2, 2, 3, 0, 9, P, 0, P) == n.RLCS_ERR_DTYPE
    assert lib.rlcs_affine_scan(FAKE, FAKE, P, FAKE2, 2, 3, 2, 0, P, 0, P) \
        == n.RLCS_ERR_INVALID_ARG  # bad direction
    assert lib.rlcs_affine_scan(FAKE, None, P, FAKE2, 2, 3, 0, 0, P, 0, P) \
        == n.RLCS_ERR_INVALID_ARG
    # bf16 data needs only 2-byte alignment; an odd address is still rejected
    assert lib.rlcs_affine_scan(MISALIGNED, FAKE, P, FAKE2, 2, 3, 0, 1, P, 0, P) \
        == n.RLCS_ERR_INVALID_ARG


def test_retrace_full_validation(lib):
    from paper_2608_17641_amd import _native as n
    P = None

    def rf(**kw):
        a = dict(r=FAKE, q=FAKE, pi=FAKE, act=FAKE, mu=FAKE, term=P, trunc=P, bv=P, boot=P,
                 delta=FAKE2, q_ret=P, N=2, T=3, A=4, gamma=0.9, lam=0.9, c_bar=1.0, dtype=0,
                 ws=P, wsb=0, s=P)
        a.update(kw)
        return lib.rlcs_retrace_full(*a.values())
    assert rf(A=0) == n.RLCS_ERR_INVALID_ARG
    assert rf(A=-5) == n.RLCS_ERR_INVALID_ARG
    assert rf(A=2 ** 31) == n.RLCS_ERR_INVALID_ARG  # actions are int32
    assert rf(N=2 ** 31, T=2 ** 20, A=2 ** 20) == n.RLCS_ERR_INVALID_ARG  # N*T*A overflows
    assert rf(act=None) == n.RLCS_ERR_INVALID_ARG
    assert rf(mu=None) == n.RLCS_ERR_INVALID_ARG
    assert rf(pi=None) == n.RLCS_ERR_INVALID_ARG
    assert rf(act=ctypes.c_void_p(0x10002)) == n.RLCS_ERR_INVALID_ARG  # int32 alignment
    assert rf(trunc=FAKE) == n.RLCS_ERR_INVALID_ARG
    assert rf(N=0, q=None) == n.RLCS_OK


def test_variant_override_range(lib):
    """The test-only variant hook (not in the public header) checks its range."""
    from paper_2608_17641_amd import _native as n
    assert lib.rlcs_testing_set_variant(5) == n.RLCS_ERR_INVALID_ARG
    assert lib.rlcs_testing_set_variant(4) == n.RLCS_OK
    assert lib.rlcs_testing_set_variant(-1) == n.RLCS_ERR_INVALID_ARG
    assert lib.rlcs_testing_set_variant(0) == n.RLCS_OK


def test_column_workspace_size(lib):
    # header and 1024 per-block counter slots, then one 16-byte record per column per
    # 32-step tile
    fixed = 64 + 1024 * 64
    assert lib.rlcs_workspace_size_columns(0, 5) == fixed
    assert lib.rlcs_workspace_size_columns(4096, 256) == fixed + 16 * 4096 * 8
    assert lib.rlcs_workspace_size_columns(3, 33) == fixed + 16 * 3 * 2
    assert lib.rlcs_workspace_size_columns(-1, 5) == 0
    assert lib.rlcs_workspace_size_columns(2 ** 62, 2 ** 30) == 0  # overflows


def gae_strided(lib, **kw):
    a = dict(r=FAKE, v=FAKE, term=None, trunc=None, bv=None, boot=None, adv=FAKE2, ret=None,
             N=4, T=8, sn=1, st=4, gamma=0.99, lam=0.95, dtype=0, ws=None, ws_bytes=0, stream=None)
    a.update(kw)
    return lib.rlcs_gae_strided(*a.values())


def test_strided_validation(lib):
    from paper_2608_17641_amd import _native as n
    assert gae_strided(lib, N=-1) == n.RLCS_ERR_INVALID_ARG
    assert gae_strided(lib, T=-1) == n.RLCS_ERR_INVALID_ARG
    assert gae_strided(lib, st=3) == n.RLCS_ERR_INVALID_ARG           # time-major ld < N
    assert gae_strided(lib, sn=7, st=1) == n.RLCS_ERR_INVALID_ARG     # row stride < T
    assert gae_strided(lib, sn=2, st=2) == n.RLCS_ERR_INVALID_ARG     # dimensions interleave
    assert gae_strided(lib, sn=0) == n.RLCS_ERR_INVALID_ARG
    assert gae_strided(lib, st=-4) == n.RLCS_ERR_INVALID_ARG
    assert gae_strided(lib, T=2 ** 30 + 1) == n.RLCS_ERR_INVALID_ARG
    assert gae_strided(lib, T=2 ** 30, st=2 ** 40) == n.RLCS_ERR_INVALID_ARG  # offsets overflow
    assert gae_strided(lib, dtype=5) == n.RLCS_ERR_DTYPE
    assert gae_strided(lib, r=None) == n.RLCS_ERR_INVALID_ARG
    assert gae_strided(lib, trunc=FAKE) == n.RLCS_ERR_INVALID_ARG
    assert gae_strided(lib, r=MISALIGNED) == n.RLCS_ERR_INVALID_ARG
    assert gae_strided(lib, gamma=1.5) == n.RLCS_ERR_INVALID_ARG
    assert gae_strided(lib, N=0) == n.RLCS_OK and gae_strided(lib, T=0) == n.RLCS_OK
    assert lib.rlcs_vtrace_strided(FAKE, FAKE, FAKE, None, None, None, None, FAKE2, None, 4, 8, 8,
                                   1, 0.99, 0.0, 1.0, 0, None, 0, None) == n.RLCS_ERR_INVALID_ARG
    assert lib.rlcs_retrace_strided(FAKE, FAKE, None, FAKE, None, None, None, None, FAKE2, None, 4,
                                    8, 1, 4, 0.99, 0.95, 1.0, 0, None, 0, None) == n.RLCS_ERR_INVALID_ARG
    assert lib.rlcs_td_lambda_strided(FAKE, FAKE, None, None, None, None, FAKE2, 4, 8, 1, 2, 0.99,
                                      0.95, 0, None, 0, None) == n.RLCS_ERR_INVALID_ARG
    assert lib.rlcs_discounted_strided(FAKE, None, FAKE, None, None, FAKE2, 4, 8, 1, 4, 0.99, 0,
                                       None, 0, None) == n.RLCS_ERR_INVALID_ARG
    assert lib.rlcs_elig_trace_strided(FAKE, None, None, FAKE2, 4, 8, 1, 4, 0.99, math.nan, 0,
                                       None, 0, None) == n.RLCS_ERR_INVALID_ARG
    assert lib.rlcs_episodic_prefix_strided(FAKE, None, None, FAKE2, 4, 8, 1, 4, 9, 0, None, 0,
                                            None) == n.RLCS_ERR_INVALID_ARG


def test_elig_trace_vec_validation(lib):
    from paper_2608_17641_amd import _native as n

    def call(**kw):
        a = dict(x=FAKE, term=None, trunc=None, z=FAKE2, N=4, T=8, F=3, gamma=0.99, lam=0.95,
                 dtype=0, ws=None, ws_bytes=0, stream=None)
        a.update(kw)
        return lib.rlcs_elig_trace_vec(*a.values())
    assert call(F=-1) == n.RLCS_ERR_INVALID_ARG
    assert call(N=-1) == n.RLCS_ERR_INVALID_ARG
    assert call(N=2 ** 40, T=2 ** 20, F=2 ** 10) == n.RLCS_ERR_INVALID_ARG  # N*T*F overflows
    assert call(dtype=3) == n.RLCS_ERR_DTYPE
    assert call(x=None) == n.RLCS_ERR_INVALID_ARG
    assert call(z=MISALIGNED) == n.RLCS_ERR_INVALID_ARG
    assert call(lam=-0.5) == n.RLCS_ERR_INVALID_ARG
    assert call(F=0) == n.RLCS_OK and call(N=0) == n.RLCS_OK


def test_gae_masked_validation(lib):
    from paper_2608_17641_amd import _native as n

    def call(**kw):
        a = dict(r=FAKE, v=FAKE, mask=None, term=None, trunc=None, bv=None, boot=None, adv=FAKE2,
                 ret=None, N=4, T=8, gamma=0.99, lam=0.95, normalize=0, eps=1e-8, dtype=0, ws=None,
                 ws_bytes=0, stream=None)
        a.update(kw)
        return lib.rlcs_gae_masked(*a.values())
    assert call(N=-1) == n.RLCS_ERR_INVALID_ARG
    assert call(dtype=4) == n.RLCS_ERR_DTYPE
    assert call(v=None) == n.RLCS_ERR_INVALID_ARG
    assert call(trunc=FAKE) == n.RLCS_ERR_INVALID_ARG
    assert call(normalize=2) == n.RLCS_ERR_INVALID_ARG
    assert call(normalize=1, eps=-1.0) == n.RLCS_ERR_INVALID_ARG
    assert call(normalize=1, eps=math.inf) == n.RLCS_ERR_INVALID_ARG
    assert call(normalize=1) == n.RLCS_ERR_WORKSPACE                 # no workspace
    assert call(normalize=1, ws=FAKE, ws_bytes=10) == n.RLCS_ERR_WORKSPACE
    assert call(lam=2.0) == n.RLCS_ERR_INVALID_ARG
    assert call(N=0) == n.RLCS_OK
    # header, 1024 one-pass moments records of 48 bytes, 64 copies of the statistics on their
    # own 128-byte lines, then the two-pass partials: one per row and one per block of 4096
    fixed = (64 + 48 * 1024 + 127) // 128 * 128 + 128 * 64
    assert lib.rlcs_workspace_size_masked(100, 7) == fixed + 32 * 100 + 32
    assert lib.rlcs_workspace_size_masked(4097, 7) == fixed + 32 * 4097 + 32 * 2
    assert lib.rlcs_workspace_size_masked(-1, 7) == 0


def test_noalloc_rejects_more_rows_than_its_workspace(lib):
    """rlcs_gae_masked_noalloc refuses calls of more rows than its built-in workspace holds,
    with or without whitening, before any HIP call."""
    from paper_2608_17641_amd import _native as n
    for norm in (0, 1):
        assert lib.rlcs_gae_masked_noalloc(FAKE, FAKE, None, None, None, None, None, FAKE2, None,
                                           65537, 4, 0.99, 0.95, norm, 1e-8, n.RLCS_F32,
                                           None) == n.RLCS_ERR_WORKSPACE
    # the argument checks of rlcs_gae_masked still apply below the limit
    assert lib.rlcs_gae_masked_noalloc(FAKE, FAKE, None, None, None, None, None, FAKE2, None,
                                       8, 4, 1.5, 0.95, 1, 1e-8, n.RLCS_F32,
                                       None) == n.RLCS_ERR_INVALID_ARG
    assert lib.rlcs_gae_masked_noalloc(FAKE, FAKE, None, None, None, None, None, FAKE2, None,
                                       8, 4, 0.99, 0.95, 1, 1e-8, 7, None) == n.RLCS_ERR_DTYPE
