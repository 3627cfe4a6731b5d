"""C-ABI checks that need no GPU: the library loads, exports every entry point
that include/bakron.h declares, and rejects invalid arguments on the host
before touching the device."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bakron.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bakron_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    import paper_2608_06291_amd as pk
    if not os.path.exists(pk.LIB_PATH):
        pytest.fail("libbakron.so is not built (run __graft_entry__.build())")
    return pk.load()


def test_header_declares_the_boundary():
    names = _declared()
    for n in ("bakron_factor", "bakron_solve", "bakron_solve_debug", "bakron_factors_free",
              "bakron_status_string"):
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    import paper_2608_06291_amd as pk
    for name in _declared():
        assert hasattr(lib, name), name
    assert set(_declared()) == set(pk.EXPORTED)


def test_status_strings(lib):
    import paper_2608_06291_amd as pk
    assert pk.status_string(0) == "BAKRON_OK"
    assert pk.status_string(2) == "BAKRON_ENOTSPD"
    assert pk.status_string(99) == "BAKRON_UNKNOWN"


def test_host_validation_needs_no_device(lib):
    """Null pointers / bad sizes / bad damping return EINVAL before any HIP call."""
    import paper_2608_06291_amd as pk
    h = ctypes.c_void_p(0)
    st = lib.bakron_factor(None, 16, None, 0, 0.01, None, ctypes.byref(h))
    assert st == pk.BAKRON_EINVAL and h.value is None
    assert b"invalid" in lib.bakron_last_error()
    st = lib.bakron_factor(ctypes.c_void_p(1), -3, None, 0, 0.01, None, ctypes.byref(h))
    assert st == pk.BAKRON_EINVAL
    st = lib.bakron_factor(ctypes.c_void_p(1), 16, None, 0, float("nan"), None, ctypes.byref(h))
    assert st == pk.BAKRON_EINVAL
    st = lib.bakron_factor(ctypes.c_void_p(1), 16, ctypes.c_void_p(1), 0, 0.01, None,
                           ctypes.byref(h))
    assert st == pk.BAKRON_EINVAL
    q = pk._lib._Quantizer(4, 1)
    assert lib.bakron_solve(ctypes.c_void_p(1), 4, 4, None, q, ctypes.c_void_p(1),
                            ctypes.c_void_p(1), None) == pk.BAKRON_EINVAL
    lib.bakron_factors_free(None)      # no-op


def test_binding_refuses_cpu_tensors():
    import torch
    import paper_2608_06291_amd as pk
    with pytest.raises(TypeError):
        pk.factor(torch.eye(4), None, 0.01)


def test_factor_construction_host_validation(lib):
    """The factor-construction calls answer workspace queries and reject bad
    arguments on the host, before any HIP call."""
    import paper_2608_06291_amd as pk
    one = ctypes.c_void_p(256)
    need = ctypes.c_size_t(0)
    # workspace query: size only, pointers unchecked; grows with the problem
    assert lib.bakron_gram(None, 1000, 200, None, 1.0, None, None, None,
                           ctypes.byref(need), None) == pk.BAKRON_OK
    small = need.value
    assert small > 0 and small % 256 == 0
    assert lib.bakron_gram(None, 100000, 1000, None, 1.0, None, None, None,
                           ctypes.byref(need), None) == pk.BAKRON_OK
    assert need.value > small
    # too small, unaligned, missing size, bad sizes
    need = ctypes.c_size_t(16)
    assert lib.bakron_gram(one, 1000, 200, None, 1.0, None, one, one, ctypes.byref(need),
                           None) == pk.BAKRON_EINVAL
    assert b"too small" in lib.bakron_last_error()
    need = ctypes.c_size_t(1 << 30)
    assert lib.bakron_gram(one, 1000, 200, None, 1.0, None, one, ctypes.c_void_p(258),
                           ctypes.byref(need), None) == pk.BAKRON_EINVAL
    assert lib.bakron_gram(one, 10, 20, None, 1.0, None, one, one, None, None) == pk.BAKRON_EINVAL
    assert lib.bakron_gram(one, -1, 20, None, 1.0, None, one, None, ctypes.byref(need),
                           None) == pk.BAKRON_EINVAL
    assert lib.bakron_gram(one, 10, (1 << 17) + 1, None, 1.0, None, one, None,
                           ctypes.byref(need), None) == pk.BAKRON_EINVAL
    assert lib.bakron_gram(None, 10, 20, None, 1.0, None, one, one, ctypes.byref(need),
                           None) == pk.BAKRON_EINVAL
    # composite calls: bad style, N = 0, shampoo needs more workspace than K-FAC
    for fn, args in ((lib.bakron_kron_factors, (one, one, 64, 32, 48)),
                     (lib.bakron_mlp_local_factors, (one, one, one, 64, 32, 48))):
        q = ctypes.c_size_t(0)
        assert fn(*args, 7, one, one, None, ctypes.byref(q), None) == pk.BAKRON_EINVAL
        assert b"style" in lib.bakron_last_error()
        bad = list(args)
        bad[-3] = 0
        assert fn(*bad, pk.BAKRON_KFAC, one, one, None, ctypes.byref(q), None) == pk.BAKRON_EINVAL
        assert fn(*args, pk.BAKRON_KFAC, one, one, None, ctypes.byref(q), None) == pk.BAKRON_OK
        kfac = q.value
        assert fn(*args, pk.BAKRON_SHAMPOO, one, one, None, ctypes.byref(q), None) == pk.BAKRON_OK
        assert q.value > kfac
        q = ctypes.c_size_t(q.value)
        assert fn(*args, pk.BAKRON_SHAMPOO, None, one, one, ctypes.byref(q),
                  None) == pk.BAKRON_EINVAL
    assert lib.bakron_sample_weights(None, 10, 4, None, one, None) == pk.BAKRON_EINVAL
    assert lib.bakron_sample_weights(one, -2, 4, None, one, None) == pk.BAKRON_EINVAL


def test_quantiser_and_scale_search_host_validation(lib):
    import paper_2608_06291_amd as pk
    one = ctypes.c_void_p(256)
    sc = ctypes.c_void_p(0)
    # the MSE search: bad bits / alphabet / grid / shrink / sizes
    for args in ((one, 4, 8, 1, 0, 0, 100, 0.5), (one, 4, 8, 4, 2, 0, 100, 0.5),
                 (one, 4, 8, 4, 0, -1, 100, 0.5), (one, 4, 8, 4, 0, 0, 256, 0.5),
                 (one, 4, 8, 4, 0, 0, 100, 1.0), (one, 0, 8, 4, 0, 0, 100, 0.5),
                 (None, 4, 8, 4, 0, 0, 100, 0.5)):
        assert lib.bakron_mse_scales(*args, one, None) == pk.BAKRON_EINVAL, args
    assert lib.bakron_mse_scales(one, 4, 8, 4, 0, 0, 100, 0.5, None, None) == pk.BAKRON_EINVAL
    # block-diagonal factor: bad block arguments
    h = ctypes.c_void_p(0)
    assert lib.bakron_factor_blockdiag(one, 8, None, 2, 4, 0.01, None,
                                       ctypes.byref(h)) == pk.BAKRON_EINVAL
    assert lib.bakron_factor_blockdiag(one, 8, one, 0, 4, 0.01, None,
                                       ctypes.byref(h)) == pk.BAKRON_EINVAL
    assert b"block" in lib.bakron_last_error()
    del sc


def test_binding_checks_quantiser_shapes():
    import torch
    import paper_2608_06291_amd as pk
    with pytest.raises(TypeError):   # CPU tensors are refused before any shape logic
        pk.mse_scales(torch.zeros(4, 4), 3)
    with pytest.raises((TypeError, ValueError)):
        pk._lib._quantizer(3, torch.zeros(4), 4, 8, "sym", 0, None)


def test_power_step_host_validation(lib):
    import paper_2608_06291_amd as pk
    one = ctypes.c_void_p(256)
    q = ctypes.c_size_t(0)
    for iters in (0, 65):
        assert lib.bakron_kron_factors_iter(one, one, 64, 32, 48, iters, one, one, None,
                                            ctypes.byref(q), None) == pk.BAKRON_EINVAL
        assert lib.bakron_mlp_local_factors_iter(one, one, one, 64, 32, 48, iters, one, one, None,
                                                 ctypes.byref(q), None) == pk.BAKRON_EINVAL
    # more steps need the quadratic-form partials (and D^T D for the MLP-local case)
    assert lib.bakron_kron_factors_iter(one, one, 4096, 32, 48, 1, one, one, None,
                                        ctypes.byref(q), None) == pk.BAKRON_OK
    one_step = q.value
    assert lib.bakron_mlp_local_factors_iter(one, one, one, 4096, 32, 48, 1, one, one, None,
                                             ctypes.byref(q), None) == pk.BAKRON_OK
    mlp1 = q.value
    assert lib.bakron_mlp_local_factors_iter(one, one, one, 4096, 32, 48, 3, one, one, None,
                                             ctypes.byref(q), None) == pk.BAKRON_OK
    assert q.value >= mlp1 + 48 * 48 * 4
    assert lib.bakron_kron_factors_iter(one, one, 4096, 32, 48, 3, one, one, None,
                                        ctypes.byref(q), None) == pk.BAKRON_OK
    assert q.value >= one_step
    assert lib.bakron_quadform_weights(None, 10, 8, None, None, None, ctypes.byref(q),
                                       None) == pk.BAKRON_OK and q.value >= 40
    q2 = ctypes.c_size_t(q.value)
    assert lib.bakron_quadform_weights(None, 10, 8, one, one, one, ctypes.byref(q2),
                                       None) == pk.BAKRON_EINVAL
