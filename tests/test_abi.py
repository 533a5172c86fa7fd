"""The C-ABI library loads and exports every symbol the header declares, and
rejects bad host-side arguments before touching the device (CPU only)."""

import ctypes
import os

import pytest

from paper_2505_07680_amd import _lib


# The argument-check tests pass placeholder addresses that must never reach a
# kernel launch; they are host-logic tests and only run where no device is visible.
no_device = pytest.mark.skipif(
    __import__("torch").cuda.device_count() > 0, reason="host-only argument checks"
)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2505_07680_amd.build import build

        build()
    return _lib.load()


def test_header_declares_the_three_calls():
    names = _lib.header_functions()
    for n in ("specrouter_verify_attention", "specrouter_accept_and_diverge", "specrouter_rollback"):
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    for name in _lib.header_functions():
        assert hasattr(lib, name), name


def test_version_and_status_strings(lib):
    assert lib.specrouter_abi_version() == 5
    for code in (0, -1, -2, -3, -4, -5, 1, 2, 4, 8, 16, 32, 64):
        s = lib.specrouter_status_string(code)
        assert s and s != b"unknown code"
    assert lib.specrouter_status_string(12345) == b"unknown code"


def _null():
    return ctypes.c_void_p(0)


@no_device
def test_attention_rejects_bad_host_arguments(lib):
    p = ctypes.c_void_p(4096)  # never dereferenced: every case fails before a launch
    args = [p, p, p, None, p, p, p, 2, 4, 8, 2, 128, 512, 0.1, None, 0, None, None]
    bad = list(args)
    bad[0] = None
    assert lib.specrouter_verify_attention(*bad) == _lib.SR_EINVAL
    bad = list(args)
    bad[9] = 3  # Hq % Hkv != 0
    assert lib.specrouter_verify_attention(*bad) == _lib.SR_EINVAL
    bad = list(args)
    bad[11] = 96  # head dim
    assert lib.specrouter_verify_attention(*bad) == _lib.SR_EUNSUPPORTED
    bad = list(args)
    bad[8] = 17  # gamma_max above 16
    assert lib.specrouter_verify_attention(*bad) == _lib.SR_EINVAL
    bad = list(args)
    bad[0] = ctypes.c_void_p(4100)  # misaligned
    assert lib.specrouter_verify_attention(*bad) == _lib.SR_EINVAL
    for scale in (0.0, -0.1, float("nan"), float("inf")):  # the score scale must be positive and finite
        bad = list(args)
        bad[13] = scale
        assert lib.specrouter_verify_attention(*bad) == _lib.SR_EINVAL


@no_device
def test_accept_rejects_bad_host_arguments(lib):
    p = ctypes.c_void_p(4096)
    B, G, V = 2, 4, 1000
    base = [p, (G + 1) * V, p, G * V, _lib.SR_F32] + [p] * 4 + [None] + [p, p] + [None] * 6 + [B, G, V, p, 1 << 20, None, None]
    bad = list(base)
    bad[4] = 7
    assert lib.specrouter_accept_and_diverge(*bad) == _lib.SR_EUNSUPPORTED
    bad = list(base)
    bad[1] = V  # batch stride too small
    assert lib.specrouter_accept_and_diverge(*bad) == _lib.SR_EINVAL
    bad = list(base)
    bad[20] = 1001  # fp32 rows of 1001 entries are not 16-byte multiples
    bad[1], bad[3] = (G + 1) * 1001, G * 1001
    assert lib.specrouter_accept_and_diverge(*bad) == _lib.SR_EUNSUPPORTED
    bad = list(base)
    bad[12] = p  # new_len without kv_len
    assert lib.specrouter_accept_and_diverge(*bad) == _lib.SR_EINVAL
    bad = list(base)
    bad[2] = None  # q_logits missing with gamma_max > 0
    assert lib.specrouter_accept_and_diverge(*bad) == _lib.SR_EINVAL


@no_device
def test_sampled_accept_rejects_bad_sampling_parameters(lib):
    p = ctypes.c_void_p(4096)
    B, G, V = 2, 4, 1000
    S = _lib.SamplingParams

    def call(sampling, u_acc=p, u_res=p):
        args = ([p, (G + 1) * V, p, G * V, _lib.SR_F32, p, p, u_acc, u_res, None, p, p] + [None] * 6
                + [B, G, V, None if sampling is None else ctypes.byref(sampling), None, 0, None, None])
        return lib.specrouter_accept_and_diverge_sampled(*args)

    # valid sampling parameters pass the argument checks and stop at the launch
    # plan (no device here) or the empty workspace
    later = (_lib.SR_EWORKSPACE, _lib.SR_ELAUNCH)
    assert call(None) in later
    assert call(S(0.7, 0, 1.0)) in later
    assert call(S(0.0, 0, 1.0), u_acc=None, u_res=None) in later  # greedy reads no uniforms
    for t in (-0.5, float("nan"), float("inf")):
        assert call(S(t, 0, 1.0)) == _lib.SR_EINVAL
    assert call(S(1.0, 5, 1.0)) in later  # top-k
    assert call(S(1.0, 0, 0.9)) in later  # top-p
    assert call(S(1.0, 40, 0.95)) in later
    for k, tp in ((-1, 1.0), (0, 0.0), (0, -0.5), (0, 1.5), (0, float("nan"))):
        assert call(S(1.0, k, tp)) == _lib.SR_EINVAL
    assert call(S(0.5, 0, 1.0), u_acc=None) == _lib.SR_EINVAL  # sampling needs the uniforms
    assert call(S(0.5, 0, 1.0), u_res=None) == _lib.SR_EINVAL


@no_device
def test_accept_and_rollback_rejects_bad_host_arguments(lib):
    p = ctypes.c_void_p(4096)
    B, G, V = 2, 4, 1000

    def call(kv=p, cache=p, L_cap=64):
        args = ([p, (G + 1) * V, p, G * V, _lib.SR_F32, p, p, p, p, kv, p, p] + [None] * 6
                + [B, G, V, None, cache, None, None, L_cap, None, 0, None, None])
        return lib.specrouter_accept_and_rollback(*args)

    assert call() in (_lib.SR_EWORKSPACE, _lib.SR_ELAUNCH)  # arguments fine, then no workspace or device
    assert call(kv=None) == _lib.SR_EINVAL  # the new lengths need kv_len
    assert call(cache=None) == _lib.SR_EINVAL
    assert call(L_cap=0) == _lib.SR_EINVAL


@no_device
def test_noalloc_accept_refuses_oversized_shapes_before_the_device(lib):
    """The size limit of the library's fixed array is checked from the shape
    alone, before any HIP call: with no device here, a shape that fits gets as
    far as the device lookup (SR_ELAUNCH), one that does not fit is refused
    with SR_ESCRATCH."""
    p = ctypes.c_void_p(4096)  # never dereferenced

    def call(B, G, V, dtype=_lib.SR_F32):
        args = ([p, (G + 1) * V, p, G * V, dtype, p, p, p, p, p, p, p] + [None] * 6
                + [B, G, V, None, p, None, None, 64, None, None])
        return lib.specrouter_accept_and_rollback_noalloc(*args)

    assert call(16, 5, 128256) == _lib.SR_ELAUNCH                     # fits: stops at the device lookup
    assert call(4096, 16, 128256) == _lib.SR_ESCRATCH                 # about 90 MB of workspace
    assert call(4096, 16, 128256, _lib.SR_BF16) == _lib.SR_ESCRATCH
    assert call(0, 5, 1000) == _lib.SR_EINVAL
    assert call(16, 5, 1000, dtype=7) == _lib.SR_EUNSUPPORTED


@no_device
def test_chain_calls_reject_bad_host_arguments(lib):
    p = ctypes.c_void_p(4096)
    win = [p, p, 4, 8, 4, None, p, p, None, None]
    for i, v in ((2, 0), (3, -1), (3, 17), (4, 0), (4, 17), (0, None), (7, None)):
        bad = list(win)
        bad[i] = v
        assert lib.specrouter_chain_window(*bad) == _lib.SR_EINVAL
    bad = list(win)
    bad[5] = p  # ctx_len without kv_len_next
    assert lib.specrouter_chain_window(*bad) == _lib.SR_EINVAL
    con = [p, p, p, 8, p, p, 4, 4, p, p, p, p, None, None]
    for i, v in ((3, -1), (6, 17), (7, 0), (0, None), (2, None), (10, None)):
        bad = list(con)
        bad[i] = v
        assert lib.specrouter_chain_consensus(*bad) == _lib.SR_EINVAL


@no_device
def test_rollback_rejects_bad_host_arguments(lib):
    p = ctypes.c_void_p(4096)
    assert lib.specrouter_rollback(None, None, p, None, 4, 16, None, None) == _lib.SR_EINVAL
    assert lib.specrouter_rollback(p, None, p, None, 0, 16, None, None) == _lib.SR_EINVAL


def test_probe_rejects_bad_arguments_without_a_device():
    lib = _lib.load()
    assert lib.specrouter_hbm_read_probe(None, 1024, None, None) == _lib.SR_EINVAL
    fake = ctypes.c_void_p(1 << 20)  # never dereferenced: the checks come first
    assert lib.specrouter_hbm_read_probe(fake, 0, None, None) == _lib.SR_EINVAL
    assert lib.specrouter_hbm_read_probe(fake, 1000, None, None) == _lib.SR_EINVAL
    assert lib.specrouter_hbm_read_probe(ctypes.c_void_p((1 << 20) + 4), 1024, None, None) == _lib.SR_EINVAL
