"""Host-side checks of the C ABI (no GPU needed).

The library is loaded with ctypes; every argument error is detected on the host
before anything is enqueued, so each error code can be forced here with fake
(never dereferenced) device pointers. A call that would pass validation is never
made in this file.
"""
import ctypes
import os
import re

import pytest

import paper_2608_03796_amd as kd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kdtopk.h")

FAKE = 0x10000          # 16-byte aligned, never dereferenced
FAKE_MISALIGNED = 0x10008


@pytest.fixture(scope="module")
def lib():
    return kd.load_library()


def test_exports_every_declared_symbol(lib):
    with open(HEADER) as f:
        text = f.read()
    declared = set(re.findall(r"^\s*(?:kd_status|const char\*|int)\s+(kd_\w+)\s*\(", text, re.M))
    assert declared == set(kd.EXPORTED)
    for name in declared:
        assert hasattr(lib, name), name


def test_abi_version(lib):
    with open(HEADER) as f:
        text = f.read()
    v = int(re.search(r"#define KDTOPK_ABI_VERSION (\d+)", text).group(1))
    assert lib.kd_abi_version() == v


def test_status_strings(lib):
    for code, name in kd.STATUS.items():
        assert lib.kd_status_string(code).decode().startswith(name)
    assert lib.kd_status_string(99) == b"unknown kd_status"


def test_profile_modes(lib):
    """0 off, 1 every kernel, 2 contraction kernels only; anything else is
    rejected. Setting a mode touches no device; reading with nothing recorded
    returns no entries."""
    for mode in (1, 2, 0):
        assert lib.kd_profile_enable(mode) == 0
    for bad in (-1, 3):
        assert lib.kd_profile_enable(bad) == 3  # KD_ERR_BAD_ARG
    assert lib.kd_profile_read((kd.KdKernelTime * 4)(), 4) == 0


def _prob(**kw):
    base = dict(N=256, D=256, V=4096, K=16, chunk=64, tau=1.0, dtype=kd.KD_F32)
    base.update(kw)
    return kd.problem(base["N"], base["D"], base["V"], base["K"], base["chunk"], base["tau"],
                      base["dtype"], base.get("flags", 0))


def _ws(lib, pr):
    out = ctypes.c_size_t(0)
    rc = lib.kd_topk_kl_workspace_size(ctypes.byref(pr), ctypes.byref(out))
    return rc, out.value


@pytest.mark.parametrize("kw,code", [
    (dict(N=-1), 2), (dict(N=2 ** 31), 2), (dict(D=0), 2), (dict(D=32), 2), (dict(D=65600), 2),
    (dict(D=96), 4), (dict(V=0), 2), (dict(V=2 ** 20 + 1), 2), (dict(K=0), 2),
    (dict(K=4097), 2), (dict(V=65536, K=4097), 2), (dict(chunk=0), 3), (dict(chunk=-5), 3), (dict(tau=0.0), 3),
    (dict(tau=-1.0), 3), (dict(tau=float("inf")), 3), (dict(tau=float("nan")), 3),
    (dict(dtype=2), 4), (dict(dtype=-1), 4), (dict(flags=4), 3), (dict(flags=-1), 3),
])
def test_workspace_size_rejects(lib, kw, code):
    rc, _ = _ws(lib, _prob(**kw))
    assert rc == code


def test_teacher_logprobs_flag_accepted(lib):
    rc, b = _ws(lib, _prob(flags=kd.KD_FLAG_TEACHER_LOGPROBS))
    rc0, b0 = _ws(lib, _prob())
    assert rc == rc0 == 0 and b == b0


def test_workspace_size_null(lib):
    pr = _prob()
    assert lib.kd_topk_kl_workspace_size(None, ctypes.byref(ctypes.c_size_t())) == 1
    assert lib.kd_topk_kl_workspace_size(ctypes.byref(pr), None) == 1


def test_workspace_linear_not_nv(lib):
    """The workspace is bounded by a constant in N (chunk-sized buffers, a dW
    group of at most 16384 gathered tokens) plus one loss partial per 4 rows."""
    sizes = {}
    for N in (4096, 32768, 262144):
        rc, b = _ws(lib, _prob(N=N, D=4096, V=131072, K=100, chunk=4096, dtype=kd.KD_BF16))
        assert rc == 0
        sizes[N] = b
    assert sizes[4096] <= sizes[32768]
    assert sizes[262144] - sizes[32768] <= (262144 - 32768) // 4 * 4 + 256
    assert sizes[32768] < 8 * 2 ** 30
    # N*V bf16 logits at 256K tokens would be 64 GiB
    assert sizes[262144] < 262144 * 131072 * 2 / 8


def test_workspace_chunk_clamped_to_N(lib):
    rc1, a = _ws(lib, _prob(N=100, chunk=100))
    rc2, b = _ws(lib, _prob(N=100, chunk=10 ** 6))
    assert rc1 == rc2 == 0 and a == b


def _call(lib, pr, hidden=FAKE, W=FAKE, idx=FAKE, logit=FAKE, ignore=None, loss=FAKE,
          lpt=None, gh=FAKE, gw=FAKE, acc=0, ws=FAKE, ws_bytes=None):
    if ws_bytes is None:
        rc, ws_bytes = _ws(lib, pr)
        if rc != 0:
            ws_bytes = 1 << 40
    v = lambda x: None if x is None else ctypes.c_void_p(x)
    return lib.kd_topk_kl_fwd_bwd(ctypes.byref(pr), v(hidden), v(W), v(idx), v(logit), v(ignore),
                                  v(loss), v(lpt), v(gh), v(gw), acc, v(ws),
                                  ctypes.c_size_t(ws_bytes), None)


@pytest.mark.parametrize("kw,code", [
    (dict(N=-3), 2), (dict(D=100), 4), (dict(K=5000), 2), (dict(chunk=0), 3),
    (dict(tau=0.0), 3), (dict(dtype=7), 4), (dict(flags=4), 3),
])
def test_fwd_bwd_rejects_problem(lib, kw, code):
    assert _call(lib, _prob(**kw)) == code


@pytest.mark.parametrize("field", ["hidden", "W", "idx", "logit", "loss", "ws"])
def test_fwd_bwd_null_pointers(lib, field):
    assert _call(lib, _prob(), **{field: None}) == 1


def test_fwd_bwd_problem_null(lib):
    v = ctypes.c_void_p(FAKE)
    assert lib.kd_topk_kl_fwd_bwd(None, v, v, v, v, None, v, None, v, v, 0, v,
                                  ctypes.c_size_t(1 << 40), None) == 1


@pytest.mark.parametrize("field", ["hidden", "W", "gh", "gw", "ws"])
def test_fwd_bwd_misaligned(lib, field):
    assert _call(lib, _prob(), **{field: FAKE_MISALIGNED}) == 4


@pytest.mark.parametrize("acc", [2, -1])
def test_fwd_bwd_bad_accumulate(lib, acc):
    assert _call(lib, _prob(), acc=acc) == 3


def test_fwd_bwd_workspace_too_small(lib):
    pr = _prob()
    rc, need = _ws(lib, pr)
    assert rc == 0 and need > 0
    assert _call(lib, pr, ws_bytes=need - 1) == 5


def test_check_indices_rejects(lib):
    pr = _prob(K=0)
    assert lib.kd_topk_kl_check_indices(ctypes.byref(pr), ctypes.c_void_p(FAKE),
                                        ctypes.c_void_p(FAKE), ctypes.c_size_t(1 << 40), None) == 2
    pr = _prob()
    assert lib.kd_topk_kl_check_indices(ctypes.byref(pr), None, ctypes.c_void_p(FAKE),
                                        ctypes.c_size_t(1 << 40), None) == 1
    assert lib.kd_topk_kl_check_indices(ctypes.byref(pr), ctypes.c_void_p(FAKE),
                                        ctypes.c_void_p(FAKE), ctypes.c_size_t(16), None) == 5


# ------------------------------------------------ split forward / backward --
def _fwd(lib, pr, hidden=FAKE, W=FAKE, idx=FAKE, logit=FAKE, ignore=None, loss=FAKE, lpt=None,
         logz=FAKE, ws=FAKE, ws_bytes=None):
    if ws_bytes is None:
        rc, ws_bytes = _ws(lib, pr)
        if rc != 0:
            ws_bytes = 1 << 40
    v = lambda x: None if x is None else ctypes.c_void_p(x)
    return lib.kd_topk_kl_fwd(ctypes.byref(pr), v(hidden), v(W), v(idx), v(logit), v(ignore),
                              v(loss), v(lpt), v(logz), v(ws), ctypes.c_size_t(ws_bytes), None)


def _bwd(lib, pr, hidden=FAKE, W=FAKE, idx=FAKE, logit=FAKE, ignore=None, logz=FAKE, gl=None,
         glt=None, gh=FAKE, gw=FAKE, acc=0, ws=FAKE, ws_bytes=None):
    if ws_bytes is None:
        rc, ws_bytes = _ws(lib, pr)
        if rc != 0:
            ws_bytes = 1 << 40
    v = lambda x: None if x is None else ctypes.c_void_p(x)
    return lib.kd_topk_kl_bwd(ctypes.byref(pr), v(hidden), v(W), v(idx), v(logit), v(ignore),
                              v(logz), v(gl), v(glt), v(gh), v(gw), acc, v(ws),
                              ctypes.c_size_t(ws_bytes), None)


@pytest.mark.parametrize("kw,code", [
    (dict(N=-3), 2), (dict(D=100), 4), (dict(K=5000), 2), (dict(chunk=0), 3),
    (dict(tau=0.0), 3), (dict(dtype=7), 4), (dict(flags=4), 3),
])
def test_split_rejects_problem(lib, kw, code):
    assert _fwd(lib, _prob(**kw)) == code
    assert _bwd(lib, _prob(**kw)) == code


@pytest.mark.parametrize("field", ["hidden", "W", "idx", "logit", "loss", "logz", "ws"])
def test_fwd_null_pointers(lib, field):
    assert _fwd(lib, _prob(), **{field: None}) == 1


@pytest.mark.parametrize("field", ["hidden", "W", "idx", "logit", "logz", "ws"])
def test_bwd_null_pointers(lib, field):
    assert _bwd(lib, _prob(), **{field: None}) == 1


@pytest.mark.parametrize("field", ["hidden", "W", "ws"])
def test_fwd_misaligned(lib, field):
    assert _fwd(lib, _prob(), **{field: FAKE_MISALIGNED}) == 4


@pytest.mark.parametrize("field", ["hidden", "W", "gh", "gw", "ws"])
def test_bwd_misaligned(lib, field):
    assert _bwd(lib, _prob(), **{field: FAKE_MISALIGNED}) == 4


def test_split_workspace_too_small(lib):
    pr = _prob()
    rc, need = _ws(lib, pr)
    assert rc == 0
    assert _fwd(lib, pr, ws_bytes=need - 1) == 5
    assert _bwd(lib, pr, ws_bytes=need - 1) == 5


@pytest.mark.parametrize("acc", [2, -1])
def test_bwd_bad_accumulate(lib, acc):
    assert _bwd(lib, _prob(), acc=acc) == 3


def test_grad_hidden_f32_flag_accepted(lib):
    for flags in (2, 3):
        rc, n = _ws(lib, _prob(flags=flags))
        assert rc == 0 and n > 0


def _scale(lib, g=FAKE, hin=None, hdt=kd.KD_F32, hout=None, nh=0, win=None, wdt=kd.KD_F32,
           wout=None, nw=0):
    return lib.kd_scale_grads(g, hin, hdt, hout, nh, win, wdt, wout, nw, None)


def test_scale_grads_rejects(lib):
    """kd_scale_grads: every argument error is found before any launch (the
    pointers below are never dereferenced)."""
    A, B = FAKE, FAKE + (1 << 20)
    assert _scale(lib, g=None, hin=A, hout=B, nh=8) == 1                  # no g
    assert _scale(lib, hin=A, hout=None, nh=8) == 1                      # half a pair
    assert _scale(lib, win=None, wout=B, nw=8) == 1
    assert _scale(lib, hin=A, hout=B, nh=-1) == 2                        # negative count
    assert _scale(lib, win=A, wout=B, nw=-8) == 2
    assert _scale(lib, hin=A, hdt=2, hout=B, nh=8) == 4                  # output dtype
    assert _scale(lib, win=A, wdt=-1, wout=B, nw=8) == 4
    assert _scale(lib, hin=FAKE_MISALIGNED, hout=B, nh=8) == 4           # alignment
    assert _scale(lib, win=A, wout=FAKE_MISALIGNED, nw=8) == 4
    assert _scale(lib, win=A, wdt=kd.KD_BF16, wout=A, nw=64) == 3        # bf16 onto its input
    assert _scale(lib, win=A, wout=A + 16, nw=64) == 3                   # partial overlap
    assert _scale(lib, hin=A, hdt=kd.KD_BF16, hout=A + 64, nh=64) == 3
    # nothing to do: no launch, KD_OK
    assert _scale(lib) == 0
    assert _scale(lib, hin=A, hout=B, nh=0, win=A, wout=B, nw=0) == 0


def test_noalloc_rejects_before_the_device(lib):
    """The allocation-free entry point refuses, on the host, a problem whose
    one-chunk workspace exceeds the library's static scratch
    (KD_ERR_WORKSPACE_TOO_SMALL), and every argument error of
    kd_topk_kl_fwd_bwd, before it touches a device (none here)."""
    v = lambda x: None if x is None else ctypes.c_void_p(x)

    def call(pr, loss=FAKE, hidden=FAKE, acc=0):
        return lib.kd_topk_kl_fwd_bwd_noalloc(ctypes.byref(pr), v(hidden), v(FAKE), v(FAKE),
                                              v(FAKE), None, v(loss), None, v(FAKE), v(FAKE),
                                              acc, None)
    big = _prob(N=8192, D=4096, V=131072, K=100, chunk=4096, dtype=kd.KD_BF16)
    assert call(big) == 5
    assert call(_prob(chunk=0)) == 3
    assert call(_prob(), loss=None) == 1
    assert call(_prob(), hidden=None) == 1
    assert call(_prob(), hidden=FAKE_MISALIGNED) == 4
    assert call(_prob(), acc=2) == 3
    assert lib.kd_topk_kl_fwd_bwd_noalloc(None, None, None, None, None, None, None, None, None,
                                          None, 0, None) == 1
