"""Host-side checks of the C ABI: the library loads, exports every declared symbol, sizes its
workspace, and rejects invalid arguments before any GPU work (no compute calls here)."""
import ctypes
import os
import re

import pytest

from paper_2608_05448_amd import dblast as D

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dblast.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dbl_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(D.LIB_PATH):
        pytest.fail("libdblast.so is not built (run `python -m paper_2608_05448_amd.build`)")
    return D.load()


def test_every_declared_symbol_is_exported_and_bound(lib):
    declared = _declared_functions()
    assert set(declared) == set(D.EXPORTED), (declared, D.EXPORTED)
    for name in declared:
        assert getattr(lib, name) is not None


def test_constants_and_status_strings(lib):
    assert lib.dbl_vtile() == 128
    assert lib.dbl_ntiles(151936) == 1187
    assert lib.dbl_ntiles(129) == 2
    assert lib.dbl_ntiles(0) == 0
    for s, name in enumerate(["DBL_OK", "DBL_EINVAL", "DBL_ESHAPE", "DBL_EDTYPE",
                              "DBL_EWORKSPACE", "DBL_EHIP"]):
        assert lib.dbl_status_string(s).decode() == name
    assert lib.dbl_status_string(99).decode() == "DBL_UNKNOWN"


def test_workspace_sizes(lib):
    S = D.Shape
    SIZE_MAX = ctypes.c_size_t(-1).value
    # Head: one uint64 argmax key per row (used only when the argmax is requested).
    assert lib.dbl_workspace_bytes(D.DBL_OP_HEAD, S(16, 16, 8, 4096, 151936)) == 2048 * 8
    assert lib.dbl_workspace_bytes(D.DBL_OP_SAMPLE_GREEDY, S(16, 16, 8, 0, 151936)) == 0
    g = lib.dbl_workspace_bytes(D.DBL_OP_VERIFY_GREEDY, S(16, 16, 8, 0, 151936))
    assert g == 2048 * 8 + 2 * -(-16 * 1187 * 8 // 256) * 256
    assert lib.dbl_workspace_bytes(D.DBL_OP_EXPECTED_LEN_GREEDY, S(16, 16, 8, 0, 151936)) == 2048 * 8
    # Sample: no workspace (the two-stage draw reads the tile masses directly).
    assert lib.dbl_workspace_bytes(D.DBL_OP_SAMPLE, S(16, 16, 8, 0, 151936)) == 0
    v = lib.dbl_workspace_bytes(D.DBL_OP_VERIFY, S(16, 16, 8, 0, 151936))
    e = lib.dbl_workspace_bytes(D.DBL_OP_EXPECTED_LEN, S(16, 16, 8, 0, 151936))
    assert v > e > 0 and v % 256 == 0 and e % 256 == 0
    # Target transform: per row, 4 segment lists of 1024 uint64 candidates and 4 int32 counts.
    assert lib.dbl_workspace_bytes(D.DBL_OP_TARGET, S(272, 1, 1, 0, 151936)) == \
        272 * 4 * 1024 * 8 + -(-272 * 4 * 4 // 256) * 256
    assert lib.dbl_workspace_bytes(D.DBL_OP_TARGET, S(16, 17, 1, 0, 151936)) == \
        lib.dbl_workspace_bytes(D.DBL_OP_TARGET, S(272, 1, 1, 0, 151936))
    assert lib.dbl_workspace_bytes(8, S(1, 1, 1, 8, 8)) == SIZE_MAX
    assert lib.dbl_workspace_bytes(D.DBL_OP_SAMPLE, S(1, 1, 65, 8, 8)) == SIZE_MAX
    assert lib.dbl_workspace_bytes(D.DBL_OP_SAMPLE, S(0, 4, 2, 8, 256)) == 0


def _fake(n=1):
    # Non-null dummy addresses. Every call made with them below is invalid in some other
    # argument and must be rejected by host validation before anything is launched.
    return [ctypes.c_void_p(0x1000 * (i + 1)) for i in range(n)]


def _err(lib):
    return lib.dbl_last_error().decode()


def test_head_validation(lib):
    S = D.Shape
    h, w, t, lm, ls = _fake(5)
    null = ctypes.c_void_p(None)
    assert lib.dbl_head_logprobs(S(1, 4, 2, 60, 256), D.DBL_BF16, h, w, t, lm, ls, null, null,
                                 0, null) == D.DBL_ESHAPE
    assert "d % 8" in _err(lib)
    assert lib.dbl_head_logprobs(S(1, 4, 2, 64, 256), 7, h, w, t, lm, ls, null, null,
                                 0, null) == D.DBL_EDTYPE
    assert lib.dbl_head_logprobs(S(1, 4, 2, 64, 256), D.DBL_F32, null, w, t, lm, ls, null, null,
                                 0, null) == D.DBL_EINVAL
    assert lib.dbl_head_logprobs(S(1, 0, 2, 64, 256), D.DBL_F32, h, w, t, lm, ls, null, null,
                                 0, null) == D.DBL_ESHAPE
    assert lib.dbl_head_logprobs(S(1, 4, 2, 64, 1 << 24), D.DBL_F32, h, w, t, lm, ls, null, null,
                                 0, null) == D.DBL_ESHAPE
    assert lib.dbl_head_logprobs(S(-1, 4, 2, 64, 256), D.DBL_F32, h, w, t, lm, ls, null, null,
                                 0, null) == D.DBL_ESHAPE


def test_head_argmax_needs_workspace(lib):
    S = D.Shape
    h, w, t, lm, ls, am = _fake(6)
    null = ctypes.c_void_p(None)
    assert lib.dbl_head_logprobs(S(1, 4, 2, 64, 256), D.DBL_F32, h, w, t, lm, ls, am, null, 0,
                                 null) == D.DBL_EWORKSPACE
    assert lib.dbl_head_logprobs(S(1, 4, 2, 64, 256), D.DBL_F32, h, w, t, lm, ls, am,
                                 ctypes.c_void_p(0x100000), 8 * 8 - 1, null) == D.DBL_EWORKSPACE


def test_greedy_validation(lib):
    S = D.Shape
    p = _fake(10)
    null = ctypes.c_void_p(None)
    shape = S(2, 4, 3, 0, 300)
    aligned = ctypes.c_void_p(0x100000)
    for zt in (-0.5, float("nan"), float("inf")):
        assert lib.dbl_sample_greedy(shape, p[0], p[1], zt, 0, 0, 0, p[2], p[3],
                                     null) == D.DBL_EINVAL
    assert lib.dbl_sample_greedy(shape, null, p[1], 1.0, 0, 0, 0, p[2], p[3],
                                 null) == D.DBL_EINVAL
    assert lib.dbl_sample_greedy(S(2, 4, 65, 0, 300), p[0], p[1], 1.0, 0, 0, 0, p[2], p[3],
                                 null) == D.DBL_ESHAPE
    vws = lib.dbl_workspace_bytes(D.DBL_OP_VERIFY_GREEDY, shape)
    for kp in (3, 6):
        assert lib.dbl_verify_greedy(shape, p[0], p[1], 1.0, p[2], p[3], kp, 0, 0, 0, p[4], p[5],
                                     null, null, null, aligned, vws, null) == D.DBL_EINVAL
    assert lib.dbl_verify_greedy(shape, p[0], p[1], 1.0, p[2], p[3], 4, 0, 0, 0, p[4], p[5],
                                 null, null, null, aligned, vws - 1, null) == D.DBL_EWORKSPACE
    ews = lib.dbl_workspace_bytes(D.DBL_OP_EXPECTED_LEN_GREEDY, shape)
    assert lib.dbl_expected_len_greedy(shape, p[0], p[1], 1.0, p[2], p[3], null, null, aligned,
                                       ews, null) == D.DBL_EINVAL
    # empty batch
    assert lib.dbl_sample_greedy(S(0, 4, 3, 0, 300), p[0], p[1], 1.0, 0, 0, 0, p[2], p[3],
                                 null) == D.DBL_OK
    assert lib.dbl_verify_greedy(S(0, 4, 3, 0, 300), p[0], p[1], 1.0, p[2], p[3], 4, 0, 0, 0,
                                 p[4], p[5], null, null, null, null, 0, null) == D.DBL_OK


def test_sample_and_verify_validation(lib):
    S = D.Shape
    p = _fake(12)
    null = ctypes.c_void_p(None)
    shape = S(2, 4, 3, 0, 300)
    ws_need = lib.dbl_workspace_bytes(D.DBL_OP_SAMPLE, shape)
    aligned = ctypes.c_void_p(0x100000)
    # Negative and NaN temperatures.
    for zt in (-0.5, float("nan"), float("inf")):
        assert lib.dbl_sample_block(shape, p[0], p[1], p[2], p[3], zt, 0, 0, 0, p[4], p[5],
                                    aligned, ws_need, null) == D.DBL_EINVAL
    # Too many categories.
    assert lib.dbl_sample_block(S(2, 4, 65, 0, 300), p[0], p[1], p[2], p[3], 1.0, 0, 0, 0, p[4],
                                p[5], aligned, 1 << 30, null) == D.DBL_ESHAPE
    vws = lib.dbl_workspace_bytes(D.DBL_OP_VERIFY, shape)
    # Kp must be K or K + 1.
    for kp in (3, 6):
        assert lib.dbl_verify_block(shape, p[0], p[1], p[2], p[3], 1.0, p[4], p[5], kp, 0, 0, 0,
                                    p[6], p[7], null, null, null, aligned, vws,
                                    null) == D.DBL_EINVAL
    assert lib.dbl_verify_block(shape, p[0], p[1], p[2], p[3], 1.0, p[4], p[5], 4, 0, 0, 0,
                                null, p[7], null, null, null, aligned, vws, null) == D.DBL_EINVAL
    ews = lib.dbl_workspace_bytes(D.DBL_OP_EXPECTED_LEN, shape)
    assert lib.dbl_expected_len(shape, p[0], p[1], p[2], p[3], 1.0, p[4], p[5], null, null,
                                aligned, ews, null) == D.DBL_EINVAL


def test_empty_batch_is_a_no_op(lib):
    S = D.Shape
    p = _fake(8)
    null = ctypes.c_void_p(None)
    assert lib.dbl_sample_block(S(0, 4, 2, 0, 256), p[0], p[1], p[2], p[3], 1.0, 0, 0, 0, p[4],
                                p[5], null, 0, null) == D.DBL_OK
    assert lib.dbl_verify_block(S(0, 4, 2, 0, 256), p[0], p[1], p[2], p[3], 1.0, p[4], p[5], 4,
                                0, 0, 0, p[6], p[7], null, null, null, null, 0, null) == D.DBL_OK
    assert lib.dbl_expected_len(S(0, 4, 2, 0, 256), p[0], p[1], p[2], p[3], 1.0, p[4], p[5],
                                null, p[6], null, 0, null) == D.DBL_OK


def test_binding_fails_loudly_without_the_library(tmp_path):
    saved = D._lib
    D._lib = None
    try:
        with pytest.raises(RuntimeError, match="not built"):
            D.load(str(tmp_path / "missing.so"))
    finally:
        D._lib = saved


def test_objective_validation(lib):
    S = D.Shape
    p = _fake(10)
    null = ctypes.c_void_p(None)
    shape = S(2, 4, 3, 0, 300)
    for tau in (0.0, -1.0, float("inf"), float("nan")):
        assert lib.dbl_acceptance_objective(shape, p[0], p[1], p[2], p[3], 1.0, p[4], p[5], tau,
                                            null, null, p[6], p[7], p[8], null) == D.DBL_EINVAL
    assert lib.dbl_acceptance_objective(shape, p[0], p[1], p[2], p[3], -1.0, p[4], p[5], 0.1,
                                        null, null, p[6], p[7], p[8], null) == D.DBL_EINVAL
    assert lib.dbl_acceptance_objective(shape, p[0], p[1], p[2], p[3], 1.0, p[4], p[5], 0.1,
                                        null, null, null, p[7], p[8], null) == D.DBL_EINVAL
    assert lib.dbl_acceptance_objective(S(0, 4, 3, 0, 300), p[0], p[1], p[2], p[3], 1.0, p[4],
                                        p[5], 0.1, null, null, p[6], p[7], p[8],
                                        null) == D.DBL_OK


def test_read_probe_validation(lib):
    p = _fake(2)
    null = ctypes.c_void_p(None)
    assert lib.dbl_stream_read_probe(null, 64, p[1], 4, null) == D.DBL_EINVAL
    assert lib.dbl_stream_read_probe(p[0], 64, null, 4, null) == D.DBL_EINVAL
    assert lib.dbl_stream_read_probe(p[0], 60, p[1], 4, null) == D.DBL_ESHAPE
    assert lib.dbl_stream_read_probe(p[0], -16, p[1], 4, null) == D.DBL_ESHAPE
    assert lib.dbl_stream_read_probe(p[0], 64, p[1], 0, null) == D.DBL_ESHAPE
    assert lib.dbl_stream_read_probe(p[0], 64, p[1], (1 << 20) + 1, null) == D.DBL_ESHAPE
    assert lib.dbl_stream_read_probe(ctypes.c_void_p(p[0].value + 4), 64, p[1], 4,
                                     null) == D.DBL_EINVAL


def test_target_validation(lib):
    p = _fake(3)
    null = ctypes.c_void_p(None)
    N, V = 4, 1000
    # logp overlapping logits (same buffer, or shifted inside it)
    assert lib.dbl_target_logprobs(N, V, p[0], 1.0, 20, 0.9, p[0], null, 0, null) == D.DBL_EINVAL
    shifted = ctypes.c_void_p(p[0].value + 4 * V)
    assert lib.dbl_target_logprobs(N, V, p[0], 1.0, 20, 0.9, shifted, null, 0, null) == \
        D.DBL_EINVAL
    far = ctypes.c_void_p(p[0].value + 4 * N * V)   # adjacent, not overlapping: only ws fails
    need = lib.dbl_workspace_bytes(D.DBL_OP_TARGET, D.Shape(N, 1, 1, 0, V))
    assert lib.dbl_target_logprobs(N, V, p[0], 1.0, 20, 0.9, far, p[2], need - 1, null) == \
        D.DBL_EWORKSPACE
    assert lib.dbl_target_logprobs(N, V, p[0], 1.0, 20, 0.9, far, null, need, null) == \
        D.DBL_EWORKSPACE
    assert lib.dbl_target_logprobs(N, V, p[0], -1.0, 20, 0.9, far, null, 0, null) == D.DBL_EINVAL
    assert lib.dbl_target_logprobs(N, V, p[0], 1.0, -1, 0.9, far, null, 0, null) == D.DBL_EINVAL
    assert lib.dbl_target_logprobs(N, V, p[0], 1.0, 20, 0.0, far, null, 0, null) == D.DBL_EINVAL
    assert lib.dbl_target_logprobs(0, V, p[0], 1.0, 20, 0.9, far, null, 0, null) == D.DBL_OK


def test_misaligned_arrays_are_rejected(lib):
    """Every array must be 16-byte aligned (the kernels use 16-byte vector accesses): a pointer
    4 bytes into an allocation is DBL_EINVAL, before anything is launched."""
    S = D.Shape
    p = _fake(12)
    null = ctypes.c_void_p(None)
    off = lambda q: ctypes.c_void_p(q.value + 4)
    aligned = ctypes.c_void_p(0x100000)
    hs = S(1, 4, 2, 64, 256)
    args = [p[0], p[1], p[2], p[3], p[4]]
    for i in range(5):
        a = list(args)
        a[i] = off(a[i])
        assert lib.dbl_head_logprobs(hs, D.DBL_BF16, *a, null, null, 0, null) == D.DBL_EINVAL
        assert "16-byte aligned" in _err(lib)
    shape = S(2, 4, 3, 0, 300)
    sws = lib.dbl_workspace_bytes(D.DBL_OP_SAMPLE, shape)
    assert lib.dbl_sample_block(shape, off(p[0]), p[1], p[2], p[3], 1.0, 0, 0, 0, p[4], p[5],
                                aligned, sws, null) == D.DBL_EINVAL
    assert lib.dbl_sample_block(shape, p[0], p[1], p[2], p[3], 1.0, 0, 0, 0, p[4], off(p[5]),
                                aligned, sws, null) == D.DBL_EINVAL
    vws = lib.dbl_workspace_bytes(D.DBL_OP_VERIFY, shape)
    assert lib.dbl_verify_block(shape, p[0], p[1], p[2], p[3], 1.0, p[4], off(p[5]), 4, 0, 0, 0,
                                p[6], p[7], null, null, null, aligned, vws, null) == D.DBL_EINVAL
    assert "logp" in _err(lib)
    assert lib.dbl_verify_block(shape, p[0], p[1], p[2], p[3], 1.0, p[4], p[5], 4, 0, 0, 0,
                                p[6], p[7], off(p[8]), null, null, aligned, vws,
                                null) == D.DBL_EINVAL
    ews = lib.dbl_workspace_bytes(D.DBL_OP_EXPECTED_LEN, shape)
    assert lib.dbl_expected_len(shape, p[0], p[1], off(p[2]), p[3], 1.0, p[4], p[5], null, p[6],
                                aligned, ews, null) == D.DBL_EINVAL
    assert lib.dbl_sample_greedy(shape, off(p[0]), p[1], 1.0, 0, 0, 0, p[2], p[3],
                                 null) == D.DBL_EINVAL
    assert lib.dbl_acceptance_objective(shape, p[0], p[1], p[2], p[3], 1.0, off(p[4]), p[5], 0.1,
                                        null, null, p[6], p[7], p[8], null) == D.DBL_EINVAL
    assert lib.dbl_expand_branches(S(1, 4, 2, 64, 1), p[0], off(p[1]), p[2], p[3],
                                   null) == D.DBL_EINVAL
    assert lib.dbl_prior_head(S(1, 1, 2, 64, 1), p[0], p[1], p[2], off(p[3]),
                              null) == D.DBL_EINVAL
    assert lib.dbl_target_logprobs(4, 1000, off(p[0]), 1.0, 20, 0.9, p[5], null, 0,
                                   null) == D.DBL_EINVAL
    assert lib.dbl_early_determinism(2, 3, 100, p[0], p[1], off(p[2]), null,
                                     null) == D.DBL_EINVAL
    # the same calls with aligned arrays fail only where something else is wrong (here: nothing
    # is checked past alignment for an empty batch, which is a no-op)
    assert lib.dbl_sample_block(S(0, 4, 3, 0, 300), p[0], p[1], p[2], p[3], 1.0, 0, 0, 0, p[4],
                                p[5], null, 0, null) == D.DBL_OK


def test_hidden_size_cap(lib):
    """The bf16 head kernels address operand rows with 32-bit byte offsets (at most 512 d within
    a tile): d above 2^20 is rejected rather than wrapping."""
    S = D.Shape
    h, w, t, lm, ls = _fake(5)
    null = ctypes.c_void_p(None)
    for dt in (D.DBL_BF16, D.DBL_F32):
        assert lib.dbl_head_logprobs(S(1, 1, 1, (1 << 20) + 8, 256), dt, h, w, t, lm, ls, null,
                                     null, 0, null) == D.DBL_ESHAPE
        assert "2^20" in _err(lib)
    assert lib.dbl_workspace_bytes(D.DBL_OP_HEAD, S(1, 1, 1, 1 << 23, 256)) == \
        ctypes.c_size_t(-1).value
    assert lib.dbl_workspace_bytes(D.DBL_OP_HEAD, S(1, 1, 1, 1 << 20, 256)) == 256  # 8, rounded up


def test_static_verify_rejects_shapes_beyond_its_scratch(lib):
    """dbl_verify_block_static has a fixed 8 MiB scratch: a shape that needs more is
    DBL_EWORKSPACE before anything is launched; invalid arguments fail as in dbl_verify_block."""
    S = D.Shape
    p = _fake(10)
    null = ctypes.c_void_p(None)
    big = S(1024, 16, 8, 0, 151936)
    assert lib.dbl_workspace_bytes(D.DBL_OP_VERIFY, big) > 8 << 20
    assert lib.dbl_verify_block_static(big, p[0], p[1], p[2], p[3], 1.0, p[4], p[5], 16, 0, 0,
                                       0, p[6], p[7], null, null, null, null) == D.DBL_EWORKSPACE
    assert "fixed scratch" in _err(lib)
    shape = S(2, 4, 3, 0, 300)
    for kp in (3, 6):
        assert lib.dbl_verify_block_static(shape, p[0], p[1], p[2], p[3], 1.0, p[4], p[5], kp, 0,
                                           0, 0, p[6], p[7], null, null, null,
                                           null) == D.DBL_EINVAL
    assert lib.dbl_verify_block_static(S(0, 4, 3, 0, 300), p[0], p[1], p[2], p[3], 1.0, p[4],
                                       p[5], 4, 0, 0, 0, p[6], p[7], null, null, null,
                                       null) == D.DBL_OK
