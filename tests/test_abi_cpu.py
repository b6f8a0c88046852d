"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function include/ff.h declares, sizes workspaces and rejects bad
arguments before touching a device."""
import ctypes
import os

import pytest

import paper_2609_14706_amd as ff


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(ff.LIB_PATH):
        from paper_2609_14706_amd.build import build
        build()
    return ff.load_library()


def cfg(m=64, n=128, N=256, dtype=ff.FF_F32, split=1):
    c = ff.ff_config()
    c.m, c.n, c.N, c.dtype, c.whiten_split = m, n, N, dtype, split
    return c


def test_every_declared_symbol_is_exported(lib):
    names = ff.header_functions()
    assert {"ff_workspace_size", "ff_init", "ff_iterate", "ff_factors", "ff_kron_apply",
            "ff_destroy", "ff_status_string"} <= set(names)
    for name in names:
        assert hasattr(lib, name), name
    # and nothing else with the ff_ prefix is exported
    out = os.popen(f"nm -D --defined-only {ff.LIB_PATH}").read().split()
    exported = {s for s in out if s.startswith("ff_")}
    assert exported == set(names)


def test_status_strings(lib):
    for code in range(6):
        assert ff.ff_status_string(code)
    assert ff.ff_status_string(99) == "unknown status"


def test_workspace_sizes(lib):
    small = ff.ff_workspace_size(cfg())
    assert small > 2 * 256 * 64 * 128 * 4            # at least the sample copies
    big = ff.ff_workspace_size(cfg(4096, 4096, 128, ff.FF_BF16))
    assert 2 * 128 * 4096 * 4096 * 2 <= big < 11e9   # transposed copy + whitened buffer + factors
    # aligned bf16 shapes need no padded copy of G; ragged ones do
    r = ff.ff_workspace_size(cfg(4000, 4096, 128, ff.FF_BF16))
    assert r > big
    split2 = ff.ff_workspace_size(cfg(4096, 4096, 128, ff.FF_BF16, split=2))
    assert split2 == big + 2 * 4096 * 4096 * 2
    # automatic split: both low parts, plus per side a flag/statistic block
    # and the statistic's partial sums (16 column blocks x 64 row chunks)
    auto = ff.ff_workspace_size(cfg(4096, 4096, 128, ff.FF_BF16, split=0))
    assert auto == split2 + 2 * (256 + 8 * 16 * 64)
    large = ff.ff_workspace_size(cfg(8192, 28672, 32, ff.FF_BF16))
    assert large < 60e9


@pytest.mark.parametrize("field,value", [("m", 0), ("n", -1), ("N", 0), ("dtype", 7),
                                         ("N", 70000)])
def test_bad_shapes_rejected(lib, field, value):
    c = cfg()
    setattr(c, field, value)
    with pytest.raises(ff.FlipFlopError) as ei:
        ff.ff_workspace_size(c)
    assert ei.value.code == ff.FF_ERR_INVALID_ARG


def test_bad_split_rejected(lib):
    with pytest.raises(ff.FlipFlopError) as ei:
        ff.ff_workspace_size(cfg(dtype=ff.FF_BF16, split=3))
    assert ei.value.code == ff.FF_ERR_INVALID_ARG
    assert ff.ff_workspace_size(cfg(dtype=ff.FF_F32, split=3)) > 0   # ignored on the fp32 path


def test_init_validates_before_any_device_call(lib):
    c = cfg()
    with pytest.raises(ff.FlipFlopError) as ei:          # NULL G
        ff.ff_init(c)
    assert ei.value.code == ff.FF_ERR_INVALID_ARG
    c.G = 0x1008                                          # misaligned G
    with pytest.raises(ff.FlipFlopError) as ei:
        ff.ff_init(c)
    assert ei.value.code == ff.FF_ERR_INVALID_ARG
    c.G = 0x1000
    c.damping = -1.0
    with pytest.raises(ff.FlipFlopError) as ei:
        ff.ff_init(c)
    assert ei.value.code == ff.FF_ERR_INVALID_ARG
    c.damping = 0.0
    c.order = 5
    with pytest.raises(ff.FlipFlopError) as ei:
        ff.ff_init(c)
    assert ei.value.code == ff.FF_ERR_INVALID_ARG
    c.order = 0
    with pytest.raises(ff.FlipFlopError) as ei:          # no workspace
        ff.ff_init(c)
    assert ei.value.code == ff.FF_ERR_WORKSPACE
    c.workspace = 0x100080                                # misaligned workspace
    c.workspace_bytes = 1 << 40
    with pytest.raises(ff.FlipFlopError) as ei:
        ff.ff_init(c)
    assert ei.value.code == ff.FF_ERR_WORKSPACE
    c.workspace = 0x100000                                # too small
    c.workspace_bytes = 1024
    with pytest.raises(ff.FlipFlopError) as ei:
        ff.ff_init(c)
    assert ei.value.code == ff.FF_ERR_WORKSPACE
    assert "too small" in ff.ff_last_error()


def test_null_handle_calls(lib):
    done = ctypes.c_int(7)
    assert lib.ff_iterate(None, 1, ctypes.byref(done), None) == ff.FF_ERR_INVALID_ARG
    assert done.value == 0
    assert lib.ff_factors(None, None, None, 1) == ff.FF_ERR_INVALID_ARG
    assert lib.ff_kron_apply(None, None, None, 1, 0) == ff.FF_ERR_INVALID_ARG
    assert lib.ff_destroy(None) == ff.FF_OK


def test_quantize_workspace_sizes(lib):
    b = ff.ff_quantize_workspace_size(4096, 4096)
    # two padded normalised inverse factors, four tile-blocked accumulators, padded codes
    assert 7 * 4096 * 4096 * 4 <= b < 7 * 4096 * 4096 * 4 + (1 << 20)
    r = ff.ff_quantize_workspace_size(100, 70)           # padded to 128 x 128 tiles
    assert 7 * 128 * 128 * 4 <= r < 7 * 128 * 128 * 4 + 8192
    assert ff.ff_quantize_workspace_size(1, 1) >= 7 * 64 * 64 * 4
    for m, n in [(0, 5), (5, 0), (-3, 4), ((1 << 20) + 1, 4)]:
        with pytest.raises(ff.FlipFlopError) as ei:
            ff.ff_quantize_workspace_size(m, n)
        assert ei.value.code == ff.FF_ERR_INVALID_ARG


def test_quantize_rejects_null_handle(lib):
    d = ctypes.c_double(0.0)
    assert lib.ff_quantize(None, None, None, None, 1.0, 0, None, None, None, None,
                           ctypes.byref(d), None, 0) == ff.FF_ERR_INVALID_ARG
    assert "handle" in ff.ff_last_error()
    assert lib.ff_objective(None, None, None, ctypes.byref(d)) == ff.FF_ERR_INVALID_ARG


def test_estimator_validation(lib):
    c = cfg()
    c.estimator = 7
    with pytest.raises(ff.FlipFlopError) as ei:
        ff.ff_workspace_size(c)
    assert ei.value.code == ff.FF_ERR_INVALID_ARG and "estimator" in ff.ff_last_error()
    for est in (ff.FF_EST_MARGINAL, ff.FF_EST_INPUT):     # token means need the rank-one form
        c.estimator = est
        with pytest.raises(ff.FlipFlopError):
            ff.ff_workspace_size(c)
        c.form = ff.FF_SAMPLES_RANK1
        assert ff.ff_workspace_size(c) > 0
        c.form = ff.FF_SAMPLES_DENSE
    c.estimator = ff.FF_EST_FROBENIUS
    assert ff.ff_workspace_size(c) == ff.ff_workspace_size(cfg())


def test_noalloc_entry_rejects_oversized_problems_before_any_device_call(lib):
    import paper_2609_14706_amd as ffe
    c = cfg(4096, 4096, 128, ff.FF_BF16)
    c.G = 0x100000                                        # never dereferenced
    assert ff.ff_workspace_size(c) > ffe.FF_NOALLOC_SCRATCH_BYTES
    with pytest.raises(ff.FlipFlopError) as ei:
        ff.ff_fit_noalloc(c, 1, 0x200000, 0x300000)
    assert ei.value.code == ff.FF_ERR_WORKSPACE
    assert "bytes of scratch" in str(ei.value)
    with pytest.raises(ff.FlipFlopError) as ei:          # outputs are checked first
        ff.ff_fit_noalloc(c, 1, 0, 0)
    assert ei.value.code == ff.FF_ERR_INVALID_ARG


def test_noalloc_scratch_size_matches_the_header(lib):
    import re
    import paper_2609_14706_amd as ffe
    from paper_2609_14706_amd.binding import HEADER
    text = open(HEADER).read()
    mo = re.search(r"#define FF_NOALLOC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", text)
    assert mo and int(mo.group(1)) << int(mo.group(2)) == ffe.FF_NOALLOC_SCRATCH_BYTES
    # the tiny workload fits, the headline one does not
    assert ff.ff_workspace_size(cfg(64, 128, 256)) < ffe.FF_NOALLOC_SCRATCH_BYTES


def test_new_entry_points_validate_handles(lib):
    with pytest.raises(ff.FlipFlopError) as ei:
        ff.ff_iterate_tol(None, 3, 1e-3)
    assert ei.value.code == ff.FF_ERR_INVALID_ARG
    with pytest.raises(ff.FlipFlopError) as ei:
        ff.ff_half_step(None, ff.FF_HALF_B, None, 0x1000)
    assert ei.value.code == ff.FF_ERR_INVALID_ARG
