"""The C ABI on the CPU: the HIP library loads, exports every symbol the
header declares, and its host-side validation answers before anything
touches a GPU (no compute calls here)."""
import ctypes
import os
import re

import pytest

from paper_2608_22643_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "neuroprefetch.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(np_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        pytest.fail("libneuroprefetch.so is not built (run __graft_entry__.build())")
    return B.lib()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) == 25, names
    for n in names:
        assert hasattr(lib, n), f"missing export {n}"
    assert set(names) == set(B.EXPORTS)


def test_status_strings(lib):
    assert B.status_name(B.NP_OK) == "NP_OK"
    assert B.status_name(B.NP_ERR_CAPACITY) == "NP_ERR_CAPACITY"
    assert B.status_name(99) == "NP_ERR_UNKNOWN"


GOOD = dict(layers=31, d_model=4096, d_ffn=11008, rank=416, k=1651, capacity=5504, wdtype="f16")


@pytest.mark.parametrize("change,status", [
    (dict(), B.NP_OK),
    (dict(k=5505), B.NP_ERR_CAPACITY),              # k > C
    (dict(k=0), B.NP_ERR_INVALID_ARG),
    (dict(capacity=11009), B.NP_ERR_INVALID_ARG),   # C > F
    (dict(d_model=4100), B.NP_ERR_INVALID_ARG),     # not a multiple of 8
    (dict(rank=420), B.NP_ERR_INVALID_ARG),
    (dict(rank=2048), B.NP_ERR_INVALID_ARG),
    (dict(d_ffn=70000, capacity=11008), B.NP_ERR_INVALID_ARG),
    (dict(layers=0), B.NP_ERR_INVALID_ARG),
    (dict(wdtype=7), B.NP_ERR_INVALID_ARG),
    (dict(k=9000, capacity=9000), B.NP_ERR_INVALID_ARG),
    (dict(act="swiglu"), B.NP_OK),
    (dict(act=2), B.NP_ERR_INVALID_ARG),
])
def test_shape_validation(lib, change, status):
    args = dict(GOOD, **change)
    shape = B.make_shape(**args)
    st = lib.np_shape_check(ctypes.byref(shape))
    assert st == status, (st, B.lib().np_last_error())


def test_mixed_dtypes_rejected(lib):
    shape = B.make_shape(**dict(GOOD, wdtype="f16"), adtype="bf16")
    assert lib.np_shape_check(ctypes.byref(shape)) == B.NP_ERR_INVALID_ARG


def test_workspace_size(lib):
    shape = B.make_shape(**GOOD)
    n = B.np_workspace_size(shape)
    # control block + z (31*416 fp32) + 512 partial rows of d fp32
    assert n >= 4096 + 31 * 416 * 4 + 512 * 4096 * 4
    assert n % 256 == 0


def test_null_and_misaligned_pointers_rejected(lib):
    shape = B.make_shape(**GOOD)
    with pytest.raises(B.NPError) as e:
        B.np_predict(shape, None, 16, 16, 16, 16, None)
    assert e.value.status == B.NP_ERR_INVALID_ARG
    with pytest.raises(B.NPError) as e:
        B.np_select(shape, 18, 16, 16, 16, None)  # misaligned scores
    assert e.value.status == B.NP_ERR_INVALID_ARG
    with pytest.raises(B.NPError) as e:
        B.np_sparse_mlp(shape, 31, 16, 16, 16, 1, 16, 16, None)  # layer out of range
    assert e.value.status == B.NP_ERR_INVALID_ARG
    with pytest.raises(B.NPError) as e:
        B.np_sparse_mlp(shape, 0, 16, 16, 16, 5505, 16, 16, None)  # n_active > C
    assert e.value.status == B.NP_ERR_INVALID_ARG
    with pytest.raises(B.NPError) as e:
        B.np_delta(shape, -2, 16, B.np_state(16, 16, 16), B.np_delta_out(*([16] * 7)), 16, None)
    assert e.value.status == B.NP_ERR_INVALID_ARG
    with pytest.raises(B.NPError) as e:  # np_select_delta: token below NP_TOKEN_AUTO
        B.np_select_delta(shape, -2, 16, 16, 16, B.np_state(16, 16, 16),
                          B.np_delta_out(*([16] * 7)), 16, None)
    assert e.value.status == B.NP_ERR_INVALID_ARG
    with pytest.raises(B.NPError) as e:  # np_select_delta: misaligned scores
        B.np_select_delta(shape, 0, 18, 16, 16, B.np_state(16, 16, 16),
                          B.np_delta_out(*([16] * 7)), 16, None)
    assert e.value.status == B.NP_ERR_INVALID_ARG
    with pytest.raises(B.NPError) as e:  # np_select_delta: a NULL output list
        B.np_select_delta(shape, 0, 16, 16, 16, B.np_state(16, 16, 16),
                          B.np_delta_out(*([16] * 6), None), 16, None)
    assert e.value.status == B.NP_ERR_INVALID_ARG
    with pytest.raises(B.NPError) as e:
        B.np_stage_gather(shape, B.np_delta_out(*([16] * 7)), 3, 2, 16, 16, 16, None)
    assert e.value.status == B.NP_ERR_INVALID_ARG
    assert "layer range" in B.lib().np_last_error().decode()


def test_stage_rows_validates_plan_before_enqueueing(lib):
    import numpy as np

    shape = B.make_shape(layers=2, d_model=64, d_ffn=100, rank=8, k=4, capacity=8, wdtype="f32")
    counts = np.zeros(8, np.int32)
    ids = np.zeros(8, np.int32)
    slots = np.zeros(8, np.int32)
    counts[0] = 1
    ids[0] = 100  # out of range: rejected on the host
    plan = B.np_stage_plan(counts.ctypes.data, ids.ctypes.data, slots.ctypes.data)
    buf = np.zeros(1 << 16, np.uint8)
    with pytest.raises(B.NPError) as e:
        B.np_stage_rows(shape, plan, 0, 2, buf.ctypes.data, 16, buf.ctypes.data, buf.nbytes, 16,
                        1 << 16, None)
    assert e.value.status == B.NP_ERR_INVALID_ARG
    ids[0] = 3
    with pytest.raises(B.NPError) as e:  # staging holds no record of 3*64*4+4 bytes per half
        B.np_stage_rows(shape, plan, 0, 2, buf.ctypes.data, 16, buf.ctypes.data, 1024, 16,
                        1 << 16, None)
    assert e.value.status == B.NP_ERR_CAPACITY


def test_centroid_select_validates_model(lib):
    shape = B.make_shape(**GOOD)
    good = dict(n_centroids=512, feat_dim=4096, heads=16, bank=16)
    for change in (dict(n_centroids=0), dict(n_centroids=5000), dict(feat_dim=4100),
                   dict(feat_dim=20000), dict(heads=18), dict(bank=0)):
        m = B.np_centroid_model(**dict(good, **change))
        with pytest.raises(B.NPError) as e:
            B.np_centroid_select(shape, m, 16, 16, 16, 16, 16, 16, 16, None)
        assert e.value.status == B.NP_ERR_INVALID_ARG, change


def test_variable_count_calls_need_counts(lib):
    shape = B.make_shape(**GOOD)
    with pytest.raises(B.NPError) as e:
        B.np_delta_n(shape, 0, 16, None, B.np_state(16, 16, 16), B.np_delta_out(*([16] * 7)), 16,
                     None)
    assert e.value.status == B.NP_ERR_INVALID_ARG
    with pytest.raises(B.NPError) as e:
        B.np_sparse_mlp_n(shape, 0, 16, 16, 16, None, 16, 16, None)
    assert e.value.status == B.NP_ERR_INVALID_ARG


def test_threshold_calls_validate_before_enqueueing(lib):
    shape = B.make_shape(**GOOD, act="swiglu")
    cases = [
        # np_sparse_mlp_t: n_active above C, misaligned thresholds
        lambda: B.np_sparse_mlp_t(shape, 0, 16, 16, 16, 5505, None, None, 16, 16),
        lambda: B.np_sparse_mlp_t(shape, 0, 16, 16, 16, 8, None, 18, 16, 16),
        lambda: B.np_sparse_mlp_t(shape, 31, 16, 16, 16, 8, None, None, 16, 16),
        # np_act_batch: n outside [1, 65536], misaligned tokens
        lambda: B.np_act_batch(shape, 16, 16, 0, 16),
        lambda: B.np_act_batch(shape, 16, 16, 70000, 16),
        lambda: B.np_act_batch(shape, 16, 24, 8, 16),
        # np_percentile: alpha outside [0, 100], no rows, NULL output, a
        # workspace without room for the error word
        lambda: B.np_percentile(16, 1, 100, 100.5, 16, 16, 4096),
        lambda: B.np_percentile(16, 1, 100, float("nan"), 16, 16, 4096),
        lambda: B.np_percentile(16, 0, 100, 50.0, 16, 16, 4096),
        lambda: B.np_percentile(16, 1, 0, 50.0, 16, 16, 4096),
        lambda: B.np_percentile(16, 1, 100, 50.0, None, 16, 4096),
        lambda: B.np_percentile(16, 1, 100, 50.0, 16, 16, 63),
        # np_threshold_active: no thresholds, no rows
        lambda: B.np_threshold_active(shape, 16, 1, None, 16, 16, 16, 16),
        lambda: B.np_threshold_active(shape, 16, 0, 16, 16, 16, 16, 16),
    ]
    for i, call in enumerate(cases):
        with pytest.raises(B.NPError) as e:
            call()
        assert e.value.status == B.NP_ERR_INVALID_ARG, i
    big = B.make_shape(layers=1, d_model=16384, d_ffn=65535, rank=8, k=8, capacity=8,
                       wdtype="f16")
    with pytest.raises(B.NPError) as e:
        B.np_act_batch(big, 16, 16, 1, 16)
    assert e.value.status == B.NP_ERR_UNSUPPORTED


def test_noalloc_rejects_rows_wider_than_its_scratch(lib):
    """The allocation-free MLP keeps partial rows of at most 8192 columns: a
    wider shape is refused before anything is enqueued."""
    s = B.make_shape(1, 16384, 2000, 16, 100, 200, "f16")
    with pytest.raises(B.NPError) as e:
        B.np_sparse_mlp_noalloc(s, 0, 256, 256, 256, 1, 256, 256)
    assert e.value.status == B.NP_ERR_CAPACITY
    assert "8192" in str(e.value)
    ok = B.make_shape(1, 8192, 2000, 16, 100, 200, "bf16")
    with pytest.raises(B.NPError) as e:  # passes the size check, fails on the error word
        B.np_sparse_mlp_noalloc(ok, 0, 256, 256, 256, 1, 256, None)
    assert e.value.status == B.NP_ERR_INVALID_ARG


def test_pinned_host_size(lib):
    """The pinned host size covers the plan copy and a staging area of at
    least four records with their row indices, in whole 4 KiB pages, for a
    small record and for the largest one (d 16384, fp16: 96 KiB)."""
    for kw in (GOOD, dict(GOOD, d_model=16384, capacity=4000)):
        shape = B.make_shape(**kw)
        dev, pinned = B.np_workspace_sizes(shape)
        assert dev == B.np_workspace_size(shape)
        rec = 3 * kw["d_model"] * 2
        plan = kw["layers"] * (4 + 2 * kw["k"]) * 4
        assert pinned % 4096 == 0
        assert pinned >= plan + 4 * rec + 4 * 4
