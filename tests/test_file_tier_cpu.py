"""The storage tier as a file, on the CPU: np_read_records (the io_uring
record reads behind np_stage_file) against the bytes written, with and
without O_DIRECT, for coalesced runs, single records, runs longer than one
read piece, any order and duplicates, at queue depth 1 and 256; and its
errors (a record past the end of the file, a bad descriptor, misaligned
direct reads, a negative id)."""
import mmap
import os

import numpy as np
import pytest

from paper_2608_22643_amd import binding as B
from paper_2608_22643_amd import workload as W

HEAD = 8192  # bytes before the records in the file (a nonzero file_offset)


def aligned(nbytes):
    """A page-aligned host buffer (anonymous mapping) and a uint8 view."""
    m = mmap.mmap(-1, max(nbytes, 1))
    return m, np.frombuffer(m, dtype=np.uint8, count=nbytes)


def ptr(a):
    return a.ctypes.data


@pytest.fixture(scope="module")
def storage_file(tmp_path_factory):
    cfg = W.Config("file", 2, 4096, 300, 8, 0.1, 0.5, "f16", "f16", 4, rho_given=0.5)
    store = W.storage(cfg)  # [2][300][3*4096] uint16: records of 24576 bytes
    path = str(tmp_path_factory.mktemp("tier") / "storage.bin")
    with open(path, "wb") as f:
        f.write(np.arange(HEAD, dtype=np.uint8).tobytes())
        f.write(store.tobytes())
    return cfg, store, path


def open_fd(path, direct):
    flags = os.O_RDONLY | (os.O_DIRECT if direct else 0)
    try:
        return os.open(path, flags)
    except OSError as e:  # a file system without direct I/O
        pytest.skip(f"O_DIRECT not supported here: {e}")


@pytest.mark.parametrize("direct", [False, True])
@pytest.mark.parametrize("qd", ["1", "256"])
def test_read_records_matches_file(storage_file, direct, qd, monkeypatch):
    monkeypatch.setenv("NP_IO_QD", qd)
    cfg, store, path = storage_file
    rec = cfg.record_bytes
    flat = store.reshape(-1, 3 * cfg.d_model)  # records of both layers, in file order
    rng = np.random.default_rng(int(qd) + direct)
    cases = [
        np.sort(rng.choice(flat.shape[0], 40, replace=False)),       # scattered
        np.arange(100, 190),                                          # one 2.1 MiB run
        np.concatenate([np.arange(5, 9), [50], np.arange(290, 310)]),  # runs across layers
        np.array([0]), np.array([flat.shape[0] - 1]),                 # first, last
        rng.permutation(60)[:25],                                     # any order
        np.array([7, 7, 8, 8, 3]),                                    # duplicates
    ]
    fd = open_fd(path, direct)
    try:
        for ids in cases:
            ids = ids.astype(np.int32)
            m, dst = aligned(ids.size * rec)
            B.np_read_records(fd, HEAD, rec, ptr(ids), ids.size, ptr(dst))
            got = dst.view(np.uint16).reshape(ids.size, -1)
            assert np.array_equal(got, flat[ids]), ids[:8]
            del got, dst
            m.close()
        B.np_read_records(fd, HEAD, rec, None, 0, None)  # nothing to read
    finally:
        os.close(fd)


def test_read_records_errors(storage_file):
    cfg, store, path = storage_file
    rec = cfg.record_bytes
    n_rec = store.shape[0] * store.shape[1]
    m, dst = aligned(4 * rec)
    fd = open_fd(path, False)
    try:
        for ids, status in (([n_rec], B.NP_ERR_IO),                  # past the end
                            ([3, n_rec + 5], B.NP_ERR_IO),
                            ([-1], B.NP_ERR_INVALID_ARG)):
            a = np.array(ids, np.int32)
            with pytest.raises(B.NPError) as e:
                B.np_read_records(fd, HEAD, rec, ptr(a), a.size, ptr(dst))
            assert e.value.status == status, ids
    finally:
        os.close(fd)
    a = np.array([0], np.int32)
    with pytest.raises(B.NPError) as e:
        B.np_read_records(fd, HEAD, rec, ptr(a), 1, ptr(dst))  # closed descriptor
    assert e.value.status == B.NP_ERR_INVALID_ARG
    dfd = open_fd(path, True)
    try:
        for off, size, shift in ((HEAD + 8, rec, 0), (HEAD, rec - 8, 0), (HEAD, rec, 8)):
            with pytest.raises(B.NPError) as e:
                B.np_read_records(dfd, off, size, ptr(a), 1, ptr(dst) + shift)
            assert e.value.status == B.NP_ERR_INVALID_ARG
    finally:
        os.close(dfd)
    del dst
    m.close()
