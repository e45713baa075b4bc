"""The storage tier's reader (I/O threads over one file of spans) against the
file's own bytes: span `key` is bytes [key*span, (key+1)*span) of the file."""
import os

import numpy as np
import pytest

import paper_2601_13631_amd as ckv


def _aligned(nbytes, align=4096):
    raw = np.empty(nbytes + align, np.uint8)
    off = (-raw.ctypes.data) % align
    return raw[off:off + nbytes]


@pytest.fixture(scope="module")
def store_file(tmp_path_factory):
    d = tmp_path_factory.mktemp("store")
    span, n = 3 << 20, 12  # 3 MiB spans: runs cross the 4 MiB read pieces
    data = np.random.default_rng(1).integers(0, 256, n * span, dtype=np.uint8)
    path = os.path.join(d, "spans.bin")
    data.tofile(path)
    return path, data, span, n


@pytest.mark.parametrize("threads", [1, 3, 16])
def test_store_reads_file_bytes(store_file, threads):
    path, data, span, n = store_file
    st = ckv.Store(path, n, span, threads)
    rng = np.random.default_rng(threads)
    for keys in ([0], [n - 1], list(range(n)), [4, 5, 6, 1, 2, 9, 9, 0],
                 list(rng.integers(0, n, 20))):
        out = np.zeros(len(keys) * span, np.uint8)
        st.read(keys, out)
        ref = np.concatenate([data[k * span:(k + 1) * span] for k in keys])
        assert np.array_equal(out, ref), keys
    st.close()


def test_store_small_spans_and_direct(tmp_path):
    span, n = 4096, 257
    data = np.random.default_rng(2).integers(0, 256, n * span, dtype=np.uint8)
    path = str(tmp_path / "small.bin")
    data.tofile(path)
    keys = np.array([256, 0, 1, 2, 100, 101, 7], np.int64)
    ref = np.concatenate([data[k * span:(k + 1) * span] for k in keys])
    st = ckv.Store(path, n, span, 4)
    out = np.zeros(keys.size * span, np.uint8)
    st.read(keys, out)
    assert np.array_equal(out, ref)
    st.close()
    try:
        direct = ckv.Store(path, n, span, 4, ckv.STORE_DIRECT)
    except ckv.CkvError:
        pytest.skip("this filesystem refuses O_DIRECT")
    out = _aligned(keys.size * span)
    direct.read(keys, out)
    assert np.array_equal(out, ref)
    odd = _aligned(2 * span)[16:16 + span]  # a destination off the 4096-byte grid
    direct.read(keys[:1], odd)
    assert np.array_equal(odd, ref[:span])
    direct.close()


def test_store_refusals(tmp_path):
    path = str(tmp_path / "short.bin")
    np.zeros(10 * 4096, np.uint8).tofile(path)
    for args in ((path, 11, 4096, 2, 0), (path, 10, 4096, 0, 0), (path, 0, 4096, 2, 0),
                 (path, 10, 4000, 2, ckv.STORE_DIRECT), (path, 10, 4096, 2, 0x8),
                 (str(tmp_path / "missing.bin"), 1, 4096, 1, 0)):
        with pytest.raises(ckv.CkvError) as e:
            ckv.Store(*args)
        assert e.value.status == ckv.EINVAL
    st = ckv.Store(path, 10, 4096, 2)
    with pytest.raises(ckv.CkvError) as e:
        st.read([3, 10], np.zeros(2 * 4096, np.uint8))
    assert e.value.status == ckv.EINVAL
    st.close()
