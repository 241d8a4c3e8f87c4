"""Host-side checks of the device ingest entry points (no GPU: every case fails or
sizes before any device call)."""

import numpy as np
import pytest

import paper_1702_06943_amd as T
from workloads import config_batches


def _infos(cfg, first, nb):
    B = config_batches(cfg, first, nb)
    encs = T.toc_encode_batches(B.n_rows, B.n_cols, B.rowptr, B.col, B.val)
    return [T.toc_phys_info_get(T.toc_enc_pack(e)) for e in encs], B.n_cols


def test_workspace_size_grows_with_batches():
    infos, m = _infos("c3", 0, 6)
    full, least = T.toc_ingest_workspace_size(infos, m)
    one_full, one_least = T.toc_ingest_workspace_size(infos[:1], m)
    assert 0 < least <= full and one_least <= one_full
    assert least >= one_least and full > one_full
    # per node and per entry of D the workspace holds at least C' (4 words per
    # node) and the inverted D (one word per entry)
    nodes = sum(f["n_nodes"] for f in infos)
    nd = sum(f["n_codes"] for f in infos)
    assert full >= 16 * nodes + 4 * nd
    assert T.toc_ingest_workspace_size([], m) == (0, 0)


def test_workspace_size_rejects_bad_counts():
    infos, m = _infos("c5", 0, 2)
    bad = dict(infos[0], max_col=m)             # a column of I at n_cols
    with pytest.raises(T.TocError) as e:
        T.toc_ingest_workspace_size([bad, infos[1]], m)
    assert e.value.status == T.TOC_EINVAL
    big = dict(infos[0], n_rows=16385)          # more tuples than C' is built for
    with pytest.raises(T.TocError) as e:
        T.toc_ingest_workspace_size([big], m)
    assert e.value.status == T.TOC_EUNSUPPORTED
    neg = dict(infos[0], n_nodes=0)
    with pytest.raises(T.TocError):
        T.toc_ingest_workspace_size([neg], m)


def test_plan_rejects_bad_offsets_before_device_work():
    infos, m = _infos("c5", 0, 2)
    blobs = np.zeros(16, np.uint8)

    class FakeTensor:       # host bytes standing in for the device blobs: never read
        def __init__(self, a):
            self.a = a

        def numel(self):
            return self.a.size

        def data_ptr(self):
            return self.a.ctypes.data

    with pytest.raises(T.TocError) as e:
        T.toc_ingest_plan(FakeTensor(blobs), np.array([0, 8, 4], np.int64), infos, m, None, 0)
    assert e.value.status == T.TOC_EINVAL
