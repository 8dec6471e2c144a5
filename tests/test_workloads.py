"""Host-side checks of the seeded workload layouts (no GPU, no oracle)."""
import numpy as np
import pytest

import workloads as W


@pytest.mark.parametrize("name", ["sep-tiny", "sep-4k", "qa-32k", "qa-124k", "docs-124k"])
def test_document_layouts(name):
    w = W.get(name)
    cl = np.asarray(w.chunk_len)
    z = np.asarray(w.zero_kv_chunks)
    # [sep][doc][sep] ... [doc][sep]: separators at even chunk indices
    assert np.array_equal(z, np.arange(0, len(cl), 2))
    assert np.all(cl[z] == 2)
    docs = cl[1::2]
    assert len(docs) == len(z) - 1 and docs.min() >= 16 and docs.max() <= 512
    row0 = np.concatenate([[0], np.cumsum(cl)[:-1]])
    want = np.concatenate([np.arange(row0[i], row0[i] + 2) for i in z])
    assert np.array_equal(w.zero_rows, want)


def test_124k_document_layouts_match_the_headline_shape():
    for name, min_docs in (("qa-124k", 700), ("docs-124k", 200)):
        w = W.get(name)
        assert (w.n_reused, w.n_rows) == (124000, 124256)
        assert len(w.zero_kv_chunks) - 1 > min_docs    # documents


def test_documents_are_seeded():
    a = W.documents("a", 5000, 150.0, 64, 8, 2, seed=3)
    b = W.documents("b", 5000, 150.0, 64, 8, 2, seed=3)
    c = W.documents("c", 5000, 150.0, 64, 8, 2, seed=4)
    assert a.chunk_len == b.chunk_len and a.chunk_len != c.chunk_len
    assert sum(a.chunk_len) == 5000


def test_plain_configs_have_no_zero_rows():
    assert len(W.get("124k").zero_rows) == 0
