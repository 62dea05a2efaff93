"""The native reader of repository-format dataset files (host code of the
library; no GPU): round trip of a synthetic dataset, 1-based ids, files
without a header, and the error paths."""
import numpy as np
import pytest

import paper_2110_07029_amd as asgd
from paper_2110_07029_amd import libsvm, synth


def test_round_trip_of_a_synthetic_dataset(tmp_path):
    ds = synth.generate(synth.TINY, n_samples=300)
    p = tmp_path / "tiny.txt"
    libsvm.save(ds, str(p))
    got = libsvm.load(str(p))
    assert (got.x.n_cols, got.y.n_cols) == (synth.TINY.n_features, synth.TINY.n_labels)
    for a, b in ((got.x, ds.x), (got.y, ds.y)):
        assert np.array_equal(a.indptr, b.indptr) and np.array_equal(a.indices, b.indices)
    assert np.array_equal(got.x.values, ds.x.values)      # %.9g round-trips float32 exactly


def test_one_based_ids_unsorted_rows_and_no_header(tmp_path):
    p = tmp_path / "small.txt"
    p.write_text("# a comment\n3,1 5:0.5 2:0.25\n\n 7 1:1\n2 3:2 4:3\n")
    info = asgd.asgd_libsvm_scan(str(p), one_based=True)
    assert (info.n_rows, info.nnz, info.label_nnz, info.header_rows) == (3, 5, 4, -1)
    assert (info.n_features, info.n_labels) == (5, 8)      # one past the largest id (shifted)
    ds = libsvm.load(str(p), one_based=True)
    assert ds.x.indptr.tolist() == [0, 2, 3, 5] and ds.x.indices.tolist() == [1, 4, 0, 2, 3]
    assert ds.x.values.tolist() == [0.25, 0.5, 1.0, 2.0, 3.0]
    assert ds.y.indptr.tolist() == [0, 2, 3, 4] and ds.y.indices.tolist() == [1, 3, 7, 2]


def test_rows_without_labels_or_features(tmp_path):
    # a row with no features is a valid batch row (A1 = b1); a row with no labels
    # is not (the loss is undefined), so it is dropped by default
    p = tmp_path / "e.txt"
    p.write_text("3 10 4\n 3:1.5\n1,2\n0 4:1 5:2\n")
    ds = libsvm.load(str(p))
    assert ds.x.n_rows == 2 and ds.workload.n_samples == 2
    assert ds.x.indptr.tolist() == [0, 0, 2] and ds.x.indices.tolist() == [4, 5]
    assert ds.y.indptr.tolist() == [0, 2, 3] and ds.y.indices.tolist() == [1, 2, 0]
    kept = libsvm.load(str(p), unlabeled="keep")
    assert kept.x.indptr.tolist() == [0, 1, 1, 3] and kept.y.indptr.tolist() == [0, 0, 2, 3]
    with pytest.raises(ValueError, match="1 rows have no labels"):
        libsvm.load(str(p), unlabeled="error")


@pytest.mark.parametrize("text,what", [
    ("1 2:x\n", "bad feature value"),
    ("1;2 3:1\n", "labels must be separated"),
    ("1 3:1 3:2\n", "repeated feature id"),
    ("1,1 3:1\n", "repeated label id"),
    ("2 5 3\n0 7:1\n1 1:1\n", "exceeds the header"),
    ("3 5 3\n0 1:1\n", "row count"),
])
def test_malformed_files_are_rejected_with_the_reason(tmp_path, text, what):
    p = tmp_path / "bad.txt"
    p.write_text(text)
    with pytest.raises(asgd.AsgdError) as e:
        libsvm.load(str(p))
    assert what in str(e.value)


def test_missing_file(tmp_path):
    with pytest.raises(asgd.AsgdError):
        asgd.asgd_libsvm_scan(str(tmp_path / "none.txt"))
