"""The planted-structure generator of the time-to-accuracy runs: seeded,
well-formed, and carrying a label signal that a simple classifier can read
(so top-1 accuracy is learnable), unlike the workload draws."""
import numpy as np

from paper_2110_07029_amd import synth


def _signatures(p):
    rng = np.random.default_rng(p.seed)
    fz = synth._BoundedZipf(p.n_features, p.feat_zipf, rng)
    return fz.draw(p.n_labels * p.sig, rng).reshape(p.n_labels, p.sig)


def test_planted_rows_are_well_formed_and_seeded():
    p = synth.PLANTED_SMALL
    a, b = synth.generate_planted(p, 500), synth.generate_planted(p, 500)
    assert np.array_equal(a.x.indices, b.x.indices) and np.array_equal(a.y.indices, b.y.indices)
    for m, n_cols in ((a.x, p.n_features), (a.y, p.n_labels)):
        ip = m.indptr
        assert ip[0] == 0 and np.all(np.diff(ip) >= 1) and m.indices.max() < n_cols
        for i in range(m.n_rows):
            assert np.all(np.diff(m.indices[ip[i]:ip[i + 1]]) > 0)      # sorted, distinct
    norms = np.sqrt(np.bincount(np.repeat(np.arange(500), np.diff(a.x.indptr)), weights=a.x.values ** 2))
    assert np.allclose(norms, 1.0, atol=1e-6)
    held = synth.generate_planted(p, 500, seed_offset=1)
    assert not np.array_equal(held.x.indices[:50], a.x.indices[:50])


def test_planted_labels_are_readable_from_features():
    # score each label by how many of its distinct signature features a row has: the best
    # label is one of the row's labels far more often than the most frequent label is
    p = synth.PLANTED_SMALL
    ds = synth.generate_planted(p, 1500, seed_offset=1)
    sig = _signatures(p)
    owner = {}
    for l in range(p.n_labels):
        for f in set(sig[l].tolist()):          # a signature may draw a hot feature twice
            owner.setdefault(int(f), []).append(l)
    hit = 0
    for i in range(ds.x.n_rows):
        score = np.zeros(p.n_labels)
        for f in ds.x.indices[ds.x.indptr[i]:ds.x.indptr[i + 1]]:
            for l in owner.get(int(f), ()):
                score[l] += 1
        hit += int(np.argmax(score) in set(ds.y.indices[ds.y.indptr[i]:ds.y.indptr[i + 1]]))
    top = np.bincount(ds.y.indices, minlength=p.n_labels).argmax()
    prior = np.mean([top in set(ds.y.indices[ds.y.indptr[i]:ds.y.indptr[i + 1]]) for i in range(ds.x.n_rows)])
    assert hit / ds.x.n_rows > 0.7 > prior + 0.3
