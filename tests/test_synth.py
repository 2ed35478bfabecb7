"""The seeded input generators: shapes, determinism, stated distributions (CPU)."""
import numpy as np

from paper_1612_08608_amd import synth


def test_dense_shard_shape_labels_and_determinism():
    wl = synth.DENSE_LR_32W.with_(samples=512, dim=64, n_workers=3)
    X, y = synth.dense_shard(wl, 1)
    X2, y2 = synth.dense_shard(wl, 1)
    assert X.shape == (512, 64) and X.dtype == np.float32 and y.dtype == np.float32
    assert np.array_equal(X, X2) and np.array_equal(y, y2)
    assert set(np.unique(y)) <= {-1.0, 1.0}
    wstar, scaled = synth.dense_planted(wl)
    assert scaled.size == round(0.1 * 64)
    # scaled columns have ~10x the spread of the others
    assert X[:, scaled].std() > 5 * np.delete(X, scaled, axis=1).std()
    agree = np.mean(np.where(X.astype(np.float64) @ wstar >= 0, 1, -1) == y)
    assert 0.93 < agree < 1.0        # 2% flips


def test_csr_shard_rows_unique_sorted_normalised():
    wl = synth.SPARSE_LR_64W.with_(samples=300, dim=1 << 12)
    rp, col, val, y = synth.csr_shard(wl, 2)
    assert rp[0] == 0 and rp[-1] == col.size and rp.dtype == np.int64 and col.dtype == np.int32
    for r in range(300):
        c = col[rp[r]:rp[r + 1]]
        assert c.size >= 1 and np.all(np.diff(c) > 0) and c.min() >= 0 and c.max() < wl.dim
        assert abs(np.linalg.norm(val[rp[r]:rp[r + 1]].astype(np.float64)) - 1) < 1e-6
    assert set(np.unique(y)) <= {-1.0, 1.0}
    rp2, col2, val2, y2 = synth.csr_shard(wl, 2)
    assert np.array_equal(col, col2) and np.array_equal(val, val2)


def test_csr_binary_values_and_concat_offsets():
    wl = synth.SPARSE_SVM_256W.with_(samples=100, dim=1 << 10, n_workers=3)
    rp, col, val, y = synth.csr_data(wl)
    assert rp.size == 301 and rp[-1] == col.size
    rp1 = synth.csr_shard(wl, 1)[0]
    assert np.array_equal(rp[100:201] - rp[100], rp1)
    for r in range(0, 300, 37):
        v = val[rp[r]:rp[r + 1]]
        assert np.allclose(v, 1 / np.sqrt(v.size), rtol=1e-6)


def test_initial_models_rows_and_column_samples():
    wl = synth.MIX_STRESS_1024W.with_(n_workers=6, dim=1000)
    W = synth.initial_models(wl)
    cols = np.array([3, 999, 0])
    assert np.array_equal(synth.initial_models(wl, rows=[4, 1], cols=cols), W[[4, 1]][:, cols])
    assert abs(W.mean()) < 0.1 and abs(W.std() - 1) < 0.1


