"""Pins for the oracle's PCA (Section 4.2: the trunk features are projected to their first 256
principal directions before the K-means).  Exact cases: rows mean +- s_j q_j for an orthonormal
q give the sample mean and covariance in closed form (eigenvalues 2 s_j^2 / (n - 1), vectors
q_j); numpy's cov as the covariance definition; the projection of the mean is zero and a full
projection keeps squared distances (an orthonormal change of basis)."""
import numpy as np


def _symmetric_design(seed, d, s):
    rs = np.random.default_rng(seed)
    Q, _ = np.linalg.qr(rs.normal(size=(d, d)))
    mu = rs.normal(size=d)
    rows = []
    for j, sj in enumerate(s):
        rows += [mu + sj * Q[:, j], mu - sj * Q[:, j]]
    return np.array(rows), mu, Q


def test_closed_form_design(orc):
    d = 12
    s = np.array([9.0, 7.0, 5.5, 4.0, 3.0, 2.0, 1.5, 1.0])
    X, mu, Q = _symmetric_design(1, d, s)
    n = X.shape[0]
    mean, comps, ev = orc.pca(X, 5)
    np.testing.assert_allclose(mean, mu, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(ev, 2 * s[:5] ** 2 / (n - 1), rtol=1e-12)
    for j in range(5):
        assert abs(abs(comps[j] @ Q[:, j]) - 1.0) < 1e-12
        k = np.argmax(np.abs(comps[j]))
        assert comps[j, k] > 0  # sign convention


def test_covariance_definition_and_projection(orc):
    rs = np.random.default_rng(2)
    X = rs.normal(size=(300, 10)) @ rs.normal(size=(10, 10)) + 3.0
    mean, comps, ev = orc.pca(X, 10)
    C = np.cov(X, rowvar=False)
    np.testing.assert_allclose(comps @ C @ comps.T, np.diag(ev), atol=1e-10 * ev[0])
    np.testing.assert_allclose(comps @ comps.T, np.eye(10), atol=1e-12)
    assert np.all(np.diff(ev) <= 0)
    Z = orc.pca_project(X, mean, comps)
    np.testing.assert_allclose(orc.pca_project(mean[None], mean, comps), 0.0, atol=1e-12)
    D = ((X[:, None] - X[None]) ** 2).sum(-1)
    Dz = ((Z[:, None] - Z[None]) ** 2).sum(-1)
    np.testing.assert_allclose(Dz, D, rtol=1e-10)
