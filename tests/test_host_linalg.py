"""The PCA fit's host steps (csrc/host_linalg.hpp: the Cholesky factor behind CholeskyQR with
the inverse of its transpose, and the Householder + implicit-QR symmetric eigensolver), built
with g++ alone and checked against LAPACK through numpy: random, clustered, repeated, diagonal
and tiny matrices, and a non-positive-definite one."""
import os
import shutil
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path_factory.mktemp("hla") / "host_linalg_driver")
    subprocess.run(["g++", "-O2", "-std=c++17", "-pthread", "-I", os.path.join(ROOT, "paper_1704_06363_amd", "csrc"),
                    os.path.join(ROOT, "tests", "host_linalg_driver.cpp"), "-o", exe], check=True)
    return exe


def _run(exe, mode, A):
    n = A.shape[0]
    text = f"{mode} {n}\n" + " ".join("%.17g" % x for x in A.ravel()) + "\n"
    out = subprocess.run([exe], input=text, capture_output=True, text=True, check=True).stdout.split()
    return out


def _matrices():
    rs = np.random.default_rng(5)
    for n in (1, 2, 3, 7, 64, 200):
        M = rs.standard_normal((n, n))
        yield f"random{n}", M + M.T
    Q, _ = np.linalg.qr(rs.standard_normal((50, 50)))
    ev = np.concatenate([np.full(20, 3.0), np.full(20, 1.0), rs.uniform(-1, 1, 10)])
    yield "repeated", (Q * ev) @ Q.T
    ev = 1.0 + 1e-9 * np.arange(40)
    Q, _ = np.linalg.qr(rs.standard_normal((40, 40)))
    yield "clustered", (Q * ev) @ Q.T
    yield "diagonal", np.diag(rs.standard_normal(30))
    yield "zero", np.zeros((5, 5))


@pytest.mark.parametrize("name,A", list(_matrices()), ids=[m[0] for m in _matrices()])
def test_sym_eigen_matches_lapack(driver, name, A):
    n = A.shape[0]
    out = np.array(_run(driver, "eig", A), dtype=np.float64)
    w, VT = out[:n], out[n:].reshape(n, n)
    scale = max(np.abs(A).max(), 1e-300)
    assert np.abs(np.sort(w) - np.linalg.eigvalsh(A)).max() <= 1e-12 * scale
    assert np.abs(VT @ VT.T - np.eye(n)).max() <= 1e-12
    assert np.abs(A @ VT.T - VT.T * w).max() <= 1e-12 * scale  # A v_j = w_j v_j


def test_sym_eigen_reports_non_convergence(driver):
    # allowed a single implicit QR step, a 64 x 64 random matrix cannot deflate: the solver must
    # say so instead of returning its partial result as eigenpairs
    M = np.random.default_rng(9).standard_normal((64, 64))
    assert _run(driver, "eigcap", M + M.T) == ["notconverged"]
    assert _run(driver, "eigcap", np.diag(np.arange(4.0))) == ["converged"]  # already diagonal


@pytest.mark.parametrize("n", [1, 5, 64, 256])
def test_chol_inverse_matches_lapack(driver, n):
    rs = np.random.default_rng(n)
    B = rs.standard_normal((n + 3, n))
    S = B.T @ B  # positive definite, like a Gram matrix Q^T Q
    out = _run(driver, "chol", S)
    assert out[0] == "ok"
    Ri = np.array(out[1:], dtype=np.float64).reshape(n, n)
    R = np.linalg.cholesky(S).T  # S = R^T R
    assert np.allclose(np.tril(Ri, -1), 0.0)
    # R^{-1} up to the tiny diagonal shift the factorisation adds (1e-12 of the mean diagonal)
    np.testing.assert_allclose(Ri @ R, np.eye(n), atol=1e-8)
    Q = B @ Ri  # orthonormal columns: the CholeskyQR step
    np.testing.assert_allclose(Q.T @ Q, np.eye(n), atol=1e-8)


def test_chol_inverse_rejects_indefinite(driver):
    S = np.diag([1.0, -1.0, 2.0])
    assert _run(driver, "chol", S)[0] == "notpd"


def test_chol_inverse_pivot_threshold(driver):
    # a Gram matrix of 8 columns spanning only 5 directions (in fp32 noise): rejected at the
    # 1e-9 relative pivot threshold the PCA fit uses to detect lost rank, accepted without it
    rs = np.random.default_rng(9)
    B = rs.standard_normal((40, 5)) @ rs.standard_normal((5, 8))
    S = (B.T @ B).astype(np.float32).astype(np.float64)
    assert _run(driver, "cholr", S)[0] == "notpd"
    full = rs.standard_normal((40, 8))
    assert _run(driver, "cholr", full.T @ full)[0] == "ok"
