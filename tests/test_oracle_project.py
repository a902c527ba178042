"""Pins for the projection oracle (Alg. 2's k = L2Norm(PCA(h)); the
datastore projection of Sec. 3.2 Eq. 6 with the PCA of the implementation
details): coordinate bases give the centred coordinates; numpy BLAS agrees;
a basis of principal directions decorrelates the data with the eigenvalues
as variances; a full orthonormal basis preserves cosine similarity; unit
norms after normalisation, a row equal to the mean stays zero."""
import numpy as np
import pytest

import oracle


def f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def test_coordinate_basis_gives_centred_coordinates():
    rng = np.random.default_rng(0)
    x = f32(rng.normal(0, 3, (50, 40)))
    mean = rng.normal(0, 1, 40)
    cols = [3, 17, 0, 39, 22]
    basis = np.zeros((5, 40))
    basis[np.arange(5), cols] = 1.0
    y = oracle.project(x, "f32", basis, mean, normalize=False)
    assert np.array_equal(y, x.astype(np.float64)[:, cols] - mean[cols])


@pytest.mark.parametrize("dt", ["f16", "bf16"])
def test_matches_numpy_blas(dt):
    rng = np.random.default_rng(1)
    xf = rng.normal(0, 2, (200, 96)).astype(np.float32)
    import torch
    t = torch.from_numpy(xf).to(torch.float16 if dt == "f16" else torch.bfloat16)
    bits = t.view(torch.int16).numpy().view(np.uint16)
    dec = t.float().numpy().astype(np.float64)
    basis = rng.normal(0, 1, (16, 96))
    mean = rng.normal(0, 0.5, 96)
    y = oracle.project(bits, dt, basis, mean, normalize=True)
    ref = (dec - mean) @ basis.T
    ref /= np.linalg.norm(ref, axis=1, keepdims=True)
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-13)


def test_principal_directions_decorrelate():
    rng = np.random.default_rng(2)
    n, d, v = 4000, 24, 6
    a = rng.normal(0, 1, (d, d))
    x = f32(rng.normal(0, 1, (n, d)) @ a + rng.normal(0, 5, d))
    xd = x.astype(np.float64)
    mean = xd.mean(axis=0)
    cov = (xd - mean).T @ (xd - mean) / n
    w, vecs = np.linalg.eigh(cov)
    top = np.argsort(w)[::-1][:v]
    basis = vecs[:, top].T
    y = oracle.project(x, "f32", basis, mean, normalize=False)
    np.testing.assert_allclose(y.mean(axis=0), 0, atol=1e-9)
    cy = y.T @ y / n
    np.testing.assert_allclose(np.diag(cy), w[top], rtol=1e-9)
    off = cy - np.diag(np.diag(cy))
    assert np.abs(off).max() < 1e-9 * w[top].max()


def test_full_orthonormal_basis_preserves_cosine():
    rng = np.random.default_rng(3)
    d = 32
    q, _ = np.linalg.qr(rng.normal(0, 1, (d, d)))
    x = f32(rng.normal(0, 1, (20, d)))
    mean = rng.normal(0, 1, d)
    y = oracle.project(x, "f32", q.T, mean, normalize=True)
    c = x.astype(np.float64) - mean
    c /= np.linalg.norm(c, axis=1, keepdims=True)
    np.testing.assert_allclose(y @ y.T, c @ c.T, atol=1e-12)


def test_unit_norms_zero_row_and_strides():
    rng = np.random.default_rng(4)
    mean = rng.normal(0, 1, 16).astype(np.float32)
    store = np.full((6, 24), 99.0, dtype=np.float32)       # stride 24, d_in 16
    store[:, :16] = rng.normal(0, 1, (6, 16))
    store[2, :16] = mean                                     # equals the mean
    basis = rng.normal(0, 1, (8, 16))
    y = oracle.project(store, "f32", basis, mean.astype(np.float64), normalize=True,
                       x_stride=24, d_in=16)
    norms = np.linalg.norm(y, axis=1)
    assert np.all(y[2] == 0.0)
    np.testing.assert_allclose(np.delete(norms, 2), 1.0, atol=1e-14)
    y2 = oracle.project(f32(store[:, :16]), "f32", basis, mean.astype(np.float64))
    assert np.array_equal(y, y2)
