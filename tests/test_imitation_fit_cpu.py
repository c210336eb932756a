"""The closed-form fit of the imitation network's second layer, against its definition: on
features with an exact linear relation to the targets the ridge solution recovers the matrix and
the bias (up to the small ridge), and it minimises the regularised squared error (no other
solution in a random neighbourhood does better)."""
import numpy as np

from paper_2510_22641_amd import imitation


def _data(seed=0, n=400, h=24, d=16):
    rng = np.random.default_rng(seed)
    phi = rng.normal(size=(n, h))
    xk = rng.normal(size=(n, d))
    A = rng.normal(size=(d, h))
    b = rng.normal(size=d)
    return phi, xk, A, b


def test_recovers_an_exact_linear_relation():
    phi, xk, A, b = _data()
    xl = xk + phi @ A.T + b  # residual form
    w2, b2 = imitation.fit(phi, xk, xl, residual=True, ridge=1e-9)
    assert np.allclose(w2, A, atol=1e-6) and np.allclose(b2, b, atol=1e-6)
    w2n, b2n = imitation.fit(phi, xk, phi @ A.T + b, residual=False, ridge=1e-9)
    assert np.allclose(w2n, A, atol=1e-6) and np.allclose(b2n, b, atol=1e-6)


def test_minimises_the_regularised_error():
    phi, xk, A, b = _data(1)
    rng = np.random.default_rng(7)
    xl = xk + phi @ A.T + b + 0.3 * rng.normal(size=xk.shape)
    ridge = 1e-2
    w2, b2 = imitation.fit(phi, xk, xl, residual=True, ridge=ridge)
    pc = phi - phi.mean(0)
    lam = ridge * np.trace(pc.T @ pc) / phi.shape[1]

    def loss(W, B):
        return np.sum(np.square(xk + phi @ W.T + B - xl)) + lam * np.sum(np.square(W))

    best = loss(w2, b2)
    for _ in range(20):
        dW = 1e-3 * rng.normal(size=w2.shape)
        dB = 1e-3 * rng.normal(size=b2.shape)
        assert loss(w2 + dW, b2 + dB) > best


def test_validated_fit_keeps_a_better_current_layer():
    phi, xk, A, b = _data(2)
    rng = np.random.default_rng(3)
    xl = xk + phi @ A.T + b + 0.1 * rng.normal(size=xk.shape)
    w2, b2, info = imitation.fit_validated(phi, xk, xl, A, b)  # the current layer is the truth
    assert w2 is None and info["val_mse"] >= info["val_mse_configured"]
    w2, b2, info = imitation.fit_validated(phi, xk, xl, 0 * A, 0 * b)
    assert w2 is not None and info["val_mse"] < info["val_mse_configured"]
    assert np.allclose(w2, A, atol=0.05)
