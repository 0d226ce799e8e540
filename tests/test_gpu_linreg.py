"""The Sec. 6.1 recovery experiment on the GPU, through the autograd
wrapper (qualitative: the paper prints no numbers for it, only Fig. 3).

With the identity initialisation, a deeper cascade fits the operator better;
with the small N(0, 1e-6) initialisation, an 8-layer cascade does not train
at all (its gradients are products of near-zero diagonals).  The thresholds
leave wide margins around a float64 CPU re-implementation of the same
training run (identity: K=1 0.62, K=8 0.20; small, K=8: 70.5 after 800
steps)."""

import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def prob():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_1511_05946_amd import linreg
    X, Y = linreg.problem(0, torch.device("cuda:0"))
    return linreg, X, Y


def test_identity_init_improves_with_depth(prob):
    linreg, X, Y = prob
    print("[case] linreg identity K=1, K=8, 800 steps", flush=True)
    _, _, h1 = linreg.train(X, Y, 1, "identity", steps=800)
    _, _, h8 = linreg.train(X, Y, 8, "identity", steps=800)
    print(f"[case]   K=1 {h1[0][1]:.4g} -> {h1[-1][1]:.4g}; K=8 {h8[0][1]:.4g} -> {h8[-1][1]:.4g}", flush=True)
    assert h8[-1][1] < 0.05 * h8[0][1]
    assert h8[-1][1] < 0.6 * h1[-1][1]
    assert h1[-1][1] < 1.0


def test_small_init_does_not_train_deep_cascades(prob):
    linreg, X, Y = prob
    print("[case] linreg small init K=8, 800 steps", flush=True)
    _, _, h = linreg.train(X, Y, 8, "small", steps=800)
    print(f"[case]   K=8 {h[0][1]:.4g} -> {h[-1][1]:.4g}", flush=True)
    assert h[-1][1] > 0.5 * h[0][1]
