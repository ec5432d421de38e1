"""Pins of the oracle's two-hidden-layer models (Section 7, Figure 3).

Pinned against PyTorch autograd in float64 (a library routine, not this
oracle) for every activation, the one-hidden-layer oracle (a second layer
with identity weights and an activation that is idempotent on its own
output reduces to it exactly), the Figure 3 example (4-1-2-2 and 4-2-3-2
packed as one network equal each model alone), the W2 = 0 closed form,
central finite differences, and the counter-based initialisation.
"""
import numpy as np
import pytest
import torch

from conftest import load_golden

ACTS = {
    0: lambda t: t,
    1: torch.relu,
    2: torch.tanh,
    3: torch.sigmoid,
    4: lambda t: torch.nn.functional.elu(t, 1.0),
    5: lambda t: torch.nn.functional.leaky_relu(t, 0.01),
    6: lambda t: torch.nn.functional.gelu(t),
    7: torch.nn.functional.silu,
    8: lambda t: torch.nn.functional.softplus(t, 1.0, 20.0),
    9: lambda t: t * torch.sigmoid(2 * t),
    10: torch.nn.functional.selu,
    11: lambda t: torch.nn.functional.hardshrink(t, 0.5),
    12: torch.nn.functional.mish,
}


def _pack(seed, M, F, O, B, hmax=4):
    rng = np.random.default_rng(seed)
    h1 = rng.integers(1, hmax + 1, M).astype(np.int32)
    h2 = rng.integers(1, hmax + 1, M).astype(np.int32)
    N1, N2, K = int(h1.sum()), int(h2.sum()), int((h1 * h2).sum())
    X = rng.standard_normal((B, F)).astype(np.float32)
    y = rng.integers(0, O, B).astype(np.int32)
    W1 = rng.uniform(-0.8, 0.8, (N1, F))
    W12 = rng.uniform(-0.8, 0.8, K)
    W2 = rng.uniform(-0.8, 0.8, (O, N2))
    return h1, h2, X, y, W1, W12, W2


def _blocks(h1, h2):
    o1 = np.concatenate([[0], np.cumsum(h1)])
    o2 = np.concatenate([[0], np.cumsum(h2)])
    ko = np.concatenate([[0], np.cumsum(np.asarray(h1, np.int64) * h2)])
    return o1, o2, ko


def _torch_model(act, X, y, w1, w12, w2):
    """loss and (dW1, dW12, dW2) of one model by autograd in float64."""
    t1 = torch.tensor(w1, requires_grad=True)
    t12 = torch.tensor(w12, requires_grad=True)
    t2 = torch.tensor(w2, requires_grad=True)
    x = torch.tensor(X, dtype=torch.float64)
    f = ACTS[act]
    logits = f(f(x @ t1.T) @ t12.T) @ t2.T
    loss = torch.nn.functional.cross_entropy(logits, torch.tensor(y, dtype=torch.long))
    loss.backward()
    return loss.item(), t1.grad.numpy(), t12.grad.numpy(), t2.grad.numpy()


def test_gradients_match_torch_autograd_for_every_activation(orc):
    F, O, B = 5, 3, 9
    h1, h2, X, y, W1, W12, W2 = _pack(1, 13, F, O, B)
    acts = np.arange(13, dtype=np.int32)
    dW1, dW12, dW2, loss, _, _, ties = orc.deep_gradients(h1, h2, acts, W1, W12, W2, X, y)
    assert ties.sum() == 0
    o1, o2, ko = _blocks(h1, h2)
    for m in range(13):
        w1 = W1[o1[m]:o1[m + 1]]
        w12 = W12[ko[m]:ko[m + 1]].reshape(h2[m], h1[m])
        w2 = W2[:, o2[m]:o2[m + 1]]
        l, g1, g12, g2 = _torch_model(m, X, y, w1, w12, w2)
        assert loss[m] == pytest.approx(l, rel=1e-12)
        np.testing.assert_allclose(dW1[o1[m]:o1[m + 1]], g1, rtol=1e-10, atol=1e-14)
        np.testing.assert_allclose(dW12[ko[m]:ko[m + 1]].reshape(h2[m], h1[m]), g12,
                                   rtol=1e-10, atol=1e-14)
        np.testing.assert_allclose(dW2[:, o2[m]:o2[m + 1]], g2, rtol=1e-10, atol=1e-14)
    logits = orc.deep_forward(h1, h2, acts, W1, W12, W2, X)
    for m in range(13):
        f = ACTS[m]
        w12 = torch.tensor(W12[ko[m]:ko[m + 1]].reshape(h2[m], h1[m]))
        ref = f(f(torch.tensor(X, dtype=torch.float64) @ torch.tensor(W1[o1[m]:o1[m + 1]]).T)
                @ w12.T) @ torch.tensor(W2[:, o2[m]:o2[m + 1]]).T
        np.testing.assert_allclose(logits[:, m, :], ref.numpy(), rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("act", [0, 1])
def test_identity_second_layer_reduces_to_one_hidden_layer(orc, act):
    """W12 = I: Z2 = H1 exactly, and identity / ReLU are idempotent, so the
    two-layer model is the one-layer model of the same W1 and W2 (bit for bit,
    ReLU'(ReLU(z)) = ReLU'(z) included)."""
    F, O, B = 6, 2, 10
    rng = np.random.default_rng(4)
    hs = np.array([3, 1, 5], np.int32)
    X = rng.standard_normal((B, F)).astype(np.float32)
    y = rng.integers(0, O, B).astype(np.int32)
    W1 = rng.uniform(-1, 1, (hs.sum(), F))
    W2 = rng.uniform(-1, 1, (O, hs.sum()))
    W12 = np.concatenate([np.eye(h).ravel() for h in hs])
    acts = np.full(3, act, np.int32)
    d = orc.deep_gradients(hs, hs, acts, W1, W12, W2, X, y)
    s = orc.gradients(hs, acts, W1, W2, X, y)
    np.testing.assert_array_equal(d[0], s[0])
    np.testing.assert_array_equal(d[2], s[1])
    np.testing.assert_array_equal(d[3], s[2])
    # one SGD step (W12 trains too, so later steps differ): W1 and W2 and the
    # loss coincide
    a = orc.deep_train(hs, hs, acts, W1, W12, W2, X, y, [(0, 4)], 0.3)
    b = orc.train(hs, acts, W1, W2, X, y, [(0, 4)], 0.3)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[2], b[1])
    np.testing.assert_array_equal(a[3], b[2])


def test_figure3_pack_equals_each_model_alone(orc):
    g = load_golden("deep_packing_example.json")
    h1, h2 = np.asarray(g["h1"], np.int32), np.asarray(g["h2"], np.int32)
    assert (h1.sum(), h2.sum(), 2 * g["O"]) == (g["packed_hidden1"], g["packed_hidden2"],
                                                g["packed_outputs"])
    rng = np.random.default_rng(11)
    F, O, B = g["F"], g["O"], 7
    X = rng.standard_normal((B, F)).astype(np.float32)
    y = rng.integers(0, O, B).astype(np.int32)
    W1, W12, W2 = orc.deep_init(F, O, h1, h2, 99)
    o1, o2, ko = _blocks(h1, h2)
    for act in range(13):
        acts = np.full(2, act, np.int32)
        pack = orc.deep_gradients(h1, h2, acts, W1, W12, W2, X, y)
        for m in range(2):
            one = orc.deep_gradients(h1[m:m + 1], h2[m:m + 1], acts[m:m + 1],
                                     W1[o1[m]:o1[m + 1]], W12[ko[m]:ko[m + 1]],
                                     W2[:, o2[m]:o2[m + 1]], X, y)
            np.testing.assert_array_equal(one[0], pack[0][o1[m]:o1[m + 1]])
            np.testing.assert_array_equal(one[1], pack[1][ko[m]:ko[m + 1]])
            np.testing.assert_array_equal(one[2], pack[2][:, o2[m]:o2[m + 1]])
            assert one[3][0] == pack[3][m]


def test_zero_output_weights_give_log_O(orc):
    h1, h2, X, y, W1, W12, W2 = _pack(5, 6, 4, 10, 8)
    acts = np.arange(6, dtype=np.int32)
    dW1, dW12, dW2, loss, _, _, _ = orc.deep_gradients(h1, h2, acts, W1, W12, np.zeros_like(W2), X, y)
    np.testing.assert_allclose(loss, np.log(10.0), rtol=1e-15)
    assert np.all(dW1 == 0.0) and np.all(dW12 == 0.0)


def test_finite_differences_of_the_summed_loss(orc):
    F, O, B = 3, 3, 6
    h1, h2, X, y, W1, W12, W2 = _pack(7, 4, F, O, B, hmax=3)
    acts = np.array([2, 3, 6, 12], np.int32)        # smooth
    dW1, dW12, dW2, _, _, _, _ = orc.deep_gradients(h1, h2, acts, W1, W12, W2, X, y)

    def total(a1, a12, a2):
        return orc.deep_gradients(h1, h2, acts, a1, a12, a2, X, y)[3].sum()

    eps = 1e-6
    for arr, grad, idx in ((W1, dW1, 0), (W12, dW12, 1), (W2, dW2, 2)):
        for i in np.ndindex(arr.shape):
            p, q = arr.copy(), arr.copy()
            p[i] += eps
            q[i] -= eps
            args_p = [W1, W12, W2]
            args_q = [W1, W12, W2]
            args_p[idx], args_q[idx] = p, q
            fd = (total(*args_p) - total(*args_q)) / (2 * eps)
            assert abs(fd - grad[i]) <= 1e-7 * max(1.0, abs(fd))


def test_init_streams(orc):
    """W1 is the one-layer stream over N1 rows; W12 entry k of model m is
    (2u - 1) * (1 / sqrt(h1_m)) with u from splitmix64 under tag 5 and index
    k (the packed block offset plus i h1_m + j)."""
    h1 = np.array([3, 1, 4], np.int32)
    h2 = np.array([2, 5, 1], np.int32)
    W1, W12, W2 = orc.deep_init(7, 3, h1, h2, 1234)
    R1, _ = orc.init_params(7, 3, h1, 1234)
    np.testing.assert_array_equal(W1, R1)
    key = orc.splitmix64(1234)
    ko = np.concatenate([[0], np.cumsum(h1 * h2)])
    for m in range(3):
        bound = np.float32(1.0 / np.sqrt(float(h1[m])))
        for k in range(ko[m], ko[m + 1]):
            r = orc.splitmix64(key ^ (5 << 60) ^ k)
            u = (r >> 40) * 2.0 ** -24
            assert W12[k] == np.float32(np.float32(2 * u - 1) * bound)
    # W2 over the N2 second-layer units, fan_in h2_m
    N2 = int(h2.sum())
    for n in (0, 2, 7):
        m = np.searchsorted(np.cumsum(h2), n, side="right")
        r = orc.splitmix64(key ^ (2 << 60) ^ (1 * N2 + n))
        u = (r >> 40) * 2.0 ** -24
        assert W2[1, n] == np.float32(np.float32(2 * u - 1) * np.float32(1 / np.sqrt(float(h2[m]))))


def test_kink_allowance_of_the_second_layer(orc):
    """A second-layer ReLU unit whose Z2 sits exactly on the kink: the
    gradients with the other one-sided derivative stay within the allowance
    (dW12 directly, dW1 through W12 and the first layer)."""
    X = np.array([[1.0, 0.5], [0.3, -1.0], [-0.7, 0.2]], np.float32)
    y = np.array([0, 1, 1], np.int32)
    W1 = np.array([[0.5, 0.25], [0.4, -0.2]])          # Z1[0] = (0.625, 0.3)
    H1 = np.maximum(X[0].astype(np.float64) @ W1.T, 0)
    W12 = np.array([H1[1], -H1[0]]) * 0.5              # Z2[0] = H1 . W12 = 0 exactly
    assert H1 @ W12 == 0.0
    W2 = np.array([[0.7], [-0.4]])
    h = np.array([2], np.int32), np.array([1], np.int32)
    d = orc.deep_gradients(h[0], h[1], [1], W1, W12, W2, X, y)
    # the other branch at sample 0: dZ2[0] = dH2[0] instead of 0
    L = orc.deep_forward(h[0], h[1], [1], W1, W12, W2, X)[:, 0, :]
    P = np.exp(L - L.max(1, keepdims=True))
    P /= P.sum(1, keepdims=True)
    G = (P - np.eye(2)[y]) / 3
    dH2 = G[0] @ W2[:, 0]
    other12 = dH2 * H1                               # change of dW12 (row 0)
    Z1 = X[0].astype(np.float64) @ W1.T
    other1 = np.outer(dH2 * W12 * (Z1 > 0), X[0].astype(np.float64))
    assert np.all(d[5] >= np.abs(other12) * (1 - 1e-12))
    assert np.all(d[4] >= np.abs(other1) * (1 - 1e-12))
