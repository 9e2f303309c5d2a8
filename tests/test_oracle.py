"""Pins of the CPU oracle against facts that do not come from the oracle.

The oracle is the plain fp64 definition of Algorithm 1 (inference) and
Algorithm 2 (training step), arXiv 2403.17607 section III-A.  Each test below
checks it against a library routine, a closed form, a hand derivation, an
invariant of the mathematics, or finite differences, chosen so that a dropped
term, a wrong sign, a wrong index or a transposed operand fails one of them.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import LINEAR, RELU, SIGMOID, SINE, Net

RNG = np.random.default_rng(12345)


def bf16_exact(a):
    """Round an array to bf16 values with torch (fp32 -> bf16 library
    conversion); used only to make test inputs bf16-exact."""
    t = torch.as_tensor(np.asarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float64).numpy()


def rand_net_inputs(net: Net, M: int, rng=RNG, scale=1.0):
    W = bf16_exact(rng.uniform(-scale, scale, net.param_count()))
    X = bf16_exact(rng.uniform(-1, 1, (M, net.in_dim)))
    T = rng.uniform(-1, 1, (M, net.out_dim)).astype(np.float32).astype(np.float64)
    return W, X, T


# --------------------------------------------------------------- rounding ---

def test_rne_bf16_matches_torch_on_fp32_values():
    """fp32 values: direct fp64->bf16 rounding equals torch's fp32->bf16."""
    vals = np.concatenate([
        RNG.standard_normal(20000).astype(np.float32),
        (RNG.standard_normal(5000) * 1e-38).astype(np.float32),   # subnormal range
        (RNG.standard_normal(5000) * 1e30).astype(np.float32),
        np.array([0.0, -0.0, 1.0, -1.0, 3.3895314e38, -3.3895314e38,
                  3.3961e38, 1e-45, -1e-45, 2.0 ** -126, 2.0 ** -133,
                  3 * 2.0 ** -134, 2.0 ** -134], dtype=np.float32),
    ])
    ref = torch.as_tensor(vals).to(torch.bfloat16).to(torch.float64).numpy()
    got = np.array([oracle.rne_bf16(float(v)) for v in vals])
    np.testing.assert_array_equal(got, ref)


def test_rne_bf16_ties_and_fp64_only_values():
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: ties go to the even (1.0).
    assert oracle.rne_bf16(1 + 2.0 ** -8) == 1.0
    # 1 + 3*2^-8 is halfway between 1 + 2^-7 (odd) and 1 + 2^-6 (even).
    assert oracle.rne_bf16(1 + 3 * 2.0 ** -8) == 1 + 2.0 ** -6
    # Just above a tie rounds up; fp32 could not even see the extra bit.
    assert oracle.rne_bf16(1 + 2.0 ** -8 + 2.0 ** -40) == 1 + 2.0 ** -7
    assert oracle.rne_bf16(-(1 + 2.0 ** -8 + 2.0 ** -40)) == -(1 + 2.0 ** -7)
    # Values beyond the largest finite bf16 by at least half an ulp overflow.
    assert math.isinf(oracle.rne_bf16(2.0 ** 128))
    assert oracle.rne_bf16(255.0 * 2.0 ** 120) == 255.0 * 2.0 ** 120
    assert math.isinf(oracle.rne_bf16(255.5 * 2.0 ** 120))
    # The smallest bf16 subnormal is 2^-133; half of it ties to zero.
    assert oracle.rne_bf16(2.0 ** -133) == 2.0 ** -133
    assert oracle.rne_bf16(2.0 ** -134) == 0.0
    assert oracle.rne_bf16(1.5 * 2.0 ** -133) == 2.0 ** -132


# --------------------------------------------------------- forward pins ---

@pytest.mark.parametrize("out_act", [LINEAR, SIGMOID, SINE, RELU])
def test_depth0_forward_is_one_gemm(out_act):
    """With no hidden layer, Algorithm 1 is sigma_out(X W_1): a library
    matmul in fp64 (bf16 products are exact in fp64)."""
    net = Net(width=64, depth=0, in_dim=48, out_dim=24, out_act=out_act)
    W, X, _ = rand_net_inputs(net, 300)
    _, Y32 = net.forward(W, X)
    C = X @ W.reshape(48, 24)
    ref = {LINEAR: C, RELU: np.maximum(C, 0), SIGMOID: 1 / (1 + np.exp(-C)),
           SINE: np.sin(C)}[out_act]
    np.testing.assert_allclose(Y32, ref, rtol=1e-13, atol=1e-14)


@pytest.mark.parametrize("out_act", [LINEAR, SIGMOID, RELU, SINE])
def test_depth0_gradient_is_one_gemm(out_act):
    """Depth 0, no rounding: G_1 = X^T D with D = 2 (Y - T) / (M out)
    times sigma_out'(C), C = X W_1 -- one library matmul.  The derivatives
    are written out here: y (1 - y) for sigmoid, [C > 0] for ReLU (0 at the
    kink), cos C for sine."""
    net = Net(width=32, depth=0, in_dim=20, out_dim=12, out_act=out_act,
              round_bf16=False)
    W, X, T = rand_net_inputs(net, 257)
    r = net.train_step(W, X, T)
    Y = r["Y32"]
    C = X @ W.reshape(20, 12)
    D = 2 * (Y - T) / (X.shape[0] * net.out_dim)
    if out_act == SIGMOID:
        D = D * Y * (1 - Y)
    elif out_act == RELU:
        assert 0 < np.mean(C > 0) < 1
        D = D * (C > 0)
    elif out_act == SINE:
        D = D * np.cos(C)
    np.testing.assert_allclose(r["G"].reshape(20, 12), X.T @ D, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(r["loss"], np.mean((Y - T) ** 2), rtol=1e-12)


@pytest.mark.parametrize("depth", [1, 3])
def test_identity_weights_give_relu_bitwise(depth):
    w = 16
    net = Net(width=w, depth=depth, in_dim=w, out_dim=w)
    W = np.concatenate([np.eye(w).ravel()] * net.L)
    _, X, _ = rand_net_inputs(net, 100)
    Y, _ = net.forward(W, X)
    np.testing.assert_array_equal(Y, np.maximum(X, 0))


@pytest.mark.parametrize("act", [RELU, SINE, LINEAR])
def test_zero_input_gives_zero_output_and_gradient(act):
    net = Net(width=8, depth=2, in_dim=5, out_dim=3, act=act)
    W, _, T = rand_net_inputs(net, 7)
    X = np.zeros((7, 5))
    r = net.train_step(W, X, T)
    np.testing.assert_array_equal(r["Y"], 0.0)
    np.testing.assert_array_equal(r["G"], 0.0)


def test_zero_input_sigmoid_output_is_one_half():
    net = Net(width=8, depth=2, in_dim=5, out_dim=3, out_act=SIGMOID)
    W, _, _ = rand_net_inputs(net, 7)
    Y, Y32 = net.forward(W, np.zeros((7, 5)))
    np.testing.assert_array_equal(Y32, 0.5)
    np.testing.assert_array_equal(Y, 0.5)


@pytest.mark.parametrize("act", [RELU, LINEAR])
@pytest.mark.parametrize("k", [3, -2])
def test_power_of_two_homogeneity_bitwise(act, k):
    """No bias and a positively homogeneous activation: scaling X or one
    weight matrix by 2^k scales Y (and G, for a fixed dY) by 2^k exactly."""
    net = Net(width=16, depth=3, in_dim=10, out_dim=6, act=act)
    W, X, _ = rand_net_inputs(net, 64)
    Y, _ = net.forward(W, X)
    Ys, _ = net.forward(W, X * 2.0 ** k)
    np.testing.assert_array_equal(Ys, Y * 2.0 ** k)
    Wl = net.split(W.copy())
    Wl[2] *= 2.0 ** k
    Yw, _ = net.forward(np.concatenate([m.ravel() for m in Wl]), X)
    np.testing.assert_array_equal(Yw, Y * 2.0 ** k)
    dY = bf16_exact(RNG.uniform(-1, 1, Y.shape))
    G = net.backward(W, X, dY)
    Gs = net.backward(W, X * 2.0 ** k, dY)
    np.testing.assert_array_equal(Gs, G * 2.0 ** k)


def test_row_permutation():
    net = Net(width=32, depth=2, in_dim=32, out_dim=16, act=SIGMOID)
    W, X, T = rand_net_inputs(net, 200)
    perm = RNG.permutation(200)
    r1 = net.train_step(W, X, T)
    r2 = net.train_step(W, X[perm], T[perm])
    np.testing.assert_array_equal(r2["Y"], r1["Y"][perm])
    np.testing.assert_allclose(r2["G"], r1["G"], rtol=1e-12, atol=1e-15)


# ------------------------------------------------------------ brute force ---

DY = [-1.0, -0.5, 0.0, 0.5, 1.0]
DW = [-1.0, -0.5, 0.5, 1.0]


def test_bruteforce_2x2_relu_net_exact():
    """Width 2, one hidden ReLU layer, linear output, one row.  Every
    quantity is dyadic with few bits, so bf16 rounding is exact and the
    oracle must equal these hand-derived scalar formulas exactly:
        h_j  = relu(x_0 W1[0,j] + x_1 W1[1,j])
        y_j  = h_0 W2[0,j] + h_1 W2[1,j]
        e_j  = 2 (y_j - t_j) / (M * out) = y_j - t_j   (M * out = 2)
        G2[i,j] = h_i e_j
        d_i  = (e_0 W2[i,0] + e_1 W2[i,1]) * [h_i > 0]
        G1[i,j] = x_i d_j
    """
    net = Net(width=2, depth=1, in_dim=2, out_dim=2)
    rng = np.random.default_rng(7)
    for _ in range(1500):
        x = rng.choice(DY, 2)
        t = rng.choice(DY, 2)
        A = rng.choice(DW, (2, 2))
        B = rng.choice(DW, (2, 2))
        h = [max(x[0] * A[0, j] + x[1] * A[1, j], 0.0) for j in range(2)]
        y = [h[0] * B[0, j] + h[1] * B[1, j] for j in range(2)]
        e = [y[j] - t[j] for j in range(2)]
        G2 = [[h[i] * e[j] for j in range(2)] for i in range(2)]
        d = [(e[0] * B[i, 0] + e[1] * B[i, 1]) * (1.0 if h[i] > 0 else 0.0)
             for i in range(2)]
        G1 = [[x[i] * d[j] for j in range(2)] for i in range(2)]
        loss = ((y[0] - t[0]) ** 2 + (y[1] - t[1]) ** 2) / 2
        W = np.concatenate([A.ravel(), B.ravel()])
        r = net.train_step(W, x[None, :], t[None, :])
        assert r["Y"][0].tolist() == y
        assert r["G"].tolist() == sum(G1, []) + sum(G2, [])
        assert r["loss"] == loss


# -------------------------------------------------------- finite differences

FD_CASES = [
    # (width, depth, in, out, act, out_act)
    (2, 0, 2, 2, LINEAR, LINEAR),
    (3, 1, 2, 3, SINE, LINEAR),
    (4, 2, 3, 2, SIGMOID, SIGMOID),
    (3, 3, 4, 1, SINE, SINE),
    (4, 2, 4, 3, RELU, LINEAR),
    (2, 1, 3, 2, LINEAR, SIGMOID),
    (3, 2, 3, 2, RELU, RELU),
    (4, 1, 2, 3, SIGMOID, RELU),
]


def away_from_relu_kinks(net, W, X, margin=1e-3):
    """True when every pre-activation that goes through a ReLU (hidden or
    output) is at least `margin` away from 0, so central differences with a
    step of 1e-6 never cross a kink."""
    acts = {LINEAR: lambda c: c, RELU: lambda c: np.maximum(c, 0), SIGMOID: lambda c: 1 / (1 + np.exp(-c)),
            SINE: np.sin}
    A = X
    mats = net.split(W)
    for l, Wl in enumerate(mats):
        C = A @ Wl
        a = net.act if l < len(mats) - 1 else net.out_act
        if a == RELU and np.min(np.abs(C)) < margin:
            return False
        A = acts[a](C)
    return True


@pytest.mark.parametrize("case", FD_CASES)
def test_gradient_matches_finite_differences(case):
    width, depth, in_dim, out_dim, act, out_act = case
    net = Net(width, depth, in_dim, out_dim, act, out_act, round_bf16=False)
    rng = np.random.default_rng(hash(case) % 2**32)
    M = 6
    W = rng.uniform(-1, 1, net.param_count())
    X = rng.uniform(-1, 1, (M, in_dim))
    T = rng.uniform(-1, 1, (M, out_dim))
    if RELU in (act, out_act):
        # stay away from the kinks: every ReLU pre-activation |c| > 1e-3
        for _ in range(200):
            ok = away_from_relu_kinks(net, W, X)
            if ok:
                break
            W = rng.uniform(-1, 1, net.param_count())
        assert ok
    G = net.train_step(W, X, T)["G"]
    h = 1e-6
    fd = np.zeros_like(W)
    for i in range(W.size):
        Wp, Wm = W.copy(), W.copy()
        Wp[i] += h
        Wm[i] -= h
        fd[i] = (net.train_step(Wp, X, T)["loss"] - net.train_step(Wm, X, T)["loss"]) / (2 * h)
    scale = np.max(np.abs(G))
    np.testing.assert_allclose(G, fd, rtol=1e-6, atol=1e-8 * scale)

    # Backward seeded with an arbitrary dY: G is the gradient of sum(dY * Y).
    dY = rng.uniform(-1, 1, (M, out_dim))
    Gb = net.backward(W, X, dY)
    fdb = np.zeros_like(W)
    for i in range(W.size):
        Wp, Wm = W.copy(), W.copy()
        Wp[i] += h
        Wm[i] -= h
        fp = np.sum(dY * net.forward(Wp, X)[1])
        fm = np.sum(dY * net.forward(Wm, X)[1])
        fdb[i] = (fp - fm) / (2 * h)
    np.testing.assert_allclose(Gb, fdb, rtol=1e-6, atol=1e-8 * np.max(np.abs(Gb)))


# ----------------------------------------------------------- input gradient

@pytest.mark.parametrize("case", FD_CASES)
def test_input_gradient_matches_finite_differences(case):
    """dX (an extension beyond Algorithm 2) is the gradient of sum(dY * Y)
    with respect to X, checked by central differences with rounding off;
    G from backward_dx equals G from backward."""
    width, depth, in_dim, out_dim, act, out_act = case
    net = Net(width, depth, in_dim, out_dim, act, out_act, round_bf16=False)
    rng = np.random.default_rng((hash(case) + 7) % 2**32)
    M = 5
    W = rng.uniform(-1, 1, net.param_count())
    X = rng.uniform(-1, 1, (M, in_dim))
    if RELU in (act, out_act):
        for _ in range(200):
            ok = away_from_relu_kinks(net, W, X)
            if ok:
                break
            X = rng.uniform(-1, 1, (M, in_dim))
        assert ok
    dY = rng.uniform(-1, 1, (M, out_dim))
    G, dX = net.backward_dx(W, X, dY)
    np.testing.assert_array_equal(G, net.backward(W, X, dY))
    h = 1e-6
    fd = np.zeros_like(X)
    for r in range(M):
        for k in range(in_dim):
            Xp, Xm = X.copy(), X.copy()
            Xp[r, k] += h
            Xm[r, k] -= h
            fd[r, k] = (np.sum(dY * net.forward(W, Xp)[1]) - np.sum(dY * net.forward(W, Xm)[1])) / (2 * h)
    np.testing.assert_allclose(dX, fd, rtol=1e-6, atol=1e-8 * np.max(np.abs(dX)))


@pytest.mark.parametrize("out_act", [LINEAR, SIGMOID])
def test_depth0_input_gradient_is_one_gemm(out_act):
    """Depth 0, no rounding: dX = (dY * sigma_out'(C)) W^T, one library
    matmul."""
    net = Net(width=32, depth=0, in_dim=20, out_dim=12, out_act=out_act, round_bf16=False)
    W, X, _ = rand_net_inputs(net, 129)
    dY = RNG.uniform(-1, 1, (129, 12))
    _, dX = net.backward_dx(W, X, dY)
    Wm = W.reshape(20, 12)
    D = dY
    if out_act == SIGMOID:
        Y = 1 / (1 + np.exp(-(X @ Wm)))
        D = dY * Y * (1 - Y)
    np.testing.assert_allclose(dX, D @ Wm.T, rtol=1e-12, atol=1e-15)


def test_identity_net_input_gradient_closed_form():
    """Identity weights, ReLU hidden, linear output, rounding on: every
    hidden delta is bf16(dY) masked by [X > 0], so dX = bf16(dY) [X > 0]
    exactly."""
    w, depth, M = 8, 3, 16
    net = Net(width=w, depth=depth, in_dim=w, out_dim=w)
    W = np.concatenate([np.eye(w).ravel()] * net.L)
    _, X, _ = rand_net_inputs(net, M)
    dY = RNG.uniform(-1, 1, (M, w))
    _, dX = net.backward_dx(W, X, dY)
    rne = np.vectorize(oracle.rne_bf16)
    np.testing.assert_array_equal(dX, rne(dY) * (X > 0))


def test_input_gradient_is_unrounded_product_of_first_delta():
    """Rounding on: dX is the first hidden layer's (rounded, separately
    pinned) delta times W_1^T, kept in fp64 (not rounded to bf16)."""
    net = Net(width=16, depth=2, in_dim=12, out_dim=5, act=SIGMOID)
    W, X, _ = rand_net_inputs(net, 40)
    dY = RNG.uniform(-1, 1, (40, 5))
    G, D = net.backward(W, X, dY, want_deltas=True)
    _, dX = net.backward_dx(W, X, dY)
    ref = D[0] @ net.split(W)[0].T
    np.testing.assert_allclose(dX, ref, rtol=1e-13, atol=1e-18)
    rne = np.vectorize(oracle.rne_bf16)
    assert np.any(rne(dX) != dX)


# ------------------------------------------------------- closed-form deltas

def test_identity_net_deltas_closed_form():
    """Identity weights, ReLU hidden, linear output:
    D_{L+1} = bf16(2 (relu(X) - T) / (M out)); every hidden delta is
    D_{L+1} masked by [X > 0]; G_1 = X^T D_2 and G_l = relu(X)^T D_{l+1}."""
    w, depth, M = 8, 3, 16
    net = Net(width=w, depth=depth, in_dim=w, out_dim=w)
    W = np.concatenate([np.eye(w).ravel()] * net.L)
    _, X, T = rand_net_inputs(net, M)
    r = net.train_step(W, X, T, want_deltas=True)
    R = np.maximum(X, 0)
    rne = np.vectorize(oracle.rne_bf16)
    Dout = rne(2 * (R - T) / (M * w))
    np.testing.assert_array_equal(r["D"][-1], Dout)
    mask = (X > 0).astype(np.float64)
    for Dl in r["D"][:-1]:
        np.testing.assert_array_equal(Dl, Dout * mask)
    G = net.split(r["G"])
    np.testing.assert_allclose(G[0], X.T @ (Dout * mask), rtol=1e-12, atol=1e-18)
    for l in range(1, net.L - 1):
        np.testing.assert_allclose(G[l], R.T @ (Dout * mask), rtol=1e-12, atol=1e-18)
    np.testing.assert_allclose(G[-1], R.T @ Dout, rtol=1e-12, atol=1e-18)


def dyadic(rng, shape):
    """Values k / 128, |k| <= 127: exact in bf16, and every sum of their
    products is exact in fp64 whatever the order, so library matmuls give
    the oracle's pre-activations bit for bit."""
    return rng.integers(-127, 128, size=shape).astype(np.float64) / 128


@pytest.mark.parametrize("act", [SINE, SIGMOID])
@pytest.mark.parametrize("out_act", [LINEAR, SIGMOID])
def test_depth1_rounding_on_closed_form(act, out_act):
    """One hidden layer, rounding on, written out by hand:
        C_1 = X W_1 (exact), A_2 = bf16(sigma(C_1)),
        Y32 = sigma_out(A_2 W_2), D_3 = bf16(2 (Y32 - T) / (M out) sigma_out'),
        D_2 = bf16((D_3 W_2^T) * s), with s = bf16(cos C_1) for sine and
              s = A_2 (1 - A_2) from the rounded A_2 for sigmoid,
        G_1 = X^T D_2,  G_2 = A_2^T D_3.
    Pins which value each derivative is taken from once rounding is on (the
    finite-difference checks run with rounding off)."""
    rng = np.random.default_rng(99 + act + 5 * out_act)
    w, i, o, M = 8, 6, 3, 11
    net = Net(width=w, depth=1, in_dim=i, out_dim=o, act=act, out_act=out_act)
    W1, W2 = dyadic(rng, (i, w)), dyadic(rng, (w, o))
    X = dyadic(rng, (M, i))
    T = rng.uniform(-1, 1, (M, o)).astype(np.float32).astype(np.float64)
    rne = np.vectorize(oracle.rne_bf16)
    C1 = X @ W1
    if act == SINE:
        A2 = rne(np.sin(C1))
        s = rne(np.cos(C1))
    else:
        A2 = rne(1 / (1 + np.exp(-C1)))
        s = A2 * (1 - A2)
    C2 = A2 @ W2
    Y32 = 1 / (1 + np.exp(-C2)) if out_act == SIGMOID else C2
    g = 2 * (Y32 - T) / (M * o)
    D3 = rne(g * (Y32 * (1 - Y32) if out_act == SIGMOID else 1.0))
    D2 = rne((D3 @ W2.T) * s)
    r = net.train_step(np.concatenate([W1.ravel(), W2.ravel()]), X, T, want_deltas=True)
    np.testing.assert_array_equal(r["Y"], rne(Y32))
    np.testing.assert_array_equal(r["D"][1], D3)
    np.testing.assert_array_equal(r["D"][0], D2)
    G1, G2 = net.split(r["G"])
    np.testing.assert_allclose(G1, X.T @ D2, rtol=1e-12, atol=1e-18)
    np.testing.assert_allclose(G2, A2.T @ D3, rtol=1e-12, atol=1e-18)
    # the readings differ from the alternatives: with an unrounded cos or an
    # unrounded sigmoid in the derivative some delta would change
    alt = np.cos(C1) if act == SINE else (1 / (1 + np.exp(-C1))) * (1 - 1 / (1 + np.exp(-C1)))
    assert np.any(rne((D3 @ W2.T) * alt) != D2)


def test_gradient_additive_over_batch_split():
    """With a fixed dY, G is a sum over rows: G(X1 u X2) = G(X1) + G(X2)."""
    net = Net(width=16, depth=2, in_dim=12, out_dim=5, act=SINE)
    W, X, _ = rand_net_inputs(net, 90)
    dY = RNG.uniform(-1, 1, (90, 5))
    G = net.backward(W, X, dY)
    G1 = net.backward(W, X[:37], dY[:37])
    G2 = net.backward(W, X[37:], dY[37:])
    np.testing.assert_allclose(G, G1 + G2, rtol=1e-12, atol=1e-15)


def test_stash_matches_forward_chain():
    """The A stash is the chain of hidden activations: A_2 is relu(X W_1)
    (a library matmul) rounded once to bf16, and Y32 = A_L W_L."""
    net = Net(width=32, depth=2, in_dim=20, out_dim=7)
    W, X, _ = rand_net_inputs(net, 50)
    _, Y32, A = net.forward(W, X, want_stash=True)
    Wl = net.split(W)
    rne = np.vectorize(oracle.rne_bf16)
    np.testing.assert_array_equal(A[0], rne(np.maximum(X @ Wl[0], 0)))
    np.testing.assert_allclose(Y32, A[-1] @ Wl[-1], rtol=1e-13, atol=1e-14)


def test_rounding_on_vs_off_close():
    net_on = Net(width=64, depth=4, in_dim=64, out_dim=16)
    net_off = Net(width=64, depth=4, in_dim=64, out_dim=16, round_bf16=False)
    rng = np.random.default_rng(3)
    W = bf16_exact(rng.uniform(-1, 1, net_on.param_count()) * math.sqrt(6 / 128))
    X = bf16_exact(rng.uniform(-1, 1, (256, 64)))
    Y_on, _ = net_on.forward(W, X)
    _, Y_off = net_off.forward(W, X)
    rel = np.linalg.norm(Y_on - Y_off) / np.linalg.norm(Y_off)
    assert rel < (net_on.L + 1) * 2.0 ** -8


def test_invalid_arguments_rejected():
    with pytest.raises(ValueError):
        Net(width=4, depth=1, in_dim=4, out_dim=4, act=9).forward(
            np.zeros(32), np.zeros((1, 4)))


# -------------------------------------------------------------- optimizer --

def test_adam_first_step_closed_form():
    """From zero moments the bias corrections cancel: the first step is
    w - lr g / (|g| + eps)."""
    g = RNG.uniform(-1, 1, 300)
    w = RNG.uniform(-1, 1, 300)
    lr, b1, b2, eps = 1e-2, 0.9, 0.999, 1e-8
    w1, m1, v1 = oracle.adam_step(w, np.zeros(300), np.zeros(300), g, lr, b1, b2, eps, 1)
    np.testing.assert_allclose(w1, w - lr * g / (np.abs(g) + eps), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(m1, (1 - b1) * g, rtol=1e-15)
    np.testing.assert_allclose(v1, (1 - b2) * g * g, rtol=1e-15)


def test_adam_matches_torch_optim():
    """Five steps against torch.optim.Adam (a library routine) in fp64."""
    lr, b1, b2, eps = 3e-3, 0.8, 0.95, 1e-6
    w0 = RNG.uniform(-1, 1, 257)
    p = torch.nn.Parameter(torch.tensor(w0, dtype=torch.float64))
    opt = torch.optim.Adam([p], lr=lr, betas=(b1, b2), eps=eps)
    w, m, v = w0.copy(), np.zeros(257), np.zeros(257)
    for t in range(1, 6):
        g = RNG.uniform(-1, 1, 257)
        p.grad = torch.tensor(g)
        opt.step()
        w, m, v = oracle.adam_step(w, m, v, g, lr, b1, b2, eps, t)
    np.testing.assert_allclose(w, p.detach().numpy(), rtol=1e-12, atol=1e-15)


def test_sgd_matches_torch_optim():
    w0 = RNG.uniform(-1, 1, 100)
    g = RNG.uniform(-1, 1, 100)
    p = torch.nn.Parameter(torch.tensor(w0, dtype=torch.float64))
    opt = torch.optim.SGD([p], lr=0.05)
    p.grad = torch.tensor(g)
    opt.step()
    np.testing.assert_allclose(oracle.sgd_step(w0, g, 0.05), p.detach().numpy(), rtol=1e-13, atol=1e-16)


def test_to_bf16_matches_torch():
    w = RNG.uniform(-3, 3, 1000).astype(np.float32).astype(np.float64)
    ref = torch.tensor(w, dtype=torch.float32).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(oracle.to_bf16(w), ref)
