"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Every case draws seeded inputs with datagen, runs the library on the GPU and
the oracle on the CPU on the same values, and compares element by element
with the bounds stated in helpers.py.  Bitwise properties (identity
weights, power-of-two scaling, row permutation, run-to-run determinism) are
checked exactly.
"""
import sys

import numpy as np
import pytest
import torch

import datagen
from helpers import (LOSS_TOL, check_dx, check_grads, check_outputs, f64, inputs, oracle_net)

pytestmark = pytest.mark.gpu


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run_case(ffmlp, dev, width, depth, in_dim, out_dim, M, act="relu", out_act="linear",
             seed=11, train=True, t_range=(-1.0, 1.0)):
    log(f"case w={width} d={depth} in={in_dim} out={out_dim} M={M} act={act} out={out_act}")
    W, X, T = inputs(seed, width, depth, in_dim, out_dim, M, t_range)
    onet = oracle_net(width, depth, in_dim, out_dim, act, out_act)
    net = ffmlp.FusedMLP(width, depth, in_dim, out_dim, act, out_act)
    Wd, Xd, Td = W.to(dev), X.to(dev), T.to(dev)
    packed = net.pack(Wd)
    Y = net.forward(packed, Xd)
    res = {"net": net, "onet": onet, "packed": packed, "W": W, "X": X, "T": T, "Y": Y}
    if train:
        ws = net.workspace(M, dev)
        Yt = torch.empty_like(Y)
        G, loss = net.train_step(packed, Xd, Td, ws, Y=Yt)
        torch.cuda.synchronize()
        ref = onet.train_step(W, X, T)
        res.update(G=G, loss=loss, Yt=Yt, ref=ref, ws=ws)
        log("  output errs", check_outputs(f64(Y), ref["Y"], onet.L))
        assert torch.equal(Y, Yt), "train-step outputs differ from inference outputs"
        errs = check_grads(f64(G), ref["G"], onet)
        log("  grad errs", ["%.2e" % e for e in errs])
        lref = ref["loss"]
        assert abs(loss.item() - lref) <= LOSS_TOL * max(abs(lref), 1e-30)
    else:
        torch.cuda.synchronize()
        Yref, _ = onet.forward(W, X)
        log("  output errs", check_outputs(f64(Y), Yref, onet.L))
    return res


# ------------------------------------------------------------------ configs --

def test_tiny_config(ffmlp, gpu):
    """Input 64, 4 hidden layers of 64, ReLU, linear output 64, batch 4096."""
    r = run_case(ffmlp, gpu, 64, 4, 64, 64, 4096, seed=1)
    Yref = r["ref"]["Y"]
    match = np.mean(f64(r["Y"]) == Yref)
    log(f"  bitwise-equal outputs: {match:.4f}")
    # the rounding points match, so only fp32-versus-fp64 sums that straddle
    # a bf16 rounding boundary can differ (measured: 0.9998)
    assert match > 0.99


@pytest.mark.parametrize("width", [16, 32, 64, 128])
@pytest.mark.parametrize("M", [1, 7, 4097])
def test_width_sweep_shapes(ffmlp, gpu, width, M):
    """The sweep shape (in = width, out 16, 4 hidden layers) at tail sizes."""
    run_case(ffmlp, gpu, width, 4, width, 16, M, seed=2)


@pytest.mark.parametrize("act", ["linear", "relu", "sigmoid", "sine"])
@pytest.mark.parametrize("out_act", ["linear", "relu", "sigmoid", "sine"])
def test_activations(ffmlp, gpu, act, out_act):
    run_case(ffmlp, gpu, 32, 3, 29, 5, 777, act, out_act, seed=4)


@pytest.mark.parametrize("width,depth", [(64, 0), (64, 1), (64, 2), (64, 16), (128, 16), (64, 24),
                                         (128, 5), (16, 0), (128, 0), (32, 7)])
def test_depths(ffmlp, gpu, width, depth):
    run_case(ffmlp, gpu, width, depth, width, width, 1000, seed=5)


def _random_shapes(n, seed=2024):
    """Seeded shapes across the launch variants: every width, depths 0-6,
    in/out widths that are and are not multiples of 8 (vector or scalar X
    and Y paths), every activation pair, ragged batches."""
    import random
    rng = random.Random(seed)
    acts = ["linear", "relu", "sigmoid", "sine"]
    out = []
    for _ in range(n):
        w = rng.choice([16, 32, 64, 128])
        out.append((w, rng.randint(0, 6), rng.randint(1, w), rng.randint(1, w), rng.choice(acts),
                    rng.choice(acts), rng.randint(1, 2600)))
    return out


@pytest.mark.parametrize("width,depth,in_dim,out_dim,act,out_act,M", _random_shapes(16))
def test_random_shapes(ffmlp, gpu, width, depth, in_dim, out_dim, act, out_act, M):
    run_case(ffmlp, gpu, width, depth, in_dim, out_dim, M, act=act, out_act=out_act,
             seed=width + depth + in_dim + out_dim + M)


def test_weights_filling_all_of_lds(ffmlp, gpu):
    """Width 128, 5 matrices of 128 x 128: the packed forward weights take
    exactly 160 KiB, all of LDS; inference keeps them resident, the training
    forward streams them."""
    run_case(ffmlp, gpu, 128, 4, 128, 128, 3000, seed=24)


@pytest.mark.parametrize("width,depth,in_dim,out_dim", [(16, 100, 16, 16), (32, 60, 5, 9)])
def test_deep_nets(ffmlp, gpu, width, depth, in_dim, out_dim):
    """Deep sine nets (the weights stream through LDS layer by layer, and the
    packed buffer has hundreds of segments, located in closed form)."""
    run_case(ffmlp, gpu, width, depth, in_dim, out_dim, 700, act="sine", seed=23)


@pytest.mark.parametrize("width,in_dim,out_dim", [(64, 1, 1), (64, 3, 3), (64, 16, 16),
                                                  (64, 8, 1), (64, 5, 64), (128, 127, 33),
                                                  (16, 1, 16), (32, 17, 31), (128, 40, 100)])
def test_in_out_dims(ffmlp, gpu, width, in_dim, out_dim):
    run_case(ffmlp, gpu, width, 2, in_dim, out_dim, 1500, seed=6)


def test_image_like(ffmlp, gpu):
    """Sinusoidal features of pixel coordinates, width 64, 2 hidden layers,
    3 sigmoid outputs, targets in [0, 1]."""
    net = ffmlp.FusedMLP(64, 2, 64, 3, "relu", "sigmoid")
    onet = oracle_net(64, 2, 64, 3, "relu", "sigmoid")
    M = 5000
    X = datagen.image_features(4, M)
    W = datagen.xavier_weights(4, 64, 2, 64, 3)
    T = datagen.targets_uniform(4, M, 3, 0.0, 1.0)
    packed = net.pack(W.to(gpu))
    ws = net.workspace(M, gpu)
    Y = torch.empty(M, 3, dtype=torch.bfloat16, device=gpu)
    G, loss = net.train_step(packed, X.to(gpu), T.to(gpu), ws, Y=Y)
    ref = onet.train_step(W, X, T)
    check_outputs(f64(Y), ref["Y"], onet.L)
    check_grads(f64(G), ref["G"], onet)


def test_pinn_like(ffmlp, gpu):
    """3-D inputs, width 64, 4 sine hidden layers, one linear output."""
    run_case(ffmlp, gpu, 64, 4, 3, 1, 3000, "sine", "linear", seed=6)


# ---------------------------------------------------- seeded backward pass --

@pytest.mark.parametrize("width,act,out_act", [(64, "relu", "linear"), (32, "sine", "sigmoid"),
                                               (128, "sigmoid", "sine"), (16, "linear", "relu")])
def test_forward_stash_then_backward(ffmlp, gpu, width, act, out_act):
    depth, in_dim, out_dim, M = 3, width, 7, 2100
    W, X, _ = inputs(7, width, depth, in_dim, out_dim, M)
    dY = datagen.uniform(7, datagen.STREAM_AUX, (M, out_dim))
    net = ffmlp.FusedMLP(width, depth, in_dim, out_dim, act, out_act)
    onet = oracle_net(width, depth, in_dim, out_dim, act, out_act)
    packed = net.pack(W.to(gpu))
    ws = net.workspace(M, gpu)
    Xd = X.to(gpu)
    Y = net.forward(packed, Xd, stash=ws)
    G = net.backward(packed, Xd, dY.to(gpu), ws)
    Yref, _ = onet.forward(W, X)
    Gref = onet.backward(W, X, dY)
    check_outputs(f64(Y), Yref, onet.L)
    check_grads(f64(G), Gref, onet)


# ------------------------------------------------------ bitwise properties --

@pytest.mark.parametrize("width", [16, 32, 64, 128])
def test_identity_weights_bitwise(ffmlp, gpu, width):
    """W_l = I with ReLU hidden and linear output gives Y = relu(X) exactly:
    any mistake in the operand layouts or the chain order scrambles it."""
    depth, M = 3, 999
    net = ffmlp.FusedMLP(width, depth, width, width, "relu")
    W = torch.eye(width, dtype=torch.bfloat16).flatten().repeat(depth + 1)
    X = datagen.inputs_uniform(8, M, width)
    Y = net.forward(net.pack(W.to(gpu)), X.to(gpu))
    assert torch.equal(Y.cpu(), torch.relu(X))


@pytest.mark.parametrize("width", [16, 128])
def test_power_of_two_homogeneity_bitwise(ffmlp, gpu, width):
    net = ffmlp.FusedMLP(width, 3, width, 16, "relu")
    W, X, _ = inputs(9, width, 3, width, 16, 3000)
    packed = net.pack(W.to(gpu))
    Xd = X.to(gpu)
    Y1 = net.forward(packed, Xd)
    Y2 = net.forward(packed, Xd * 4)
    assert torch.equal(Y2, Y1 * 4)


def test_row_permutation_bitwise(ffmlp, gpu):
    net = ffmlp.FusedMLP(64, 4, 64, 16, "sigmoid")
    W, X, _ = inputs(10, 64, 4, 64, 16, 5000)
    packed = net.pack(W.to(gpu))
    perm = torch.randperm(5000, generator=torch.Generator().manual_seed(0))
    Y = net.forward(packed, X.to(gpu))
    Yp = net.forward(packed, X[perm].contiguous().to(gpu))
    assert torch.equal(Yp, Y[perm.to(gpu)])


@pytest.mark.parametrize("width", [16, 32, 128])
def test_gradients_deterministic(ffmlp, gpu, width):
    """Fixed-order partial sums: G and the loss are bitwise the same from
    run to run (width 128: fused backward and reduce; widths 16 and 32: the
    one-kernel step and reduce)."""
    net = ffmlp.FusedMLP(width, 4, width, 16, "relu")
    M = 70000
    W, X, T = inputs(12, width, 4, width, 16, M)
    packed = net.pack(W.to(gpu))
    ws = net.workspace(M, gpu)
    Xd, Td = X.to(gpu), T.to(gpu)
    G1, l1 = net.train_step(packed, Xd, Td, ws)
    G1, l1 = G1.clone(), l1.clone()
    G2, l2 = net.train_step(packed, Xd, Td, ws)
    assert torch.equal(G1, G2) and torch.equal(l1, l2)


def test_empty_batch(ffmlp, gpu):
    net = ffmlp.FusedMLP(32, 2, 32, 16, "relu")
    W, _, _ = inputs(13, 32, 2, 32, 16, 1)
    packed = net.pack(W.to(gpu))
    X = torch.empty(0, 32, dtype=torch.bfloat16, device=gpu)
    T = torch.empty(0, 16, dtype=torch.float32, device=gpu)
    ws = net.workspace(0, gpu)
    G = torch.full((net.param_count(),), 7.0, device=gpu)
    G, loss = net.train_step(packed, X, T, ws, G=G)
    assert torch.count_nonzero(G).item() == 0 and loss.item() == 0.0
    assert net.forward(packed, X).shape == (0, 16)


# ----------------------------------------------------- input gradient dX --

def dx_case(ffmlp, dev, width, depth, in_dim, out_dim, M, act="relu", out_act="linear", seed=21):
    log(f"dx case w={width} d={depth} in={in_dim} out={out_dim} M={M} act={act} out={out_act}")
    W, X, _ = inputs(seed, width, depth, in_dim, out_dim, M)
    dY = datagen.uniform(seed, datagen.STREAM_AUX, (M, out_dim))
    net = ffmlp.FusedMLP(width, depth, in_dim, out_dim, act, out_act)
    onet = oracle_net(width, depth, in_dim, out_dim, act, out_act)
    packed = net.pack(W.to(dev))
    ws = net.workspace(M, dev)
    Xd, dYd = X.to(dev), dY.to(dev)
    net.forward(packed, Xd, stash=ws)
    G, dX = net.backward_dx(packed, Xd, dYd, ws)
    G0 = net.backward(packed, Xd, dYd, ws)
    torch.cuda.synchronize()
    Gref, dXref = onet.backward_dx(W, X, dY)
    log("  dx errs", check_dx(f64(dX), dXref, onet.L))
    check_grads(f64(G), Gref, onet)
    # mlp_backward may take the fused kernel (another summation order of G)
    check_grads(f64(G0), Gref, onet)
    d = (G - G0).norm() / G0.norm().clamp_min(1e-30)
    assert d.item() < 1e-5, "G of mlp_backward_dx and mlp_backward differ beyond fp32 rounding"


@pytest.mark.parametrize("width,depth,in_dim,out_dim,act,out_act", [
    (16, 2, 16, 16, "relu", "linear"), (32, 3, 32, 7, "sine", "sigmoid"),
    (64, 4, 64, 16, "relu", "linear"), (128, 4, 128, 16, "relu", "linear"),
    (128, 1, 100, 3, "sigmoid", "linear"), (64, 0, 40, 12, "linear", "sigmoid"),
    (64, 2, 3, 1, "sine", "linear"), (128, 5, 127, 33, "relu", "relu")])
def test_input_gradient(ffmlp, gpu, width, depth, in_dim, out_dim, act, out_act):
    """dX = D_1 W_1^T against the oracle, G unchanged by asking for dX;
    both delta-buffer parities, depth 0, in_dim not a multiple of 4."""
    dx_case(ffmlp, gpu, width, depth, in_dim, out_dim, 4097, act, out_act)


@pytest.mark.parametrize("width,depth,in_dim,out_dim,act,out_act,M", _random_shapes(8, seed=77))
def test_random_shapes_input_gradient(ffmlp, gpu, width, depth, in_dim, out_dim, act, out_act, M):
    dx_case(ffmlp, gpu, width, depth, in_dim, out_dim, M, act=act, out_act=out_act,
            seed=width + depth + in_dim + out_dim + M)


def test_input_gradient_streaming(ffmlp, gpu):
    """Weights too large for LDS (staged layer by layer) with dX."""
    dx_case(ffmlp, gpu, 128, 16, 128, 128, 3000)


def test_chained_nets_nerf_like(ffmlp, gpu):
    """A density net (in 32 Gaussian features, width 64, 1 hidden layer,
    16 linear outputs) feeds a color net (its 16 outputs + 16 direction
    features, width 64, 2 hidden layers, 3 sigmoid outputs).  The color
    net's dX, first 16 columns, seeds the density net's backward pass;
    the density net's G matches the oracle's chain."""
    M = 4096
    Xd = datagen.gaussian_features(5, datagen.STREAM_X, M, 32)
    dirs = datagen.gaussian_features(5, datagen.STREAM_AUX, M, 16)
    Wd = datagen.xavier_weights(5, 64, 1, 32, 16)
    Wc = datagen.xavier_weights(6, 64, 2, 32, 3)
    dYc = datagen.uniform(5, datagen.STREAM_T, (M, 3))
    dens = ffmlp.FusedMLP(64, 1, 32, 16, "relu", "linear")
    col = ffmlp.FusedMLP(64, 2, 32, 3, "relu", "sigmoid")
    odens = oracle_net(64, 1, 32, 16, "relu", "linear")
    ocol = oracle_net(64, 2, 32, 3, "relu", "sigmoid")
    pd, pc = dens.pack(Wd.to(gpu)), col.pack(Wc.to(gpu))
    wsd, wsc = dens.workspace(M, gpu), col.workspace(M, gpu)
    Yd = dens.forward(pd, Xd.to(gpu), stash=wsd)
    Xc = torch.cat([Yd, dirs.to(gpu)], dim=1).contiguous()
    col.forward(pc, Xc, stash=wsc)
    Gc, dXc = col.backward_dx(pc, Xc, dYc.to(gpu), wsc)
    Gd = dens.backward(pd, Xd.to(gpu), dXc[:, :16].contiguous(), wsd)
    torch.cuda.synchronize()
    Yd_ref, _ = odens.forward(Wd, Xd)
    Xc_ref = np.concatenate([Yd_ref, f64(dirs)], axis=1)
    Gc_ref, dXc_ref = ocol.backward_dx(Wc, Xc_ref, dYc)
    Gd_ref = odens.backward(Wd, Xd, dXc_ref[:, :16])
    check_outputs(f64(Yd), Yd_ref, odens.L)
    log("  color dx errs", check_dx(f64(dXc), dXc_ref, ocol.L))
    check_grads(f64(Gc), Gc_ref, ocol)
    log("  density grad errs", ["%.2e" % e for e in check_grads(f64(Gd), Gd_ref, odens)])


# ------------------------------------------------ HIP graph capture (NEXT-3) --

def test_graph_capture_replays_bitwise(ffmlp, gpu):
    """The library neither allocates nor synchronizes, so a forward pass, a
    training step and an Adam step can be captured in one HIP graph (what a
    small-batch loop needs to shed launch overhead).  Every replay, with
    other work and synchronizations between replays, equals the eager
    results bit for bit."""
    width, depth, in_dim, out_dim, M = 64, 4, 64, 16, 4096
    W, X, T = inputs(12, width, depth, in_dim, out_dim, M)
    net = ffmlp.FusedMLP(width, depth, in_dim, out_dim, "relu")
    n = net.param_count()
    Xd, Td = X.to(gpu), T.to(gpu)
    ws = net.workspace(M, gpu)

    def step(packed, master, m, v, Wb, G, loss, Yt, Yf):
        net.train_step(packed, Xd, Td, ws, G=G, loss=loss, Y=Yt)
        net.forward(packed, Xd, Y=Yf)
        net.adam_step(master, m, v, G, Wb, packed, 1e-3, (0.9, 0.999), 1e-8, 1)

    def state():
        Wb = W.to(gpu).clone()
        return dict(packed=net.pack(Wb), master=Wb.float(), m=torch.zeros(n, device=gpu),
                    v=torch.zeros(n, device=gpu), Wb=Wb,
                    G=torch.empty(n, device=gpu), loss=torch.empty(1, device=gpu),
                    Yt=torch.empty(M, out_dim, dtype=torch.bfloat16, device=gpu),
                    Yf=torch.empty(M, out_dim, dtype=torch.bfloat16, device=gpu))

    eager = state()
    step(**eager)  # also fills the launch caches before capture
    torch.cuda.synchronize()
    cap = state()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(**cap)
    for rep in range(3):
        fresh = state()  # reset the captured buffers' inputs
        for k in ("packed", "master", "m", "v", "Wb"):
            cap[k].copy_(fresh[k])
        torch.cuda.synchronize()
        graph.replay()
        other = state()
        step(**other)  # eager work between replays
        torch.cuda.synchronize()
        for k in eager:
            assert torch.equal(cap[k], eager[k]), (rep, k)
            assert torch.equal(other[k], eager[k]), (rep, k)


# ---------------------------------------------------- optimizer (NEXT-4) --

def test_optimizer_steps_match_oracle(ffmlp, gpu):
    """Three Adam steps, then one SGD step, on fp32 master weights: master
    weights and moments against the fp64 definitions, W bitwise the bf16
    rounding of the GPU's own master weights (and of the oracle's on all
    but boundary cases), and the re-packed buffer equal to a fresh pack."""
    import oracle
    net = ffmlp.FusedMLP(64, 3, 40, 10, "relu")
    n = net.param_count()
    W0 = datagen.xavier_weights(8, 64, 3, 40, 10)
    Gs = [datagen.uniform(8 + t, datagen.STREAM_AUX, (n,)) * 1e-2 for t in range(4)]
    master = W0.float().to(gpu)
    m = torch.zeros(n, dtype=torch.float32, device=gpu)
    v = torch.zeros_like(m)
    W = torch.empty(n, dtype=torch.bfloat16, device=gpu)
    packed = torch.empty(net.packed_bytes(), dtype=torch.uint8, device=gpu)
    wo, mo, vo = f64(W0), np.zeros(n), np.zeros(n)
    lr, b1, b2, eps = 1e-2, 0.9, 0.99, 1e-8
    for t in range(1, 4):
        net.adam_step(master, m, v, Gs[t - 1].to(gpu), W, packed, lr, (b1, b2), eps, t)
        wo, mo, vo = oracle.adam_step(wo, mo, vo, f64(Gs[t - 1]), lr, b1, b2, eps, t)
    torch.cuda.synchronize()
    np.testing.assert_allclose(f64(master), wo, rtol=0, atol=1e-6)
    # fp32 against fp64: a few fp32 ulps of the moments' scale (m can cancel
    # to near zero, so the bound is absolute)
    np.testing.assert_allclose(f64(m), mo, rtol=0, atol=1e-6 * np.abs(mo).max())
    np.testing.assert_allclose(f64(v), vo, rtol=0, atol=1e-6 * np.abs(vo).max())
    assert np.array_equal(f64(W), oracle.to_bf16(f64(master)))
    assert np.mean(f64(W) == oracle.to_bf16(wo)) > 0.999
    assert torch.equal(packed, net.pack(W))
    net.sgd_step(master, Gs[3].to(gpu), W, None, 0.5)
    torch.cuda.synchronize()
    np.testing.assert_allclose(f64(master), oracle.sgd_step(wo, f64(Gs[3]), 0.5), rtol=0, atol=2e-6)
    assert np.array_equal(f64(W), oracle.to_bf16(f64(master)))


def test_adam_training_loop_matches_oracle(ffmlp, gpu):
    """Five training steps (train step, then Adam with re-packing) on the
    GPU against the same loop on the oracle: losses agree and fall."""
    import oracle
    width, depth, in_dim, out_dim, M = 32, 2, 32, 8, 2048
    W0, X, T = inputs(9, width, depth, in_dim, out_dim, M)
    net = ffmlp.FusedMLP(width, depth, in_dim, out_dim, "relu")
    onet = oracle_net(width, depth, in_dim, out_dim, "relu")
    n = net.param_count()
    master = W0.float().to(gpu)
    m = torch.zeros(n, dtype=torch.float32, device=gpu)
    v = torch.zeros_like(m)
    W = W0.to(gpu).clone()
    packed = net.pack(W)
    ws = net.workspace(M, gpu)
    Xd, Td = X.to(gpu), T.to(gpu)
    wo, mo, vo, Wb = f64(W0), np.zeros(n), np.zeros(n), f64(W0)
    lr, b1, b2, eps = 2e-2, 0.9, 0.999, 1e-8
    gl, ol = [], []
    for t in range(1, 6):
        G, loss = net.train_step(packed, Xd, Td, ws)
        net.adam_step(master, m, v, G, W, packed, lr, (b1, b2), eps, t)
        gl.append(loss.item())
        r = onet.train_step(Wb, X, T)
        ol.append(r["loss"])
        wo, mo, vo = oracle.adam_step(wo, mo, vo, r["G"], lr, b1, b2, eps, t)
        Wb = oracle.to_bf16(wo)
    log("  losses gpu", ["%.6f" % x for x in gl], "oracle", ["%.6f" % x for x in ol])
    np.testing.assert_allclose(gl, ol, rtol=1e-2)
    assert gl[-1] < gl[0] and ol[-1] < ol[0]


# ------------------------------------------- full sizes, sampled rows only --

def sampled_rows(M, n, seed):
    g = torch.Generator().manual_seed(seed)
    return torch.unique(torch.randint(0, M, (n,), generator=g))


@pytest.mark.parametrize("width,depth,in_dim,out_dim,M", [
    (128, 4, 128, 16, 1 << 20),       # width sweep at 2^20
    (64, 4, 64, 16, (1 << 20) + 37),  # ragged tail
    (32, 4, 32, 16, 1 << 20),
    (16, 4, 16, 16, 1 << 22),         # width sweep at 2^22
    (128, 4, 128, 16, 1 << 22),       # the largest sweep batch at width 128
    (128, 16, 128, 128, 1 << 20),     # depth/width stress: weights stream through LDS
    (128, 3, 128, 16, (1 << 20) + 100),  # even matrix count, ragged tail
    (64, 5, 64, 16, 1 << 20),         # even matrix count at width 64
])
def test_full_size_sampled(ffmlp, gpu, width, depth, in_dim, out_dim, M):
    """At benchmark sizes: Y on sampled rows against the oracle, inference Y
    bitwise equal to the stashing forward's on every row, and G and dX from
    mlp_backward_dx with dY nonzero only on the sampled rows (G is a sum
    over rows and dX a function of each row, so the oracle needs only those
    rows; every other row's dX is exactly 0)."""
    log(f"full-size w={width} d={depth} M={M}")
    net = ffmlp.FusedMLP(width, depth, in_dim, out_dim, "relu")
    onet = oracle_net(width, depth, in_dim, out_dim, "relu")
    W = datagen.xavier_weights(14, width, depth, in_dim, out_dim)
    Xd = datagen.inputs_uniform(14, M, in_dim, device=gpu)
    rows = sampled_rows(M, 2048, 14)
    # the same rows drawn on the CPU must be the same bits
    Xs = torch.stack([datagen.uniform(14, datagen.STREAM_X, (in_dim,), device="cpu",
                                      start=int(r) * in_dim) for r in rows]).to(torch.bfloat16)
    assert torch.equal(Xs, Xd[rows.to(gpu)].cpu())
    packed = net.pack(W.to(gpu))
    ws = net.workspace(M, gpu)
    Y = net.forward(packed, Xd, stash=ws)
    # inference (its own kernel and tile loop) computes every row the same
    Yi = net.forward(packed, Xd)
    assert torch.equal(Yi, Y), "inference outputs differ from the stashing forward's"
    dYs = datagen.uniform(14, datagen.STREAM_AUX, (len(rows), out_dim))
    dY = torch.zeros(M, out_dim, dtype=torch.float32, device=gpu)
    dY[rows.to(gpu)] = dYs.to(gpu)
    G, dX = net.backward_dx(packed, Xd, dY, ws)
    Yref, _ = onet.forward(W, Xs)
    log("  output errs", check_outputs(f64(Y[rows.to(gpu)]), Yref, onet.L))
    Gref, dXref = onet.backward_dx(W, Xs, dYs)
    errs = check_grads(f64(G), Gref, onet)
    log("  dx errs", check_dx(f64(dX[rows.to(gpu)]), dXref, onet.L))
    # rows with dY = 0 have dX = 0 exactly
    others = torch.ones(M, dtype=torch.bool, device=gpu)
    others[rows.to(gpu)] = False
    assert torch.count_nonzero(dX[others]).item() == 0
    log("  grad errs", ["%.2e" % e for e in errs])
    del ws
    torch.cuda.empty_cache()


@pytest.mark.parametrize("width,depth,in_dim,out_dim,M", [
    (128, 4, 128, 16, 1 << 20),       # the benchmark's training step
    (128, 16, 128, 128, 1 << 20),     # depth/width stress net (streamed weights)
    (64, 4, 64, 16, (1 << 20) + 37),  # ragged tail
    (16, 4, 16, 16, 1 << 22),         # the largest sweep batch at width 16
])
def test_train_step_full_batch(ffmlp, gpu, width, depth, in_dim, out_dim, M):
    """The timed training call at benchmark sizes, where every workgroup
    loops over many row tiles: Y on every row, every layer's G over the
    full batch and the loss against the oracle's training step, and the
    inference outputs bitwise equal to the training forward's."""
    log(f"train-step full batch w={width} d={depth} in={in_dim} out={out_dim} M={M}")
    net = ffmlp.FusedMLP(width, depth, in_dim, out_dim, "relu")
    onet = oracle_net(width, depth, in_dim, out_dim, "relu")
    W = datagen.xavier_weights(16, width, depth, in_dim, out_dim)
    Xd = datagen.inputs_uniform(16, M, in_dim, device=gpu)
    Td = datagen.targets_uniform(16, M, out_dim, device=gpu)
    packed = net.pack(W.to(gpu))
    ws = net.workspace(M, gpu)
    Y = torch.empty(M, out_dim, dtype=torch.bfloat16, device=gpu)
    G, loss = net.train_step(packed, Xd, Td, ws, Y=Y)
    Yi = net.forward(packed, Xd)
    torch.cuda.synchronize()
    assert torch.equal(Yi, Y), "inference outputs differ from the training forward's"
    X, T = Xd.cpu(), Td.cpu()
    del ws, Xd, Td, Yi
    torch.cuda.empty_cache()
    ref = onet.train_step(W, X, T)
    log("  output errs (all rows)", check_outputs(f64(Y), ref["Y"], onet.L))
    errs = check_grads(f64(G), ref["G"], onet)
    log("  grad errs (full batch)", ["%.2e" % e for e in errs])
    lerr = abs(loss.item() - ref["loss"]) / ref["loss"]
    log(f"  loss {loss.item():.7f} oracle {ref['loss']:.7f} rel err {lerr:.2e}")
    assert lerr <= LOSS_TOL


@pytest.mark.parametrize("width,depth,in_dim,out_dim,act,out_act", [
    (128, 1, 128, 16, "relu", "linear"), (128, 2, 100, 3, "relu", "sigmoid"),
    (128, 3, 128, 16, "relu", "relu"), (128, 4, 64, 1, "relu", "linear"),
    (64, 1, 32, 16, "relu", "linear"), (64, 2, 64, 3, "relu", "sigmoid"),
    (64, 3, 60, 64, "relu", "linear"), (64, 4, 64, 40, "relu", "sine"),
    (32, 1, 8, 32, "relu", "linear"), (32, 4, 32, 17, "relu", "sigmoid"),
    (32, 4, 30, 32, "sine", "linear"), (32, 2, 32, 1, "sigmoid", "sigmoid"),
    (16, 2, 16, 5, "relu", "linear"), (16, 4, 12, 16, "relu", "relu"),
    (16, 3, 7, 16, "sine", "sine"), (16, 1, 16, 16, "linear", "relu"),
])
def test_fused_backward_shapes(ffmlp, gpu, width, depth, in_dim, out_dim, act, out_act):
    """Nets of 2 to 5 matrices take the fused backward kernel (deltas kept
    on chip, weight gradients in registers): every width, both output-strip
    classes at width 64, input widths that are multiples of 4 and ones that
    are not (7, 30), every hidden activation at the narrow widths, every
    output activation, and a batch of several tiles per workgroup with a
    ragged tail.  The training step and the seeded backward (after a
    stashing forward) against the oracle."""
    M = 70001
    log(f"fused w={width} d={depth} in={in_dim} out={out_dim} act={act} out_act={out_act} M={M}")
    r = run_case(ffmlp, gpu, width, depth, in_dim, out_dim, M, act, out_act, seed=40 + depth)
    net, onet, packed, W, X = r["net"], r["onet"], r["packed"], r["W"], r["X"]
    dY = datagen.uniform(41, datagen.STREAM_AUX, (M, out_dim))
    ws = r["ws"]
    Xd = X.to(gpu)
    net.forward(packed, Xd, stash=ws)
    G = net.backward(packed, Xd, dY.to(gpu), ws)
    torch.cuda.synchronize()
    errs = check_grads(f64(G), onet.backward(W, X, dY), onet)
    log("  seeded grad errs", ["%.2e" % e for e in errs])


@pytest.mark.parametrize("width,depth,in_dim,out_dim,act,out_act,M", [
    (16, 1, 5, 3, "sine", "sigmoid", 1), (16, 4, 16, 16, "relu", "linear", 257),
    (16, 3, 12, 7, "sigmoid", "relu", 4099),
    (32, 2, 31, 32, "sigmoid", "relu", 513), (32, 3, 8, 4, "linear", "sine", 1025),
    (32, 4, 32, 20, "sine", "linear", 9000),
    (64, 1, 1, 1, "relu", "linear", 129), (64, 4, 64, 64, "sine", "linear", 3000),
    (64, 3, 12, 17, "sigmoid", "sigmoid", 700), (64, 2, 40, 16, "linear", "relu", 65541),
])
def test_one_kernel_step_shapes(ffmlp, gpu, width, depth, in_dim, out_dim, act, out_act, M):
    """The one-kernel training step (widths 16, 32, 64 with 2 to 5 matrices)
    across its variants: vector and per-element X, T and Y paths (in_dim a
    multiple of 8 or not, out_dim a multiple of 4 or not), one and several
    output strips, every hidden and output activation, a single row, ragged
    tiles and several tiles per workgroup.  Y (bitwise equal to inference),
    G and the loss against the oracle."""
    run_case(ffmlp, gpu, width, depth, in_dim, out_dim, M, act, out_act, seed=50 + width + depth)


def test_argument_errors_on_device(ffmlp, gpu):
    net = ffmlp.FusedMLP(64, 2, 64, 16, "relu")
    W, X, T = inputs(15, 64, 2, 64, 16, 100)
    packed = net.pack(W.to(gpu))
    Xd = torch.empty(100 * 64 + 8, dtype=torch.bfloat16, device=gpu)[1:1 + 100 * 64].view(100, 64)
    with pytest.raises(ffmlp.FFMLPError) as e:
        net.forward(packed, Xd)
    assert e.value.code == ffmlp.MLP_ERR_INVALID_ARG


def test_binding_size_and_dtype_checks(ffmlp, gpu):
    """Buffers too small for M, wrong dtypes or shapes, and mixed devices are
    refused with ValueError before anything is enqueued (the C ABI derives
    every offset from M and cannot see buffer sizes)."""
    net = ffmlp.FusedMLP(64, 2, 64, 16, "relu")
    M = 300
    W, X, T = inputs(15, 64, 2, 64, 16, M)
    packed = net.pack(W.to(gpu))
    Xd, Td = X.to(gpu), T.to(gpu)
    ws = net.workspace(M, gpu)
    small_ws = net.workspace(M // 2, gpu)
    bad = [
        lambda: net.train_step(packed, Xd, Td, small_ws),                        # workspace for M/2
        lambda: net.forward(packed, Xd, stash=small_ws),
        lambda: net.train_step(packed[:-1024], Xd, Td, ws),                      # short packed
        lambda: net.train_step(packed, Xd, Td[:-1], ws),                         # T rows
        lambda: net.train_step(packed, Xd, Td.double(), ws),                     # T dtype
        lambda: net.train_step(packed, Xd.float(), Td, ws),                      # X dtype
        lambda: net.train_step(packed, Xd[:, :32].contiguous(), Td, ws),         # X columns
        lambda: net.train_step(packed, Xd, Td, ws, Y=torch.empty(M - 1, 16, dtype=torch.bfloat16,
                                                                 device=gpu)),   # Y rows
        lambda: net.forward(packed, Xd, Y=torch.empty(M, 16, dtype=torch.float32, device=gpu)),
        lambda: net.backward(packed, Xd, torch.zeros(M, 15, device=gpu), ws),    # dY columns
        lambda: net.backward_dx(packed, Xd, torch.zeros(M, 16, device=gpu), ws,
                                dX=torch.empty(M, 63, device=gpu)),              # dX columns
        lambda: net.train_step(packed, Xd, Td, ws, G=torch.empty(7, device=gpu)),  # G size
        lambda: net.pack(W.to(gpu)[:-1]),                                        # W size
        lambda: net.train_step(packed, Xd, T, ws),                               # T on the host
    ]
    for i, f in enumerate(bad):
        with pytest.raises(ValueError):
            f()
            pytest.fail(f"case {i} was accepted")
    torch.cuda.synchronize()
    G, loss = net.train_step(packed, Xd, Td, ws)  # the good call still works
    torch.cuda.synchronize()
    assert torch.isfinite(G).all()
