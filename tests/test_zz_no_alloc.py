"""mlp_train_step_noalloc: the training step on the library's static scratch
array instead of a caller workspace, for callers that cannot allocate.  Its
results must equal mlp_train_step's bit for bit (the same kernels on the
same inputs), on consecutive calls whose batch shrinks (the array keeps the
previous call's contents), and an oversized batch must be refused before
anything is enqueued."""
import ctypes

import pytest
import torch

import datagen

pytestmark = pytest.mark.gpu


def _case(ffmlp, dev, net, W, M, seed):
    X = datagen.inputs_uniform(seed, M, net.in_dim, device=dev)
    T = datagen.targets_uniform(seed, M, net.out_dim, device=dev)
    packed = net.pack(W)
    ws = net.workspace(M, dev)
    Y0 = torch.empty(M, net.out_dim, dtype=torch.bfloat16, device=dev)
    G0, l0 = net.train_step(packed, X, T, ws, Y=Y0)
    G1 = torch.full_like(G0, float("nan"))
    l1 = torch.full_like(l0, float("nan"))
    Y1 = torch.full_like(Y0, float("nan"))
    net.train_step_noalloc(packed, X, T, G1, l1, Y=Y1)
    torch.cuda.synchronize()
    assert torch.equal(G1, G0), (M, (G1 - G0).abs().max().item())
    assert torch.equal(l1, l0) and torch.equal(Y1, Y0)
    return G1


@pytest.mark.parametrize("width,depth,in_dim,out_dim,act,M1,M2", [
    (128, 4, 128, 16, "relu", 15000, 4097),
    (64, 3, 40, 7, "sine", 9000, 333),
    (16, 2, 16, 16, "sigmoid", 20000, 1),
])
def test_noalloc_matches_train_step(ffmlp, gpu, width, depth, in_dim, out_dim, act, M1, M2):
    net = ffmlp.FusedMLP(width, depth, in_dim, out_dim, act)
    assert net.workspace_bytes(M1) <= ffmlp.MLP_SCRATCH_BYTES
    W = datagen.xavier_weights(31, width, depth, in_dim, out_dim, device=gpu)
    _case(ffmlp, gpu, net, W, M1, 31)
    _case(ffmlp, gpu, net, W, M2, 32)  # smaller batch on the reused array


def test_noalloc_refuses_oversized_batch(ffmlp, gpu):
    net = ffmlp.FusedMLP(128, 4, 128, 16, "relu")
    M = 1
    while net.workspace_bytes(M) <= ffmlp.MLP_SCRATCH_BYTES:
        M *= 2
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: the size check fails first
    rc = ffmlp.lib().mlp_train_step_noalloc(net.handle, fake, fake, fake, None, fake, None, M, None)
    assert rc == ffmlp.MLP_ERR_WORKSPACE
    assert "static scratch" in ffmlp.last_error()
