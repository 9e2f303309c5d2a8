"""Host-side checks of the C-ABI library (no GPU needed): it loads, it
exports every function include/ffmlp.h declares, and its shape queries and
argument checks behave as the header states.  Nothing here launches a
kernel."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ffmlp.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mlp_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ["mlp_create", "mlp_forward", "mlp_backward", "mlp_backward_dx", "mlp_train_step",
                     "mlp_sgd_step", "mlp_adam_step",
                     "mlp_pack_weights", "mlp_workspace_bytes", "mlp_destroy"]:
        assert required in names


def test_library_exports_every_declared_symbol(ffmlp):
    handle = ctypes.CDLL(ffmlp.LIB_PATH)
    for name in declared_functions():
        assert hasattr(handle, name), name
    assert set(declared_functions()) == set(ffmlp._SIGNATURES)


def create(ffmlp, *args):
    h = ctypes.c_void_p()
    rc = ffmlp.lib().mlp_create(*args, ctypes.byref(h))
    return rc, h


@pytest.mark.parametrize("width", [16, 32, 64, 128])
def test_shapes_and_offsets(ffmlp, width):
    depth, in_dim, out_dim = 3, max(1, width // 2 - 1), 3
    net = ffmlp.FusedMLP(width, depth, in_dim, out_dim, "relu")
    shapes = [net.layer_shape(l) for l in range(depth + 1)]
    assert [s[:2] for s in shapes] == [(in_dim, width), (width, width), (width, width),
                                       (width, out_dim)]
    offs = [s[2] for s in shapes]
    assert offs == [0, in_dim * width, in_dim * width + width * width,
                    in_dim * width + 2 * width * width]
    assert net.param_count() == offs[-1] + width * out_dim
    # packed: forward strips(fan_out) + backward layers 1..L-1 and 0 strips(fan_in),
    # each with the width's k-blocks, 1 KiB per fragment.
    st = lambda n: (n + 15) // 16
    kb = (width + 31) // 32
    fwd = sum(st(fo) * kb for fi, fo, _ in shapes)
    bwd = sum(st(fi) * kb for fi, fo, _ in shapes[1:])
    bwd += st(shapes[0][0]) * kb  # backward layer 0, for the input gradient
    assert net.packed_bytes() == (fwd + bwd) * 1024


def test_deepest_net_is_accepted(ffmlp):
    net = ffmlp.FusedMLP(16, 65534, 16, 16, "relu")
    assert net.param_count() == 65535 * 256
    assert net.layer_shape(65534) == (16, 16, 65534 * 256)


def test_depth0_single_matrix(ffmlp):
    net = ffmlp.FusedMLP(32, 0, 20, 7, "sine")
    assert net.layer_shape(0) == (20, 7, 0)
    assert net.param_count() == 140
    with pytest.raises(ffmlp.FFMLPError):
        net.layer_shape(1)


def test_workspace_sizes(ffmlp):
    net = ffmlp.FusedMLP(64, 4, 64, 16, "relu")
    assert net.workspace_bytes(1 << 17, ffmlp.MLP_MODE_INFER) == 0
    small, big = net.workspace_bytes(1000), net.workspace_bytes(1 << 20)
    # at least the activation and delta stashes: 2 x depth x M x width bf16
    assert big >= 2 * 4 * (1 << 20) * 64 * 2
    assert small < big and small % 256 == 0
    # sine adds the bf16 cos stash; ReLU instead keeps one 32-bit mask word
    # per lane of every 16-row block and hidden activation
    sine = ffmlp.FusedMLP(64, 4, 64, 16, "sine")
    relu_masks = 4 * ((1 << 20) // 16) * 64 * 4
    assert sine.workspace_bytes(1 << 20) >= big - relu_masks + 4 * (1 << 20) * 64 * 2
    lin = ffmlp.FusedMLP(64, 4, 64, 16, "linear")
    assert big - lin.workspace_bytes(1 << 20) == relu_masks


@pytest.mark.parametrize("args,code", [
    ((48, 2, 8, 8, 1), -2),     # width not supported
    ((64, 2, 8, 8, 7), -2),     # unknown activation
    ((64, -1, 8, 8, 1), -1),    # negative depth
    ((64, 65535, 8, 8, 1), -1), # deeper than one grid dimension holds
    ((64, 2, 0, 8, 1), -1),     # in_dim < 1
    ((64, 2, 65, 8, 1), -1),    # in_dim > width
    ((64, 2, 8, 65, 1), -1),    # out_dim > width
])
def test_create_rejects_bad_shapes(ffmlp, args, code):
    rc, h = create(ffmlp, *args)
    assert rc == code
    assert not h.value
    assert ffmlp.last_error()


def test_null_and_bad_arguments_fail_before_any_launch(ffmlp):
    L = ffmlp.lib()
    net = ffmlp.FusedMLP(64, 2, 64, 16, "relu")
    h = net.handle
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: checks fail first
    assert L.mlp_forward(None, fake, fake, fake, 10, None, None) == ffmlp.MLP_ERR_INVALID_ARG
    assert L.mlp_forward(h, None, fake, fake, 10, None, None) == ffmlp.MLP_ERR_INVALID_ARG
    assert L.mlp_forward(h, fake, fake, fake, -1, None, None) == ffmlp.MLP_ERR_INVALID_ARG
    assert L.mlp_forward(h, fake, ctypes.c_void_p(0x1002), fake, 10, None, None) == \
        ffmlp.MLP_ERR_INVALID_ARG  # misaligned X
    assert "aligned" in ffmlp.last_error()
    assert L.mlp_forward(h, None, None, None, 0, None, None) == ffmlp.MLP_OK  # empty batch
    assert L.mlp_backward(h, fake, fake, fake, None, 10, fake, None) == ffmlp.MLP_ERR_INVALID_ARG
    assert L.mlp_train_step(h, fake, fake, None, None, fake, None, 10, fake, None) == \
        ffmlp.MLP_ERR_INVALID_ARG
    assert L.mlp_pack_weights(h, None, fake, None) == ffmlp.MLP_ERR_INVALID_ARG
    assert L.mlp_set_output_activation(h, 9) == ffmlp.MLP_ERR_UNSUPPORTED
    assert L.mlp_backward_dx(h, fake, fake, fake, fake, ctypes.c_void_p(0x1004), 10, fake, None) == \
        ffmlp.MLP_ERR_INVALID_ARG  # misaligned dX
    # optimizer: every check happens before the launch
    inv = ffmlp.MLP_ERR_INVALID_ARG
    assert L.mlp_sgd_step(h, None, fake, fake, None, 0.1, None) == inv
    assert L.mlp_sgd_step(h, fake, fake, fake, None, float("nan"), None) == inv
    assert L.mlp_sgd_step(h, ctypes.c_void_p(0x1002), fake, fake, None, 0.1, None) == inv
    assert L.mlp_adam_step(h, fake, fake, fake, fake, fake, None, 1e-3, 0.9, 0.999, 1e-8, 0, None) == inv
    assert "t = 0" in ffmlp.last_error()
    assert L.mlp_adam_step(h, fake, fake, fake, fake, fake, None, 1e-3, 1.0, 0.999, 1e-8, 1, None) == inv
    assert L.mlp_adam_step(h, fake, fake, fake, fake, fake, None, 1e-3, 0.9, 0.999, 0.0, 1, None) == inv
    assert L.mlp_adam_step(h, fake, None, fake, fake, fake, None, 1e-3, 0.9, 0.999, 1e-8, 1, None) == inv
    assert L.mlp_adam_step(h, fake, fake, fake, fake, fake, ctypes.c_void_p(0x1008), 1e-3, 0.9,
                           0.999, 1e-8, 1, None) == inv  # misaligned packed
    L.mlp_destroy(None)  # ignored


def test_binding_rejects_host_tensors_before_any_call(ffmlp):
    """The binding checks every tensor before calling into the library: a
    host tensor is refused with ValueError (no pointer reaches the C ABI)."""
    import torch
    net = ffmlp.FusedMLP(32, 2, 32, 16, "relu")
    X = torch.zeros(10, 32, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="GPU"):
        net.forward(torch.zeros(net.packed_bytes(), dtype=torch.uint8), X)
    with pytest.raises(ValueError, match="GPU"):
        net.pack(torch.zeros(net.param_count(), dtype=torch.bfloat16))
    with pytest.raises(ValueError):
        net.forward(None, X[0])  # not 2-D
