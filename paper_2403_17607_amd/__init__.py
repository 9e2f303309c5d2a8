"""Fully-fused narrow MLPs on AMD Instinct MI355X (gfx950).

Python binding of libffmlp.so, the C-ABI library declared in
include/ffmlp.h.  Every computation runs in the library's HIP kernels; this
module only marshals arguments (tensor data pointers, the current HIP
stream) and allocates device memory through PyTorch.  If the library is not
built, importing the low-level functions raises: there is no fallback.

Operations (arXiv 2403.17607, section III-A):
  * forward      -- Algorithm 1, inference; optionally keeps the training
                    stash for a later backward.
  * backward     -- the backward half of Algorithm 2 seeded with dY: weight
                    gradients G_i = A_i^T D_{i+1}, no input gradient.
  * train_step   -- Algorithm 2 with the mean-squared-error loss.

Example::

    net = FusedMLP(width=64, depth=4, in_dim=64, out_dim=16, activation="relu")
    packed = net.pack(W)              # W: bf16 [param_count] on the GPU
    Y = net.forward(packed, X)        # X: bf16 [M, in_dim]
    ws = net.workspace(M)
    G, loss = net.train_step(packed, X, T, ws)
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libffmlp.so")

MLP_OK = 0
MLP_ERR_INVALID_ARG = -1
MLP_ERR_UNSUPPORTED = -2
MLP_ERR_WORKSPACE = -3
MLP_ERR_HIP = -4
MLP_SCRATCH_BYTES = 64 << 20
MLP_MODE_INFER = 0
MLP_MODE_TRAIN = 1

ACTIVATIONS = {"linear": 0, "relu": 1, "sigmoid": 2, "sine": 3}
WIDTHS = (16, 32, 64, 128)

# Every exported symbol of include/ffmlp.h with its ctypes signature.
_VP = ctypes.c_void_p
_SIGNATURES = {
    "mlp_create": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                   ctypes.c_int, ctypes.POINTER(_VP)]),
    "mlp_set_output_activation": (ctypes.c_int, [_VP, ctypes.c_int]),
    "mlp_destroy": (None, [_VP]),
    "mlp_param_count": (ctypes.c_int64, [_VP]),
    "mlp_layer_shape": (ctypes.c_int, [_VP, ctypes.c_int, ctypes.POINTER(ctypes.c_int),
                                       ctypes.POINTER(ctypes.c_int),
                                       ctypes.POINTER(ctypes.c_int64)]),
    "mlp_packed_bytes": (ctypes.c_size_t, [_VP]),
    "mlp_pack_weights": (ctypes.c_int, [_VP, _VP, _VP, _VP]),
    "mlp_workspace_bytes": (ctypes.c_size_t, [_VP, ctypes.c_int64, ctypes.c_int]),
    "mlp_forward": (ctypes.c_int, [_VP, _VP, _VP, _VP, ctypes.c_int64, _VP, _VP]),
    "mlp_backward": (ctypes.c_int, [_VP, _VP, _VP, _VP, _VP, ctypes.c_int64, _VP, _VP]),
    "mlp_backward_dx": (ctypes.c_int, [_VP, _VP, _VP, _VP, _VP, _VP, ctypes.c_int64, _VP, _VP]),
    "mlp_train_step": (ctypes.c_int, [_VP, _VP, _VP, _VP, _VP, _VP, _VP, ctypes.c_int64,
                                      _VP, _VP]),
    "mlp_train_step_noalloc": (ctypes.c_int, [_VP, _VP, _VP, _VP, _VP, _VP, _VP, ctypes.c_int64,
                                              _VP]),
    "mlp_sgd_step": (ctypes.c_int, [_VP, _VP, _VP, _VP, _VP, ctypes.c_float, _VP]),
    "mlp_adam_step": (ctypes.c_int, [_VP, _VP, _VP, _VP, _VP, _VP, _VP, ctypes.c_float,
                                     ctypes.c_float, ctypes.c_float, ctypes.c_float,
                                     ctypes.c_int64, _VP]),
    "mlp_last_error": (ctypes.c_char_p, []),
}

_lib = None


class FFMLPError(RuntimeError):
    """A library call returned an error code."""

    def __init__(self, code: int, msg: str):
        super().__init__(f"ffmlp error {code}: {msg}")
        self.code = code


def lib() -> ctypes.CDLL:
    """The loaded libffmlp.so.  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2403_17607_amd.build`")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def last_error() -> str:
    return lib().mlp_last_error().decode()


def _check(rc: int) -> None:
    if rc != MLP_OK:
        raise FFMLPError(rc, last_error())


def _ptr(t) -> int | None:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensor must be on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


def _require(t, name: str, dtype, shape=None, min_numel=None, device=None) -> None:
    """Raise ValueError unless tensor `t` is a contiguous GPU tensor of
    `dtype` (and `shape`, at least `min_numel` elements, on `device`).  The
    C ABI derives every offset from M and the handle's dims and cannot see
    buffer sizes, so these checks are what stands between a short or
    mistyped buffer and an out-of-bounds access on the GPU; they run before
    any launch and survive `python -O`."""
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on the GPU")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if min_numel is not None and t.numel() < min_numel:
        raise ValueError(f"{name} holds {t.numel()} elements, needs at least {min_numel}")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, the other arguments on {device}")


_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)


def _stream(device) -> int:
    """The current HIP stream of `device` as an integer handle.  torch's
    raw accessor takes about 0.2 us where current_stream() takes 2, which
    matters for small batches, whose kernels run for a few microseconds."""
    if _raw_stream is not None and device.index is not None:
        return _raw_stream(device.index)
    return torch.cuda.current_stream(device).cuda_stream


def _act(a) -> int:
    if isinstance(a, int):
        return a
    return ACTIVATIONS[a]


class FusedMLP:
    """A handle on an MLP shape: `depth` hidden layers of `width` neurons,
    `depth + 1` weight matrices, hidden activation `activation` and output
    activation `output_activation`.  Holds no device memory."""

    def __init__(self, width: int, depth: int, in_dim: int, out_dim: int,
                 activation="relu", output_activation="linear"):
        h = _VP()
        _check(lib().mlp_create(width, depth, in_dim, out_dim, _act(activation), ctypes.byref(h)))
        self._h = h
        _check(lib().mlp_set_output_activation(h, _act(output_activation)))
        self.width, self.depth, self.in_dim, self.out_dim = width, depth, in_dim, out_dim
        self.activation = _act(activation)
        self.output_activation = _act(output_activation)

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and _lib is not None:
            _lib.mlp_destroy(h)
            self._h = None

    # ------------------------------------------------------------ shapes --
    @property
    def handle(self):
        return self._h

    @property
    def n_layers(self) -> int:
        return self.depth + 1

    def param_count(self) -> int:
        return int(lib().mlp_param_count(self._h))

    def layer_shape(self, l: int):
        fi, fo, off = ctypes.c_int(), ctypes.c_int(), ctypes.c_int64()
        _check(lib().mlp_layer_shape(self._h, l, ctypes.byref(fi), ctypes.byref(fo),
                                     ctypes.byref(off)))
        return fi.value, fo.value, off.value

    def packed_bytes(self) -> int:
        return int(lib().mlp_packed_bytes(self._h))

    def workspace_bytes(self, M: int, mode: int = MLP_MODE_TRAIN) -> int:
        return int(lib().mlp_workspace_bytes(self._h, M, mode))

    def workspace(self, M: int, device="cuda") -> torch.Tensor:
        """A training workspace for a batch of exactly M rows."""
        return torch.empty(max(self.workspace_bytes(M), 1), dtype=torch.uint8, device=device)

    # -------------------------------------------------------------- calls --
    def pack(self, W: torch.Tensor, out: torch.Tensor | None = None) -> torch.Tensor:
        """Pack bf16 weights [param_count] (concatenated row-major matrices)."""
        _require(W, "W", torch.bfloat16, shape=(self.param_count(),))
        if out is None:
            out = torch.empty(self.packed_bytes(), dtype=torch.uint8, device=W.device)
        _require(out, "packed", torch.uint8, min_numel=self.packed_bytes(), device=W.device)
        _check(lib().mlp_pack_weights(self._h, _ptr(W), _ptr(out), _stream(W.device)))
        return out

    def forward(self, packed: torch.Tensor, X: torch.Tensor, Y: torch.Tensor | None = None,
                stash: torch.Tensor | None = None) -> torch.Tensor:
        """Algorithm 1.  X bf16 [M, in_dim] -> Y bf16 [M, out_dim].  With a
        training workspace as `stash`, also keeps the activations."""
        M = self._check_x(X)
        self._check_packed(packed, X.device)
        if Y is None:
            Y = torch.empty(M, self.out_dim, dtype=torch.bfloat16, device=X.device)
        _require(Y, "Y", torch.bfloat16, shape=(M, self.out_dim), device=X.device)
        if stash is not None:
            self._check_ws(stash, M, X.device, "stash")
        _check(lib().mlp_forward(self._h, _ptr(packed), _ptr(X), _ptr(Y), M, _ptr(stash),
                                 _stream(X.device)))
        return Y

    def backward(self, packed: torch.Tensor, X: torch.Tensor, dY: torch.Tensor,
                 ws: torch.Tensor, G: torch.Tensor | None = None) -> torch.Tensor:
        """Weight gradients for a caller-given dY (fp32 [M, out_dim]) after
        forward(..., stash=ws)."""
        M = self._check_x(X)
        self._check_packed(packed, X.device)
        _require(dY, "dY", torch.float32, shape=(M, self.out_dim), device=X.device)
        self._check_ws(ws, M, X.device)
        if G is None:
            G = torch.empty(self.param_count(), dtype=torch.float32, device=X.device)
        _require(G, "G", torch.float32, shape=(self.param_count(),), device=X.device)
        _check(lib().mlp_backward(self._h, _ptr(packed), _ptr(X), _ptr(dY), _ptr(G), X.shape[0],
                                  _ptr(ws), _stream(X.device)))
        return G

    def sgd_step(self, master: torch.Tensor, G: torch.Tensor, W: torch.Tensor,
                 packed: torch.Tensor | None, lr: float) -> None:
        """master -= lr G (fp32); W = bf16(master); re-packs into `packed`
        when given."""
        self._check_params(master, G, W, packed)
        _check(lib().mlp_sgd_step(self._h, _ptr(master), _ptr(G), _ptr(W), _ptr(packed), lr,
                                  _stream(master.device)))

    def adam_step(self, master: torch.Tensor, m: torch.Tensor, v: torch.Tensor, G: torch.Tensor,
                  W: torch.Tensor, packed: torch.Tensor | None, lr: float,
                  betas=(0.9, 0.999), eps: float = 1e-8, t: int = 1) -> None:
        """One Adam step t (1, 2, ...) on fp32 master weights and moments;
        W = bf16(master); re-packs into `packed` when given."""
        self._check_params(master, G, W, packed)
        for name, b in (("m", m), ("v", v)):
            _require(b, name, torch.float32, shape=(self.param_count(),), device=master.device)
        _check(lib().mlp_adam_step(self._h, _ptr(master), _ptr(m), _ptr(v), _ptr(G), _ptr(W),
                                   _ptr(packed), lr, betas[0], betas[1], eps, t,
                                   _stream(master.device)))

    # ------------------------------------------------- argument checks --
    def _check_params(self, master, G, W, packed):
        n = self.param_count()
        _require(master, "master", torch.float32, shape=(n,))
        _require(G, "G", torch.float32, shape=(n,), device=master.device)
        _require(W, "W", torch.bfloat16, shape=(n,), device=master.device)
        if packed is not None:
            self._check_packed(packed, master.device)

    def _check_x(self, X) -> int:
        """X must be bf16 [M, in_dim] on the GPU; returns M."""
        if not isinstance(X, torch.Tensor) or X.dim() != 2:
            raise ValueError("X must be a 2-D tensor [M, in_dim]")
        _require(X, "X", torch.bfloat16, shape=(X.shape[0], self.in_dim))
        return X.shape[0]

    def _check_packed(self, packed, device):
        _require(packed, "packed", torch.uint8, min_numel=self.packed_bytes(), device=device)

    def _check_ws(self, ws, M, device, name="ws"):
        _require(ws, name, torch.uint8, min_numel=self.workspace_bytes(M), device=device)

    def backward_dx(self, packed: torch.Tensor, X: torch.Tensor, dY: torch.Tensor,
                    ws: torch.Tensor, G: torch.Tensor | None = None,
                    dX: torch.Tensor | None = None):
        """backward() plus the input gradient dX (fp32 [M, in_dim]); returns
        (G, dX)."""
        M = self._check_x(X)
        self._check_packed(packed, X.device)
        _require(dY, "dY", torch.float32, shape=(M, self.out_dim), device=X.device)
        self._check_ws(ws, M, X.device)
        if G is None:
            G = torch.empty(self.param_count(), dtype=torch.float32, device=X.device)
        _require(G, "G", torch.float32, shape=(self.param_count(),), device=X.device)
        if dX is None:
            dX = torch.empty(M, self.in_dim, dtype=torch.float32, device=X.device)
        _require(dX, "dX", torch.float32, shape=(M, self.in_dim), device=X.device)
        _check(lib().mlp_backward_dx(self._h, _ptr(packed), _ptr(X), _ptr(dY), _ptr(G), _ptr(dX),
                                     M, _ptr(ws), _stream(X.device)))
        return G, dX

    def train_step(self, packed: torch.Tensor, X: torch.Tensor, T: torch.Tensor,
                   ws: torch.Tensor, G: torch.Tensor | None = None, Y: torch.Tensor | None = None,
                   loss: torch.Tensor | None = None):
        """Algorithm 2 with the MSE loss.  Returns (G, loss) as device
        tensors; Y, if given, receives the bf16 outputs."""
        M = self._check_x(X)
        dev = X.device
        self._check_packed(packed, dev)
        _require(T, "T", torch.float32, shape=(M, self.out_dim), device=dev)
        self._check_ws(ws, M, dev)
        if G is None:
            G = torch.empty(self.param_count(), dtype=torch.float32, device=dev)
        _require(G, "G", torch.float32, shape=(self.param_count(),), device=dev)
        if loss is None:
            loss = torch.empty(1, dtype=torch.float32, device=dev)
        _require(loss, "loss", torch.float32, min_numel=1, device=dev)
        if Y is not None:
            _require(Y, "Y", torch.bfloat16, shape=(M, self.out_dim), device=dev)
        _check(lib().mlp_train_step(self._h, _ptr(packed), _ptr(X), _ptr(T), _ptr(Y), _ptr(G),
                                    _ptr(loss), X.shape[0], _ptr(ws), _stream(dev)))
        return G, loss

    def train_step_noalloc(self, packed: torch.Tensor, X: torch.Tensor, T: torch.Tensor,
                           G: torch.Tensor, loss: torch.Tensor, Y: torch.Tensor | None = None):
        """train_step with the library's static scratch array as the
        workspace: nothing is allocated, so the caller passes G and loss.
        Batches needing more than MLP_SCRATCH_BYTES of workspace are refused
        by the library (FFMLPError, MLP_ERR_WORKSPACE)."""
        M = self._check_x(X)
        dev = X.device
        self._check_packed(packed, dev)
        _require(T, "T", torch.float32, shape=(M, self.out_dim), device=dev)
        _require(G, "G", torch.float32, shape=(self.param_count(),), device=dev)
        _require(loss, "loss", torch.float32, min_numel=1, device=dev)
        if Y is not None:
            _require(Y, "Y", torch.bfloat16, shape=(M, self.out_dim), device=dev)
        _check(lib().mlp_train_step_noalloc(self._h, _ptr(packed), _ptr(X), _ptr(T), _ptr(Y),
                                            _ptr(G), _ptr(loss), M, _stream(dev)))
        return G, loss
