"""Python access to the CPU oracle (oracle.c) for fully-fused MLPs.

TEST INFRASTRUCTURE ONLY.  This is the plain fp64 definition of Algorithm 1
(inference) and Algorithm 2 (training step) of arXiv 2403.17607, section
III-A, with bf16 rounding at the points where the GPU stores bf16 values.
Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import it; the GPU library never does, and this module imports nothing from
the GPU package.

Parity status of each oracle function (every one is pinned by a CPU test in
tests/test_oracle.py, against facts that do not come from the oracle):
  rne_bf16      pinned: torch's fp32 -> bf16 conversion (library) on fp32
                values, and hand-picked ties, subnormals and overflow.
  forward       pinned: depth 0 equals one library matmul; identity weights
                give relu(X) bitwise; zero input; power-of-two homogeneity;
                row permutation; brute force on 2x2 nets with hand-derived
                scalar formulas.
  backward /    pinned: finite differences of the loss (rounding off;
  train_step    every hidden and output activation, ReLU output included),
                the 2x2 brute-force formulas, depth 0 against a library
                matmul (all four output derivatives), the closed-form deltas
                of the identity net, rounding-on closed forms of depth-1 sine
                and sigmoid nets (bf16 cos C and A (1 - A) from the rounded
                A as the derivative sources), and additivity of G over a
                split batch.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

LINEAR, RELU, SIGMOID, SINE = 0, 1, 2, 3
ACTS = {"linear": LINEAR, "relu": RELU, "sigmoid": SIGMOID, "sine": SINE}


def build(force: bool = False) -> str:
    """Compile oracle.c into liboracle.so with gcc (fp64, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + f".tmp{os.getpid()}"
        cmd = ["gcc", "-std=c11", "-O2", "-ffp-contract=off", "-fopenmp",
               "-fPIC", "-shared", "-Wall", "-Wextra", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class _Net(ctypes.Structure):
    _fields_ = [("width", ctypes.c_int), ("depth", ctypes.c_int),
                ("in_dim", ctypes.c_int), ("out_dim", ctypes.c_int),
                ("act", ctypes.c_int), ("out_act", ctypes.c_int),
                ("round_bf16", ctypes.c_int), ("threads", ctypes.c_int)]


_lib = None


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        dp = ctypes.POINTER(ctypes.c_double)
        np_ = ctypes.POINTER(_Net)
        lib.orc_rne_bf16.argtypes = [ctypes.c_double]
        lib.orc_rne_bf16.restype = ctypes.c_double
        lib.orc_param_count.argtypes = [np_]
        lib.orc_param_count.restype = ctypes.c_int64
        lib.orc_forward.argtypes = [np_, dp, dp, ctypes.c_int64, dp, dp, dp]
        lib.orc_backward.argtypes = [np_, dp, dp, ctypes.c_int64, dp, dp, dp]
        lib.orc_backward_dx.argtypes = [np_, dp, dp, ctypes.c_int64, dp, dp, dp, dp]
        lib.orc_train_step.argtypes = [np_, dp, dp, dp, ctypes.c_int64, dp, dp,
                                       dp, dp, dp]
        for f in (lib.orc_forward, lib.orc_backward, lib.orc_backward_dx, lib.orc_train_step):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


def _f64(a) -> np.ndarray:
    if hasattr(a, "detach"):  # torch tensor
        a = a.detach().to("cpu").double().numpy()
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def rne_bf16(x: float) -> float:
    """Round one fp64 value to bf16, ties to even."""
    return _load().orc_rne_bf16(float(x))


@dataclass
class Net:
    """An MLP shape: depth hidden layers of ``width``, depth + 1 matrices."""
    width: int
    depth: int
    in_dim: int
    out_dim: int
    act: int = RELU
    out_act: int = LINEAR
    round_bf16: bool = True
    threads: int = 0

    def _c(self) -> _Net:
        return _Net(self.width, self.depth, self.in_dim, self.out_dim,
                    self.act, self.out_act, int(self.round_bf16), self.threads)

    @property
    def L(self) -> int:
        return self.depth + 1

    def shapes(self):
        return [(self.in_dim if l == 0 else self.width,
                 self.out_dim if l == self.L - 1 else self.width)
                for l in range(self.L)]

    def param_count(self) -> int:
        return int(_load().orc_param_count(ctypes.byref(self._c())))

    def split(self, flat):
        """Split a concatenated parameter vector into per-layer matrices."""
        flat = np.asarray(flat)
        out, off = [], 0
        for fi, fo in self.shapes():
            out.append(flat[off: off + fi * fo].reshape(fi, fo))
            off += fi * fo
        return out

    def forward(self, W, X, want_stash: bool = False):
        """Algorithm 1.  Returns (Y, Y32[, A]) as fp64 arrays; A has shape
        [depth, M, width] (the hidden activations A_2..A_L)."""
        W, X = _f64(W), _f64(X)
        M = X.shape[0]
        assert X.shape == (M, self.in_dim) and W.size == self.param_count()
        Y = np.zeros((M, self.out_dim))
        Y32 = np.zeros((M, self.out_dim))
        A = np.zeros((self.depth, M, self.width)) if want_stash else None
        rc = _load().orc_forward(ctypes.byref(self._c()), _ptr(W), _ptr(X), M,
                                 _ptr(Y), _ptr(Y32), _ptr(A))
        if rc != 0:
            raise ValueError("orc_forward rejected its arguments")
        return (Y, Y32, A) if want_stash else (Y, Y32)

    def _deltas(self, D, M):
        hidden = D[: self.depth * M * self.width].reshape(self.depth, M, self.width)
        out = D[self.depth * M * self.width:].reshape(M, self.out_dim)
        return list(hidden) + [out]

    def backward(self, W, X, dY, want_deltas: bool = False):
        """Backward pass of Algorithm 2 seeded with dY.  Returns G (flat fp64)
        and, if asked, the deltas [D_2, ..., D_{L+1}]."""
        W, X, dY = _f64(W), _f64(X), _f64(dY)
        M = X.shape[0]
        assert dY.shape == (M, self.out_dim)
        G = np.zeros(self.param_count())
        D = np.zeros(self.depth * M * self.width + M * self.out_dim) if want_deltas else None
        rc = _load().orc_backward(ctypes.byref(self._c()), _ptr(W), _ptr(X), M,
                                  _ptr(dY), _ptr(G), _ptr(D))
        if rc != 0:
            raise ValueError("orc_backward rejected its arguments")
        return (G, self._deltas(D, M)) if want_deltas else G

    def backward_dx(self, W, X, dY):
        """backward() plus the input gradient: returns (G, dX), dX [M, in_dim]
        fp64, the first hidden layer's delta times W_1^T (no rounding)."""
        W, X, dY = _f64(W), _f64(X), _f64(dY)
        M = X.shape[0]
        assert dY.shape == (M, self.out_dim)
        G = np.zeros(self.param_count())
        dX = np.zeros((M, self.in_dim))
        rc = _load().orc_backward_dx(ctypes.byref(self._c()), _ptr(W), _ptr(X), M,
                                     _ptr(dY), _ptr(G), None, _ptr(dX))
        if rc != 0:
            raise ValueError("orc_backward_dx rejected its arguments")
        return G, dX

    def train_step(self, W, X, T, want_deltas: bool = False):
        """Algorithm 2 with the MSE loss.  Returns dict with Y, Y32, G (flat),
        loss and, if asked, deltas."""
        W, X, T = _f64(W), _f64(X), _f64(T)
        M = X.shape[0]
        assert T.shape == (M, self.out_dim)
        Y = np.zeros((M, self.out_dim))
        Y32 = np.zeros((M, self.out_dim))
        G = np.zeros(self.param_count())
        loss = ctypes.c_double(0.0)
        D = np.zeros(self.depth * M * self.width + M * self.out_dim) if want_deltas else None
        rc = _load().orc_train_step(ctypes.byref(self._c()), _ptr(W), _ptr(X),
                                    _ptr(T), M, _ptr(Y), _ptr(Y32), _ptr(G),
                                    ctypes.byref(loss), _ptr(D))
        if rc != 0:
            raise ValueError("orc_train_step rejected its arguments")
        out = {"Y": Y, "Y32": Y32, "G": G, "loss": loss.value}
        if want_deltas:
            out["D"] = self._deltas(D, M)
        return out


# ------------------------------------------------------------- optimizer --
# The paper leaves the optimizer out of the training step (section III-A);
# applications need one.  These are the plain definitions, elementwise in
# fp64 numpy: SGD, and Adam as in Kingma & Ba (2015), Algorithm 1, with the
# bias corrections applied to the moment estimates.

def sgd_step(w, g, lr):
    """w - lr g."""
    return np.asarray(w, np.float64) - lr * np.asarray(g, np.float64)


def adam_step(w, m, v, g, lr, beta1, beta2, eps, t):
    """One Adam step (t = 1, 2, ...): returns (w, m, v).
    m <- beta1 m + (1 - beta1) g;  v <- beta2 v + (1 - beta2) g^2;
    w <- w - lr * (m / (1 - beta1^t)) / (sqrt(v / (1 - beta2^t)) + eps)."""
    w, m, v, g = (np.asarray(a, np.float64) for a in (w, m, v, g))
    m = beta1 * m + (1.0 - beta1) * g
    v = beta2 * v + (1.0 - beta2) * g * g
    mhat = m / (1.0 - beta1 ** t)
    vhat = v / (1.0 - beta2 ** t)
    return w - lr * mhat / (np.sqrt(vhat) + eps), m, v


def to_bf16(w):
    """Round every value to bf16 (round to nearest, ties to even)."""
    return np.vectorize(rne_bf16, otypes=[np.float64])(np.asarray(w, np.float64))
