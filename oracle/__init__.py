"""fp64 CPU oracle for the LoRA-adapted linear layer -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its binding in ``paper_2606_19528_amd``) never imports, links or calls it, and
this package imports nothing from the product.

The arithmetic lives in ``lora_oracle.c`` (plain fp64 loops, ascending-index
sums).  This module only marshals numpy float64 arrays into it and composes the
per-definition functions into the forward and backward passes:

    forward:   U = X A^T ;  Y = X W^T + s U B^T
    backward:  G = dY B ; dU = s G ; dX = dY W + dU A ; dA = dU^T X ;
               dB = s dY^T U
    quantized base:  W = S * W_q + Bo per group (dequant), then as above
    table:     row i = the k tokens most cosine-similar to token i (topk_table)
    LM head:   J = union of top-k table rows of the trainable targets;
               loss_t = logsumexp_{j in J} h_t.w_j - h_t.w_{y_t};  dH (ce_reduced)

(LoRA as described in the paper's background on parameter-efficient
fine-tuning, with r and alpha from its hyperparameter table; frozen-base
forward and input gradient as in its "On-the-fly Dequantization" algorithm,
with tokens as rows.)

If the shared object has not been built yet it is compiled here with gcc.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "lora_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liblora_oracle.so")

GCC_FLAGS = ["-O2", "-fPIC", "-shared", "-fopenmp", "-std=c11"]


def build_shared(src: str = _SRC, out: str = _LIB_PATH) -> str:
    """Compile the oracle source into a shared object (gcc -O2, no fast-math)."""
    cmd = ["gcc", *GCC_FLAGS, "-o", out, src, "-lm"]
    subprocess.run(cmd, check=True)
    return out


_i64 = ctypes.c_int64
_dp = ctypes.POINTER(ctypes.c_double)
_lp = ctypes.POINTER(ctypes.c_int64)


def _declare(lib: ctypes.CDLL) -> ctypes.CDLL:
    lib.oracle_lora_u.argtypes = [_dp, _dp, _i64, _i64, _i64, _dp]
    lib.oracle_lora_y_rows.argtypes = [_dp, _dp, _dp, _dp, _i64, _i64, _i64, _i64,
                                       ctypes.c_double, _lp, _i64, _dp]
    lib.oracle_lora_grad_u.argtypes = [_dp, _dp, _i64, _i64, _i64, ctypes.c_double, _dp, _dp]
    lib.oracle_lora_dx_rows.argtypes = [_dp, _dp, _dp, _dp, _i64, _i64, _i64, _i64,
                                        _lp, _i64, _dp]
    lib.oracle_lora_da.argtypes = [_dp, _dp, _i64, _i64, _i64, _dp]
    lib.oracle_lora_db.argtypes = [_dp, _dp, _i64, _i64, _i64, ctypes.c_double, _dp]
    lib.oracle_dequant.argtypes = [ctypes.POINTER(ctypes.c_uint8), _dp, _dp, _i64, _i64,
                                   ctypes.c_int, _i64, _dp]
    lib.oracle_ce_reduced.argtypes = [_dp, _dp, _i64, _i64, _lp, _i64, _lp, _i64, _lp, _dp, _dp]
    lib.oracle_topk_table.argtypes = [_dp, _i64, _i64, _i64, _lp, _i64, _lp, _dp]
    for name in ("oracle_lora_u", "oracle_lora_y_rows", "oracle_lora_grad_u",
                 "oracle_lora_dx_rows", "oracle_lora_da", "oracle_lora_db", "oracle_dequant",
                 "oracle_ce_reduced", "oracle_topk_table"):
        getattr(lib, name).restype = None
    lib.oracle_threads.argtypes = []
    lib.oracle_threads.restype = ctypes.c_int
    lib.oracle_set_threads.argtypes = [ctypes.c_int]
    lib.oracle_set_threads.restype = None
    return lib


def load(path: str | None = None) -> "Oracle":
    """Load an oracle shared object (default: the in-tree build, built on demand)."""
    if path is None:
        path = _LIB_PATH
        if not os.path.exists(path):
            build_shared()
    return Oracle(_declare(ctypes.CDLL(path)))


def _f64(a) -> np.ndarray:
    """Exact upcast to a C-contiguous float64 array (accepts numpy or torch CPU)."""
    if hasattr(a, "detach"):
        a = a.detach().to("cpu")
        import torch  # local: only needed for torch inputs

        a = a.to(torch.float64).numpy()
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(_dp)


def _rows(rows):
    if rows is None:
        return None, 0, None
    r = np.ascontiguousarray(rows, dtype=np.int64)
    return r.ctypes.data_as(_lp), r.size, r


class Oracle:
    """Thin marshalling wrapper over one loaded oracle shared object."""

    def __init__(self, lib: ctypes.CDLL):
        self.lib = lib

    def threads(self) -> int:
        return int(self.lib.oracle_threads())

    def set_threads(self, n: int) -> None:
        """OpenMP threads of the following calls (timing only)."""
        self.lib.oracle_set_threads(int(n))

    # --- one definition per call -------------------------------------------------
    def u(self, X, A):
        X, A = _f64(X), _f64(A)
        T, K = X.shape
        r = A.shape[0]
        U = np.zeros((T, r), np.float64)
        if r:
            self.lib.oracle_lora_u(_ptr(X), _ptr(A), T, K, r, _ptr(U))
        return U

    def y(self, X, W, U, B, s, rows=None):
        X, W, U, B = _f64(X), _f64(W), _f64(U), _f64(B)
        T, K = X.shape
        N = W.shape[0]
        r = U.shape[1]
        rp, nr, keep = _rows(rows)
        Y = np.zeros((nr if rows is not None else T, N), np.float64)
        self.lib.oracle_lora_y_rows(_ptr(X), _ptr(W), _ptr(U), _ptr(B.reshape(N, r) if r else np.zeros((N, 1))),
                                    T, K, N, r, float(s), rp, nr, _ptr(Y))
        del keep
        return Y

    def grad_u(self, dY, B, s):
        dY, B = _f64(dY), _f64(B)
        T, N = dY.shape
        r = B.shape[1] if B.ndim == 2 else 0
        G = np.zeros((T, r), np.float64)
        dU = np.zeros((T, r), np.float64)
        if r:
            self.lib.oracle_lora_grad_u(_ptr(dY), _ptr(B), T, N, r, float(s), _ptr(G), _ptr(dU))
        return G, dU

    def dx(self, dY, W, dU, A, rows=None):
        dY, W, dU, A = _f64(dY), _f64(W), _f64(dU), _f64(A)
        T, N = dY.shape
        K = W.shape[1]
        r = dU.shape[1]
        rp, nr, keep = _rows(rows)
        dX = np.zeros((nr if rows is not None else T, K), np.float64)
        self.lib.oracle_lora_dx_rows(_ptr(dY), _ptr(W), _ptr(dU), _ptr(A if r else np.zeros((1, K))),
                                     T, K, N, r, rp, nr, _ptr(dX))
        del keep
        return dX

    def da(self, dU, X):
        dU, X = _f64(dU), _f64(X)
        T, K = X.shape
        r = dU.shape[1]
        dA = np.zeros((r, K), np.float64)
        if r:
            self.lib.oracle_lora_da(_ptr(dU), _ptr(X), T, K, r, _ptr(dA))
        return dA

    def db(self, dY, U, s):
        dY, U = _f64(dY), _f64(U)
        T, N = dY.shape
        r = U.shape[1]
        dB = np.zeros((N, r), np.float64)
        if r:
            self.lib.oracle_lora_db(_ptr(dY), _ptr(U), T, N, r, float(s), _ptr(dB))
        return dB

    # --- composed passes ---------------------------------------------------------
    def forward(self, X, W, A, B, s, rows=None):
        """Returns (U [T,r], Y) where Y holds the requested rows (all if None)."""
        U = self.u(X, A)
        return U, self.y(X, W, U, B, s, rows=rows)

    def backward(self, X, W, A, B, dY, s, U=None, dx_rows=None, want_dx=True):
        """Returns dict with U, G, dU, dX (requested rows), dA, dB."""
        if U is None:
            U = self.u(X, A)
        G, dU = self.grad_u(dY, B, s)
        out = {"U": U, "G": G, "dU": dU, "dA": self.da(dU, X), "dB": self.db(dY, U, s)}
        if want_dx:
            out["dX"] = self.dx(dY, W, dU, A, rows=dx_rows)
        return out

    def topk_table(self, W, k, rows=None):
        """(A [n, k] int64, C [n, k] fp64): each token's k most cosine-similar
        tokens (itself first for distinct directions) and their similarities,
        for every token (rows None) or the listed ones."""
        W = _f64(W)
        V, D = W.shape
        rp, nr, keep = _rows(rows)
        n = V if rows is None else nr
        A = np.empty((n, k), dtype=np.int64)
        C = np.empty((n, k), dtype=np.float64)
        self.lib.oracle_topk_table(_ptr(W), V, D, k, rp, nr, A.ctypes.data_as(_lp), _ptr(C))
        del keep
        return A, C

    def chain(self, X0, nodes, G_last):
        """A chain of LoRA linears, x_i = f_i(x_{i-1}) with f_i the LoRA
        forward above (nodes: dicts W, A, B, s), and its backward from
        G_last = dL/dx_n by the chain rule (dy_i = dx_{i+1}).  Returns the
        outputs [x_1 .. x_n] and per node dA, dB, plus dx_0.  (The paper's
        checkpointed schedule recomputes and reloads, but computes exactly
        these values.)"""
        xs = [_f64(X0)]
        for nd in nodes:
            _, Y = self.forward(xs[-1], nd["W"], nd["A"], nd["B"], nd["s"])
            xs.append(Y)
        g = _f64(G_last)
        grads = [None] * len(nodes)
        for i in range(len(nodes) - 1, -1, -1):
            nd = nodes[i]
            bw = self.backward(xs[i], nd["W"], nd["A"], nd["B"], g, nd["s"])
            grads[i] = {"dA": bw["dA"], "dB": bw["dB"]}
            g = bw["dX"]
        return xs[1:], grads, g

    def dequant(self, Wq, S, Bo, bits, G):
        """W = S * q + Bo per group of G inputs (fp64 [N, K]) from the codes in
        Wq ([N, K*bits/8] uint8) and the per-group scales S / offsets Bo."""
        if hasattr(Wq, "detach"):
            Wq = Wq.detach().to("cpu").numpy()
        Wq = np.ascontiguousarray(Wq, dtype=np.uint8)
        S, Bo = _f64(S), _f64(Bo)
        N = Wq.shape[0]
        K = Wq.shape[1] * 8 // bits
        assert bits in (4, 8) and K % G == 0 and S.shape == (N, K // G) == Bo.shape
        W = np.empty((N, K), dtype=np.float64)
        self.lib.oracle_dequant(Wq.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)), _ptr(S),
                                _ptr(Bo), N, K, bits, G, _ptr(W))
        return W

    # --- reduced-vocabulary LM head with logits masking ---------------------------
    @staticmethod
    def reduced_vocab(table, k, targets, rows):
        """J = union over the listed positions t of the first k entries of the
        table row of the target y_t (sorted ascending), and the position of
        each listed target in J."""
        table = np.asarray(table)
        targets = np.asarray(targets, dtype=np.int64)
        rows = np.asarray(rows, dtype=np.int64)
        J = np.unique(table[targets[rows], :k].reshape(-1)).astype(np.int64)
        tpos = np.searchsorted(J, targets[rows]).astype(np.int64)
        return J, tpos

    def ce_reduced(self, H, W, rows, J, tpos):
        """Per-position losses (for the listed rows) and dH (fp64 [T, D]) of the
        reduced-vocabulary cross entropy; see oracle_ce_reduced."""
        H, W = _f64(H), _f64(W)
        T, D = H.shape
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        J = np.ascontiguousarray(J, dtype=np.int64)
        tpos = np.ascontiguousarray(tpos, dtype=np.int64)
        assert W.shape[1] == D and rows.size == tpos.size
        loss = np.empty(rows.size, dtype=np.float64)
        dH = np.empty((T, D), dtype=np.float64)
        self.lib.oracle_ce_reduced(_ptr(H), _ptr(W), T, D, rows.ctypes.data_as(_lp), rows.size,
                                   J.ctypes.data_as(_lp), J.size, tpos.ctypes.data_as(_lp),
                                   _ptr(loss), _ptr(dH))
        return loss, dH

    def frozen_dx(self, dY, W, rows=None):
        """Rank-0 frozen linear input gradient dX = dY W."""
        dY, W = _f64(dY), _f64(W)
        T = dY.shape[0]
        K = W.shape[1]
        return self.dx(dY, W, np.zeros((T, 0)), np.zeros((0, K)), rows=rows)
