"""Pins for the fp64 oracle: checks against facts fixed by the mathematics,
not against the oracle's own formulas.

Each pin takes a loaded oracle (``oracle.Oracle``) and raises AssertionError on
failure.  ``ALL_PINS`` is run by ``test_oracle.py`` on the real oracle and by
``test_oracle_mutants.py`` on deliberately broken copies of it, where at least
one pin must fail for every planted mistake.

The definitions being pinned (LoRA: frozen W plus a scaled rank-r update, from
the paper's background on parameter-efficient fine-tuning; frozen-base forward
and input gradient with no weight gradient, from its "On-the-fly
Dequantization" algorithm; tokens as rows):
    Y = X W^T + s (X A^T) B^T,  dX = dY W + s (dY B) A,
    dA = s (dY B)^T X,          dB = s dY^T (X A^T).
A quantized frozen base is dequantized first, as in that algorithm:
    W = s W_q + b, one scale s and offset b per group of G inputs of a row.
The frozen LM head's reduced-vocabulary cross entropy with logits masking
(its "Softmax Approximation" and "Logits Masking" sections):
    loss_t = logsumexp_{j in J} h_t.w_j - h_t.w_{y_t} for trainable t,
    J = union of the first k entries of the similarity-table rows of the targets.
"""
from __future__ import annotations

import json
import os

import numpy as np

TIGHT = 1e-12
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden(name):
    """A hand-worked example from tests/golden (inputs, expected values, the
    passage that defines the operation and the derivation)."""
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _rng(seed):
    return np.random.default_rng(seed)


def _rand_case(T, K, N, r, seed=0):
    g = _rng(seed)
    return dict(X=g.standard_normal((T, K)), W=g.standard_normal((N, K)),
                A=g.standard_normal((r, K)), B=g.standard_normal((N, r)),
                dY=g.standard_normal((T, N)))


def _relmax(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    den = np.max(np.abs(ref)) if ref.size else 0.0
    num = np.max(np.abs(got - ref)) if ref.size else 0.0
    return num / den if den > 0 else num


def _full(o, c, s):
    U, Y = o.forward(c["X"], c["W"], c["A"], c["B"], s)
    bw = o.backward(c["X"], c["W"], c["A"], c["B"], c["dY"], s, U=U)
    return U, Y, bw


def pin_lora_worked_examples(o):
    """Hand-worked LoRA forward and backward (golden/lora_closed_form.json): a
    1x1x1 rank-1 case and a 1x2 -> 3 case with distinct entries, so that a
    transposed or mis-indexed operand changes the answer.  Exact in fp64."""
    for c in _golden("lora_closed_form.json")["cases"]:
        X, W, A, B, dY = (np.array(c[k], np.float64) for k in ("X", "W", "A", "B", "dY"))
        U, Y = o.forward(X, W, A, B, c["s"])
        bw = o.backward(X, W, A, B, dY, c["s"], U=U)
        got = {"U": U, "Y": Y, "G": bw["G"], "dU": bw["dU"], "dX": bw["dX"], "dA": bw["dA"], "dB": bw["dB"]}
        for k, v in c["expect"].items():
            assert got[k].tolist() == v, (c["name"], k, got[k].tolist(), v)


def pin_rank0_textbook_gemm(o):
    """r = 0 reduces to the plain GEMMs Y = X W^T and dX = dY W (numpy matmul)."""
    c = _rand_case(7, 5, 6, 0, seed=1)
    U, Y = o.forward(c["X"], c["W"], c["A"], c["B"], 2.0)
    assert U.shape == (7, 0)
    assert _relmax(Y, c["X"] @ c["W"].T) <= TIGHT
    dX = o.frozen_dx(c["dY"], c["W"])
    assert _relmax(dX, c["dY"] @ c["W"]) <= TIGHT


def pin_down_projection_gemm(o):
    """U = X A^T is itself a plain GEMM (numpy matmul)."""
    c = _rand_case(9, 11, 4, 3, seed=2)
    assert _relmax(o.u(c["X"], c["A"]), c["X"] @ c["A"].T) <= TIGHT


def pin_finite_differences(o):
    """L = sum(Y * dY) is affine in each of X, A, B, W taken alone, so central
    differences are exact up to rounding: they must reproduce dX, dA, dB."""
    T, K, N, r, s = 3, 5, 4, 2, 1.7
    c = _rand_case(T, K, N, r, seed=3)
    U, Y, bw = _full(o, c, s)

    def loss(X, W, A, B):
        _, Yp = o.forward(X, W, A, B, s)
        return float(np.sum(Yp * c["dY"]))

    h = 0.5
    for name, grad in (("X", bw["dX"]), ("A", bw["dA"]), ("B", bw["dB"])):
        base = c[name]
        fd = np.zeros_like(base)
        for idx in np.ndindex(base.shape):
            args = {k: c[k].copy() for k in ("X", "W", "A", "B")}
            args[name][idx] += h
            lp = loss(args["X"], args["W"], args["A"], args["B"])
            args[name][idx] -= 2 * h
            lm = loss(args["X"], args["W"], args["A"], args["B"])
            fd[idx] = (lp - lm) / (2 * h)
        assert _relmax(grad, fd) <= 1e-9, (name, _relmax(grad, fd))


def pin_dense_identities(o):
    """With W_eff = W + s B A (the merged LoRA weight):
    Y = X W_eff^T, dX = dY W_eff, dA = s B^T (dY^T X), dB = s (dY^T X) A^T."""
    T, K, N, r, s = 6, 8, 5, 3, 2.0
    c = _rand_case(T, K, N, r, seed=4)
    U, Y, bw = _full(o, c, s)
    W_eff = c["W"] + s * (c["B"] @ c["A"])
    G_xy = c["dY"].T @ c["X"]            # the dW that the method never forms, [N, K]
    assert _relmax(Y, c["X"] @ W_eff.T) <= TIGHT
    assert _relmax(bw["dX"], c["dY"] @ W_eff) <= TIGHT
    assert _relmax(bw["dA"], s * (c["B"].T @ G_xy)) <= TIGHT
    assert _relmax(bw["dB"], s * (G_xy @ c["A"].T)) <= TIGHT


def pin_zero_B(o):
    """B = 0: Y equals the rank-0 result bitwise, dA is exactly 0, dB = s dY^T U."""
    c = _rand_case(5, 8, 6, 2, seed=5)
    c["B"][:] = 0.0
    s = 2.0
    U, Y, bw = _full(o, c, s)
    _, Y0 = o.forward(c["X"], c["W"], c["A"][:0], c["B"][:, :0], s)
    assert np.array_equal(Y, Y0)
    assert np.all(bw["dA"] == 0.0)
    assert _relmax(bw["dB"], s * (c["dY"].T @ (c["X"] @ c["A"].T))) <= TIGHT
    assert np.any(bw["dB"] != 0.0)


def pin_zero_A(o):
    """A = 0: U = 0, Y = X W^T, dB is exactly 0, dA = s (dY B)^T X."""
    c = _rand_case(5, 8, 6, 2, seed=6)
    c["A"][:] = 0.0
    s = 2.0
    U, Y, bw = _full(o, c, s)
    assert np.all(U == 0.0)
    assert _relmax(Y, c["X"] @ c["W"].T) <= TIGHT
    assert np.all(bw["dB"] == 0.0)
    assert _relmax(bw["dA"], s * ((c["dY"] @ c["B"]).T @ c["X"])) <= TIGHT


def pin_zero_W(o):
    """W = 0 isolates the LoRA branch: Y = s U B^T, dX = dU A."""
    c = _rand_case(5, 8, 6, 3, seed=7)
    c["W"][:] = 0.0
    s = 3.0
    U, Y, bw = _full(o, c, s)
    assert _relmax(Y, s * (c["X"] @ c["A"].T) @ c["B"].T) <= TIGHT
    assert _relmax(bw["dX"], (s * (c["dY"] @ c["B"])) @ c["A"]) <= TIGHT


def pin_linear_in_scale(o):
    """Y(s) - Y(0) is proportional to s; dA, dB and dU are proportional to s."""
    c = _rand_case(4, 8, 5, 2, seed=8)
    _, Y0, _ = _full(o, c, 0.0)
    _, Y1, b1 = _full(o, c, 1.0)
    _, Y3, b3 = _full(o, c, 3.0)
    assert _relmax(Y3 - Y0, 3.0 * (Y1 - Y0)) <= 1e-11
    for k in ("dA", "dB", "dU"):
        assert _relmax(b3[k], 3.0 * b1[k]) <= TIGHT, k


def pin_token_split_additivity(o):
    """dA and dB are sums over tokens: the gradient over T equals the sum of the
    gradients over a split T = T1 + T2 (the data-parallel decomposition)."""
    c = _rand_case(9, 8, 6, 3, seed=9)
    s = 2.0
    _, _, full = _full(o, c, s)
    parts = []
    for sl in (slice(0, 4), slice(4, 9)):
        cc = dict(c, X=c["X"][sl], dY=c["dY"][sl])
        parts.append(_full(o, cc, s)[2])
    for k in ("dA", "dB"):
        assert _relmax(full[k], parts[0][k] + parts[1][k]) <= TIGHT, k
    # per-token outputs are the concatenation of the parts
    assert _relmax(full["dX"], np.concatenate([parts[0]["dX"], parts[1]["dX"]])) <= TIGHT


def pin_row_permutation(o):
    """Permuting token rows permutes Y, dX, U, G and leaves dA, dB unchanged."""
    c = _rand_case(8, 8, 6, 2, seed=10)
    s = 2.0
    U, Y, bw = _full(o, c, s)
    perm = _rng(11).permutation(8)
    cp = dict(c, X=c["X"][perm], dY=c["dY"][perm])
    Up, Yp, bwp = _full(o, cp, s)
    assert _relmax(Yp, Y[perm]) <= TIGHT
    assert _relmax(Up, U[perm]) <= TIGHT
    assert _relmax(bwp["dX"], bw["dX"][perm]) <= TIGHT
    assert _relmax(bwp["G"], bw["G"][perm]) <= TIGHT
    for k in ("dA", "dB"):
        assert _relmax(bwp[k], bw[k]) <= TIGHT, k


def pin_row_sampling(o):
    """Row-sampled Y and dX equal the corresponding rows of the full result."""
    c = _rand_case(10, 8, 6, 2, seed=12)
    s = 2.0
    U, Y, bw = _full(o, c, s)
    rows = [0, 3, 9]
    _, Ys = o.forward(c["X"], c["W"], c["A"], c["B"], s, rows=rows)
    assert np.array_equal(Ys, Y[rows])
    dXs = o.dx(c["dY"], c["W"], bw["dU"], c["A"], rows=rows)
    assert np.array_equal(dXs, bw["dX"][rows])


def pin_torch_autograd(o):
    """Independent library route: torch fp64 autograd of the LoRA forward."""
    import torch

    T, K, N, r, s = 6, 10, 7, 3, 2.0
    c = _rand_case(T, K, N, r, seed=13)
    t = {k: torch.tensor(v, dtype=torch.float64, requires_grad=(k in ("X", "A", "B")))
         for k, v in c.items()}
    Y_t = torch.nn.functional.linear(t["X"], t["W"]) + \
        s * torch.nn.functional.linear(torch.nn.functional.linear(t["X"], t["A"]), t["B"])
    Y_t.backward(t["dY"])
    U, Y, bw = _full(o, c, s)
    assert _relmax(Y, Y_t.detach().numpy()) <= TIGHT
    assert _relmax(bw["dX"], t["X"].grad.numpy()) <= TIGHT
    assert _relmax(bw["dA"], t["A"].grad.numpy()) <= TIGHT
    assert _relmax(bw["dB"], t["B"].grad.numpy()) <= TIGHT


# --- dequantization of a quantized frozen base (W = s W_q + b per group) --------
def pin_dequant_worked_example(o):
    """Codes and parameters worked by hand (golden/dequant_worked_example.json):
    4-bit codes two per byte across two groups, and 8-bit codes."""
    c4, c8 = _golden("dequant_worked_example.json")["cases"]
    Wq = np.zeros((1, c4["nbytes"]), np.uint8)
    for b, v in c4["bytes"].items():
        Wq[0, int(b)] = v
    W = o.dequant(Wq, np.array(c4["scale"]), np.array(c4["offset"]), c4["bits"], c4["group"])
    assert W.shape == (1, c4["K"])
    for k, v in c4["expect"].items():
        assert W[0, int(k)] == v, (k, W[0, int(k)], v)
    W8 = o.dequant(np.array([c8["codes"]], np.uint8), np.array(c8["scale"]), np.array(c8["offset"]),
                   c8["bits"], c8["group"])
    assert list(W8[0]) == c8["expect_row"]


def pin_dequant_unit_scale_is_the_codes(o):
    """With s = 1 and b = 0 the weight is the integer codes themselves, read out
    of the bytes with numpy's own bit operations (low nibble = even k)."""
    g = _rng(40)
    Wq = g.integers(0, 256, size=(5, 48), dtype=np.uint8)
    W8 = o.dequant(Wq, np.ones((5, 3)), np.zeros((5, 3)), 8, 16)
    assert np.array_equal(W8, Wq.astype(np.float64))
    W4 = o.dequant(Wq, np.ones((5, 6)), np.zeros((5, 6)), 4, 16)
    assert np.array_equal(W4[:, 0::2], (Wq & 0x0F).astype(np.float64))
    assert np.array_equal(W4[:, 1::2], (Wq >> 4).astype(np.float64))


def pin_dequant_groups(o):
    """Groups are G consecutive inputs of one row: with every code 1 and b = 0
    the weight is each group's scale repeated G times (numpy repeat); with
    s = 0 it is each group's offset repeated."""
    g = _rng(41)
    N, K, G = 4, 96, 32
    S, Bo = g.standard_normal((N, K // G)), g.standard_normal((N, K // G))
    ones4 = np.full((N, K // 2), 0x11, np.uint8)
    assert np.array_equal(o.dequant(ones4, S, np.zeros_like(Bo), 4, G), np.repeat(S, G, axis=1))
    codes = g.integers(0, 256, size=(N, K // 2), dtype=np.uint8)
    assert np.array_equal(o.dequant(codes, np.zeros_like(S), Bo, 4, G), np.repeat(Bo, G, axis=1))
    ones8 = np.ones((N, K), np.uint8)
    assert np.array_equal(o.dequant(ones8, S, np.zeros_like(Bo), 8, G), np.repeat(S, G, axis=1))


# --- reduced-vocabulary LM head cross entropy with logits masking --------------
def pin_ce_worked_example(o):
    """Hand-worked reduced-vocabulary cross entropy and dh
    (golden/ce_worked_example.json): D = 1, embeddings (1, 0, -1), hidden
    states 1 and 2 with targets 0 and 2."""
    c = _golden("ce_worked_example.json")
    loss, dH = o.ce_reduced(np.array(c["H"]), np.array(c["W"]), c["rows"], c["cols"], c["targets"])
    tol = c["tolerance"]
    assert np.abs(np.asarray(loss) - np.array(c["expect"]["loss"])).max() < tol
    assert np.abs(np.asarray(dH) - np.array(c["expect"]["dH"])).max() < tol


def _torch_ce(H, W, cols, rows, targets_local):
    """Cross entropy of the logits H[rows] W[cols]^T through torch (fp64) and
    the gradient of its sum with respect to H."""
    import torch
    h = torch.tensor(H, dtype=torch.float64, requires_grad=True)
    z = h[rows] @ torch.tensor(W, dtype=torch.float64)[cols].T
    l = torch.nn.functional.cross_entropy(z, torch.tensor(targets_local), reduction="none")
    l.sum().backward()
    return l.detach().numpy(), h.grad.numpy()


def pin_ce_full_vocab_is_torch_cross_entropy(o):
    """J = the whole vocabulary and every position trainable: the ordinary
    softmax cross entropy (torch) and its gradient."""
    g = _rng(50)
    T, V, D = 7, 23, 5
    H, W = g.standard_normal((T, D)), g.standard_normal((V, D))
    y = g.integers(0, V, size=T)
    rows, J = np.arange(T), np.arange(V)
    loss, dH = o.ce_reduced(H, W, rows, J, y)
    l_t, g_t = _torch_ce(H, W, J, rows, y)
    assert _relmax(loss, l_t) <= TIGHT
    assert _relmax(dH, g_t) <= TIGHT


def pin_ce_reduced_vocab_is_restricted_softmax(o):
    """A reduced J: the cross entropy of the logits restricted to the columns J
    with the target's position in J as the class (torch)."""
    g = _rng(51)
    T, V, D = 6, 40, 4
    H, W = g.standard_normal((T, D)), g.standard_normal((V, D))
    J = np.sort(g.choice(V, size=13, replace=False))
    tpos = g.integers(0, J.size, size=T)
    loss, dH = o.ce_reduced(H, W, np.arange(T), J, tpos)
    l_t, g_t = _torch_ce(H, W, J, np.arange(T), tpos)
    assert _relmax(loss, l_t) <= TIGHT
    assert _relmax(dH, g_t) <= TIGHT


def pin_ce_logits_masking_identity(o):
    """Logits masking (only the trainable rows) gives the same per-position
    losses and gradients as computing every row and masking the loss: the
    listed rows match, the others have zero gradient."""
    g = _rng(52)
    T, V, D = 9, 30, 6
    H, W = g.standard_normal((T, D)), g.standard_normal((V, D))
    J = np.arange(0, V, 2)
    tpos_all = g.integers(0, J.size, size=T)
    l_all, d_all = o.ce_reduced(H, W, np.arange(T), J, tpos_all)
    keep = np.array([1, 4, 5, 8])
    l_m, d_m = o.ce_reduced(H, W, keep, J, tpos_all[keep])
    assert np.array_equal(l_m, l_all[keep])
    assert np.array_equal(d_m[keep], d_all[keep])
    drop = np.setdiff1d(np.arange(T), keep)
    assert not np.any(d_m[drop])


def pin_ce_finite_differences(o):
    """d(sum of losses)/dH by central differences (the loss is smooth)."""
    g = _rng(53)
    T, V, D = 3, 8, 3
    H, W = g.standard_normal((T, D)), g.standard_normal((V, D))
    J, tpos = np.array([0, 2, 3, 7]), np.array([1, 3, 0])
    _, dH = o.ce_reduced(H, W, np.arange(T), J, tpos)
    eps = 1e-6
    for t in range(T):
        for d in range(D):
            Hp, Hm = H.copy(), H.copy()
            Hp[t, d] += eps
            Hm[t, d] -= eps
            fd = (o.ce_reduced(Hp, W, np.arange(T), J, tpos)[0].sum()
                  - o.ce_reduced(Hm, W, np.arange(T), J, tpos)[0].sum()) / (2 * eps)
            assert abs(fd - dH[t, d]) <= 1e-7 * max(1.0, abs(dH[t, d]))


def pin_reduced_vocab_union(o):
    """J is the union of the first k entries of the targets' table rows; with
    a table whose first entry of row i is i itself, J holds every target."""
    table = np.array([[0, 5, 2], [1, 0, 4], [2, 3, 1], [3, 2, 6], [4, 1, 0], [5, 0, 6], [6, 3, 5]])
    targets = np.array([3, 3, 5, 1, 6])
    J, tpos = o.reduced_vocab(table, 2, targets, np.array([0, 2, 3]))
    assert list(J) == [0, 1, 2, 3, 5]          # {3,2} | {5,0} | {1,0}
    assert list(J[tpos]) == [3, 5, 1]
    J1, _ = o.reduced_vocab(table, 1, targets, np.arange(5))
    assert list(J1) == [1, 3, 5, 6]


# --- top-k similarity table ------------------------------------------------------
def pin_topk_table_worked_example(o):
    """Four 2-d embeddings at angles 0, 30, 90 and 180 degrees, scaled
    differently (the table depends on directions only):
    golden/topk_worked_example.json."""
    c = _golden("topk_worked_example.json")
    A, C = o.topk_table(np.array(c["W"]), c["k"])
    assert [list(r) for r in A] == c["expect_table"]
    for i, m, v in c["expect_cos"]:
        assert abs(C[i, m] - v) < c["tolerance"], (i, m, C[i, m], v)


def pin_topk_table_is_argsort(o):
    """Against numpy: a stable argsort of each row of the normalised Gram
    matrix (descending), first k columns; the first entry of row i is i."""
    g = _rng(70)
    V, D, k = 60, 7, 9
    W = g.standard_normal((V, D))
    Wn = W / np.linalg.norm(W, axis=1, keepdims=True)
    S = Wn @ Wn.T
    ref = np.argsort(-S, axis=1, kind="stable")[:, :k]
    A, C = o.topk_table(W, k)
    assert np.array_equal(A, ref)
    assert np.array_equal(A[:, 0], np.arange(V))
    assert _relmax(C, np.take_along_axis(S, ref, axis=1)) <= 1e-13


def pin_topk_table_invariances(o):
    """Rescaling embeddings leaves the table unchanged; permuting the tokens
    permutes it accordingly."""
    g = _rng(71)
    V, D, k = 40, 5, 6
    W = g.standard_normal((V, D))
    A, _ = o.topk_table(W, k)
    A2, _ = o.topk_table(W * g.uniform(0.5, 3.0, size=(V, 1)), k)
    assert np.array_equal(A, A2)
    perm = g.permutation(V)
    Ap, _ = o.topk_table(W[perm], k)
    inv = np.argsort(perm)
    assert np.array_equal(perm[Ap], A[perm])
    del inv
    # a sample of rows is those rows of the full table
    rows = [3, 17, 39]
    Ar, Cr = o.topk_table(W, k, rows=rows)
    Af, Cf = o.topk_table(W, k)
    assert np.array_equal(Ar, Af[rows]) and np.array_equal(Cr, Cf[rows])


# --- chain of LoRA linears (checkpointed step) ----------------------------------
def pin_chain_finite_differences(o):
    """L = sum(x_2 * G) for a two-node chain: its gradients with respect to
    x_0, A_1 and B_2 by central differences match the chained backward (the
    loss is polynomial in each of them)."""
    g = _rng(60)
    T, d0, d1, d2, r = 3, 4, 5, 3, 2
    X0 = g.standard_normal((T, d0))
    n1 = dict(W=g.standard_normal((d1, d0)), A=g.standard_normal((r, d0)),
              B=g.standard_normal((d1, r)), s=0.7)
    n2 = dict(W=g.standard_normal((d2, d1)), A=g.standard_normal((r, d1)),
              B=g.standard_normal((d2, r)), s=1.3)
    G = g.standard_normal((T, d2))
    xs, grads, dX0 = o.chain(X0, [n1, n2], G)

    def loss(X0_, A1, B2):
        return float(np.sum(o.chain(X0_, [dict(n1, A=A1), dict(n2, B=B2)], G)[0][-1] * G))

    eps = 1e-5
    for name, arr, grad in (("X0", X0, dX0), ("A1", n1["A"], grads[0]["dA"]),
                            ("B2", n2["B"], grads[1]["dB"])):
        for idx in np.ndindex(arr.shape):
            P, M = arr.copy(), arr.copy()
            P[idx] += eps
            M[idx] -= eps
            args_p = {"X0": (P, n1["A"], n2["B"]), "A1": (X0, P, n2["B"]), "B2": (X0, n1["A"], P)}[name]
            args_m = {"X0": (M, n1["A"], n2["B"]), "A1": (X0, M, n2["B"]), "B2": (X0, n1["A"], M)}[name]
            fd = (loss(*args_p) - loss(*args_m)) / (2 * eps)
            assert abs(fd - grad[idx]) <= 1e-6 * max(1.0, abs(grad[idx])), (name, idx)


def pin_chain_of_one_is_one_layer(o):
    """A one-node chain is the single LoRA linear."""
    c = _rand_case(4, 6, 5, 2, seed=61)
    xs, grads, dX0 = o.chain(c["X"], [dict(W=c["W"], A=c["A"], B=c["B"], s=0.5)], c["dY"])
    U, Y, bw = _full(o, c, 0.5)
    assert np.array_equal(xs[0], Y) and np.array_equal(dX0, bw["dX"])
    assert np.array_equal(grads[0]["dA"], bw["dA"]) and np.array_equal(grads[0]["dB"], bw["dB"])


ALL_PINS = [
    pin_lora_worked_examples, pin_rank0_textbook_gemm,
    pin_down_projection_gemm, pin_finite_differences, pin_dense_identities,
    pin_zero_B, pin_zero_A, pin_zero_W, pin_linear_in_scale,
    pin_token_split_additivity, pin_row_permutation, pin_row_sampling,
    pin_torch_autograd, pin_dequant_worked_example, pin_dequant_unit_scale_is_the_codes,
    pin_dequant_groups, pin_ce_worked_example, pin_ce_full_vocab_is_torch_cross_entropy,
    pin_ce_reduced_vocab_is_restricted_softmax, pin_ce_logits_masking_identity,
    pin_ce_finite_differences, pin_reduced_vocab_union, pin_chain_finite_differences,
    pin_chain_of_one_is_one_layer, pin_topk_table_worked_example, pin_topk_table_is_argsort,
    pin_topk_table_invariances,
]


def run_all(o) -> list:
    """Run every pin; return the names of those that failed (or raised)."""
    failed = []
    for pin in ALL_PINS:
        try:
            pin(o)
        except Exception:  # noqa: BLE001 -- any error means the pin caught something
            failed.append(pin.__name__)
    return failed
