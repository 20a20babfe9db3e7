"""GPU parity of the frozen LM head's reduced-vocabulary cross entropy with
logits masking against the fp64 oracle: the reduced vocabulary J and the
targets' positions bit-exact; per-position losses, their sum and dh within the
bf16 tolerance (max relative error per tensor <= 2e-2)."""
import sys

import numpy as np
import pytest
import torch

from gpu_helpers import TOL, relerr
from workloads import head_inputs

pytestmark = pytest.mark.gpu

import paper_2606_19528_amd as lm  # noqa: E402


def _announce(msg):
    print(f"[case] {msg}", file=sys.stderr, flush=True)


def _gpu(d, k, want_dh=True, rows=None, J=None, tpos=None, dscale=1.0):
    g = {key: v.cuda() for key, v in d.items()}
    rows = g["rows"] if rows is None else rows.cuda()
    if J is None:
        J, tpos = lm.lm_head_build_vocab(g["table"], k, g["targets"], rows)
    else:
        J, tpos = J.cuda(), tpos.cuda()
    T, D = g["h"].shape
    loss = torch.empty(rows.shape[0], dtype=torch.float32, device="cuda")
    total = torch.empty(1, dtype=torch.float32, device="cuda")
    dh = torch.empty(T, D, dtype=torch.bfloat16, device="cuda") if want_dh else None
    lm.lm_head_reduced_ce(g["h"], g["W"], rows, J, tpos, loss, total, dh, dscale)
    torch.cuda.synchronize()
    return (J.cpu(), tpos.cpu(), loss.cpu(), total.cpu(), None if dh is None else dh.cpu())


def _case(orc, T, V, D, k, trainable=0.3, clusters=16, spread=8, seed=0):
    _announce(f"head T={T} V={V} D={D} k={k} trainable={trainable}")
    d = head_inputs(T, V, D, max(k, 4), trainable, clusters, spread, seed=seed)
    J, tpos, loss, total, dh = _gpu(d, k)
    Jr, tr = orc.reduced_vocab(d["table"].numpy(), k, d["targets"].numpy(), d["rows"].numpy())
    assert np.array_equal(J.numpy().astype(np.int64), Jr), "reduced vocabulary"
    assert np.array_equal(tpos.numpy().astype(np.int64), tr), "target positions"
    lr, dhr = orc.ce_reduced(d["h"], d["W"], d["rows"].numpy(), Jr, tr)
    tol = TOL[torch.bfloat16]
    e_loss = relerr(loss.double().numpy(), lr)
    e_tot = abs(float(total[0]) - lr.sum()) / abs(lr.sum())
    e_dh = relerr(dh.double().numpy(), dhr)
    _announce(f"  |J|={J.numel()} err loss {e_loss:.2e} total {e_tot:.2e} dh {e_dh:.2e}")
    assert e_loss <= tol and e_tot <= tol and e_dh <= tol
    return J.numel()


@pytest.mark.parametrize("shape", [
    (64, 500, 64, 4), (129, 3000, 136, 40), (200, 7000, 256, 300), (37, 1000, 24, 1),
])
def test_head_small(orc, shape):
    T, V, D, k = shape
    _case(orc, T, V, D, k, seed=T + V)


def test_head_all_positions_trainable(orc):
    _case(orc, 96, 2048, 128, 64, trainable=1.0, seed=5)


def test_head_several_backward_chunks(orc):
    # |J| above 8192: the backward recomputes the logits in several chunks
    nJ = _case(orc, 150, 40000, 128, 1000, clusters=24, spread=200, seed=9)
    assert nJ > 2 * 8192


def test_head_logits_masking_identity(orc):
    """Only the trainable positions' logits: their losses and dh rows equal
    those of the computation over every position with the same J, and every
    other dh row is zero (the paper's claim of identical losses and gradients)."""
    T, V, D, k = 160, 4000, 128, 100
    _announce("head logits-masking identity")
    d = head_inputs(T, V, D, k, 0.4, 8, 8, seed=13)
    all_rows = torch.arange(T, dtype=torch.int32)
    J, tpos_all = lm.lm_head_build_vocab(d["table"].cuda(), k, d["targets"].cuda(), all_rows.cuda())
    _, _, l_all, _, dh_all = _gpu(d, k, rows=all_rows, J=J.cpu(), tpos=tpos_all.cpu())
    keep = d["rows"].long()
    _, _, l_m, _, dh_m = _gpu(d, k, rows=d["rows"], J=J.cpu(), tpos=tpos_all.cpu()[keep])
    assert torch.equal(l_m, l_all[keep])
    assert torch.equal(dh_m[keep], dh_all[keep])
    drop = torch.ones(T, dtype=torch.bool)
    drop[keep] = False
    assert not dh_m[drop].float().abs().sum()


def test_head_invalid_target_gives_nan_loss(orc):
    # a target outside [0, V) is skipped, never followed: its loss is NaN, the
    # others are unaffected
    T, V, D, k = 64, 700, 64, 8
    d = head_inputs(T, V, D, k, 0.5, 4, 4, seed=17)
    d["targets"][-1] = V + 5
    _, tpos, loss, _, _ = _gpu(d, k, want_dh=False)
    assert int(tpos[-1]) == -1
    assert torch.isnan(loss[-1]) and torch.isfinite(loss[:-1]).all()


def test_head_deterministic(orc):
    d = head_inputs(120, 3000, 128, 50, 0.5, 8, 16, seed=19)
    a = _gpu(d, 50)
    b = _gpu(d, 50)
    for x, y in zip(a, b):
        assert torch.equal(x, y)
