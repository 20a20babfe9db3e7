"""CPU tests of the C ABI's host logic: the library loads, exports every symbol
its header declares, sizes workspaces and rejects bad arguments before any
device work (fake, never-dereferenced pointers are used, so no GPU is needed).
"""
import ctypes
import os
import re

import pytest

import paper_2606_19528_amd as lm
from paper_2606_19528_amd import lora as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lora_mi355x.h")

EINVAL, EUNSUP, EWS = L.LORA_EINVAL, L.LORA_EUNSUPPORTED, L.LORA_EWORKSPACE


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    names = re.findall(r"^[A-Za-z_][\w \t\*]*?\b([a-z_][a-z0-9_]*)\s*\(", src, flags=re.M)
    return sorted(set(n for n in names if n not in ("if", "defined")))


def test_library_exports_every_declared_symbol():
    lib = lm.lib()
    names = declared_functions()
    assert {"lora_linear_fwd", "lora_linear_bwd", "frozen_linear_bwd_dx",
            "lora_linear_workspace_bytes"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings_and_kernel_names():
    lib = lm.lib()
    for s in range(5):
        assert lib.lora_status_str(s)
    names = lm.kernel_names()
    assert "gemm_fwd" in names and "gemm_bwd_dx" in names and "gemm_frozen_dx" in names
    assert lib.lora_kernel_name(len(names)) is None


def ws(op, T, K, N, r, dt=L.LORA_BF16):
    return lm.lib().lora_linear_workspace_bytes(op, T, K, N, r, dt)


BAD = ctypes.c_size_t(-1).value


def test_workspace_query():
    assert ws(L.LORA_OP_FROZEN_DX, 4096, 3072, 128256, 0) == 0
    assert ws(L.LORA_OP_FWD, 128, 256, 256, 0) == 0
    # forward: partial sums of u (at most ldt / r of them over the split
    # reduction axis), the bf16 LoRA-step operand (ldt = 64 columns) and B
    # repeated once per partial; backward: partial sums of u and du, the
    # LoRA-step operand, A repeated once per partial, and where the dA / dB
    # items run as token parts their counts and part tiles (at most an eighth
    # of the fp32 dW) -- all far below the fp32 dW the method never forms.
    assert ws(L.LORA_OP_BWD, 128, 256, 256, 0) == 0
    for T, K, N, r in [(128, 256, 256, 8), (1024, 3072, 3072, 16), (2048, 3072, 8192, 16),
                       (4096, 8192, 3072, 32), (2048, 2048, 256, 8), (16, 4096, 4096, 128),
                       (4096, 3072, 1024, 32), (1500, 1544, 2056, 12)]:
        ldt = (r + 63) // 64 * 64
        S = ldt // r
        f = ws(L.LORA_OP_FWD, T, K, N, r)
        assert T * r * 4 <= f <= S * T * r * 4 + (T + N) * ldt * 2 + 3 * 256, (T, K, N, r, f)
        b = ws(L.LORA_OP_BWD, T, K, N, r)
        side = (-(-K // 128) - (-N // 128)) * -(-r // 32) * 4 + 256 + K * N // 2
        assert 8 * T * r <= b <= 2 * S * T * r * 4 + T * ldt * 2 + S * r * K * 2 + side + 4 * 256, (T, K, N, r, b)
        assert b < N * K * 4, (T, K, N, r, b)
    # fp32 check mode pads the LoRA step to 32 columns
    assert 64 * 16 * 4 <= ws(L.LORA_OP_FWD, 64, 256, 256, 16, dt=L.LORA_F32) <= 2 * 64 * 16 * 4 + (64 + 256) * 32 * 4 + 768
    # rejected shapes
    assert ws(L.LORA_OP_BWD, 0, 256, 256, 8) == BAD
    assert ws(L.LORA_OP_BWD, 16, 250, 256, 8) == BAD
    assert ws(L.LORA_OP_BWD, 16, 256, 256, 129) == BAD
    assert ws(L.LORA_OP_BWD, 16, 256, 256, 8, dt=7) == BAD


# fake, 16-byte aligned device addresses in disjoint ranges (never dereferenced)
def P(i):
    return ctypes.c_void_p(0x7F0000000000 + i * 0x100000000)


def fwd(**kw):
    a = dict(x=P(1), W=P(2), A=P(3), B=P(4), y=P(5), u=P(6), T=64, K=256, N=256, r=8, s=2.0,
             dt=L.LORA_BF16, ws=P(7), wsb=1 << 20)
    a.update(kw)
    return lm.lib().lora_linear_fwd(a["x"], a["W"], a["A"], a["B"], a["y"], a["u"], a["T"], a["K"],
                                    a["N"], a["r"], a["s"], a["dt"], a["ws"], a["wsb"], None)


def bwd(**kw):
    a = dict(x=P(1), W=P(2), A=P(3), B=P(4), u=P(6), dy=P(8), dx=P(9), dA=P(10), dB=P(11), T=64,
             K=256, N=256, r=8, s=2.0, dt=L.LORA_BF16, ws=P(7), wsb=1 << 24)
    a.update(kw)
    return lm.lib().lora_linear_bwd(a["x"], a["W"], a["A"], a["B"], a["u"], a["dy"], a["dx"],
                                    a["dA"], a["dB"], a["T"], a["K"], a["N"], a["r"], a["s"],
                                    a["dt"], a["ws"], a["wsb"], None)


def frozen(**kw):
    a = dict(dy=P(8), W=P(2), dx=P(9), T=64, K=256, N=256, dt=L.LORA_BF16)
    a.update(kw)
    return lm.lib().frozen_linear_bwd_dx(a["dy"], a["W"], a["dx"], a["T"], a["K"], a["N"], a["dt"],
                                         None, 0, None)


def misaligned(i):
    return ctypes.c_void_p(P(i).value + 8)


@pytest.mark.parametrize("kw,code", [
    (dict(x=None), EINVAL), (dict(W=None), EINVAL), (dict(y=None), EINVAL),
    (dict(A=None), EINVAL), (dict(B=None), EINVAL),
    (dict(x=misaligned(1)), EINVAL), (dict(u=misaligned(6)), EINVAL),
    (dict(T=0), EINVAL), (dict(K=0), EINVAL), (dict(r=-1), EINVAL), (dict(r=129), EINVAL),
    (dict(K=250), EUNSUP), (dict(N=12), EUNSUP), (dict(T=1 << 22, K=1024), EUNSUP),
    (dict(s=float("inf")), EINVAL), (dict(s=float("nan")), EINVAL),
    (dict(dt=5), EINVAL),
    (dict(ws=None), EWS), (dict(wsb=100), EWS),
    (dict(y=P(1)), EINVAL),                     # y aliases x
    (dict(u=ctypes.c_void_p(P(5).value + 64)), EINVAL),   # u inside y
    (dict(ws=P(2)), EINVAL),                    # workspace aliases W
])
def test_fwd_rejects(kw, code):
    assert fwd(**kw) == code
    assert lm.lib().lora_last_error()


@pytest.mark.parametrize("kw,code", [
    (dict(dy=None), EINVAL), (dict(W=None), EINVAL), (dict(dA=None), EINVAL), (dict(dB=None), EINVAL),
    (dict(x=None), EINVAL), (dict(r=0, dx=None), EINVAL),
    (dict(dA=misaligned(10)), EINVAL), (dict(K=20), EUNSUP), (dict(wsb=1000), EWS),
    (dict(dx=P(8)), EINVAL),                    # dx aliases dy
    (dict(dB=P(10)), EINVAL),                   # dB aliases dA
    (dict(dA=P(6)), EINVAL),                    # dA aliases u_saved
    (dict(s=float("-inf")), EINVAL),
])
def test_bwd_rejects(kw, code):
    assert bwd(**kw) == code


@pytest.mark.parametrize("kw,code", [
    (dict(dy=None), EINVAL), (dict(dx=None), EINVAL), (dict(dx=P(2)), EINVAL),
    (dict(W=misaligned(2)), EINVAL), (dict(N=100), EUNSUP), (dict(T=0), EINVAL),
])
def test_frozen_rejects(kw, code):
    assert frozen(**kw) == code


def fwd_q(**kw):
    a = dict(x=P(1), codes=P(2), sc=P(11), off=P(12), bits=4, group=128, A=P(3), B=P(4), y=P(5),
             u=P(6), T=64, K=256, N=256, r=8, s=2.0, ws=P(7), wsb=1 << 24)
    a.update(kw)
    return lm.lib().lora_linear_fwd_q(a["x"], a["codes"], a["sc"], a["off"], a["bits"], a["group"],
                                      a["A"], a["B"], a["y"], a["u"], a["T"], a["K"], a["N"],
                                      a["r"], a["s"], a["ws"], a["wsb"], None)


def bwd_q(**kw):
    a = dict(x=P(1), codes=P(2), sc=P(11), off=P(12), bits=8, group=64, A=P(3), B=P(4), u=P(6),
             dy=P(8), dx=P(9), dA=P(10), dB=P(13), T=64, K=256, N=256, r=8, s=2.0, ws=P(7),
             wsb=1 << 24)
    a.update(kw)
    return lm.lib().lora_linear_bwd_q(a["x"], a["codes"], a["sc"], a["off"], a["bits"], a["group"],
                                      a["A"], a["B"], a["u"], a["dy"], a["dx"], a["dA"], a["dB"],
                                      a["T"], a["K"], a["N"], a["r"], a["s"], a["ws"], a["wsb"],
                                      None)


def frozen_q(**kw):
    a = dict(dy=P(8), codes=P(2), sc=P(11), off=P(12), bits=8, group=128, dx=P(9), T=64, K=256,
             N=256)
    a.update(kw)
    return lm.lib().frozen_linear_bwd_dx_q(a["dy"], a["codes"], a["sc"], a["off"], a["bits"],
                                           a["group"], a["dx"], a["T"], a["K"], a["N"], None, 0,
                                           None)


@pytest.mark.parametrize("kw,code", [
    (dict(bits=3), EINVAL), (dict(bits=16), EINVAL), (dict(codes=None), EINVAL),
    (dict(sc=None), EINVAL), (dict(off=misaligned(12)), EINVAL),
    (dict(group=8), EUNSUP), (dict(group=96), EUNSUP), (dict(group=512), EUNSUP),
    (dict(r=65), EUNSUP), (dict(K=250), EUNSUP), (dict(x=None), EINVAL),
    (dict(y=P(2)), EINVAL),                     # y aliases the codes
    (dict(wsb=10), EWS),
])
def test_fwd_q_rejects(kw, code):
    assert fwd_q(**kw) == code
    assert lm.lib().lora_last_error()


@pytest.mark.parametrize("kw,code", [
    (dict(bits=2), EINVAL), (dict(group=48), EUNSUP), (dict(r=80), EUNSUP),
    (dict(dx=P(11)), EINVAL),                   # dx aliases the scales
    (dict(dy=None), EINVAL), (dict(dA=None), EINVAL),
])
def test_bwd_q_rejects(kw, code):
    assert bwd_q(**kw) == code


@pytest.mark.parametrize("kw,code", [
    (dict(bits=5), EINVAL), (dict(group=1024), EUNSUP), (dict(dx=P(2)), EINVAL),
    (dict(codes=misaligned(2)), EINVAL), (dict(dy=None), EINVAL),
])
def test_frozen_q_rejects(kw, code):
    assert frozen_q(**kw) == code


def vocab(**kw):
    a = dict(table=P(1), V=1000, ldtab=16, k=8, targets=P(2), T=64, rows=P(3), nrows=20, J=P(4),
             tpos=P(5), nJ=ctypes.byref(ctypes.c_int64(0)), ws=P(6), wsb=1 << 24)
    a.update(kw)
    return lm.lib().lm_head_build_vocab(a["table"], a["V"], a["ldtab"], a["k"], a["targets"], a["T"],
                                        a["rows"], a["nrows"], a["J"], a["tpos"], a["nJ"], a["ws"],
                                        a["wsb"], None)


def head_ce(**kw):
    a = dict(h=P(1), W=P(2), T=64, V=1000, D=256, rows=P(3), nrows=20, J=P(4), nJ=300, tpos=P(5),
             loss=P(6), total=P(7), dh=P(8), dscale=1.0, ws=P(9), wsb=1 << 28)
    a.update(kw)
    return lm.lib().lm_head_reduced_ce(a["h"], a["W"], a["T"], a["V"], a["D"], a["rows"], a["nrows"],
                                       a["J"], a["nJ"], a["tpos"], a["loss"], a["total"], a["dh"],
                                       a["dscale"], a["ws"], a["wsb"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(table=None), EINVAL), (dict(nJ=None), EINVAL), (dict(k=0), EINVAL), (dict(k=17), EINVAL),
    (dict(nrows=65), EINVAL), (dict(V=0), EINVAL), (dict(rows=misaligned(3)), EINVAL),
    (dict(wsb=100), EWS), (dict(J=P(1)), EINVAL),   # J aliases the table
])
def test_build_vocab_rejects(kw, code):
    assert vocab(**kw) == code


@pytest.mark.parametrize("kw,code", [
    (dict(h=None), EINVAL), (dict(loss=None), EINVAL), (dict(nJ=0), EINVAL), (dict(nJ=1001), EINVAL),
    (dict(nrows=0), EINVAL), (dict(D=12), EUNSUP), (dict(dscale=float("nan")), EINVAL),
    (dict(dh=misaligned(8)), EINVAL), (dict(wsb=1000), EWS),
    (dict(dh=P(1)), EINVAL),                    # dh aliases h
    (dict(loss=P(5)), EINVAL),                  # losses alias tpos
])
def test_reduced_ce_rejects(kw, code):
    assert head_ce(**kw) == code


def test_head_workspace_query():
    w = lm.lib().lm_head_workspace_bytes
    assert w(0, 64, 1000, 256, 20, 0) >= 2 * 1000 * 4
    loss = w(1, 4096, 128256, 3072, 1229, 40000)
    both = w(2, 4096, 128256, 3072, 1229, 40000)
    # gathered operands + partials; the backward adds one 8192-column chunk of
    # dz, the fp32 dh rows and the position map -- never the full logits
    tiles = (40000 + 127) // 128
    assert 1229 * 3072 * 2 + 40000 * 3072 * 2 <= loss
    assert loss <= 1229 * 3072 * 2 + 40000 * 3072 * 2 + 2 * tiles * 1229 * 4 + 2 * 1229 * 4 + 6 * 256
    assert both - loss <= 1229 * 8192 * 2 + 1229 * 3072 * 4 + 4096 * 4 + 1024
    assert w(1, 64, 1000, 256, 20, 1001) == BAD
    assert w(3, 64, 1000, 256, 20, 10) == BAD


def _chain(dims, r=8):
    nodes = (L._Node * (len(dims) - 1))()
    for i in range(len(dims) - 1):
        nodes[i] = L._Node(P(20 + i).value, P(40 + i).value, P(60 + i).value, P(80 + i).value,
                           P(100 + i).value, dims[i], dims[i + 1], r, 2.0)
    return nodes


def test_ckpt_sizes_and_rejects():
    lib = lm.lib()
    nodes = _chain([256, 512, 256, 384])
    ws = lib.lora_ckpt_workspace_bytes(nodes, 3, 128)
    host = lib.lora_ckpt_host_bytes(nodes, 3, 128)
    assert host == 128 * (256 + 512 + 256) * 2
    # two activation + two gradient buffers of the widest node and one LoRA workspace
    assert 4 * 128 * 512 * 2 <= ws <= 4 * 128 * 512 * 2 + 4 * 256 + (1 << 20)
    # ... independent of the chain's depth
    deep = _chain([256, 512] * 10 + [256])
    assert lib.lora_ckpt_workspace_bytes(deep, 20, 128) == ws
    bad = _chain([256, 512, 264])
    bad[1].d_in = 520                            # does not follow node 0's d_out
    assert lib.lora_ckpt_workspace_bytes(bad, 2, 128) == BAD
    big = 1 << 40
    x0, out, stash, wsp = P(1), P(2), P(3), ctypes.c_void_p(P(4).value)
    assert lib.lora_ckpt_forward(nodes, 0, 128, x0, out, stash, big, wsp, big, None, None) == EINVAL
    assert lib.lora_ckpt_forward(nodes, 3, 128, None, out, stash, big, wsp, big, None, None) == EINVAL
    assert lib.lora_ckpt_forward(nodes, 3, 128, x0, out, stash, host - 1, wsp, big, None, None) == EWS
    assert lib.lora_ckpt_forward(nodes, 3, 128, x0, out, stash, big, wsp, ws - 1, None, None) == EWS
    assert lib.lora_ckpt_backward(nodes, 3, 128, None, None, stash, big, wsp, big, None, None) == EINVAL
    assert lib.lora_ckpt_backward(nodes, 3, 128, x0, None, stash, big,
                                  ctypes.c_void_p(P(4).value + 16), big, None, None) == EINVAL
    nodes[1].A = None
    assert lib.lora_ckpt_forward(nodes, 3, 128, x0, out, stash, big, wsp, big, None, None) == EINVAL


def test_topk_table_sizes_and_rejects():
    lib = lm.lib()
    w = lib.topk_table_workspace_bytes
    # norms + per batch of rows (at most 16384) 8192 - 1024 candidate slots per
    # row (k = 1000: the final sort takes 1024), which exceeds k + one chunk
    n = w(128256, 3072, 1000)
    R = 16384
    assert R * 7168 * 8 <= n <= R * 7168 * 8 + 128256 * 4 + 2 * R * 4 + 6 * 256
    assert w(5000, 64, 2048) >= 5000 * 6144 * 8 and 6144 >= 2048 + 4096
    assert w(1000, 64, 1001) == BAD and w(5000, 64, 2049) == BAD and w(100, 12, 5) == BAD
    t = lib.topk_table_build
    assert t(None, 1000, 64, 10, P(2), None, P(3), 1 << 30, None) == EINVAL
    assert t(P(1), 1000, 64, 0, P(2), None, P(3), 1 << 30, None) == EINVAL
    assert t(P(1), 1000, 60, 10, P(2), None, P(3), 1 << 30, None) == EUNSUP
    assert t(P(1), 1000, 64, 10, P(2), None, P(3), 100, None) == EWS
    assert t(P(1), 1000, 64, 10, P(1), None, P(3), 1 << 30, None) == EINVAL   # table aliases W
    assert t(P(1), 1000, 64, 10, misaligned(2), None, P(3), 1 << 30, None) == EINVAL


def test_rank0_ignores_lora_pointers():
    # r = 0: A, B, u, dA, dB are ignored, so NULL or misaligned values do not matter
    # (the call would then launch; only validation failures are exercised on the CPU,
    # so check that the same call with a bad *required* pointer still fails).
    assert fwd(r=0, A=None, B=None, u=None, x=None) == EINVAL
    assert bwd(r=0, A=None, B=None, u=None, dA=None, dB=None, dy=None) == EINVAL


def test_python_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(L, "_lib", None)
    monkeypatch.setattr(L, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="not built"):
        L.lib()


def test_plan_coverage():
    """The W = 0 / B = 0 isolation cases of the GPU tests together select every
    kernel configuration (GEMM tile, fused or not, one or several partial
    sums) that any workload linear runs, in both directions."""
    from test_gpu_isolation import CASES, signatures
    from workloads import WORKLOADS

    fwd = {c[1] for c in CASES}
    bwd = {c[2] for c in CASES}
    for w in WORKLOADS.values():
        for lin in w.linears:
            f, b = signatures(w.tokens, lin.d_in, lin.d_out, lin.rank)
            assert f in fwd, (w.key, lin.name, f)
            assert b in bwd, (w.key, lin.name, b)


def test_plan_query():
    p = lm.lora_linear_plan(1024, 3072, 3072, 16)
    assert (p["fwd_tile_m"], p["fwd_tile_n"], p["fwd_fused"]) == (128, 128, 1)
    p = lm.lora_linear_plan(300, 520, 392, 16, L.LORA_F32)
    assert (p["fwd_tile_m"], p["fwd_tile_n"], p["fwd_fused"], p["bwd_fused"]) == (128, 128, 0, 0)
    p = lm.lora_linear_plan(64, 128, 128, 0)
    assert p["fwd_fused"] == 0 and p["fwd_u_parts"] == 0 and p["bwd_du_parts"] == 0
    lib = lm.lib()
    plan = L._Plan()
    assert lib.lora_linear_plan(0, 128, 128, 8, 0, ctypes.byref(plan)) == EINVAL
    assert lib.lora_linear_plan(64, 100, 128, 8, 0, ctypes.byref(plan)) == EUNSUP
    assert lib.lora_linear_plan(64, 128, 128, 8, 0, None) == EINVAL


def test_handover_hooks_reject_bad_arguments():
    lib = lm.lib()
    assert lib.lora_debug_set_handover(-1) == EINVAL
    assert lib.lora_debug_set_handover(2) == EINVAL
    assert lib.lora_handover_giveups(None, 0) == EINVAL
    assert lib.lora_debug_set_handover(0) == L.LORA_OK
