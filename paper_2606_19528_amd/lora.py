"""Python binding of ``liblora_mi355x.so`` (the C ABI in include/lora_mi355x.h).

Argument marshalling only: every step of the LoRA forward and backward runs in
the library's HIP kernels on the caller's stream.  PyTorch provides device
memory and the current HIP stream.  If the library has not been built the
binding raises -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "liblora_mi355x.so")

LORA_OK, LORA_EINVAL, LORA_EUNSUPPORTED, LORA_EWORKSPACE, LORA_EHIP = range(5)
LORA_BF16, LORA_F32 = 0, 1
LORA_OP_FWD, LORA_OP_BWD, LORA_OP_FROZEN_DX = 0, 1, 2

_lib = None


class _Node(ctypes.Structure):
    """lora_node_t of the C ABI."""
    _fields_ = [("W", ctypes.c_void_p), ("A", ctypes.c_void_p), ("B", ctypes.c_void_p),
                ("dA", ctypes.c_void_p), ("dB", ctypes.c_void_p), ("d_in", ctypes.c_int64),
                ("d_out", ctypes.c_int64), ("r", ctypes.c_int64), ("scale", ctypes.c_float)]


class _Plan(ctypes.Structure):
    """lora_plan_t of the C ABI."""
    _fields_ = [(n, ctypes.c_int) for n in ("fwd_tile_m", "fwd_tile_n", "fwd_fused", "fwd_u_parts",
                                             "bwd_tile_m", "bwd_tile_n", "bwd_fused", "bwd_du_parts",
                                             "bwd_side_parts")]


class LoraError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: status {status} ({detail})")
        self.status = status


def lib() -> ctypes.CDLL:
    """Load the HIP library (once).  Raises if it is missing: build it with
    ``python -m paper_2606_19528_amd.build``."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"HIP library not built: {LIB_PATH} is missing "
                           "(run python -m paper_2606_19528_amd.build)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i64, f32, sz, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t, ctypes.c_int
    L.lora_linear_workspace_bytes.argtypes = [i32, i64, i64, i64, i64, i32]
    L.lora_linear_workspace_bytes.restype = sz
    L.lora_linear_fwd.argtypes = [vp, vp, vp, vp, vp, vp, i64, i64, i64, i64, f32, i32, vp, sz, vp]
    L.lora_linear_fwd.restype = i32
    L.lora_linear_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, i64, i64, i64, i64, f32, i32,
                                  vp, sz, vp]
    L.lora_linear_bwd.restype = i32
    L.lora_linear_bwd_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, i64, i64, i64, i64, f32, i32,
                                          vp]
    L.lora_linear_bwd_noalloc.restype = i32
    L.frozen_linear_bwd_dx.argtypes = [vp, vp, vp, i64, i64, i64, i32, vp, sz, vp]
    L.frozen_linear_bwd_dx.restype = i32
    L.lora_linear_fwd_q.argtypes = [vp, vp, vp, vp, i32, i64, vp, vp, vp, vp, i64, i64, i64, i64,
                                    f32, vp, sz, vp]
    L.lora_linear_fwd_q.restype = i32
    L.lora_linear_bwd_q.argtypes = [vp, vp, vp, vp, i32, i64, vp, vp, vp, vp, vp, vp, vp, i64, i64,
                                    i64, i64, f32, vp, sz, vp]
    L.lora_linear_bwd_q.restype = i32
    L.frozen_linear_bwd_dx_q.argtypes = [vp, vp, vp, vp, i32, i64, vp, i64, i64, i64, vp, sz, vp]
    L.frozen_linear_bwd_dx_q.restype = i32
    L.lm_head_workspace_bytes.argtypes = [i32, i64, i64, i64, i64, i64]
    L.lm_head_workspace_bytes.restype = sz
    L.lm_head_build_vocab.argtypes = [vp, i64, i64, i64, vp, i64, vp, i64, vp, vp,
                                      ctypes.POINTER(i64), vp, sz, vp]
    L.lm_head_build_vocab.restype = i32
    L.lm_head_reduced_ce.argtypes = [vp, vp, i64, i64, i64, vp, i64, vp, i64, vp, vp, vp, vp, f32,
                                     vp, sz, vp]
    L.lm_head_reduced_ce.restype = i32
    NP = ctypes.POINTER(_Node)
    L.lora_ckpt_workspace_bytes.argtypes = [NP, i32, i64]
    L.lora_ckpt_workspace_bytes.restype = sz
    L.lora_ckpt_host_bytes.argtypes = [NP, i32, i64]
    L.lora_ckpt_host_bytes.restype = sz
    L.lora_ckpt_forward.argtypes = [NP, i32, i64, vp, vp, vp, sz, vp, sz, vp, vp]
    L.lora_ckpt_forward.restype = i32
    L.lora_ckpt_backward.argtypes = [NP, i32, i64, vp, vp, vp, sz, vp, sz, vp, vp]
    L.lora_ckpt_backward.restype = i32
    L.topk_table_workspace_bytes.argtypes = [i64, i64, i64]
    L.topk_table_workspace_bytes.restype = sz
    L.topk_table_build.argtypes = [vp, i64, i64, i64, vp, vp, vp, sz, vp]
    L.topk_table_build.restype = i32
    L.lora_status_str.argtypes = [i32]
    L.lora_status_str.restype = ctypes.c_char_p
    L.lora_last_error.argtypes = []
    L.lora_last_error.restype = ctypes.c_char_p
    L.lora_profiler_enable.argtypes = [i32]
    L.lora_profiler_enable.restype = i32
    L.lora_profiler_reset.argtypes = []
    L.lora_profiler_reset.restype = i32
    L.lora_profiler_read.argtypes = [i32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i64)]
    L.lora_profiler_read.restype = i32
    L.lora_kernel_name.argtypes = [i32]
    L.lora_kernel_name.restype = ctypes.c_char_p
    L.lora_kernel_count.argtypes = []
    L.lora_kernel_count.restype = i32
    L.lora_linear_plan.argtypes = [i64, i64, i64, i64, i32, ctypes.POINTER(_Plan)]
    L.lora_linear_plan.restype = i32
    L.lora_handover_giveups.argtypes = [ctypes.POINTER(ctypes.c_uint64), i32]
    L.lora_handover_giveups.restype = i32
    L.lora_debug_set_handover.argtypes = [i32]
    L.lora_debug_set_handover.restype = i32
    _lib = L
    return L


def _check(status: int, where: str):
    if status != LORA_OK:
        detail = lib().lora_last_error().decode()
        raise LoraError(status, where, detail)


def _dtype_code(t) -> int:
    import torch

    if t.dtype == torch.bfloat16:
        return LORA_BF16
    if t.dtype == torch.float32:
        return LORA_F32
    raise TypeError(f"unsupported dtype {t.dtype} (bf16 or fp32)")


def _ptr(t):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous (row-major, no padding)")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch

    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _ws(ws, nbytes: int, like, stream=None):
    """The caller's workspace, or a temporary one.  A temporary is allocated on
    the stream the call is enqueued on, so the caching allocator does not hand
    its block to another tensor while that stream's kernels still use it."""
    import torch

    if nbytes == 0:
        return None, 0
    if ws is None:
        if stream is None:
            ws = torch.empty(nbytes, dtype=torch.uint8, device=like.device)
        else:
            with torch.cuda.stream(stream):
                ws = torch.empty(nbytes, dtype=torch.uint8, device=like.device)
    return ws, ws.numel() * ws.element_size()


def lora_linear_workspace_bytes(op: int, T: int, d_in: int, d_out: int, r: int, dt: int) -> int:
    n = lib().lora_linear_workspace_bytes(op, T, d_in, d_out, r, dt)
    if n == ctypes.c_size_t(-1).value:
        raise LoraError(LORA_EINVAL, "lora_linear_workspace_bytes", lib().lora_last_error().decode())
    return int(n)


def lora_linear_fwd(x, W, A, B, y, u_save=None, scale: float = 1.0, ws=None, stream=None):
    """y = x W^T + scale (x A^T) B^T; u_save (fp32 [T, r]) receives x A^T."""
    T, d_in = x.shape
    d_out = W.shape[0]
    r = 0 if A is None else A.shape[0]
    dt = _dtype_code(x)
    ws, ws_bytes = _ws(ws, lora_linear_workspace_bytes(LORA_OP_FWD, T, d_in, d_out, r, dt), x, stream)
    st = lib().lora_linear_fwd(_ptr(x), _ptr(W), _ptr(A), _ptr(B), _ptr(y), _ptr(u_save), T, d_in,
                               d_out, r, float(scale), dt, _ptr(ws), ws_bytes, _stream(stream))
    _check(st, "lora_linear_fwd")
    return y


def lora_linear_bwd(x, W, A, B, u_saved, dy, dx, dA, dB, scale: float = 1.0, ws=None, stream=None):
    """dx = dy W + du A, dA = du^T x, dB = scale dy^T u with du = scale dy B."""
    T, d_out = dy.shape
    d_in = W.shape[1]
    r = 0 if A is None else A.shape[0]
    dt = _dtype_code(dy)
    ws, ws_bytes = _ws(ws, lora_linear_workspace_bytes(LORA_OP_BWD, T, d_in, d_out, r, dt), dy, stream)
    st = lib().lora_linear_bwd(_ptr(x), _ptr(W), _ptr(A), _ptr(B), _ptr(u_saved), _ptr(dy),
                               _ptr(dx), _ptr(dA), _ptr(dB), T, d_in, d_out, r, float(scale), dt,
                               _ptr(ws), ws_bytes, _stream(stream))
    _check(st, "lora_linear_bwd")
    return dx, dA, dB


def lora_linear_bwd_noalloc(x, W, A, B, u_saved, dy, dx, dA, dB, scale: float = 1.0, stream=None):
    """lora_linear_bwd with the library's static device scratch as workspace
    (no allocation by the library or by this wrapper)."""
    T, d_out = dy.shape
    d_in = W.shape[1]
    r = 0 if A is None else A.shape[0]
    dt = _dtype_code(dy)
    st = lib().lora_linear_bwd_noalloc(_ptr(x), _ptr(W), _ptr(A), _ptr(B), _ptr(u_saved), _ptr(dy),
                                       _ptr(dx), _ptr(dA), _ptr(dB), T, d_in, d_out, r, float(scale), dt,
                                       _stream(stream))
    _check(st, "lora_linear_bwd_noalloc")
    return dx, dA, dB


def frozen_linear_bwd_dx(dy, W, dx, ws=None, stream=None):
    """Rank-0 frozen linear input gradient dx = dy W."""
    T, d_out = dy.shape
    d_in = W.shape[1]
    dt = _dtype_code(dy)
    st = lib().frozen_linear_bwd_dx(_ptr(dy), _ptr(W), _ptr(dx), T, d_in, d_out, dt, _ptr(ws),
                                    0 if ws is None else ws.numel() * ws.element_size(),
                                    _stream(stream))
    _check(st, "frozen_linear_bwd_dx")
    return dx


# --- quantized frozen base (codes + per-group scale / offset) ----------------------
def _qw(Wq):
    """(codes, scale, offset, bits, group, d_out, d_in) of a quantized weight given
    as a dict with keys codes (uint8 [d_out, d_in*bits/8]), scale and offset
    (fp32 [d_in/group, d_out], group-major) and bits."""
    codes, sc, off, bits = Wq["codes"], Wq["scale"], Wq["offset"], int(Wq["bits"])
    d_out = codes.shape[0]
    d_in = codes.shape[1] * 8 // bits
    group = d_in // sc.shape[0]
    return codes, sc, off, bits, group, d_out, d_in


def lora_linear_fwd_q(x, Wq, A, B, y, u_save=None, scale: float = 1.0, ws=None, stream=None):
    """lora_linear_fwd with the frozen W quantized (dict, see _qw)."""
    codes, sc, off, bits, group, d_out, d_in = _qw(Wq)
    T = x.shape[0]
    r = 0 if A is None else A.shape[0]
    ws, ws_bytes = _ws(ws, lora_linear_workspace_bytes(LORA_OP_FWD, T, d_in, d_out, r, LORA_BF16), x, stream)
    st = lib().lora_linear_fwd_q(_ptr(x), _ptr(codes), _ptr(sc), _ptr(off), bits, group, _ptr(A),
                                 _ptr(B), _ptr(y), _ptr(u_save), T, d_in, d_out, r, float(scale),
                                 _ptr(ws), ws_bytes, _stream(stream))
    _check(st, "lora_linear_fwd_q")
    return y


def lora_linear_bwd_q(x, Wq, A, B, u_saved, dy, dx, dA, dB, scale: float = 1.0, ws=None,
                      stream=None):
    """lora_linear_bwd with the frozen W quantized (dict, see _qw)."""
    codes, sc, off, bits, group, d_out, d_in = _qw(Wq)
    T = dy.shape[0]
    r = 0 if A is None else A.shape[0]
    ws, ws_bytes = _ws(ws, lora_linear_workspace_bytes(LORA_OP_BWD, T, d_in, d_out, r, LORA_BF16), dy, stream)
    st = lib().lora_linear_bwd_q(_ptr(x), _ptr(codes), _ptr(sc), _ptr(off), bits, group, _ptr(A),
                                 _ptr(B), _ptr(u_saved), _ptr(dy), _ptr(dx), _ptr(dA), _ptr(dB), T,
                                 d_in, d_out, r, float(scale), _ptr(ws), ws_bytes, _stream(stream))
    _check(st, "lora_linear_bwd_q")
    return dx, dA, dB


def frozen_linear_bwd_dx_q(dy, Wq, dx, ws=None, stream=None):
    """frozen_linear_bwd_dx with W quantized (dict, see _qw)."""
    codes, sc, off, bits, group, d_out, d_in = _qw(Wq)
    T = dy.shape[0]
    st = lib().frozen_linear_bwd_dx_q(_ptr(dy), _ptr(codes), _ptr(sc), _ptr(off), bits, group,
                                      _ptr(dx), T, d_in, d_out, _ptr(ws),
                                      0 if ws is None else ws.numel() * ws.element_size(),
                                      _stream(stream))
    _check(st, "frozen_linear_bwd_dx_q")
    return dx


# --- frozen LM head: reduced-vocabulary cross entropy with logits masking -----------
LM_HEAD_OP_VOCAB, LM_HEAD_OP_LOSS, LM_HEAD_OP_LOSS_DH = 0, 1, 2


def lm_head_workspace_bytes(op: int, T: int, V: int, D: int, nrows: int, nJ: int = 1) -> int:
    n = lib().lm_head_workspace_bytes(op, T, V, D, nrows, nJ)
    if n == ctypes.c_size_t(-1).value:
        raise LoraError(LORA_EINVAL, "lm_head_workspace_bytes", "sizes rejected")
    return int(n)


def lm_head_build_vocab(table, k: int, targets, rows, ws=None, stream=None):
    """(J [nJ] int32, tpos [nrows] int32) on the device; waits for the stream."""
    import torch

    V, ldtab = table.shape
    T = targets.shape[0]
    nrows = rows.shape[0]
    J = torch.empty(V, dtype=torch.int32, device=table.device)
    tpos = torch.empty(nrows, dtype=torch.int32, device=table.device)
    ws, ws_bytes = _ws(ws, lm_head_workspace_bytes(LM_HEAD_OP_VOCAB, T, V, 8, nrows), table, stream)
    nJ = ctypes.c_int64(0)
    st = lib().lm_head_build_vocab(_ptr(table), V, ldtab, k, _ptr(targets), T, _ptr(rows), nrows,
                                   _ptr(J), _ptr(tpos), ctypes.byref(nJ), _ptr(ws), ws_bytes,
                                   _stream(stream))
    _check(st, "lm_head_build_vocab")
    return J[: nJ.value], tpos


def lm_head_reduced_ce(h, W, rows, J, tpos, loss_rows, loss_total=None, dh=None,
                       dscale: float = 1.0, ws=None, stream=None):
    """Per-position losses (and their sum, and dh) of the reduced-vocabulary
    cross entropy over the trainable positions `rows`."""
    T, D = h.shape
    V = W.shape[0]
    nrows, nJ = rows.shape[0], J.shape[0]
    op = LM_HEAD_OP_LOSS if dh is None else LM_HEAD_OP_LOSS_DH
    ws, ws_bytes = _ws(ws, lm_head_workspace_bytes(op, T, V, D, nrows, nJ), h, stream)
    st = lib().lm_head_reduced_ce(_ptr(h), _ptr(W), T, V, D, _ptr(rows), nrows, _ptr(J), nJ,
                                  _ptr(tpos), _ptr(loss_rows), _ptr(loss_total), _ptr(dh),
                                  float(dscale), _ptr(ws), ws_bytes, _stream(stream))
    _check(st, "lm_head_reduced_ce")
    return loss_rows


# --- top-k similarity table ---------------------------------------------------------
def topk_table_build(W, k: int, table=None, values=None, ws=None, stream=None):
    """table [V, k] int32 (and optionally values [V, k] fp32) of each token's k
    most cosine-similar tokens."""
    import torch

    V, D = W.shape
    if table is None:
        table = torch.empty(V, k, dtype=torch.int32, device=W.device)
    n = lib().topk_table_workspace_bytes(V, D, k)
    if n == ctypes.c_size_t(-1).value:
        raise LoraError(LORA_EINVAL, "topk_table_workspace_bytes", "sizes rejected")
    ws, ws_bytes = _ws(ws, int(n), W, stream)
    st = lib().topk_table_build(_ptr(W), V, D, k, _ptr(table), _ptr(values), _ptr(ws), ws_bytes,
                                _stream(stream))
    _check(st, "topk_table_build")
    return table


# --- checkpointed step over a chain of LoRA linears ---------------------------------
def _nodes(nodes):
    arr = (_Node * len(nodes))()
    for i, nd in enumerate(nodes):
        W, A, B = nd["W"], nd.get("A"), nd.get("B")
        r = 0 if A is None else A.shape[0]
        arr[i] = _Node(W.data_ptr(), None if A is None else A.data_ptr(),
                       None if B is None else B.data_ptr(),
                       None if nd.get("dA") is None else nd["dA"].data_ptr(),
                       None if nd.get("dB") is None else nd["dB"].data_ptr(),
                       W.shape[1], W.shape[0], r, float(nd.get("scale", 1.0)))
    return arr


def lora_ckpt_sizes(nodes, T: int):
    """(device workspace bytes, pinned host stash bytes) of a checkpointed step."""
    arr = _nodes(nodes)
    w = lib().lora_ckpt_workspace_bytes(arr, len(nodes), T)
    h = lib().lora_ckpt_host_bytes(arr, len(nodes), T)
    if w == ctypes.c_size_t(-1).value:
        raise LoraError(LORA_EINVAL, "lora_ckpt_workspace_bytes", "chain rejected")
    return int(w), int(h)


def lora_ckpt_forward(nodes, x0, out, host_stash, ws, compute_stream=None, copy_stream=None):
    """Checkpointed forward: out = x_n; every node input goes to host_stash
    (pinned) on copy_stream.  nodes: dicts W, A, B, dA, dB, scale."""
    arr = _nodes(nodes)
    T = x0.shape[0]
    st = lib().lora_ckpt_forward(arr, len(nodes), T, _ptr(x0), _ptr(out), _ptr(host_stash),
                                 host_stash.numel() * host_stash.element_size(), _ptr(ws),
                                 ws.numel() * ws.element_size(), _stream(compute_stream),
                                 _stream(copy_stream))
    _check(st, "lora_ckpt_forward")
    return out


def lora_ckpt_backward(nodes, g_n, dx0, host_stash, ws, compute_stream=None, copy_stream=None):
    """Checkpointed backward from g_n = dL/dx_n: fills every node's dA, dB and dx0."""
    arr = _nodes(nodes)
    T = g_n.shape[0]
    st = lib().lora_ckpt_backward(arr, len(nodes), T, _ptr(g_n), _ptr(dx0), _ptr(host_stash),
                                  host_stash.numel() * host_stash.element_size(), _ptr(ws),
                                  ws.numel() * ws.element_size(), _stream(compute_stream),
                                  _stream(copy_stream))
    _check(st, "lora_ckpt_backward")
    return dx0


# --- kernel timing hook (benchmarks) -----------------------------------------------
def kernel_names() -> list:
    L = lib()
    return [L.lora_kernel_name(i).decode() for i in range(L.lora_kernel_count())]


def profiler_enable(on: bool = True):
    _check(lib().lora_profiler_enable(1 if on else 0), "lora_profiler_enable")


def profiler_reset():
    _check(lib().lora_profiler_reset(), "lora_profiler_reset")


def profiler_read(name: str):
    """(total milliseconds, launches) recorded for the kernel `name`."""
    idx = kernel_names().index(name)
    ms = ctypes.c_double(0.0)
    n = ctypes.c_int64(0)
    _check(lib().lora_profiler_read(idx, ctypes.byref(ms), ctypes.byref(n)), "lora_profiler_read")
    return ms.value, n.value


# --- plan and hand-over diagnostics -------------------------------------------------
def lora_linear_plan(T: int, d_in: int, d_out: int, r: int, dt: int = LORA_BF16) -> dict:
    """Kernel configuration of lora_linear_fwd / lora_linear_bwd for these sizes:
    GEMM output tiles, whether the rank-r pass is fused, number of partial sums."""
    p = _Plan()
    _check(lib().lora_linear_plan(T, d_in, d_out, r, dt, ctypes.byref(p)), "lora_linear_plan")
    return {n: getattr(p, n) for n, _ in _Plan._fields_}


def handover_giveups(reset: bool = False) -> int:
    """Hand-over waits that gave up on the current device (synchronises it)."""
    n = ctypes.c_uint64(0)
    _check(lib().lora_handover_giveups(ctypes.byref(n), 1 if reset else 0), "lora_handover_giveups")
    return n.value


def debug_set_handover(hold: int = 0):
    """Test hook: 1 makes every tile's hand-over wait give up (results invalid)."""
    _check(lib().lora_debug_set_handover(hold), "lora_debug_set_handover")
