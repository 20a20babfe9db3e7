// ckpt.cpp -- the checkpointed training step over a chain of LoRA linears
// (the paper's algorithm "Memory-Efficient Checkpointing for LoRA
// Fine-tuning" on one GPU): the forward saves no LoRA activation and moves
// each node's input to pinned host memory while the following nodes run; the
// backward brings each input back one node ahead of its use, recomputes u
// from it and backpropagates.  Device memory holds two activation buffers
// and two gradient buffers, whatever the depth of the chain.
//
// Streams: compute work on `compute_stream`, host copies on `copy_stream`,
// ordered by events (a copy out waits for the node that produced its data;
// a node that overwrites a buffer waits for the copy out of it; a copy in
// waits for the node that last read its buffer).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <vector>

#include "../../include/lora_mi355x.h"
#include "launch.hpp"

namespace {

struct Events {
  std::vector<hipEvent_t> ev;
  ~Events() {
    for (hipEvent_t e : ev) (void)hipEventDestroy(e);
  }
  hipError_t make(size_t n) {
    for (size_t i = 0; i < n; ++i) {
      hipEvent_t e;
      hipError_t r = hipEventCreateWithFlags(&e, hipEventDisableTiming);
      if (r != hipSuccess) return r;
      ev.push_back(e);
    }
    return hipSuccess;
  }
};

struct Plan {
  int64_t maxd = 0;        // widest activation
  size_t act_bytes = 0;    // one activation / gradient buffer
  size_t op_ws = 0;        // workspace of the widest LoRA call
  size_t total = 0;
  std::vector<size_t> stash_off;  // host offset of each node's input
  size_t stash_bytes = 0;
};

lora_status_t plan(const lora_node_t *nodes, int n, int64_t T, Plan *p) {
  if (!nodes || n < 1 || T < 1) return LORA_EINVAL;
  p->stash_off.assign(n, 0);
  for (int i = 0; i < n; ++i) {
    const lora_node_t &nd = nodes[i];
    if (i > 0 && nd.d_in != nodes[i - 1].d_out) return LORA_EINVAL;
    const size_t fw = lora_linear_workspace_bytes(LORA_OP_FWD, T, nd.d_in, nd.d_out, nd.r, LORA_BF16);
    const size_t bw = lora_linear_workspace_bytes(LORA_OP_BWD, T, nd.d_in, nd.d_out, nd.r, LORA_BF16);
    if (fw == (size_t)-1 || bw == (size_t)-1) return LORA_EUNSUPPORTED;
    p->op_ws = std::max({p->op_ws, fw, bw});
    p->maxd = std::max({p->maxd, nd.d_in, nd.d_out});
    p->stash_off[i] = p->stash_bytes;
    p->stash_bytes += (size_t)T * nd.d_in * 2;
  }
  p->act_bytes = ((size_t)T * p->maxd * 2 + 255) & ~size_t(255);
  p->total = 4 * p->act_bytes + ((p->op_ws + 255) & ~size_t(255));
  return LORA_OK;
}

lora_status_t fail(lora_status_t s, const char *msg) {
  lora::set_last_error(msg);
  return s;
}

lora_status_t hipfail(hipError_t e, const char *what) {
  char buf[256];
  std::snprintf(buf, sizeof buf, "%s: %s", what, hipGetErrorString(e));
  lora::set_last_error(buf);
  return LORA_EHIP;
}

lora_status_t check_common(const lora_node_t *nodes, int n, int64_t T, void *host_stash,
                           size_t host_bytes, void *ws, size_t ws_bytes, Plan *p) {
  lora_status_t s = plan(nodes, n, T, p);
  if (s == LORA_EINVAL) return fail(s, "need n >= 1, T >= 1 and d_in of each node = d_out of the one before");
  if (s != LORA_OK) return fail(s, "a node's shape is not supported (see lora_linear_workspace_bytes)");
  for (int i = 0; i < n; ++i) {
    const lora_node_t &nd = nodes[i];
    if (!nd.W || (nd.r > 0 && (!nd.A || !nd.B || !nd.dA || !nd.dB)))
      return fail(LORA_EINVAL, "each node needs W, and A, B, dA, dB when r > 0");
  }
  if (!host_stash || host_bytes < p->stash_bytes) return fail(LORA_EWORKSPACE, "host stash missing or too small");
  if (!ws || ws_bytes < p->total) return fail(LORA_EWORKSPACE, "device workspace missing or too small");
  if ((reinterpret_cast<uintptr_t>(ws) & 255u) != 0) return fail(LORA_EINVAL, "workspace not 256-byte aligned");
  return LORA_OK;
}

}  // namespace

extern "C" {

size_t lora_ckpt_workspace_bytes(const lora_node_t *nodes, int n, int64_t T) {
  Plan p;
  return plan(nodes, n, T, &p) == LORA_OK ? p.total : (size_t)-1;
}

size_t lora_ckpt_host_bytes(const lora_node_t *nodes, int n, int64_t T) {
  Plan p;
  return plan(nodes, n, T, &p) == LORA_OK ? p.stash_bytes : (size_t)-1;
}

lora_status_t lora_ckpt_forward(const lora_node_t *nodes, int n, int64_t T, const void *x0,
                                void *out, void *host_stash, size_t host_bytes, void *ws,
                                size_t ws_bytes, void *compute_stream, void *copy_stream) {
  Plan p;
  lora_status_t s = check_common(nodes, n, T, host_stash, host_bytes, ws, ws_bytes, &p);
  if (s != LORA_OK) return s;
  if (!x0 || !out) return fail(LORA_EINVAL, "x0 and out are required");
  hipStream_t cs = (hipStream_t)compute_stream, xs = (hipStream_t)copy_stream;
  char *wsb = (char *)ws;
  void *act[2] = {wsb, wsb + p.act_bytes};
  void *opws = wsb + 4 * p.act_bytes;
  Events E;
  // produced[i]: input of node i ready; copied[i]: its copy to the host done
  hipError_t e = E.make(2 * (size_t)n);
  if (e != hipSuccess) return hipfail(e, "event creation");
  hipEvent_t *produced = E.ev.data(), *copied = E.ev.data() + n;
  const void *cur = x0;
  for (int i = 0; i < n; ++i) {
    const lora_node_t &nd = nodes[i];
    // the node's input leaves for the host as soon as it exists
    if ((e = hipEventRecord(produced[i], cs)) != hipSuccess) return hipfail(e, "event");
    if ((e = hipStreamWaitEvent(xs, produced[i], 0)) != hipSuccess) return hipfail(e, "wait");
    if ((e = hipMemcpyAsync((char *)host_stash + p.stash_off[i], cur, (size_t)T * nd.d_in * 2,
                            hipMemcpyDeviceToHost, xs)) != hipSuccess)
      return hipfail(e, "copy to host");
    if ((e = hipEventRecord(copied[i], xs)) != hipSuccess) return hipfail(e, "event");
    // output buffer: the caller's for the last node, else the one that held
    // the input of node i-1, which must have reached the host
    void *dst = i == n - 1 ? out : act[i % 2];
    if (i >= 1 && i < n - 1)
      if ((e = hipStreamWaitEvent(cs, copied[i - 1], 0)) != hipSuccess) return hipfail(e, "wait");
    s = lora_linear_fwd(cur, nd.W, nd.A, nd.B, dst, nullptr, T, nd.d_in, nd.d_out, nd.r, nd.scale,
                        LORA_BF16, opws, p.op_ws, cs);
    if (s != LORA_OK) return s;  // message set by lora_linear_fwd
    cur = dst;
  }
  // the stash must be complete before the backward reads it back
  if ((e = hipStreamWaitEvent(cs, copied[n - 1], 0)) != hipSuccess) return hipfail(e, "wait");
  return LORA_OK;
}

lora_status_t lora_ckpt_backward(const lora_node_t *nodes, int n, int64_t T, const void *g_n,
                                 void *dx0, const void *host_stash, size_t host_bytes, void *ws,
                                 size_t ws_bytes, void *compute_stream, void *copy_stream) {
  Plan p;
  lora_status_t s = check_common(nodes, n, T, (void *)host_stash, host_bytes, ws, ws_bytes, &p);
  if (s != LORA_OK) return s;
  if (!g_n) return fail(LORA_EINVAL, "g_n is required");
  hipStream_t cs = (hipStream_t)compute_stream, xs = (hipStream_t)copy_stream;
  char *wsb = (char *)ws;
  void *act[2] = {wsb, wsb + p.act_bytes};
  void *grad[2] = {wsb + 2 * p.act_bytes, wsb + 3 * p.act_bytes};
  void *opws = wsb + 4 * p.act_bytes;
  Events E;
  // loaded[i]: input of node i back on the device; done[i]: node i's backward issued
  hipError_t e = E.make(2 * (size_t)n + 1);
  if (e != hipSuccess) return hipfail(e, "event creation");
  hipEvent_t *loaded = E.ev.data(), *done = E.ev.data() + n, start = E.ev[2 * (size_t)n];
  // the copies must not overtake work already queued on the compute stream
  if ((e = hipEventRecord(start, cs)) != hipSuccess) return hipfail(e, "event");
  if ((e = hipStreamWaitEvent(xs, start, 0)) != hipSuccess) return hipfail(e, "wait");
  auto load = [&](int i) -> hipError_t {
    // buffer act[i % 2] last held the input of node i + 2
    hipError_t r;
    if (i + 2 < n && (r = hipStreamWaitEvent(xs, done[i + 2], 0)) != hipSuccess) return r;
    if ((r = hipMemcpyAsync(act[i % 2], (const char *)host_stash + p.stash_off[i],
                            (size_t)T * nodes[i].d_in * 2, hipMemcpyHostToDevice, xs)) != hipSuccess)
      return r;
    return hipEventRecord(loaded[i], xs);
  };
  if ((e = load(n - 1)) != hipSuccess) return hipfail(e, "copy to device");
  const void *g = g_n;
  for (int i = n - 1; i >= 0; --i) {
    const lora_node_t &nd = nodes[i];
    if (i >= 1 && (e = load(i - 1)) != hipSuccess) return hipfail(e, "copy to device");  // one ahead
    if ((e = hipStreamWaitEvent(cs, loaded[i], 0)) != hipSuccess) return hipfail(e, "wait");
    void *gout = i == 0 ? dx0 : grad[i % 2];
    s = lora_linear_bwd(act[i % 2], nd.W, nd.A, nd.B, nullptr, g, gout, nd.dA, nd.dB, T, nd.d_in,
                        nd.d_out, nd.r, nd.scale, LORA_BF16, opws, p.op_ws, cs);
    if (s != LORA_OK) return s;  // message set by lora_linear_bwd
    if ((e = hipEventRecord(done[i], cs)) != hipSuccess) return hipfail(e, "event");
    g = gout;
  }
  return LORA_OK;
}

}  // extern "C"
