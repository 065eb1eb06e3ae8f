"""A hybrid schedule's stack through the library alone (Section 3.3: the
sparse backbone with a few layers replaced by standard multi-head attention).

The schedule is a list whose entries are sparse layer codes (hypercube layers
or hcmix.LAYER_NEAR) or "attn".  Runs of sparse layers are one hcmix stack
each; an attention layer is the library's linear map (query/key/value
projection), attention core and linear map (output projection).  Backward:
each sparse run's dX chain (hcmix_stack_backward_data), each attention
layer's three backward products, and at the end the weight gradients of all
sparse layers in one hcmix_stack_weight_gradients call.  No arithmetic is
done here: every step is a library call on device tensors.

    h = HybridStack(schedule, w_self, w_off, attn_w, heads)
    y = h.forward(x)             # x [batch, n, width] bf16
    dx = h.backward(dy)          # then h.dw_self, h.dw_off, h.dw_attn (fp32)
"""
from __future__ import annotations

import torch

from . import hcmix


class HybridStack:
    def __init__(self, schedule, w_self, w_off, attn_w, heads, causal=True):
        self.schedule = list(schedule)
        self.w_self, self.w_off = list(w_self), list(w_off)
        self.attn_w = [tuple(p) for p in attn_w]
        self.heads = heads
        self.causal = causal
        self.segments = []
        cur, ns, na = [], 0, 0
        for e in self.schedule:
            if e == "attn":
                if cur:
                    self.segments.append(("sparse", cur))
                self.segments.append(("attn", na))
                cur, na = [], na + 1
            else:
                cur.append((ns, e))
                ns += 1
        if cur:
            self.segments.append(("sparse", cur))
        if na != len(self.attn_w) or ns > len(self.w_self):
            raise ValueError("schedule does not match the weights given")
        self.num_sparse = ns
        self._saved = []
        self._dw_in = []
        self.dw_self = self.dw_off = self.dw_attn = None

    # ---- one segment at a time (so that a caller can time each) ----

    def forward_segment(self, k, x):
        kind, arg = self.segments[k]
        if kind == "sparse":
            xs = hcmix.stack_forward(x, [self.w_self[j] for j, _ in arg],
                                     [self.w_off[j] for j, _ in arg], [c for _, c in arg],
                                     self.causal)
            self._saved.append(xs)
            return xs[-1]
        wqkv, wout = self.attn_w[arg]
        batch, n, width = x.shape
        hd = wqkv.shape[0] // (3 * self.heads)
        qkv = hcmix.linear_forward(x.view(batch * n, width), wqkv)
        o, lse = hcmix.attention_forward(qkv.view(batch, n, 3, self.heads, hd))
        y = hcmix.linear_forward(o.view(batch * n, self.heads * hd), wout)
        self._saved.append((x, qkv, o, lse))
        return y.view(batch, n, -1)

    def backward_segment(self, k, g):
        kind, arg = self.segments[k]
        sv = self._saved[k]
        if kind == "sparse":
            g_out = g
            g, grads = hcmix.stack_backward_data([self.w_self[j] for j, _ in arg],
                                                 [self.w_off[j] for j, _ in arg],
                                                 [c for _, c in arg], g_out, self.causal)
            self._dw_in.append((arg, sv[:len(arg)], [*grads, g_out]))
            return g
        x, qkv, o, lse = sv
        wqkv, wout = self.attn_w[arg]
        batch, n, width = x.shape
        hd = wqkv.shape[0] // (3 * self.heads)
        rows = batch * n
        d_o, d_wout = hcmix.linear_backward(o.view(rows, -1), wout, g.reshape(rows, -1))
        dqkv = hcmix.attention_backward(qkv.view(batch, n, 3, self.heads, hd), o, lse,
                                        d_o.view(batch, n, self.heads, hd))
        dx, d_wqkv = hcmix.linear_backward(x.view(rows, width), wqkv, dqkv.view(rows, -1))
        self.dw_attn[arg] = (d_wqkv, d_wout)
        return dx.view(batch, n, width)

    def sparse_weight_gradients(self):
        """All sparse layers' weight gradients in one library call (fp32)."""
        xs, gs, codes, order = [], [], [], []
        for arg, xin, gout in self._dw_in:
            xs += xin
            gs += gout
            codes += [c for _, c in arg]
            order += [j for j, _ in arg]
        dws, dwo = hcmix.stack_weight_gradients(xs, gs, codes, self.causal)
        self.dw_self = [None] * self.num_sparse
        self.dw_off = [None] * self.num_sparse
        for k, j in enumerate(order):
            self.dw_self[j], self.dw_off[j] = dws[k], dwo[k]

    # ---- whole step ----

    def forward(self, x):
        self._saved = []
        for k in range(len(self.segments)):
            x = self.forward_segment(k, x)
        return x

    def backward(self, dy):
        self._dw_in = []
        self.dw_attn = [None] * len(self.attn_w)
        g = dy
        for k in reversed(range(len(self.segments))):
            g = self.backward_segment(k, g)
        self.sparse_weight_gradients()
        return g
