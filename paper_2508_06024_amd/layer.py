"""One group-gated MoE layer with the low-rank codec at the end-cloud cut, on device.

The step follows the paper's pipeline (EC2MoE Overall Design; HL-GGN then PO-ECC):
the end side routes the hidden states X with the hardware-aware group gate and
compresses them, Z = U^T X V (per slice of h = T / c rows); the cloud side
reconstructs X_hat = U_hat Z V_hat^T and
runs the sparse MoE layer of Eq. 1 on X_hat with the end side's routing:

    route = group_gate(X, mask);  Z = encode(X);  X_hat = decode(Z);  y = moe(X_hat, route)

All four are calls into libec2moe; this class only owns the device buffers (allocated
once) and issues the calls on the current stream.

overlap=True runs the routing (gate, then the index permutation), which like the codec
depends only on X, on a second stream (default priority) forked from and joined back into
the current one, so that it overlaps the codec; the expert GEMMs and the combine follow on
the current stream. The kernels and their inputs are those of the one-stream order, so
the results are bit-identical. It is off by default: the cross-stream join costs about as
much as the overlap saves on the workloads measured, and more on the small ones.
"""
from __future__ import annotations

import torch

from . import ec2moe as E


class Ec2moeLayer:
    def __init__(self, x, mask_words, w_global, b_global, w_local, b_local, w_gate_up, w_down, u, v,
                 u_hat=None, v_hat=None, n_groups=1, top_k=1, renormalize=True, activation="swiglu",
                 codec_slices=1, top_groups=0, group_sizes=None, overlap=False):
        T, d = x.shape
        M, _, H = w_down.shape
        dt = x.dtype
        dev = x.device
        self.x, self.mask = x, list(mask_words)
        self.w_global, self.b_global, self.w_local, self.b_local = w_global, b_global, w_local, b_local
        self.w_gate_up, self.w_down = w_gate_up, w_down
        self.u, self.v = u, v
        self.u_hat = u if u_hat is None else u_hat
        self.v_hat = v if v_hat is None else v_hat
        if tuple(w_gate_up.shape) != (M, E.w_in_rows(H, activation), d):
            raise ValueError(f"w_gate_up has shape {tuple(w_gate_up.shape)} for {activation} experts of width {H}")
        self.moe_desc = E.moe_desc(T, M, n_groups, d, H, top_k, dt, renormalize, activation)
        # gate options: top-G groups, unequal groups and the gate workspace that lets a small
        # batch split d over more workgroups
        self.gate_ws = E.workspace(E.gate_workspace_size(self.moe_desc), dev)
        self.gate_opts = E.gate_opts(top_groups, group_sizes, self.gate_ws)
        if T % codec_slices or u.shape[0] != T // codec_slices:
            raise ValueError(f"u has {u.shape[0]} rows for {codec_slices} slices of {T} tokens")
        self.codec_desc = E.codec_desc(T // codec_slices, d, u.shape[1], v.shape[1], dt, codec_slices)
        self.topk_idx = torch.empty((T, top_k), dtype=torch.int32, device=dev)
        self.topk_w = torch.empty((T, top_k), dtype=torch.float32, device=dev)
        self.z = torch.empty((codec_slices, u.shape[1], v.shape[1]), dtype=torch.float32, device=dev)
        self.x_hat = torch.empty((T, d), dtype=dt, device=dev)
        self.y = torch.empty((T, d), dtype=dt, device=dev)
        self.moe_ws = E.workspace(E.moe_workspace_size(self.moe_desc), dev)
        self.overlap = overlap
        if overlap:
            A = T * top_k
            self.seg = torch.empty(M + 1, dtype=torch.int32, device=dev)
            self.perm_src = torch.empty(A, dtype=torch.int32, device=dev)
            self.inv_perm = torch.empty(A, dtype=torch.int32, device=dev)
            self.y_perm = torch.empty((A, d), dtype=dt, device=dev)
            self.side = torch.cuda.Stream(device=dev)
            self.forked = torch.cuda.Event()
            self.routed = torch.cuda.Event()
        self.codec_ws = E.workspace(E.lowrank_workspace_size(self.codec_desc), dev)

    def set_input(self, x, mask_words=None):
        """Point the layer at another [T][d] input (and candidate mask) of the same shape."""
        assert x.shape == self.x.shape and x.dtype == self.x.dtype
        self.x = x
        if mask_words is not None:
            self.mask = list(mask_words)

    def _gate(self):
        E.group_gate_ex(self.moe_desc, self.gate_opts, self.mask, self.x, self.w_global, self.b_global,
                        self.w_local, self.b_local, self.topk_idx, self.topk_w)

    def route(self):
        """The gate alone on the current input: (topk_idx, topk_w), the routing step() uses."""
        self._gate()
        return self.topk_idx, self.topk_w

    def _codec(self):
        E.lowrank_encode_into(self.codec_desc, self.x, self.u, self.v, self.z, self.codec_ws)
        E.lowrank_decode_into(self.codec_desc, self.z, self.u_hat, self.v_hat, self.x_hat, self.codec_ws)

    def step(self):
        if not self.overlap:
            self._gate()
            self._codec()
            E.moe_forward_into(self.moe_desc, self.x_hat, self.topk_idx, self.topk_w, self.w_gate_up,
                               self.w_down, self.y, self.moe_ws)
            return self.y
        main = torch.cuda.current_stream()
        # the fork orders this step's routing after everything the current stream holds, the
        # previous step's experts and combine (readers of the routing buffers) included
        self.forked.record(main)
        self.side.wait_event(self.forked)
        with torch.cuda.stream(self.side):
            self._gate()
            E.permute_into(self.moe_desc, self.topk_idx, self.seg, self.perm_src, self.inv_perm, self.moe_ws)
            self.routed.record(self.side)
        self._codec()
        main.wait_event(self.routed)
        E.expert_ffn_into(self.moe_desc, self.x_hat, self.seg, self.perm_src, self.w_gate_up, self.w_down,
                          self.y_perm, self.moe_ws)
        E.combine_into(self.moe_desc, self.y_perm, self.inv_perm, self.topk_w, self.y)
        return self.y
