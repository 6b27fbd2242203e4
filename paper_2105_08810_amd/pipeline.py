"""A whole network through libsnn: LIF forward of every layer, readout loss, active-set
compaction, the sparse backward chain and the dense baseline chain.

This is orchestration only -- allocation and the order of C-ABI calls; every number is
computed by the HIP kernels. The network is the paper's fully connected stack (Sec. 3): L LIF
layers then an infinite-threshold readout with a cross-entropy loss (App. E).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional

import torch

from . import snn

INF = float("inf")


@dataclass
class Network:
    X: torch.Tensor  # [T, B, N_in] uint8
    Ws: List[torch.Tensor]
    W_out: torch.Tensor
    alphas: List[float]
    alpha_out: float
    labels: torch.Tensor  # [B] int32
    loss_mode: int  # 0 = max over t, 1 = sum over t
    theta: float = 1.0
    beta: float = 100.0
    # forward state
    V: List[torch.Tensor] = field(default_factory=list)
    S: List[torch.Tensor] = field(default_factory=list)
    trace: List[torch.Tensor] = field(default_factory=list)
    V_out: Optional[torch.Tensor] = None
    S_out: Optional[torch.Tensor] = None
    trace_out: Optional[torch.Tensor] = None
    bits: List[torch.Tensor] = field(default_factory=list)  # active bitsets of the LIF layers
    bits_bth: Optional[float] = None
    # trace recompute: with recompute_k = K > 0 the LIF layers' input traces are not stored; the
    # forward keeps the trace at every K-th step (ck) and the sparse dW rebuilds the rest from the
    # input spikes (snn_sparse_dw_spikes). The dense baseline needs the stored traces.
    recompute_k: int = 0
    ck: List[torch.Tensor] = field(default_factory=list)
    _aux2: Optional[torch.cuda.Stream] = None  # second dW stream of the pipelined schedule

    @property
    def T(self):
        return self.X.shape[0]

    @property
    def B(self):
        return self.X.shape[1]

    @property
    def L(self):
        return len(self.Ws)

    def allocate(self):
        """Forward buffers, allocated once so repeated steps reuse them."""
        dev = self.X.device
        T, B = self.T, self.B
        sizes = [self.X.shape[2]] + [W.shape[1] for W in self.Ws]
        self.V = [torch.empty((T, B, n), dtype=torch.float32, device=dev) for n in sizes[1:]]
        self.S = [torch.empty((T, B, n), dtype=torch.uint8, device=dev) for n in sizes[1:]]
        if self.recompute_k > 0:
            nck = snn.snn_trace_checkpoint_count(T, self.recompute_k)
            self.trace = [None] * self.L
            self.ck = [torch.empty((nck, B, n), dtype=torch.float32, device=dev) for n in sizes[:-1]]
        else:
            self.trace = [torch.empty((T, B, n), dtype=torch.float32, device=dev) for n in sizes[:-1]]
        C = self.W_out.shape[1]
        self.V_out = torch.empty((T, B, C), dtype=torch.float32, device=dev)
        self.S_out = torch.empty((T, B, C), dtype=torch.uint8, device=dev)
        self.trace_out = torch.empty((T, B, sizes[-1]), dtype=torch.float32, device=dev)
        return self

    def forward(self, b_th: Optional[float] = None):
        """Forward of every layer. With b_th, the LIF layers also mark their active sets (bitsets
        that compact() then turns into CSR without reading V again)."""
        if not self.V:
            self.allocate()
        x = self.X
        T, B = self.T, self.B
        if b_th is not None and not self.bits:
            self.bits = [torch.empty(snn.snn_active_bits_words(T, B, W.shape[1]), dtype=torch.int64,
                                     device=self.X.device) for W in self.Ws]
        self.bits_bth = b_th
        L = len(self.Ws)
        top = None
        for l, W in enumerate(self.Ws):
            if self.recompute_k > 0:
                snn.trace_checkpoints(x, self.alphas[l], self.recompute_k, ck=self.ck[l])
            # A top layer whose width is whole 64-bit bitset words takes the fused forward, which
            # absorbs the stores of the readout's input trace written from its spikes as it makes
            # them, and the readout then walks no trace (three 1024-wide layers, a 1024 -> 100
            # readout, T = 500, B = 256: forward 1.81 -> 1.77 ms). In the two-kernel form the top layer's recurrence is the critical
            # path and the readout's own trace blocks run beside its short recurrence, so the
            # readout keeps writing it (2312 -> 200 -> 10, T = 300, B = 256: 0.446 against 0.453 ms).
            top = self.trace_out if l == L - 1 and W.shape[1] % 64 == 0 else None
            snn.snn_lif_forward_traces(x, W, T, B, W.shape[0], W.shape[1], self.alphas[l], self.theta,
                                       0.0 if b_th is None else b_th, self.V[l], self.S[l], self.trace[l], top,
                                       self.alpha_out, None if b_th is None else self.bits[l])
            x = self.S[l]
        snn.snn_lif_forward(x, self.W_out, T, B, self.W_out.shape[0], self.W_out.shape[1], self.alpha_out, INF,
                            self.V_out, self.S_out, None if top is not None else self.trace_out)
        return self

    def readout(self, dense=False):
        """Readout CSR, eps at its entries, loss (device scalar) and, if asked, dL/dV_out densely."""
        return snn.readout_ce(self.V_out, self.labels, self.loss_mode, dense=dense)

    def compact(self, b_th, capacities: Optional[List[int]] = None) -> List[snn.Csr]:
        """CSR of every LIF layer's active set: from the forward's bitsets when they were marked
        with this b_th, else from V."""
        caps = capacities or [None] * self.L
        return [self.compact_layer(l, b_th, caps[l]) for l in range(self.L)]

    def compact_layer(self, l, b_th, capacity: Optional[int] = None) -> snn.Csr:
        """CSR of layer l's active set (as compact())."""
        if self.bits and self.bits_bth == b_th:
            return snn.active_compact_bits(self.bits[l], self.V[l], self.theta, self.beta, capacity)
        return snn.active_compact(self.V[l], self.theta, b_th, self.beta, capacity)

    def activity(self, reg: "Penalty", want_zeta=False):
        """Activity penalties of every LIF layer (App. E) on the forward's spikes.
        Returns a list of (coef [B, N_l], penalty [1], zeta or None), all on the device."""
        return [snn.activity_reg(S, reg.lam_low, reg.nu_low, reg.lam_up, reg.nu_up, want_zeta) for S in self.S]

    def sparse_backward(self, csrs: List[snn.Csr], ro=None, aux_stream=None, workspaces=None, reg_coefs=None):
        """Readout backward, then every LIF layer top down. Returns (dW list, dW_out, eps list)
        where eps[l] is the gradient w.r.t. layer l's spikes at its active entries. reg_coefs[l]
        ([B, N_l], from activity()) joins layer l's spike gradient before its backward."""
        if ro is None:
            ro = self.readout()
        ro_csr, ro_eps = ro[0], ro[1]
        ws = workspaces or [None] * (self.L + 1)
        if aux_stream is not None and self.L >= 2 and self.recompute_k == 0 and workspaces is None:
            return self._sparse_backward_pipelined(csrs, ro_csr, ro_eps, aux_stream, reg_coefs)
        dW_out, eps = snn.sparse_backward(self.W_out, self.trace_out, self.alpha_out, ro_csr, ro_eps,
                                          inp=csrs[self.L - 1], ws=ws[self.L], aux_stream=aux_stream)
        dWs: List[Optional[torch.Tensor]] = [None] * self.L
        epss: List[Optional[torch.Tensor]] = [None] * self.L
        for l in range(self.L - 1, -1, -1):
            if reg_coefs is not None:
                snn.activity_reg_grad(reg_coefs[l], self.T, eps, csrs[l])
            epss[l] = eps
            if self.recompute_k > 0:
                dWs[l], eps = self._layer_backward_recompute(l, csrs, eps, aux_stream)
            else:
                dWs[l], eps = snn.sparse_backward(self.Ws[l], self.trace[l], self.alphas[l], csrs[l], eps,
                                                  inp=csrs[l - 1] if l > 0 else None, ws=ws[l],
                                                  aux_stream=aux_stream)
        return dWs, dW_out, epss

    def _sparse_backward_pipelined(self, csrs, ro_csr, ro_eps, aux, reg_coefs=None):
        """The spike gradients form a chain down the layers (each needs the one above), while a
        layer's dW needs only its own eps, and the structure-only part of every dW call needs only
        the active sets. The layouts run on aux from the start, beside the readout's backward.
        When a dW call fills the GPU by itself (big layers), the dW calls then run on the current
        stream, each after its layer's spike gradient (a dW beside a spike gradient would only take
        CUs from it, and the chain then starts without waiting for a layout); for small layers every dW runs on a dW stream as soon as its eps is there, beside
        the chain."""
        main = torch.cuda.current_stream()
        T, B, L = self.T, self.B, self.L
        big = max(csrs[l].capacity * self.Ws[l].shape[0] for l in range(L)) >= 10 ** 9  # multiply-adds
        if not big and self._aux2 is None:
            self._aux2 = torch.cuda.Stream()  # default priority
        streams = [main] if big else [aux, self._aux2]
        aux.wait_stream(main)  # the active sets are ready: the dW parts that need only them start on aux
        wss, laid = [], []
        with torch.cuda.stream(aux):
            for l in range(L - 1, -1, -1):  # top layer first: its dW comes first
                n_in, n_out = self.Ws[l].shape
                ws = snn.workspace(snn.snn_sparse_dw_workspace(T, B, n_in, n_out, csrs[l].capacity), self.X.device)
                snn.sparse_dw_layout((T, B, n_in), csrs[l], n_out, ws, stream=aux)
                ev = torch.cuda.Event()
                ev.record(aux)
                wss.insert(0, ws)
                laid.insert(0, ev)
        eps = snn.sparse_grad_in(self.W_out, self.alpha_out, T, B, ro_csr, ro_eps, csrs[L - 1], share_cu=not big,
                                 stream=main)
        dWs: List[Optional[torch.Tensor]] = [None] * L
        epss: List[Optional[torch.Tensor]] = [None] * L
        for l in range(L - 1, -1, -1):
            if reg_coefs is not None:
                snn.activity_reg_grad(reg_coefs[l], T, eps, csrs[l])
            epss[l] = eps
            eps_below = None
            if big and l > 0:  # one stream: the spike gradient first, it needs no layout
                eps_below = snn.sparse_grad_in(self.Ws[l], self.alphas[l], T, B, csrs[l], eps, csrs[l - 1],
                                               share_cu=False, stream=main)
            sd = streams[(L - 1 - l) % len(streams)]
            sd.wait_stream(main)  # eps of layer l is ready
            sd.wait_event(laid[l])  # and its layout
            with torch.cuda.stream(sd):
                dWs[l] = snn.sparse_dw_prepared(self.trace[l], csrs[l], eps, self.Ws[l].shape[1], wss[l], stream=sd)
            if l > 0:
                eps = eps_below if big else snn.sparse_grad_in(self.Ws[l], self.alphas[l], T, B, csrs[l], eps,
                                                               csrs[l - 1], share_cu=True, stream=main)
        with torch.cuda.stream(aux):  # the readout's dW last: nothing below waits for it
            dW_out = snn.sparse_dw(self.trace_out, ro_csr, ro_eps, self.W_out.shape[1], stream=aux)
        for sd in [aux] + streams:
            if sd is not main:
                main.wait_stream(sd)
        for t in dWs + [dW_out] + wss:
            t.record_stream(main)
        return dWs, dW_out, epss

    def _layer_backward_recompute(self, l, csrs, eps, aux_stream=None):
        """Layer l's sparse backward with the trace rebuilt from its input spikes: the spike
        gradient (on aux_stream when given) beside dW from snn_sparse_dw_spikes."""
        s_in = self.X if l == 0 else self.S[l - 1]
        W = self.Ws[l]
        main = torch.cuda.current_stream()
        eps_in = None
        if l > 0:
            side = aux_stream if aux_stream is not None else main
            side.wait_stream(main)
            with torch.cuda.stream(side):
                eps_in = snn.sparse_grad_in(W, self.alphas[l], self.T, self.B, csrs[l], eps, csrs[l - 1],
                                            share_cu=aux_stream is not None, stream=side)
        dW = snn.sparse_dw_spikes(s_in, self.ck[l], self.recompute_k, self.alphas[l], csrs[l], eps, W.shape[1],
                                  stream=main)
        if l > 0 and aux_stream is not None:
            main.wait_stream(aux_stream)
            eps_in.record_stream(main)
        return dW, eps_in

    def dense_backward(self, b_th, ro=None, reg_coefs=None):
        """The dense baseline chain (b_th = inf: full-surrogate BPTT). Returns (dW list, dW_out,
        eps_dense list); reg_coefs as in sparse_backward."""
        if self.recompute_k > 0:
            raise ValueError("dense_backward needs the stored input traces (recompute_k = 0)")
        if ro is None or ro[3] is None:
            ro = self.readout(dense=True)
        dW_out, eps = snn.dense_backward_ref(self.W_out, self.trace_out, self.V_out, ro[3], self.alpha_out, INF,
                                             INF, self.beta, grad_in=True)
        dWs: List[Optional[torch.Tensor]] = [None] * self.L
        epss: List[Optional[torch.Tensor]] = [None] * self.L
        for l in range(self.L - 1, -1, -1):
            if reg_coefs is not None:
                snn.activity_reg_grad(reg_coefs[l], self.T, eps)
            epss[l] = eps
            dWs[l], eps = snn.dense_backward_ref(self.Ws[l], self.trace[l], self.V[l], eps, self.alphas[l],
                                                 self.theta, b_th, self.beta, grad_in=l > 0)
        return dWs, dW_out, epss


    def params(self) -> List[torch.Tensor]:
        return list(self.Ws) + [self.W_out]

    def train_step(self, opt: "Adam", b_th: float, reg: Optional["Penalty"] = None, sparse: bool = True,
                   aux_stream=None, events=None):
        """One training step (App. E): forward, cross-entropy plus activity penalties, the sparse
        (or, with sparse=False, the dense) backward with truncation band b_th, and an Adam step on
        every weight matrix in place. b_th = inf with sparse=False is full-surrogate BPTT.
        events: optional list of 6 timing events recorded on the current stream at the phase
        boundaries (start, after forward, after loss and penalties, after compaction, after the
        backward, after Adam).
        Returns a dict of device tensors: ce [1], penalty [1] (all layers), grads (list), nnz."""
        mark = (lambda k: events[k].record()) if events is not None else (lambda k: None)
        mark(0)
        self.forward(b_th if sparse and math.isfinite(b_th) else None)
        mark(1)
        acts = self.activity(reg) if reg is not None else None
        coefs = [a[0] for a in acts] if acts else None
        ro = self.readout(dense=not sparse)
        mark(2)
        if sparse:
            csrs = self.compact(b_th)
            mark(3)
            dWs, dW_out, _ = self.sparse_backward(csrs, ro, aux_stream=aux_stream, reg_coefs=coefs)
            nnz = [c.nnz_dev for c in csrs]
        else:
            mark(3)
            dWs, dW_out, _ = self.dense_backward(b_th, ro, reg_coefs=coefs)
            nnz = None
        mark(4)
        grads = list(dWs) + [dW_out]
        opt.step(grads)
        mark(5)
        pen = sum(a[1] for a in acts) if acts else torch.zeros(1, device=self.X.device)
        return {"ce": ro[2], "penalty": pen, "grads": grads, "nnz": nnz}


@dataclass
class Penalty:
    """Activity penalty weights and bounds of App. E (its parameter table: F-MNIST / N-MNIST
    values by default; SHD uses nu_up = 10)."""
    lam_low: float = 100.0
    nu_low: float = 0.001
    lam_up: float = 0.06
    nu_up: float = 1.0


class Adam:
    """Adam state for a list of float32 device tensors, updated in place by snn_adam_step."""

    def __init__(self, params: List[torch.Tensor], lr: float, betas=(0.9, 0.999), eps: float = 1e-8):
        self.params = params
        self.lr, self.betas, self.eps = float(lr), tuple(betas), float(eps)
        self.m = [torch.zeros_like(p) for p in params]
        self.v = [torch.zeros_like(p) for p in params]
        self.k = 0

    def step(self, grads: List[torch.Tensor]):
        self.k += 1
        for p, g, m, v in zip(self.params, grads, self.m, self.v):
            snn.adam_step(p, g, m, v, self.k, self.lr, self.betas, self.eps)


@dataclass
class ConvNetwork:
    """The convolutional network of Sec. 3's convolutional experiment (App. E): a convolutional
    LIF layer (3x3, stride 1, padding 1, F filters) on input spikes [T, B, H, W, C], 2x2 max
    pooling of its spikes, and the infinite-threshold readout on the flattened pooled spikes."""
    X: torch.Tensor  # [T, B, H, W, C] uint8
    Wc: torch.Tensor  # [3, 3, C, F]
    W_out: torch.Tensor  # [(H/2)(W/2)F, classes]
    alpha: float
    alpha_out: float
    labels: torch.Tensor
    loss_mode: int
    theta: float = 1.0
    beta: float = 100.0
    V: Optional[torch.Tensor] = None
    S: Optional[torch.Tensor] = None
    trace: Optional[torch.Tensor] = None
    bits: Optional[torch.Tensor] = None
    bits_bth: Optional[float] = None
    P: Optional[torch.Tensor] = None
    arg: Optional[torch.Tensor] = None
    pbits: Optional[torch.Tensor] = None
    V_out: Optional[torch.Tensor] = None
    S_out: Optional[torch.Tensor] = None
    trace_out: Optional[torch.Tensor] = None

    @property
    def dims(self):
        T, B, H, W, C = self.X.shape
        return T, B, H, W, C, self.Wc.shape[3]

    @property
    def N(self):
        _, _, H, W, _, F = self.dims
        return H * W * F

    @property
    def Np(self):
        _, _, H, W, _, F = self.dims
        return (H // 2) * (W // 2) * F

    def allocate(self):
        T, B, H, W, C, F = self.dims
        dev = self.X.device
        self.V = torch.empty((T, B, self.N), dtype=torch.float32, device=dev)
        self.S = torch.empty((T, B, self.N), dtype=torch.uint8, device=dev)
        self.trace = torch.empty((T, B, H * W * C), dtype=torch.float32, device=dev)
        self.bits = torch.empty(snn.snn_active_bits_words(T, B, self.N), dtype=torch.int64, device=dev)
        self.P = torch.empty((T, B, self.Np), dtype=torch.uint8, device=dev)
        self.arg = torch.empty((T, B, self.Np), dtype=torch.uint8, device=dev)
        self.pbits = torch.empty(snn.snn_active_bits_words(T, B, self.Np), dtype=torch.int64, device=dev)
        Cl = self.W_out.shape[1]
        self.V_out = torch.empty((T, B, Cl), dtype=torch.float32, device=dev)
        self.S_out = torch.empty((T, B, Cl), dtype=torch.uint8, device=dev)
        self.trace_out = torch.empty((T, B, self.Np), dtype=torch.float32, device=dev)
        return self

    def forward(self, b_th: Optional[float] = None):
        """Conv layer (marking its active set when b_th is given), pooling, readout."""
        if self.V is None:
            self.allocate()
        T, B, H, W, C, F = self.dims
        snn.snn_conv_lif_forward(self.X, self.Wc, T, B, H, W, C, F, self.alpha, self.theta,
                                 0.0 if b_th is None else b_th, self.V, self.S, self.trace,
                                 None if b_th is None else self.bits)
        self.bits_bth = b_th
        snn.snn_maxpool_spikes(self.S, T, B, H, W, F, self.P, self.arg)
        snn.snn_lif_forward(self.P, self.W_out, T, B, self.Np, self.W_out.shape[1], self.alpha_out, INF, self.V_out,
                            self.S_out, self.trace_out)
        return self

    def readout(self, dense=False):
        return snn.readout_ce(self.V_out, self.labels, self.loss_mode, dense=dense)

    def compact(self, b_th, capacities: Optional[List[int]] = None):
        """[conv CSR (with g), pooled CSR (the readout's input-active entries)]; the forward must
        have marked the active set with this b_th."""
        if self.bits_bth != b_th:
            raise ValueError("compact(b_th): run forward(b_th) first")
        T, B, H, W, C, F = self.dims
        caps = capacities or [None, None]
        conv = snn.active_compact_bits(self.bits, self.V, self.theta, self.beta, caps[0])
        snn.snn_pool_route_bits(self.bits, self.arg, T, B, H, W, F, self.pbits)
        pool = snn.active_compact_bits(self.pbits, None, self.theta, self.beta, caps[1], with_g=False,
                                       shape=(T, B, self.Np))
        return [conv, pool]

    def params(self) -> List[torch.Tensor]:
        return [self.Wc, self.W_out]

    def activity(self, reg: "Penalty", want_zeta=False):
        """Activity penalties (App. E) of the conv layer's spikes: (coef [B, N], penalty [1], zeta)."""
        return snn.activity_reg(self.S, reg.lam_low, reg.nu_low, reg.lam_up, reg.nu_up, want_zeta)

    def sparse_backward(self, csrs, ro=None, ws=None, reg_coef=None):
        """Readout backward at the pooled entries, routed to the conv layer's active entries, and
        the sparse filter gradient. reg_coef ([B, N], from activity()) joins the conv spikes'
        gradient before the filter gradient. Returns (dWc, dW_out, eps at the conv entries)."""
        if ro is None:
            ro = self.readout()
        conv, pool = csrs
        dW_out, eps_pool = snn.sparse_backward(self.W_out, self.trace_out, self.alpha_out, ro[0], ro[1], inp=pool)
        dWc, eps = self._route_and_filter(conv, pool, eps_pool, ws, reg_coef)
        return dWc, dW_out, eps

    def compact_and_backward(self, b_th, ro=None, capacities: Optional[List[int]] = None, ws=None, reg_coef=None,
                             aux_stream=None, events=None):
        """compact() then sparse_backward(), with the conv layer's compaction on aux_stream beside
        the pooled entries' compaction and the readout's backward, which need only the pooled
        entries; the routing to the conv entries waits for both. events: optional dict of timing
        events, "conv0"/"conv1" recorded around the conv layer's compaction (on its stream) and
        "pool0"/"pool1" around the pooled entries' compaction. Returns (csrs, (dWc, dW_out, eps))."""
        mark = (lambda k, st: events[k].record(st)) if events is not None else (lambda k, st: None)
        if self.bits_bth != b_th:
            raise ValueError("compact_and_backward(b_th): run forward(b_th) first")
        if ro is None:
            ro = self.readout()
        T, B, H, W, C, F = self.dims
        caps = capacities or [None, None]
        main = torch.cuda.current_stream()
        side = aux_stream if aux_stream is not None else main
        side.wait_stream(main)
        with torch.cuda.stream(side):
            mark("conv0", side)
            conv = snn.active_compact_bits(self.bits, self.V, self.theta, self.beta, caps[0])
            mark("conv1", side)
        mark("pool0", main)
        snn.snn_pool_route_bits(self.bits, self.arg, T, B, H, W, F, self.pbits)
        pool = snn.active_compact_bits(self.pbits, None, self.theta, self.beta, caps[1], with_g=False,
                                       shape=(T, B, self.Np))
        mark("pool1", main)
        dW_out, eps_pool = snn.sparse_backward(self.W_out, self.trace_out, self.alpha_out, ro[0], ro[1], inp=pool)
        if side is not main:
            main.wait_stream(side)
            conv.record_stream(main)
        dWc, eps = self._route_and_filter(conv, pool, eps_pool, ws, reg_coef)
        return [conv, pool], (dWc, dW_out, eps)

    def pooled_backward(self, b_th, ro=None, pool_capacity: Optional[int] = None, ws=None, events=None):
        """The sparse backward from the pooled entries alone, for a loss that reaches the conv
        spikes only through the pooling (no activity penalty): the pooled entries' compaction, the
        readout's backward at them, and the filter gradient of the conv neurons the pooling picked
        (snn_conv_sparse_dw_pooled); every other conv neuron, active or not, has a zero gradient,
        so no conv-layer compaction and no routing are needed. events: optional dict of timing
        events, "pool0"/"pool1" recorded around the pooled entries' compaction. Returns
        (pooled CSR, (dWc, dW_out, eps at the pooled entries))."""
        if self.bits_bth != b_th:
            raise ValueError("pooled_backward(b_th): run forward(b_th) first")
        mark = (lambda k: events[k].record()) if events is not None else (lambda k: None)
        if ro is None:
            ro = self.readout()
        T, B, H, W, C, F = self.dims
        mark("pool0")
        snn.snn_pool_route_bits(self.bits, self.arg, T, B, H, W, F, self.pbits)
        pool = snn.active_compact_bits(self.pbits, None, self.theta, self.beta, pool_capacity, with_g=False,
                                       shape=(T, B, self.Np))
        mark("pool1")
        dW_out, eps_pool = snn.sparse_backward(self.W_out, self.trace_out, self.alpha_out, ro[0], ro[1], inp=pool)
        dWc = torch.empty_like(self.Wc)
        if ws is None:
            ws = snn.workspace(snn.snn_conv_sparse_dw_workspace(T, B, H, W, C, F), self.X.device)
        snn.snn_conv_sparse_dw_pooled(self.trace, self.V, self.arg, T, B, H, W, C, F, self.theta, b_th, self.beta,
                                      pool.row_ptr, pool.col_idx, eps_pool, pool.capacity, dWc, ws)
        return pool, (dWc, dW_out, eps_pool)

    def _route_and_filter(self, conv, pool, eps_pool, ws, reg_coef):
        """The pooled gradient routed to the conv entries, the penalty term, the filter gradient."""
        T, B, H, W, C, F = self.dims
        eps = torch.empty(conv.capacity, dtype=torch.float32, device=self.X.device)
        snn.snn_pool_scatter_eps(T, B, H, W, F, pool.row_ptr, pool.col_idx, pool.capacity, eps_pool, self.arg,
                                 conv.row_ptr, conv.col_idx, conv.capacity, eps)
        if reg_coef is not None:
            snn.activity_reg_grad(reg_coef, T, eps, conv)
        dWc = torch.empty_like(self.Wc)
        if ws is None:
            ws = snn.workspace(snn.snn_conv_sparse_dw_workspace(T, B, H, W, C, F), self.X.device)
        snn.snn_conv_sparse_dw(self.trace, T, B, H, W, C, F, conv.row_ptr, conv.col_idx, conv.g, eps, conv.capacity,
                               dWc, ws)
        return dWc, eps

    def dense_backward(self, b_th, ro=None, ws=None, reg_coef=None):
        """The dense chain: dense readout backward, dense routing, dense filter gradient (b_th =
        inf: full surrogate); reg_coef as in sparse_backward. Returns (dWc, dW_out, eps dense
        [T, B, N])."""
        if ro is None or ro[3] is None:
            ro = self.readout(dense=True)
        T, B, H, W, C, F = self.dims
        dW_out, eps_pool = snn.dense_backward_ref(self.W_out, self.trace_out, self.V_out, ro[3], self.alpha_out, INF,
                                                  INF, self.beta, grad_in=True)
        eps = torch.empty((T, B, self.N), dtype=torch.float32, device=self.X.device)
        snn.snn_pool_scatter_eps_dense(eps_pool, self.arg, T, B, H, W, F, eps)
        if reg_coef is not None:
            snn.activity_reg_grad(reg_coef, T, eps)
        dWc = torch.empty_like(self.Wc)
        if ws is None:
            ws = snn.workspace(snn.snn_conv_dense_dw_workspace(T, B, H, W, C, F), self.X.device)
        snn.snn_conv_dense_dw(self.trace, self.V, eps, T, B, H, W, C, F, self.theta, b_th, self.beta, dWc, ws)
        return dWc, dW_out, eps

    def train_step(self, opt: "Adam", b_th: float, reg: Optional["Penalty"] = None, sparse: bool = True,
                   aux_stream=None, events=None):
        """One training step of the conv network (App. E), as Network.train_step: forward,
        cross-entropy plus the conv layer's activity penalties, the sparse (or dense) backward with
        band b_th, Adam on Wc and W_out in place. aux_stream is accepted for a common interface
        and not used. Returns a dict of device tensors: ce [1], penalty [1], grads [dWc, dW_out],
        nnz ([conv layer's active-entry count] or None)."""
        mark = (lambda k: events[k].record()) if events is not None else (lambda k: None)
        mark(0)
        self.forward(b_th if sparse and math.isfinite(b_th) else None)
        mark(1)
        act = self.activity(reg) if reg is not None else None
        coef = act[0] if act else None
        ro = self.readout(dense=not sparse)
        mark(2)
        if sparse:
            csrs = self.compact(b_th)
            mark(3)
            dWc, dW_out, _ = self.sparse_backward(csrs, ro, reg_coef=coef)
            nnz = [csrs[0].nnz_dev]
        else:
            mark(3)
            dWc, dW_out, _ = self.dense_backward(b_th, ro, reg_coef=coef)
            nnz = None
        mark(4)
        grads = [dWc, dW_out]
        opt.step(grads)
        mark(5)
        pen = act[1] if act else torch.zeros(1, device=self.X.device)
        return {"ce": ro[2], "penalty": pen, "grads": grads, "nnz": nnz}


class Graphed:
    """Library calls captured once as a HIP graph and replayed. fn makes its calls on the current
    stream (the capture stream) and returns what later work reads; those tensors stay the
    outputs of every replay. Capture records work without running it, so replay before reading."""

    def __init__(self, fn, stream=None):
        self.graph = torch.cuda.CUDAGraph()
        cur = stream or torch.cuda.current_stream()
        cap = torch.cuda.Stream()  # default priority
        cap.wait_stream(cur)
        with torch.cuda.graph(self.graph, stream=cap):
            self.out = fn()
        cur.wait_stream(cap)

    def __call__(self, stream=None):
        with torch.cuda.stream(stream or torch.cuda.current_stream()):
            self.graph.replay()
        return self.out


def from_inputs(inp, device="cuda") -> Network:
    """Network on the device from a synth.Inputs bundle (host arrays)."""
    dev = torch.device(device)
    cfg = inp.cfg
    return Network(
        X=torch.from_numpy(inp.X).to(dev),
        Ws=[torch.from_numpy(W).to(dev) for W in inp.Ws],
        W_out=torch.from_numpy(inp.W_out).to(dev),
        alphas=[float(a) for a in inp.alphas],
        alpha_out=float(inp.alpha_out),
        labels=torch.from_numpy(inp.labels.astype("int32")).to(dev),
        loss_mode=0 if cfg.loss_mode == "max" else 1,
        theta=float(cfg.theta),
        beta=float(cfg.beta),
    )
