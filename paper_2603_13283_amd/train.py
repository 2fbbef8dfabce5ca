"""One training step of the paper's two-layer network (App. E): sorted input
queue -> LIF layer 1 -> merge -> LIF layer 2 -> merge -> weighted leaky-
integrator readout with temperature cross-entropy (Sec. 3.3, App. C), the
backward pass chained through both merges (App. D.3), and an Adam update of
the weight matrices.  Options the paper's models use (App. E.5
hyperparameter table): spike-count regularisers on both hidden layers (App.
E.1, Eq. loss) and learnable synaptic delays on both hidden layers (Sec.
3.1 Eq. spike_input, softplus activation, their own Adam learning rate),
each alone or both together.
Every step is a call of liblif.so; this module only holds the device buffers
and orders the calls on one stream."""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Sequence

from . import (LiParams, Params, adam_step, add_, backward, backward_delayed, delay_queues, forward,
               forward_delayed, li_readout, merge, merge_grad, softplus, softplus_grad, spike_count_reg_backward,
               spike_count_reg_delayed_backward, lif_layer_forward_workspace_size,
               lif_layer_backward_workspace_size, lif_li_readout_workspace_size,
               lif_spike_count_reg_backward_workspace_size, lif_spike_count_reg_delayed_workspace_size,
               LIF_MERGE_MAX, _torch)


@dataclass
class AdamParams:
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8


@dataclass
class RegConfig:
    """Spike-count regularisers of the hidden layers (App. E.1): target spike
    counts per layer, lambda_reg and lambda_over-reg.  L_reg and L_over
    average over all hidden neurons of the network, so each layer's terms
    are weighted by its share of them."""
    c_target: Sequence[float] = (14.0, 14.0)
    lam_reg: float = 1e-3
    lam_over: float = 5e-5


@dataclass
class DelayConfig:
    """Learnable delays of both hidden layers: raw parameters X1 [C, N1] and
    X2 [N1, N2] (float32 device tensors, W^T layout), delays d = softplus(X)
    with sharpness beta, updated by Adam with their own learning rate."""
    X1: "object"
    X2: "object"
    beta: float = 5.0
    adam: AdamParams = field(default_factory=lambda: AdamParams(lr=1e-3))


@dataclass
class StepResult:
    loss: "object"                       # float32 [1] device: the readout's cross-entropy
    logits: "object"                     # float32 [B, K]
    grads: dict = field(default_factory=dict)
    fwd1: "object" = None
    fwd2: "object" = None
    queue2: tuple = ()
    queue3: tuple = ()
    reg_losses: tuple = ()               # per hidden layer float32 [2] device: (L_reg, L_over) of its neurons
    delays: tuple = ()                   # per hidden layer: the delays used (float32 device tensors)


class TwoLayerNet:
    """Weights W1 [C, N1], W2 [N1, N2], Wo [N2, K] (W^T layouts, float32
    device tensors) with their Adam moments, and workspaces sized for a
    batch of B queues of at most E_max events."""

    def __init__(self, W1, W2, Wo, B: int, E_max: int, P1: Params = Params(), P2: Params = Params(),
                 q: LiParams = LiParams(), adam: AdamParams = AdamParams(), E2_max: int = LIF_MERGE_MAX,
                 E3_max: int = LIF_MERGE_MAX, reg: Optional[RegConfig] = None, delays: Optional[DelayConfig] = None):
        torch = _torch()
        self.W = [W1, W2, Wo]
        self.m1 = [torch.zeros_like(w) for w in self.W]
        self.m2 = [torch.zeros_like(w) for w in self.W]
        self.P1, self.P2, self.q, self.adam = P1, P2, q, adam
        self.E2_max, self.E3_max = E2_max, E3_max
        self.reg, self.delays = reg, delays
        if delays is not None:
            self.dm1 = [torch.zeros_like(x) for x in (delays.X1, delays.X2)]
            self.dm2 = [torch.zeros_like(x) for x in (delays.X1, delays.X2)]
        self.t = 0
        dev = W1.device
        C, N1 = W1.shape
        N2, K = Wo.shape
        u8 = lambda n: torch.empty(max(int(n), 1), dtype=torch.uint8, device=dev)
        self.ws_f1 = u8(lif_layer_forward_workspace_size(B, E_max, C, N1, P1.c()))
        self.ws_f2 = u8(lif_layer_forward_workspace_size(B, E2_max, N1, N2, P2.c()))
        self.ws_b1 = u8(lif_layer_backward_workspace_size(B, E_max, C, N1, P1.c()))
        self.ws_b2 = u8(lif_layer_backward_workspace_size(B, E2_max, N1, N2, P2.c()))
        self.ws_ro = u8(lif_li_readout_workspace_size(B, E3_max, N2, K))
        if reg is not None:
            size = lif_spike_count_reg_delayed_workspace_size if delays is not None else \
                lif_spike_count_reg_backward_workspace_size
            self.ws_r1 = u8(size(B, E_max, C, N1))
            self.ws_r2 = u8(size(B, E2_max, N1, N2))

    def _layer(self, l, ev_t, ev_src, ev_n, W, P, sequential, stream, ws):
        """Forward of hidden layer l (0 or 1); with delays also its queues."""
        if self.delays is None:
            return forward(ev_t, ev_src, ev_n, W, P, sequential=sequential, stream=stream, ws=ws), None, None
        X = (self.delays.X1, self.delays.X2)[l]
        d = softplus(X, self.delays.beta, stream=stream)
        qs = delay_queues(ev_t, ev_src, ev_n, d, stream=stream)
        out = forward_delayed(qs, ev_src, ev_n, W, P, sequential=sequential, stream=stream)
        out.queues = qs
        return out, qs, d

    def _layer_backward(self, l, ev_t, ev_src, ev_n, W, out, g, P, stream, ws, ws_reg, want_time_grad):
        """Backward of hidden layer l for the spike-time gradient g (with the
        layer's regulariser terms when configured).  Returns (grad_W,
        grad_ev_t or None, grad of the raw delays or None, reg loss or None)."""
        reg_loss = None
        if self.reg is not None:
            n_all = self.W[0].shape[1] + self.W[1].shape[1]
            share = W.shape[1] / n_all
            c, lr, lo = self.reg.c_target[l], self.reg.lam_reg * share, self.reg.lam_over * share
            if self.delays is not None:
                reg_loss, g, gWd, gDd, gTd = spike_count_reg_delayed_backward(
                    out.queues, ev_src, ev_n, W, out, c, lr, lo, P, grad_spike=g, want_time_grad=want_time_grad,
                    stream=stream, ws=ws_reg)
            else:
                reg_loss, g, gWd, gTd = spike_count_reg_backward(
                    ev_t, ev_src, ev_n, W, out, c, lr, lo, P, grad_spike=g, want_time_grad=want_time_grad,
                    stream=stream, ws=ws_reg)
        if self.delays is not None:
            qs, X = out.queues, (self.delays.X1, self.delays.X2)[l]
            gW, gD, gT = backward_delayed(qs, ev_src, ev_n, W, out, g, P, stream=stream, want_time_grad=want_time_grad)
            if self.reg is not None:
                add_(gW, gWd, stream=stream)
                add_(gD, gDd, stream=stream)
                if want_time_grad:
                    add_(gT, gTd, stream=stream)
            return gW, gT, softplus_grad(X, gD, self.delays.beta, stream=stream), reg_loss
        gW, gT = backward(ev_t, ev_src, ev_n, W, out, g, P, stream=stream, want_time_grad=want_time_grad, ws=ws)
        if self.reg is not None:
            add_(gW, gWd, stream=stream)
            if want_time_grad:
                add_(gT, gTd, stream=stream)
        return gW, gT, None, reg_loss

    def step(self, ev_t, ev_src, ev_n, labels, sequential: bool = False, update: bool = True,
             stream=None) -> StepResult:
        """Forward, loss, backward and (update=True) the Adam update; the
        forward passes run the parallel layer, or the sequential baseline
        with sequential=True (everything else is the same)."""
        W1, W2, Wo = self.W
        o1, q1, d1 = self._layer(0, ev_t, ev_src, ev_n, W1, self.P1, sequential, stream, self.ws_f1)
        t2, s2, n2, perm2, _ = merge(o1, self.E2_max, stream=stream)
        o2, q2, d2 = self._layer(1, t2, s2, n2, W2, self.P2, sequential, stream, self.ws_f2)
        t3, s3, n3, perm3, _ = merge(o2, self.E3_max, stream=stream)
        logits, loss, gWo, gT3 = li_readout(t3, s3, n3, Wo, self.q, labels=labels, stream=stream, ws=self.ws_ro)
        g2 = merge_grad(gT3, perm3, n3, W2.shape[1], self.P2.s_max, stream=stream)
        gW2, gT2, gX2, r2 = self._layer_backward(1, t2, s2, n2, W2, o2, g2, self.P2, stream, self.ws_b2,
                                                 getattr(self, "ws_r2", None), True)
        g1 = merge_grad(gT2, perm2, n2, W1.shape[1], self.P1.s_max, stream=stream)
        gW1, _, gX1, r1 = self._layer_backward(0, ev_t, ev_src, ev_n, W1, o1, g1, self.P1, stream, self.ws_b1,
                                               getattr(self, "ws_r1", None), False)
        grads = {"W1": gW1, "W2": gW2, "Wo": gWo}
        if self.delays is not None:
            grads.update({"X1": gX1, "X2": gX2})
        if update:
            self.t += 1
            a = self.adam
            for w, g, m1, m2 in zip(self.W, (gW1, gW2, gWo), self.m1, self.m2):
                adam_step(w, g, m1, m2, self.t, a.lr, a.beta1, a.beta2, a.eps, stream=stream)
            if self.delays is not None:
                a = self.delays.adam
                for x, g, m1, m2 in zip((self.delays.X1, self.delays.X2), (gX1, gX2), self.dm1, self.dm2):
                    adam_step(x, g, m1, m2, self.t, a.lr, a.beta1, a.beta2, a.eps, stream=stream)
        regs = (r1, r2) if self.reg is not None else ()
        return StepResult(loss, logits, grads, o1, o2, (t2, s2, n2, perm2), (t3, s3, n3, perm3), regs,
                          (d1, d2) if self.delays is not None else ())
