"""One training step of the paper's two-layer network (App. E): sorted input
queue -> LIF layer 1 -> merge -> LIF layer 2 -> merge -> weighted leaky-
integrator readout with temperature cross-entropy (Sec. 3.3, App. C), the
backward pass chained through both merges (App. D.3), and an Adam update of
the three weight matrices.  Every step is a call of liblif.so; this module
only holds the device buffers and orders the calls on one stream."""
from __future__ import annotations

from dataclasses import dataclass, field

from . import (LiParams, Params, adam_step, backward, forward, li_readout, merge, merge_grad,
               lif_layer_forward_workspace_size, lif_layer_backward_workspace_size, lif_li_readout_workspace_size,
               LIF_MERGE_MAX, _torch)


@dataclass
class AdamParams:
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8


@dataclass
class StepResult:
    loss: "object"                       # float32 [1] device
    logits: "object"                     # float32 [B, K]
    grads: dict = field(default_factory=dict)
    fwd1: "object" = None
    fwd2: "object" = None
    queue2: tuple = ()
    queue3: tuple = ()


class TwoLayerNet:
    """Weights W1 [C, N1], W2 [N1, N2], Wo [N2, K] (W^T layouts, float32
    device tensors) with their Adam moments, and workspaces sized for a
    batch of B queues of at most E_max events."""

    def __init__(self, W1, W2, Wo, B: int, E_max: int, P1: Params = Params(), P2: Params = Params(),
                 q: LiParams = LiParams(), adam: AdamParams = AdamParams(), E2_max: int = LIF_MERGE_MAX,
                 E3_max: int = LIF_MERGE_MAX):
        torch = _torch()
        self.W = [W1, W2, Wo]
        self.m1 = [torch.zeros_like(w) for w in self.W]
        self.m2 = [torch.zeros_like(w) for w in self.W]
        self.P1, self.P2, self.q, self.adam = P1, P2, q, adam
        self.E2_max, self.E3_max = E2_max, E3_max
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

    def step(self, ev_t, ev_src, ev_n, labels, sequential: bool = False, update: bool = True,
             stream=None) -> StepResult:
        """Forward, loss, backward and (update=True) the Adam update; the
        forward passes run the parallel layer, or the sequential baseline
        with sequential=True (everything else is the same)."""
        W1, W2, Wo = self.W
        o1 = forward(ev_t, ev_src, ev_n, W1, self.P1, sequential=sequential, stream=stream, ws=self.ws_f1)
        t2, s2, n2, perm2, _ = merge(o1, self.E2_max, stream=stream)
        o2 = forward(t2, s2, n2, W2, self.P2, sequential=sequential, stream=stream, ws=self.ws_f2)
        t3, s3, n3, perm3, _ = merge(o2, self.E3_max, stream=stream)
        logits, loss, gWo, gT3 = li_readout(t3, s3, n3, Wo, self.q, labels=labels, stream=stream, ws=self.ws_ro)
        g2 = merge_grad(gT3, perm3, n3, W2.shape[1], self.P2.s_max, stream=stream)
        gW2, gT2 = backward(t2, s2, n2, W2, o2, g2, self.P2, stream=stream, ws=self.ws_b2)
        g1 = merge_grad(gT2, perm2, n2, W1.shape[1], self.P1.s_max, stream=stream)
        gW1, _ = backward(ev_t, ev_src, ev_n, W1, o1, g1, self.P1, stream=stream, want_time_grad=False,
                          ws=self.ws_b1)
        grads = {"W1": gW1, "W2": gW2, "Wo": gWo}
        if update:
            self.t += 1
            a = self.adam
            for w, g, m1, m2 in zip(self.W, (gW1, gW2, gWo), self.m1, self.m2):
                adam_step(w, g, m1, m2, self.t, a.lr, a.beta1, a.beta2, a.eps, stream=stream)
        return StepResult(loss, logits, grads, o1, o2, (t2, s2, n2, perm2), (t3, s3, n3, perm3))
