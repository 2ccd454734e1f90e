"""Reverse-mode reference for pinning the oracle (CPU, float64 autograd).

The same network function the oracle differentiates, written as a plain
forward pass in PyTorch and differentiated by backpropagation through time
(the adjoint recursion, Eq. 6-7 of the paper) instead of the forward RTRL
recursion of Eq. (5).  The three gradient stops of the method are
``detach()`` calls: the recurrent spikes (Sec. III-B, the stop_gradient
footnote), the reset term (kept when the shape has ``reset_grad=1``), and in
two-layer stacks the spikes passed from layer 1 to layer 2.  With these stops the forward recursion of e-prop and
backpropagation give the same gradient, which is what the paper checks in
Table II for a feed-forward layer.

The spike nonlinearity is the Heaviside step with the triangular surrogate
in the backward pass (the footnote on the surrogate in Sec. III-C).
"""
from __future__ import annotations

import numpy as np
import torch

F64 = torch.float64


class _Spike(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, gamma, thr):
        ctx.save_for_backward(x)
        ctx.gamma, ctx.thr = gamma, thr
        return (x > 0).to(x.dtype)

    @staticmethod
    def backward(ctx, g):
        (x,) = ctx.saved_tensors
        psi = (ctx.gamma / ctx.thr) * torch.clamp(1.0 - x.abs() / ctx.thr, min=0.0)
        return g * psi, None, None


class _Readout(torch.autograd.Function):
    """y = z W_out^T whose backward sends dy to z through a fixed feedback
    matrix F [K, N] instead of W_out (F = W_out gives the ordinary product);
    the gradient of W_out itself is the ordinary one."""

    @staticmethod
    def forward(ctx, z, wo, fb):
        ctx.save_for_backward(z, fb)
        return z @ wo.T

    @staticmethod
    def backward(ctx, g):
        z, fb = ctx.saved_tensors
        return g @ fb, g.T @ z, None


def bptt_grads(shape, W, Wout, x, labels, T=None, reset=None, stop=True, feedback=None,
               schedule=None):
    """Returns (dW list, dWout list, loss) as float64 numpy arrays.

    ``stop=False`` keeps every path (true surrogate gradient); it is only used
    to show the gradient stops matter.  ``feedback``: per layer a matrix of
    W_out's shape that carries the readout's gradient back to the spikes in
    place of W_out (random-feedback learning signal).  ``schedule``: a list
    of (t_start, W list, Wout list) in increasing t_start; from step t_start
    on, the network uses those values in place of W, Wout.  The gradient is
    still taken with respect to W and W_out: each use adds its derivative,
    which is what a forward recursion accumulates while the weights change.
    With a schedule the learning signal is e-prop's online one: the error at
    step t reaches the spikes of steps s <= t through the readout weights in
    use at step t (kappa^(t-s) W_out(t)^T delta_t), not those in use at s;
    the readout value and its gradient stay exact.  With both, the feedback
    matrices take the place of W_out(t) in that signal and do not change.
    """
    T = x.shape[0] if T is None else T
    L, B, N = shape.n_layers, shape.batch, shape.n_rec
    keep_reset = bool(getattr(shape, "reset_grad", 0))   # the reset path kept in the gradient
    reset = shape.thr if reset is None else reset
    sg = (lambda v: v.detach()) if stop else (lambda v: v)
    Ws = [torch.tensor(np.asarray(w, dtype=np.float64), requires_grad=True) for w in W]
    Wos = [torch.tensor(np.asarray(w, dtype=np.float64), requires_grad=True) for w in Wout]
    # a None entry: that layer's learning signal through its own readout weights
    Fbs = None if feedback is None else [None if f is None else torch.tensor(np.asarray(f, dtype=np.float64))
                                         for f in feedback]
    beta = torch.zeros(N, dtype=F64)
    beta[: shape.n_adaptive] = shape.beta
    lab = torch.tensor(np.asarray(labels, dtype=np.int64))
    xs = torch.tensor(np.asarray(x[:T], dtype=np.float64))
    v = [torch.zeros(B, N, dtype=F64) for _ in range(L)]
    a = [torch.zeros(B, N, dtype=F64) for _ in range(L)]
    zp = [torch.zeros(B, N, dtype=F64) for _ in range(L)]
    y = [torch.zeros(B, shape.n_out, dtype=F64) for _ in range(L)]
    zh = [torch.zeros(B, N, dtype=F64) for _ in range(L)]   # kappa-filtered spikes (schedule)
    loss = torch.zeros((), dtype=F64)
    sched = [(t0, [torch.tensor(np.asarray(w, dtype=np.float64)) for w in Wv],
              [torch.tensor(np.asarray(w, dtype=np.float64)) for w in Wov])
             for t0, Wv, Wov in (schedule or [])]
    for t in range(T):
        z_now = []
        cur = [e for e in sched if e[0] <= t]
        if cur:
            # the values in use at this step; the derivative still flows to W, W_out
            _, Wv, Wov = cur[-1]
            Wuse = [w + (wv - w).detach() for w, wv in zip(Ws, Wv)]
            Wouse = [w + (wv - w).detach() for w, wv in zip(Wos, Wov)]
        else:
            Wuse, Wouse = Ws, Wos
        for l in range(L):
            inp = xs[t] if l == 0 else sg(z_now[l - 1])
            p = torch.cat([inp, sg(zp[l])], dim=1) if shape.recurrent else inp
            I = p @ Wuse[l].T
            if getattr(shape, "neuron_model", 0) == 1:
                # two-compartment neuron: v is the soma, a the dendrite; the
                # own spike reaches the dendrite (kept) and resets the soma
                al = shape.alpha_d * a[l]
                al = al + I
                al = al + shape.bap * zp[l]
                vl = shape.alpha * v[l]
                vl = vl + shape.coupling * a[l]
                vl = vl - reset * (zp[l] if keep_reset else sg(zp[l]))
                z = _Spike.apply(vl - shape.thr, shape.gamma, shape.thr)
            else:
                vl = shape.alpha * v[l]
                vl = vl + I
                vl = vl - reset * (zp[l] if keep_reset else sg(zp[l]))
                al = shape.rho * a[l]
                al = al + zp[l]                 # spike -> adaptation path is kept
                A = beta * al
                A = shape.thr + A
                z = _Spike.apply(vl - A, shape.gamma, shape.thr)
            if schedule is None:
                yz = z @ Wouse[l].T if Fbs is None or Fbs[l] is None else _Readout.apply(z, Wouse[l], Fbs[l])
                y[l] = shape.kappa * y[l] + yz
                logits = y[l]
            else:
                # value: the exact leaky readout (gradient to W_out only); the
                # spikes' gradient: filtered spikes through today's W_out
                y[l] = shape.kappa * y[l] + z.detach() @ Wouse[l].T
                zh[l] = shape.kappa * zh[l] + z
                back = Wouse[l].detach() if Fbs is None or Fbs[l] is None else Fbs[l]   # fixed feedback
                logits = y[l] + (zh[l] - zh[l].detach()) @ back.T
            loss = loss + torch.nn.functional.cross_entropy(logits, lab, reduction="sum")
            v[l], a[l] = vl, al
            z_now.append(z)
        zp = z_now
    loss.backward()
    dW = [w.grad.numpy().copy() for w in Ws]
    if shape.recurrent:
        for l in range(L):
            n_in_l = shape.n_in if l == 0 else N
            idx = np.arange(N)
            dW[l][idx, n_in_l + idx] = 0.0   # no self-connections
    return dW, [w.grad.numpy().copy() for w in Wos], float(loss.detach())


def rel_l2(a, b) -> float:
    a = np.asarray(a, dtype=np.float64).ravel()
    b = np.asarray(b, dtype=np.float64).ravel()
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (den if den > 0 else 1.0))
