"""Double-precision torch autograd model of a network given as layer tuples.

Used only to pin the CPU oracle: it is an independent implementation of the same definitions
(torch's conv2d / max_pool2d / linear / batch_norm / cross_entropy and autograd), run on the
CPU in float64.
"""
import torch
import torch.nn.functional as F


def split_params(geo, w):
    """Views of the flat parameter vector as per-layer (W, b) tensors in logical layout."""
    out = []
    for g in geo:
        if g["kind"] in (2, 4):
            out.append(None)
            continue
        c, h, wd = g["in_shape"]
        oc = g["out_shape"][0]
        W = w[g["w_off"]:g["w_off"] + g["w_len"]]
        b = w[g["b_off"]:g["b_off"] + g["b_len"]]
        out.append((W, b))
    return out


def forward(layers, geo, wt, x):
    a = x
    acts = []
    for (kind, o, k, s, p, gr, relu), g, pr in zip(layers, geo, split_params(geo, wt)):
        if kind == 1:
            c = g["in_shape"][0]
            W = pr[0].view(o, c // gr, k, k)
            a = F.conv2d(a, W, pr[1], stride=s, padding=p, groups=gr)
        elif kind == 0:
            a = a.reshape(a.shape[0], -1)
            a = F.linear(a, pr[0].view(o, -1), pr[1])
        elif kind == 3:  # batch statistics of this forward's samples (one shard)
            a = F.batch_norm(a, None, None, pr[0], pr[1], training=True, eps=1e-3)
        elif kind == 4:
            a = a + acts[k]
        elif kind == 5:  # projection shortcut: 1x1 convolution of stride s of layer k's output
            cs = acts[k].shape[1]
            a = a + F.conv2d(acts[k], pr[0].view(o, cs, 1, 1), pr[1], stride=s)
        else:
            a = F.max_pool2d(a, k, s)
        if relu:
            a = torch.relu(a)
        acts.append(a)
    return a, acts


def shard_grads(layers, geo, w, x, y, R):
    """Per-shard gradients of the shard-mean cross-entropy, in float64. Returns ([R,P], losses)."""
    w = torch.as_tensor(w, dtype=torch.float64)
    x = torch.as_tensor(x, dtype=torch.float64)
    y = torch.as_tensor(y, dtype=torch.long)
    Nb = x.shape[0] // R
    gs, ls = [], []
    for r in range(R):
        wt = w.clone().requires_grad_(True)
        z, _ = forward(layers, geo, wt, x[r * Nb:(r + 1) * Nb])
        loss = F.cross_entropy(z, y[r * Nb:(r + 1) * Nb], reduction="mean")
        loss.backward()
        gs.append(wt.grad.detach().clone())
        ls.append(loss.item())
    return torch.stack(gs).to(torch.float64).numpy(), ls


def fp32_evaluation_bf16(layers, geo, w, x, y):
    """One shard in float32 arithmetic (torch CPU: fp32 sums in torch's own order) with the bf16
    mode's storage points -- an evaluation of the same step that is as legitimate as the GPU's.
    Returns (gradient [P] as float64, stored outputs per layer, pool decisions, ReLU decisions)
    in the oracle's layouts."""
    wt = torch.as_tensor(w, dtype=torch.float32).clone().requires_grad_(True)
    dec = []
    z, acts = forward_bf16(layers, geo, wt, torch.as_tensor(x, dtype=torch.float32),
                           decisions=dec)
    F.cross_entropy(z, torch.as_tensor(y, dtype=torch.long), reduction="mean").backward()
    pools = [d for k, d in dec if k == "pool"]
    relus = [d for k, d in dec if k == "relu"]
    import numpy as np
    return (wt.grad.detach().to(torch.float64).numpy(),
            [a.detach().to(torch.float64).numpy().ravel() for a in acts],
            np.concatenate(pools).astype(np.int32) if pools else np.zeros(0, np.int32),
            np.concatenate(relus).astype(np.int8) if relus else np.zeros(0, np.int8))


# ---- bfloat16 storage emulation (the rounding points of the bf16 mode) -------------------------

def bf16(t):
    """Round to bfloat16 as an fp32 accumulator is stored: first to float, then to nearest even
    bfloat16 (torch's float -> bfloat16 conversion), returned in t's dtype."""
    return t.to(torch.float32).to(torch.bfloat16).to(t.dtype)


def f32(t):
    return t.to(torch.float32).to(t.dtype)


class _RoundValue(torch.autograd.Function):
    """Round the forward value; the gradient passes unchanged (the stored value is the one the
    layer above reads, and its gradient is that of the stored value)."""

    @staticmethod
    def forward(ctx, t, to_bf16):
        return bf16(t) if to_bf16 else f32(t)

    @staticmethod
    def backward(ctx, g):
        return g, None


class _RoundGrad(torch.autograd.Function):
    """Identity forward; the incoming gradient is rounded to bfloat16 (a stored data gradient)."""

    @staticmethod
    def forward(ctx, t):
        return t.clone()

    @staticmethod
    def backward(ctx, g):
        return bf16(g)


def forward_bf16(layers, geo, wt, x, round_grads=True, round_loss_grad=True, decisions=None):
    """The network's forward pass with the bf16 mode's storage: x and every W rounded to bf16
    (biases and batch-normalisation scales stay float); every hidden layer's output rounded to
    bf16 after bias and ReLU, and the gradient reaching it rounded to bf16 (a stored data
    gradient; at a residual source the next layer's data gradient is stored, the residual
    addition's gradient added to it and the sum stored again); the logits rounded
    to float and the gradient of the loss with respect to them rounded to bf16.  The two flags
    drop the gradient-side roundings (used to show that a test can see them).  The arithmetic
    is that of x's dtype: float64, or float32 for an evaluation with fp32 sums.  With a list as
    `decisions`, the max-pool window positions (u*k + v, int32) and ReLU decisions (int8) are
    appended to it per layer as ("pool" | "relu", array) in the oracle's layout."""
    a = _RoundValue.apply(x, True)
    acts = []
    n = len(layers)
    for li, ((kind, o, k, s, p, gr, relu), g, pr) in enumerate(zip(layers, geo, split_params(geo, wt))):
        if kind == 1:
            c = g["in_shape"][0]
            W = _RoundValue.apply(pr[0].view(o, c // gr, k, k), True)
            a = F.conv2d(a, W, pr[1], stride=s, padding=p, groups=gr)
        elif kind == 0:
            a = a.reshape(a.shape[0], -1)
            a = F.linear(a, _RoundValue.apply(pr[0].view(o, -1), True), pr[1])
        elif kind == 3:
            a = F.batch_norm(a, None, None, pr[0], pr[1], training=True, eps=1e-3)
        elif kind == 4:
            a = a + acts[k]
        elif kind == 5:  # the projection's output is stored, then added; its data gradient
            cs = acts[k].shape[1]  # is stored before it joins the source's other gradient
            src = _RoundGrad.apply(acts[k]) if round_grads else acts[k]
            pj = F.conv2d(src, _RoundValue.apply(pr[0].view(o, cs, 1, 1), True), pr[1], stride=s)
            a = a + _RoundValue.apply(pj, True)
        else:
            W_ = a.shape[3]
            a, idx = F.max_pool2d(a, k, s, return_indices=True)
            if decisions is not None:
                oh, ow = a.shape[2], a.shape[3]
                u = idx // W_ - (torch.arange(oh) * s).view(1, 1, oh, 1)
                v = idx % W_ - (torch.arange(ow) * s).view(1, 1, 1, ow)
                decisions.append(("pool", (u * k + v).to(torch.int32).numpy().ravel()))
        if relu:
            if decisions is not None:
                decisions.append(("relu", (a > 0).to(torch.int8).numpy().ravel()))
            a = torch.relu(a)
        last = li == n - 1
        if kind != 2:  # a pooled value is one of its (already stored) inputs
            a = _RoundValue.apply(a, not last)
        if (round_loss_grad if last else round_grads):
            a = _RoundGrad.apply(a)
        acts.append(a)  # what a residual addition reads
        if round_grads and not last:
            # the next layer's data gradient is stored before a residual addition's gradient is
            # added to it (a no-op where the next layer is the only reader)
            a = _RoundGrad.apply(a)
    return a, acts


def shard_grads_bf16(layers, geo, w, x, y, R, dtype=torch.float64, **kw):
    """Per-shard gradients of the shard-mean cross-entropy with the bf16 mode's storage, in
    float64 (or `dtype`) arithmetic.  Returns ([R,P], losses)."""
    w = torch.as_tensor(w, dtype=dtype)
    x = torch.as_tensor(x, dtype=dtype)
    y = torch.as_tensor(y, dtype=torch.long)
    Nb = x.shape[0] // R
    gs, ls = [], []
    for r in range(R):
        wt = w.clone().requires_grad_(True)
        z, _ = forward_bf16(layers, geo, wt, x[r * Nb:(r + 1) * Nb], **kw)
        loss = F.cross_entropy(z, y[r * Nb:(r + 1) * Nb], reduction="mean")
        loss.backward()
        gs.append(wt.grad.detach().clone())
        ls.append(loss.item())
    return torch.stack(gs).to(torch.float64).numpy(), ls


def fp32_evaluation_bf16(layers, geo, w, x, y):
    """One shard in float32 arithmetic (torch CPU: fp32 sums in torch's own order) with the bf16
    mode's storage points -- an evaluation of the same step that is as legitimate as the GPU's.
    Returns (gradient [P] as float64, stored outputs per layer, pool decisions, ReLU decisions)
    in the oracle's layouts."""
    wt = torch.as_tensor(w, dtype=torch.float32).clone().requires_grad_(True)
    dec = []
    z, acts = forward_bf16(layers, geo, wt, torch.as_tensor(x, dtype=torch.float32),
                           decisions=dec)
    F.cross_entropy(z, torch.as_tensor(y, dtype=torch.long), reduction="mean").backward()
    pools = [d for k, d in dec if k == "pool"]
    relus = [d for k, d in dec if k == "relu"]
    import numpy as np
    return (wt.grad.detach().to(torch.float64).numpy(),
            [a.detach().to(torch.float64).numpy().ravel() for a in acts],
            np.concatenate(pools).astype(np.int32) if pools else np.zeros(0, np.int32),
            np.concatenate(relus).astype(np.int8) if relus else np.zeros(0, np.int8))
