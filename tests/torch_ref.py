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
    return torch.stack(gs).numpy(), ls
