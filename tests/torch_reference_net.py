"""A float64 PyTorch (CPU) implementation of the workload networks, used only to pin the oracle.

It builds f(theta, x) from torch's own layer routines (linear, conv2d with
padding 1 -- grouped per channel for the depthwise layer, 1x1 for the pointwise one --,
avg_pool2d, relu,
erf, mean) so that torch autograd provides an independent
Jacobian against which the oracle's hand-written reverse-mode Jacobian is
checked.
"""
import torch
import torch.nn.functional as F


def torch_forward(spec, flat_params, X):
    """f(theta, X) with theta given as a list of float64 tensors (spec order)."""
    h = X
    i = 0
    for L in spec["layers"]:
        if L["kind"] == "dense":
            w = flat_params[i]
            i += 1
            b = None
            if L["bias"]:
                b = flat_params[i]
                i += 1
            h = F.linear(h, w, b)
        elif L["kind"] == "conv3x3":
            w = flat_params[i]
            i += 1
            b = None
            if L["bias"]:
                b = flat_params[i]
                i += 1
            # NHWC activations, OHWI weights -> torch's NCHW / OIHW
            y = F.conv2d(h.permute(0, 3, 1, 2), w.permute(0, 3, 1, 2), b, stride=1, padding=1)
            h = y.permute(0, 2, 3, 1)
        elif L["kind"] == "conv1x1":
            w = flat_params[i]
            i += 1
            b = None
            if L["bias"]:
                b = flat_params[i]
                i += 1
            # weights [Cout, Cin] -> torch's OIHW with a 1x1 kernel
            y = F.conv2d(h.permute(0, 3, 1, 2), w[:, :, None, None], b)
            h = y.permute(0, 2, 3, 1)
        elif L["kind"] == "dwconv3x3":
            w = flat_params[i]
            i += 1
            b = None
            if L["bias"]:
                b = flat_params[i]
                i += 1
            # weights [3, 3, C] -> torch's grouped [C, 1, 3, 3]
            C = w.shape[2]
            y = F.conv2d(h.permute(0, 3, 1, 2), w.permute(2, 0, 1).unsqueeze(1), b,
                         stride=1, padding=1, groups=C)
            h = y.permute(0, 2, 3, 1)
        elif L["kind"] == "scale":
            w = flat_params[i]
            i += 1
            h = h * w
            if L["bias"]:
                h = h + flat_params[i]
                i += 1
        elif L["kind"] == "avgpool2":
            h = F.avg_pool2d(h.permute(0, 3, 1, 2), kernel_size=2, stride=2).permute(0, 2, 3, 1)
            continue
        elif L["kind"] == "gap":
            h = h.mean(dim=(1, 2))
            continue
        act = L["act"]
        if act == "relu":
            h = torch.relu(h)
        elif act == "erf":
            h = torch.erf(h)
    return h


def torch_jacobian(spec, params, X):
    """[N, O, P] Jacobian of f w.r.t. all parameters (flattened in spec order), float64."""
    ps = [torch.tensor(p, dtype=torch.float64) for p in params]
    x = torch.tensor(X, dtype=torch.float64)
    shapes = [p.shape for p in ps]
    sizes = [p.numel() for p in ps]

    def f_of_flat(flat):
        chunks = torch.split(flat, sizes)
        return torch_forward(spec, [c.reshape(s) for c, s in zip(chunks, shapes)], x)

    flat = torch.cat([p.reshape(-1) for p in ps])
    J = torch.autograd.functional.jacobian(f_of_flat, flat)   # [N, O, P]
    return J.numpy()
