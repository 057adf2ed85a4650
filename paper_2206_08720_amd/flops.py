"""Analytic operation counts of one NTK evaluation (host logic, no GPU needed).

Counts use 2*M*N*K floating-point operations per M x N x K product, i.e. twice
the paper's multiply-add count (appendix "Experimental Details" counts a
(M,K) x (K,P) product as M*K*P).  The stages are those the library runs:

FCN (dense layers 0..L, d_0 = input size, d_{L+1} = O; M = N1 + N2 stacked rows,
or N when X2 is X1):
  forward      sum_{l<L} 2 M d_l d_{l+1}                 (part of N O [FP], Section 3.4)
  backward     sum_{1<=l<L} 2 (M O) d_{l+1} d_l          (the N O L W^2 term of Table "FCN")
  gram         sum_{l<=L} 2 N1 N2 d_l                    (the x1.x2 scalars)
  contraction  sum_{l<L} 2 (N1 O)(N2 O) d_{l+1}          (the N^2 O^2 L W term)
CNN (conv3x3 layers l with Cin_l -> Cout_l on D pixels, GAP, dense readout; the further
layer kinds are listed in `cnn_flops`):
  forward      sum_l 2 M D 9 Cin_l Cout_l
  backward     sum_{l>=1} 2 (M O D) 9 Cout_l Cin_l
  wgrad        sum_l 2 M (O Cout_l) (9 Cin_l) D           (outside-in weight-space Jacobian)
  contraction  2 (N1 O)(N2 O) sum_l Cout_l 9 Cin_l + readout gram 2 N1 N2 C

Variants (output = "trace" | "logit", batch = "diagonal"): the backward pass and the
weight-space cotangents run for Oe = 1 output with "logit" (O otherwise); the contraction
covers `pairs` input pairs (N1 N2, or N on the batch diagonal) and Oc output pairs per input
pair (O^2 full, O for the trace, 1 for one logit).

Symmetric schedule (X2 is X1, N1 = N2 = N): the stacked rows are the N samples once, and the
contraction runs for the N (N + 1) / 2 pairs n1 <= n2 (the mirror image fills the rest), so
its count uses that many pairs.

Jacobian contraction (method = "jacobian", the baseline of Section 3.2): the same forward
and backward passes (and, for the CNN, the weight-space Jacobians of every conv layer), then
the explicit contraction, 2 pairs Oc P for P parameters in total.
"""
from __future__ import annotations


def _variant(O, n1, n2, output, batch, symmetric=False):
    """(cotangent rows per sample, output pairs per input pair, input pairs contracted)."""
    Oe = 1 if output == "logit" else O
    Oc = {"full": O * O, "trace": O, "logit": 1}[output]
    if batch == "diagonal":
        pairs = n1
    elif symmetric:
        pairs = n1 * (n1 + 1) // 2
    else:
        pairs = n1 * n2
    return Oe, Oc, pairs


def fcn_flops(spec, n1, n2, symmetric=False, output="full", batch="full"):
    layers = spec["layers"]
    L = len(layers) - 1
    d = [layers[0]["in"]] + [Lr["out"] for Lr in layers]
    O = d[-1]
    Oe, Oc, pairs = _variant(O, n1, n2, output, batch, symmetric)
    gpairs = n1 if batch == "diagonal" else n1 * n2     # the Gram kernels form the full block
    M = n1 if symmetric else n1 + n2
    st = {
        "forward": sum(2.0 * M * d[l] * d[l + 1] for l in range(L)),
        "backward": sum(2.0 * M * Oe * d[l + 1] * d[l] for l in range(1, L)),
        "gram": sum(2.0 * gpairs * d[l] for l in range(L + 1)),
        "contraction": sum(2.0 * pairs * Oc * d[l + 1] for l in range(L)),
    }
    st["total"] = sum(st.values())
    return st


def _spatial_layers(spec):
    """(kind, Cin, Cout, D = pixels of the layer's input, bias) of each layer before the global
    pool, and the channels that reach the pool."""
    H, W, c = spec["input_shape"]
    out = []
    for Lr in spec["layers"]:
        k = Lr["kind"]
        if k in ("gap", "dense"):
            continue
        if k == "avgpool2":
            out.append((k, c, c, H * W, False))
            H, W = H // 2, W // 2
        else:
            out.append((k, c, Lr["out"], H * W, bool(Lr.get("bias"))))
            c = Lr["out"]
    return out, c


def _weight_cols(kind, cin, cout):
    return {"conv3x3": 9 * cin * cout, "conv1x1": cin * cout, "dwconv3x3": 9 * cout,
            "scale": cout}.get(kind, 0)


# Time per executed matrix-core multiply-add of the inside-out kernel relative to the outside-in
# products, as in the library's cost model.
INSIDE_OUT_TIME_WEIGHT = 1.0


def inside_out_cost(pairs, D, cin, cout, Oe, trace=False):
    """The library's cost of the inside-out order of one convolution: the multiply-adds its
    matrix-core kernel executes, with the pixels padded to Dp = 16 ceil(D / 16), the outputs to
    blocks of 16 and the input channels to steps of 16 (per block of 16 x 16 outputs: the pixel
    Gram Dp^2 Cin, the product with the patch-pair Gram 16 Dp^2 C, the output product 256 Dp C),
    times INSIDE_OUT_TIME_WEIGHT."""
    Dp, ci, nob = 16 * -(-D // 16), 16 * -(-cin // 16), -(-Oe // 16)
    gram_blocks, out_blocks = (1, nob) if trace else (nob * nob, nob * nob)
    return INSIDE_OUT_TIME_WEIGHT * pairs * (gram_blocks * Dp * Dp * ci
                                             + out_blocks * (16 * Dp * Dp * cout + 256 * Dp * cout))


def _inside_out(kind, D, cin, cout, M, Oe, Oc, gpairs, order, trace=False):
    """Whether a 3x3 or pointwise convolution is contracted inside-out: forced by `order`, or
    (order "auto") the library's per-layer choice by the cost model of the appendix "CNN NTK
    Complexity": outside-in gpairs Oc F Cin Cout plus forming J, M Oe D F Cin Cout, against the
    inside-out kernel's cost (inside_out_cost); inside-out only for images of at most 64 pixels
    (the kernel's limit)."""
    if kind not in ("conv3x3", "conv1x1") or order == "outside_in":
        return False
    if order == "inside_out":
        return True
    F = 9 if kind == "conv3x3" else 1
    oi = gpairs * Oc * F * cin * cout + M * Oe * D * F * cin * cout
    return D <= 64 and inside_out_cost(gpairs, D, cin, cout, Oe, trace) < oi


def _conv_orders(sp, O, n1, n2, output, batch, M, Oe, Oc, gpairs, order):
    """Per spatial layer whether it is contracted inside-out, and whether the last convolution is
    folded, as the library decides: _inside_out per layer; the fold (the last convolution's
    cotangent is the readout's through the global pool, so its weight-space columns factor into
    Wr[o, c] times O-free per-channel rows and its summand into per-channel Grams) for a last 3x3
    or pointwise convolution, the full O x O output or its trace (O >= 2), on the full batch or its
    diagonal, with other
    weight-space columns in the contraction (a bias, a depthwise or scale layer, an outside-in
    convolution); with order "auto" the last convolution then goes outside-in when the fold's
    M D F Cin Cout + N1 N2 (F Cin Cout + O^2 Cout) is below its inside-out cost."""
    trace = output == "trace"
    io = [_inside_out(k, D, cin, cout, M, Oe, Oc, gpairs, order, trace) for (k, cin, cout, D, bias) in sp]
    if not sp or O < 2 or output not in ("full", "trace") or sp[-1][0] not in ("conv3x3", "conv1x1"):
        return io, False
    others = bool(sp[-1][4]) or any(b or k in ("dwconv3x3", "scale") or (k in ("conv3x3", "conv1x1") and not io[i])
                                    for i, (k, ci, co, D, b) in enumerate(sp[:-1]))
    if not others:
        return io, False
    k, cin, cout, D, bias = sp[-1]
    if io[-1] and order == "auto":
        F = 9 if k == "conv3x3" else 1
        folded = M * D * F * cin * cout + gpairs * (F * cin * cout + O * O * cout)
        if folded < inside_out_cost(gpairs, D, cin, cout, Oe, trace):
            io[-1] = False
    return io, not io[-1]


def cnn_flops(spec, n1, n2, symmetric=False, order="outside_in", output="full", batch="full", fold=True):
    """CNN counts per stage.  3x3 convolutions as in the module docstring; the further layer
    kinds (memory-bound, counted for completeness, in the struct_* stages): depthwise 3x3
    forward, backward and weight-space cotangent 2 M (Oe) D 9 C each; scale forward M D C (2 M D C
    with a bias), backward M Oe D C, cotangent 2 M Oe D C; a 2x2 pool M D C forward and
    M Oe D C backward (D: its input pixels); a bias M D C forward and its cotangent (a pixel sum)
    M Oe D C.  The contraction covers every weight-space column (9 Cin Cout, 9 C, C, and C per
    bias).  `order` is "outside_in", "inside_out" or "auto" (the library's
    per-layer choice, _inside_out) for the 3x3 and pointwise convolutions; a layer contracted
    inside-out forms no J columns and counts its own operations in the stage "pairsum": the
    pixel Gram D^2 Cin, the F D^2 tap sums of the patch-pair Gram (one FLOP each), and the
    products Oe D^2 Cout and Oc D Cout (the form of the appendix "CNN NTK Complexity" with the
    patch-pair Gram built from the pixel Gram instead of D^2 F Cin patch products).  With `fold`
    (the library's schedule, _conv_orders) the last convolution forms O-free rows A [M, C, F Cin]
    ("wgrad"), no J columns, and per-channel Grams plus their O x O sums, or for the trace their
    sum weighted by sum_o Wr[o, c]^2 ("gram"); fold=False counts
    every outside-in layer alike, as the paper's table does (and the orders of the plain cost
    model)."""
    layers = spec["layers"]
    sp, C = _spatial_layers(spec)
    O = layers[-1]["out"]
    Oe, Oc, pairs = _variant(O, n1, n2, output, batch, symmetric)
    gpairs = n1 if batch == "diagonal" else n1 * n2
    M = n1 if symmetric else n1 + n2
    # the 3x3 convolutions' stages ("forward", "backward", "wgrad"), and those of the other kinds
    # and of the biases (memory-bound kernels of their own: "struct_forward", "struct_backward",
    # "struct_wgrad"); a conv bias is added in the conv forward kernel's epilogue
    fwd = bwd = wg = sfwd = sbwd = swg = cols = io = fold_gram = 0.0
    inside, can_fold = _conv_orders(sp, O, n1, n2, output, batch, M, Oe, Oc, gpairs, order)
    if not fold and can_fold and order == "auto":   # the unfolded count keeps the plain cost model
        inside = [_inside_out(k, D, cin, cout, M, Oe, Oc, gpairs, order, output == "trace")
                  for (k, cin, cout, D, bias) in sp]
    fold = fold and can_fold
    for i, (k, cin, cout, D, bias) in enumerate(sp):
        if k in ("conv1x1", "conv3x3"):
            F = 9 if k == "conv3x3" else 1
            fwd += 2.0 * M * D * F * cin * cout + (1.0 * M * D * cout if bias else 0.0)
            if i >= 1:
                bwd += 2.0 * M * Oe * D * F * cout * cin
            if fold and i == len(sp) - 1:
                # the folded last convolution: A [M, C, F Cin] (one row block per sample instead
                # of O), the per-channel Grams of every input pair, and the O x O sums over C
                wg += 2.0 * M * cout * (F * cin) * D
                if output == "trace":   # weights sum_o Wr[o, c]^2, then one weighted sum per pair
                    fold_gram = 2.0 * gpairs * cout * F * cin + 2.0 * O * cout + 2.0 * gpairs * cout
                else:
                    fold_gram = 2.0 * gpairs * cout * F * cin + 3.0 * gpairs * O * O * cout
            elif not inside[i]:
                wg += 2.0 * M * (Oe * cout) * (F * cin) * D
                cols += F * cin * cout
            else:  # inside-out (every input pair, also on the symmetric schedule): the pixel Gram,
                # the F-tap sums forming the patch-pair Gram, the one-sided cotangent product and
                # the O x O product
                io += gpairs * (2.0 * D * D * cin + F * D * D + 2.0 * Oe * D * D * cout + 2.0 * Oc * D * cout)
        elif k == "dwconv3x3":
            sfwd += 2.0 * M * D * 9 * cout + (1.0 * M * D * cout if bias else 0.0)
            if i >= 1:
                sbwd += 2.0 * M * Oe * D * 9 * cout
            swg += 2.0 * M * Oe * D * 9 * cout
            cols += 9 * cout
        elif k == "scale":
            sfwd += 2.0 * M * D * cout if bias else 1.0 * M * D * cout
            if i >= 1:
                sbwd += 1.0 * M * Oe * D * cout
            swg += 2.0 * M * Oe * D * cout
            cols += cout
        else:  # avgpool2
            sfwd += 1.0 * M * D * cout
            if i >= 1:
                sbwd += 1.0 * M * Oe * D * cout
        if bias:
            swg += 1.0 * M * Oe * D * cout
            cols += cout
    st = {"forward": fwd, "backward": bwd, "gram": 2.0 * gpairs * C + fold_gram}
    if wg:
        st["wgrad"] = wg
    for key, v in (("struct_forward", sfwd), ("struct_backward", sbwd), ("struct_wgrad", swg)):
        if v:
            st[key] = v
    st["contraction"] = 2.0 * pairs * Oc * cols
    if io:
        st["pairsum"] = io
    st["total"] = sum(st.values())
    return st


def param_total(spec):
    P = 0
    for Lr in spec["layers"]:
        k = Lr["kind"]
        if k == "dense":
            P += Lr["out"] * Lr["in"]
        elif k in ("conv3x3", "conv1x1", "dwconv3x3", "scale"):
            P += _weight_cols(k, Lr["in"], Lr["out"])
        else:
            continue
        P += Lr["out"] if Lr.get("bias") else 0
    return P


def ntk_flops(spec, n1, n2, symmetric=False, method="structured", **kw):
    cnn = any(Lr["kind"] != "dense" for Lr in spec["layers"])
    if method == "jacobian":
        kw["order"] = "outside_in"
    if cnn:
        st = cnn_flops(spec, n1, n2, symmetric, **kw)
    else:
        kw.pop("order", None)
        st = fcn_flops(spec, n1, n2, symmetric, **kw)
    if method == "jacobian":
        O = spec["layers"][-1]["out"]
        _, Oc, pairs = _variant(O, n1, n2, kw.get("output", "full"), kw.get("batch", "full"), symmetric)
        st.pop("gram", None)
        st.pop("total")
        st["contraction"] = 2.0 * pairs * Oc * param_total(spec)
        st["total"] = sum(st.values())
    return st


def ntk_entries(spec, n1, n2, output="full", batch="full"):
    O = spec["layers"][-1]["out"]
    pairs = n1 if batch == "diagonal" else n1 * n2
    return pairs * (O * O if output == "full" else 1)


def vp_flops(spec, n1, n2, symmetric=False):
    """Operation count of one NTK-vector product Theta(X1, X2) v (ntk_vector_product), by the
    kernel groups that run it: the forward pass of both batches, the VJP of batch 2 (one
    cotangent row per sample), the weight-space cotangent (sum over batch 2) and the JVP of
    batch 1.  FCN: `gram_products` is the weight-space cotangent plus the JVP (both run on the
    Gram kernel).  CNN: `forward_and_jvp` is the forward pass plus the JVP convolutions."""
    M = n1 if symmetric else n1 + n2
    layers = spec["layers"]
    if any(Lr["kind"] != "dense" for Lr in layers):
        # the 3x3 and 1x1 convolutions' matrix-core work (D: each layer's own pixels); the memory-bound
        # depthwise, scale, bias and pool steps are not counted
        sp, C = _spatial_layers(spec)
        O = layers[-1]["out"]
        conv = [(i, D, _weight_cols(k, cin, cout)) for i, (k, cin, cout, D, _) in enumerate(sp)
                if k in ("conv3x3", "conv1x1")]
        first = min([i for i, (k, *_r) in enumerate(sp) if k != "avgpool2"] or [0])
        st = {
            "forward_and_jvp": sum(2.0 * M * D * k for _, D, k in conv) + sum(2.0 * n1 * D * k for _, D, k in conv)
            + sum(2.0 * n1 * D * k for i, D, k in conv if i > first),
            "vjp_backward": sum(2.0 * n2 * D * k for i, D, k in conv if i >= 1),
            "weight_cotangent": sum(2.0 * n2 * D * k for _, D, k in conv),
            "gram": 2.0 * n2 * O * C * 2 + 2.0 * n1 * O * C * 2,
        }
    else:
        L = len(layers) - 1
        d = [layers[0]["in"]] + [Lr["out"] for Lr in layers]
        st = {
            "forward": sum(2.0 * M * d[l] * d[l + 1] for l in range(L)),
            "vjp_backward": sum(2.0 * n2 * d[l + 1] * d[l] for l in range(1, L + 1)),
            "gram_products": sum(2.0 * n2 * d[l + 1] * d[l] for l in range(L + 1))
            + sum(2.0 * n1 * d[l] * d[l + 1] for l in range(L + 1))
            + sum(2.0 * n1 * d[l] * d[l + 1] for l in range(1, L + 1)),
        }
    st["total"] = sum(st.values())
    return st
