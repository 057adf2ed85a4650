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
CNN (conv3x3 layers l with Cin_l -> Cout_l on D pixels, GAP, dense readout):
  forward      sum_l 2 M D 9 Cin_l Cout_l
  backward     sum_{l>=1} 2 (M O D) 9 Cout_l Cin_l
  wgrad        sum_l 2 M (O Cout_l) (9 Cin_l) D           (outside-in weight-space Jacobian)
  contraction  2 (N1 O)(N2 O) sum_l Cout_l 9 Cin_l + readout gram 2 N1 N2 C
"""
from __future__ import annotations


def fcn_flops(spec, n1, n2, symmetric=False):
    layers = spec["layers"]
    L = len(layers) - 1
    d = [layers[0]["in"]] + [Lr["out"] for Lr in layers]
    O = d[-1]
    M = n1 if symmetric else n1 + n2
    st = {
        "forward": sum(2.0 * M * d[l] * d[l + 1] for l in range(L)),
        "backward": sum(2.0 * M * O * d[l + 1] * d[l] for l in range(1, L)),
        "gram": sum(2.0 * n1 * n2 * d[l] for l in range(L + 1)),
        "contraction": sum(2.0 * (n1 * O) * (n2 * O) * d[l + 1] for l in range(L)),
    }
    st["total"] = sum(st.values())
    return st


def cnn_flops(spec, n1, n2, symmetric=False, order="outside_in"):
    layers = spec["layers"]
    H, W, _ = spec["input_shape"]
    D = H * W
    convs = [Lr for Lr in layers if Lr["kind"] == "conv3x3"]
    O = layers[-1]["out"]
    C = convs[-1]["out"]
    M = n1 if symmetric else n1 + n2
    st = {
        "forward": sum(2.0 * M * D * 9 * c["in"] * c["out"] for c in convs),
        "backward": sum(2.0 * M * O * D * 9 * c["out"] * c["in"] for c in convs[1:]),
        "gram": 2.0 * n1 * n2 * C,
    }
    if order == "outside_in":
        st["wgrad"] = sum(2.0 * M * (O * c["out"]) * (9 * c["in"]) * D for c in convs)
        st["contraction"] = 2.0 * (n1 * O) * (n2 * O) * sum(c["out"] * 9 * c["in"] for c in convs)
    else:  # inside-out: patch Gram, one-sided cotangent contraction, then the O x O product
        st["contraction"] = sum(2.0 * n1 * n2 * (D * D * 9 * c["in"] + O * D * D * c["out"]
                                                 + O * O * D * c["out"]) for c in convs)
    st["total"] = sum(st.values())
    return st


def ntk_flops(spec, n1, n2, symmetric=False, **kw):
    if any(Lr["kind"] == "conv3x3" for Lr in spec["layers"]):
        return cnn_flops(spec, n1, n2, symmetric, **kw)
    return fcn_flops(spec, n1, n2, symmetric)


def ntk_entries(spec, n1, n2):
    O = spec["layers"][-1]["out"]
    return n1 * n2 * O * O
