"""Writes hand_derived.json: tiny cases whose loss and gradients were derived by
hand from the definition of softmax cross-entropy (no code from oracle/ or the
HIP path is used; the closed forms below are evaluated with math only)."""
import json
import math
import os

e = math.e
cases = [
    {
        "name": "three_classes_one_ignored_mean",
        "derivation": "z0 = W x0 = [1,0,0]; lse0 = ln(e+2); loss = ln(e+2) - 1 (one valid token); "
                      "dZ0 = softmax - onehot = [-2,1,1]/(e+2); dH0 = dZ0 W = [-2,1]/(e+2); dH1 = 0; "
                      "dW_v = dZ0_v x0 = [dZ0_v, 0]",
        "hidden": [[1.0, 0.0], [0.0, 2.0]],
        "weight": [[1.0, 0.0], [0.0, 1.0], [0.0, 0.0]],
        "labels": [0, -100], "ignore_index": -100, "reduction": "mean",
        "loss": math.log(e + 2) - 1,
        "dH": [[-2 / (e + 2), 1 / (e + 2)], [0.0, 0.0]],
        "dW": [[-2 / (e + 2), 0.0], [1 / (e + 2), 0.0], [1 / (e + 2), 0.0]],
    },
    {
        "name": "two_classes_sum",
        "derivation": "z0 = [0,1], y0 = 1: l0 = ln(1+e^-1); z1 = [0,2], y1 = 0: l1 = ln(1+e^2); "
                      "dZ0 = [1,-1]/(1+e); dZ1 = [-e^2, e^2]/(1+e^2); dH_i = dZ_i1 (W = [[0],[1]]); "
                      "dW_0 = dZ00*1 + dZ10*2, dW_1 = dZ01*1 + dZ11*2",
        "hidden": [[1.0], [2.0]],
        "weight": [[0.0], [1.0]],
        "labels": [1, 0], "ignore_index": -100, "reduction": "sum",
        "loss": math.log1p(math.exp(-1)) + math.log1p(e * e),
        "dH": [[-1 / (1 + e)], [e * e / (1 + e * e)]],
        "dW": [[1 / (1 + e) - 2 * e * e / (1 + e * e)], [-1 / (1 + e) + 2 * e * e / (1 + e * e)]],
    },
]
with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "hand_derived.json"), "w") as f:
    json.dump({"source": "hand-derived closed forms of softmax cross-entropy; the paper prints "
                         "no worked example for its fused linear + cross-entropy kernel",
               "cases": cases}, f, indent=1)
