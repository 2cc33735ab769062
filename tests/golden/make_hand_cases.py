"""Writes hand_cases.json: tiny hand-worked trees with closed-form states.

Every expected number below comes from the derivation printed next to it,
evaluated with scalar ``math`` functions only (no oracle, no HIP code).  The
inputs are dyadic rationals, exact in float32, so float64 evaluation of the
same formula is exact up to libm rounding.  The cells follow the standard
published forms the paper cites (TreeRNN/TreeFC, N-ary and child-sum
TreeLSTM, MV-RNN, DAG-RNN; Sec. 7.1 "Models and datasets").

Run:  python tests/golden/make_hand_cases.py
"""
import json
import math
import os


def sig(z):
    return 1.0 / (1.0 + math.exp(-z))


cases = {}

# TreeRNN, H = 1: h = tanh(W_l h_l + W_r h_r + b) = tanh(0.5*1 - 0.25*2 + 0.125)
cases["tree_rnn_h1"] = {
    "cell": "tree_rnn", "K": 2, "H": 1, "children": [-1, -1, -1, -1, 0, 1],
    "inputs": {"x_index": [0, 1, -1], "x_table": [[1.0], [2.0]], "W": [[0.5, -0.25]], "b": [0.125]},
    "derivation": "h2 = tanh(0.5*1 - 0.25*2 + 0.125) = tanh(0.125); swapped halves would give tanh(0.875)",
    "expect": {"h": {"0": 1.0, "1": 2.0, "2": math.tanh(0.125)}},
}

# binary N-ary TreeLSTM, H = 1, leaves (1, 0) and (-1, 0).
# U_l = 0.5 for all gates; U_r = (-0.5, 0.25, 0.25, 0.25, 1.0) for (i, f_l, f_r, o, u); b = 0
# a = (1.0, 0.25, 0.25, 0.25, -0.5); c = sig(1) tanh(-0.5); h = sig(0.25) tanh(c)
c = sig(1.0) * math.tanh(-0.5)
cases["nary_treelstm_h1"] = {
    "cell": "nary_treelstm", "K": 2, "H": 1, "children": [-1, -1, -1, -1, 0, 1],
    "inputs": {"x_index": [0, 1, -1], "x_table": [[1.0], [-1.0]],
               "U": [[[[0.5]]] * 5, [[[-0.5]], [[0.25]], [[0.25]], [[0.25]], [[1.0]]]],
               "b": [[0.0]] * 5},
    "derivation": "a=(1,.25,.25,.25,-.5); c=sig(1)tanh(-.5); h=sig(.25)tanh(c); leaf c=0",
    "expect": {"h": {"0": 1.0, "1": -1.0, "2": sig(0.25) * math.tanh(c)},
               "c": {"0": 0.0, "1": 0.0, "2": c}},
}

# child-sum TreeLSTM leaf, H = 1, x = 1: W = (W_i, W_f, W_o, W_u) = (0, .75, 0, .5),
# b = (.25, 0, -.25, 0): i = sig(.25), o = sig(-.25), u = tanh(.5); c = i u; h = o tanh(c)
cl = sig(0.25) * math.tanh(0.5)
cases["childsum_leaf_h1"] = {
    "cell": "childsum_treelstm", "K": 4, "H": 1, "children": [-1, -1, -1, -1],
    "inputs": {"x_index": [0], "x_table": [[1.0]],
               "W": [[[0.0]], [[0.75]], [[0.0]], [[0.5]]], "U": [[[0.25]]] * 4,
               "b": [[0.25], [0.0], [-0.25], [0.0]]},
    "derivation": "leaf: h~=0, no forget terms; c = sig(.25) tanh(.5), h = sig(-.25) tanh(c)",
    "expect": {"c": {"0": cl}, "h": {"0": sig(-0.25) * math.tanh(cl)}},
}
# child-sum TreeLSTM, two leaves under a root, H = 1.
# W = (0, 0, 0, 1), U = (1, 1, 0, 0), b = 0.  Emb = [1, 2, -1]; leaves x = 2, -1; root x = 1.
# leaf k: i = o = 1/2, u = tanh(x_k): c_k = tanh(x_k)/2, h_k = tanh(c_k)/2
# root: i = sig(h1 + h2), f_k = sig(h_k), o = 1/2, u = tanh(1)
c1, c2 = 0.5 * math.tanh(2.0), 0.5 * math.tanh(-1.0)
h1, h2 = 0.5 * math.tanh(c1), 0.5 * math.tanh(c2)
cr = sig(h1 + h2) * math.tanh(1.0) + sig(h1) * c1 + sig(h2) * c2
cases["childsum_two_children_h1"] = {
    "cell": "childsum_treelstm", "K": 4, "H": 1,
    "children": [-1, -1, -1, -1, -1, -1, -1, -1, 0, 1, -1, -1],
    "inputs": {"x_index": [1, 2, 0], "x_table": [[1.0], [2.0], [-1.0]],
               "W": [[[0.0]], [[0.0]], [[0.0]], [[1.0]]], "U": [[[1.0]], [[1.0]], [[0.0]], [[0.0]]],
               "b": [[0.0]] * 4},
    "derivation": "c = sig(h1+h2) tanh(1) + sig(h1) c1 + sig(h2) c2, h = tanh(c)/2; "
                  "a forget gate on h~ instead of h_k would give sig(h1+h2)(c1+c2)",
    "expect": {"h": {"0": h1, "1": h2, "2": 0.5 * math.tanh(cr)}, "c": {"0": c1, "1": c2, "2": cr}},
}

# MV-RNN, H = 1: left (a, A) = (1, 2), right (b, B) = (3, 4), W = [.125, -.0625], W_M = [.5, .25]
# p = tanh(W [B a; A b]) = tanh(.125*4 - .0625*6) = tanh(.125); P = .5*2 + .25*4 = 2
cases["mvrnn_h1"] = {
    "cell": "mvrnn", "K": 2, "H": 1, "children": [-1, -1, -1, -1, 0, 1],
    "inputs": {"x_index": [0, 1, -1], "x_table": [[1.0], [3.0]], "leaf_mat": [[[2.0]], [[4.0]]],
               "W": [[0.125, -0.0625]], "W_M": [[0.5, 0.25]]},
    "derivation": "p = tanh(.125*B*a - .0625*A*b) = tanh(.125); (A a, B b) would give tanh(-.5); P = 2",
    "expect": {"h": {"2": math.tanh(0.125)}, "P": {"2": 2.0}},
}

# DAG-RNN on a 2x2 grid, H = 1: W = 1, U_up = .5, U_left = -.5, b = 0, x = [[.125, .25], [.375, .5]]
h00 = math.tanh(0.125)
h01 = math.tanh(0.25 - 0.5 * h00)
h10 = math.tanh(0.375 + 0.5 * h00)
h11 = math.tanh(0.5 + 0.5 * h01 - 0.5 * h10)
cases["dagrnn_2x2_h1"] = {
    "cell": "dagrnn", "K": 2, "H": 1, "children": [-1, -1, -1, 0, 0, -1, 1, 2],
    "inputs": {"x": [[0.125], [0.25], [0.375], [0.5]], "W": [[1.0]], "U": [[[0.5]], [[-0.5]]], "b": [0.0]},
    "derivation": "h(i,j) = tanh(x + .5 h(i-1,j) - .5 h(i,j-1)), absent neighbours = 0",
    "expect": {"h": {"0": h00, "1": h01, "2": h10, "3": h11}},
}

# child-sum TreeGRU and SimpleTreeGRU, two leaves under a root, H = 1.
# W = (W_z, W_r, W_h) = (0, .25, 1), U = (U_z, U_r, U_h) = (.5, 1, .5), b = 0.
# Emb = [1, 2, -1]; leaves x = 2, -1; root x = 1.
# leaf k (no child): z = sig(0) = 1/2, h' = tanh(x_k), h_k = tanh(x_k)/2 (both variants)
# root: z = sig(.5 (h1 + h2)); r_k = sig(.25 + h_k); m = r_1 h1 + r_2 h2;
#       h' = tanh(1 + .5 m); TreeGRU h = z (h1 + h2) + (1 - z) h';  Simple h = (1 - z) h'
g1, g2 = 0.5 * math.tanh(2.0), 0.5 * math.tanh(-1.0)
gz = sig(0.5 * (g1 + g2))
gm = sig(0.25 + g1) * g1 + sig(0.25 + g2) * g2
gcand = math.tanh(1.0 + 0.5 * gm)
gru_inputs = {"x_index": [1, 2, 0], "x_table": [[1.0], [2.0], [-1.0]],
              "W": [[[0.0]], [[0.25]], [[1.0]]], "U": [[[0.5]], [[1.0]], [[0.5]]], "b": [[0.0]] * 3}
gru_children = [-1, -1, -1, -1, -1, -1, -1, -1, 0, 1, -1, -1]
cases["childsum_treegru_two_children_h1"] = {
    "cell": "childsum_treegru", "K": 4, "H": 1, "children": gru_children, "inputs": gru_inputs,
    "derivation": "h = z(h1+h2) + (1-z) tanh(1 + .5(r1 h1 + r2 h2)), r_k = sig(.25 + h_k); "
                  "one reset gate on h~ would give sig(.25 + h~) h~ inside the tanh",
    "expect": {"h": {"0": g1, "1": g2, "2": gz * (g1 + g2) + (1.0 - gz) * gcand}},
}
cases["simple_treegru_two_children_h1"] = {
    "cell": "simple_treegru", "K": 4, "H": 1, "children": gru_children, "inputs": gru_inputs,
    "derivation": "h = (1-z) tanh(1 + .5(r1 h1 + r2 h2)); leaves as in the TreeGRU case",
    "expect": {"h": {"0": g1, "1": g2, "2": (1.0 - gz) * gcand}},
}

# child-sum TreeGRU, H = 2, one leaf under a root: where the reset gate sits.
# W = (W_z, W_r, W_h) = (0, 0, I), U = (U_z, U_r, U_h) = (0, 0, [[0, 1], [1, 0]]),
# b = (0, (1, -2), 0).  Leaf x = (1, -.5): z = 1/2, h_c = tanh(x)/2.  Root x = 0:
# h~ = h_c, z = 1/2, r = (sig(1), sig(-2)), m = r * h_c, h' = tanh(U_h m) =
# (tanh(r_1 h_c1), tanh(r_0 h_c0)); h = h_c/2 + h'/2.  A reset applied after U_h
# (r * (U_h h_c)) would give (tanh(r_0 h_c1), tanh(r_1 h_c0)) instead.
hc0, hc1 = 0.5 * math.tanh(1.0), 0.5 * math.tanh(-0.5)
r0, r1 = sig(1.0), sig(-2.0)
cases["childsum_treegru_reset_placement_h2"] = {
    "cell": "childsum_treegru", "K": 4, "H": 2, "children": [-1, -1, -1, -1, 0, -1, -1, -1],
    "inputs": {"x_index": [1, 0], "x_table": [[0.0, 0.0], [1.0, -0.5]],
               "W": [[[0.0, 0.0], [0.0, 0.0]], [[0.0, 0.0], [0.0, 0.0]], [[1.0, 0.0], [0.0, 1.0]]],
               "U": [[[0.0, 0.0], [0.0, 0.0]], [[0.0, 0.0], [0.0, 0.0]], [[0.0, 1.0], [1.0, 0.0]]],
               "b": [[0.0, 0.0], [1.0, -2.0], [0.0, 0.0]]},
    "derivation": "h' = tanh(U_h (r * h_c)) with U_h the swap: (tanh(r1 hc1), tanh(r0 hc0)); h = hc/2 + h'/2",
    "expect": {"h": {"0": [hc0, hc1],
                     "1": [0.5 * hc0 + 0.5 * math.tanh(r1 * hc1), 0.5 * hc1 + 0.5 * math.tanh(r0 * hc0)]}},
}

out = os.path.join(os.path.dirname(os.path.abspath(__file__)), "hand_cases.json")
with open(out, "w") as f:
    json.dump(cases, f, indent=1, sort_keys=True)
    f.write("\n")
print("wrote", out)
