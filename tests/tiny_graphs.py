"""Small dgir graphs covering every op kind and attribute of the vocabulary,
plus shrunken versions of the five workloads and of the paper's example.
Sized so that perturbation over every leaf element and autograd over every
output element finish in seconds."""

from __future__ import annotations

from paper_2609_19611_amd.workloads import (GraphText, c5_reference_text, c5_variant_text,
                                            paper_kernel_text, paper_reference_text)


def _g(leaves, ops, out, shape):
    g = GraphText()
    for n, s in leaves:
        g.leaf(n, s)
    for name, kind, operands, attrs in ops:
        g.op(name, kind, *operands, **attrs)
    g.output(out, shape)
    return g.text()


# Graphs whose reads couple two dims of one operand (a grouped transposed
# convolution feeds its weight's first two dims from the output channel; a
# reshape that merges dims feeds them from one coordinate): the library
# compiles them over merged dims.  MERGED_DIMS lists the catalogue's such
# graphs.
MERGED_DIMS = {"convT1d_groups", "views", "convT2d_groups", "convT3d_groups", "conv_flatten_softmax",
               "reshape_split_merge", "reshape_refine", "unflatten_linear"}

# A reshape between two factorisations of one block of dims with no common
# refinement ([2,3,4] -> [4,3,2]: 4 does not divide 6): the library refuses
# it (DG_E_UNSUPPORTED_OP); the oracle takes it.
UNREFINABLE_RESHAPE = ("dgir 1\nleaf x 2,3,4\nleaf z 4,3,2\nop r reshape x ; shape=4,3,2\n"
                       "op y mul r z\noutput y 4,3,2\n")


def catalogue():
    """name -> (dgir text, masks) where masks says whether a saturating or
    selecting op may hide a dependence from perturbation."""
    G = {}
    G["matmul2d"] = (_g([("A", [3, 4]), ("B", [4, 2])], [("y", "matmul", ["A", "B"], {})], "y", [3, 2]), False)
    G["matmul_bcast"] = (_g([("A", [2, 1, 3, 4]), ("B", [3, 4, 2])],
                            [("y", "matmul", ["A", "B"], {})], "y", [2, 3, 3, 2]), False)
    G["linear"] = (_g([("x", [2, 3, 4]), ("W", [5, 4]), ("b", [5])],
                      [("y", "linear", ["x", "W", "b"], {})], "y", [2, 3, 5]), False)
    G["conv1d_groups"] = (_g([("x", [2, 4, 7]), ("W", [6, 2, 3]), ("b", [6])],
                             [("y", "conv", ["x", "W", "b"], dict(stride=[2], pad=[1], dilation=[2], groups=2))],
                             "y", [2, 6, 3]), False)
    G["conv2d_asym"] = (_g([("x", [1, 2, 5, 6]), ("W", [3, 2, 3, 2])],
                           [("y", "conv", ["x", "W"], dict(stride=[1, 2], pad=[1, 0], dilation=[1, 1], groups=1))],
                           "y", [1, 3, 5, 3]), False)
    G["conv3d_groups"] = (_g([("x", [1, 2, 3, 4, 4]), ("W", [2, 1, 2, 2, 3]), ("b", [2])],
                             [("y", "conv", ["x", "W", "b"], dict(stride=[1, 1, 1], pad=[0, 1, 1], dilation=[1, 1, 1], groups=2))],
                             "y", [1, 2, 2, 5, 4]), False)
    G["convT1d_groups"] = (_g([("x", [1, 4, 5]), ("W", [4, 3, 3]), ("b", [6])],
                              [("y", "conv_transpose", ["x", "W", "b"],
                                dict(stride=[2], pad=[1], output_padding=[1], dilation=[1], groups=2))],
                              "y", [1, 6, 10]), False)
    G["convT2d_dil"] = (_g([("x", [1, 3, 3, 4]), ("W", [3, 2, 3, 2])],
                           [("y", "conv_transpose", ["x", "W"],
                             dict(stride=[2, 3], pad=[1, 0], output_padding=[1, 2], dilation=[1, 2], groups=1))],
                           "y", [1, 2, 6, 14]), False)
    G["convT3d"] = (_g([("x", [1, 2, 2, 3, 3]), ("W", [2, 2, 3, 3, 3]), ("b", [2])],
                       [("y", "conv_transpose", ["x", "W", "b"],
                         dict(stride=[2, 2, 2], pad=[1, 1, 1], output_padding=[1, 1, 1], dilation=[1, 1, 1], groups=1))],
                       "y", [1, 2, 4, 6, 6]), False)
    G["maxpool2d"] = (_g([("x", [1, 2, 5, 5])],
                         [("y", "max_pool", ["x"], dict(kernel=[3, 3], stride=[2, 2], pad=[1, 1], dilation=[1, 1]))],
                         "y", [1, 2, 3, 3]), True)
    G["maxpool2d_dil"] = (_g([("x", [1, 1, 7, 7])],
                             [("y", "max_pool", ["x"], dict(kernel=[2, 2], stride=[1, 1], pad=[0, 0], dilation=[2, 2]))],
                             "y", [1, 1, 5, 5]), True)
    G["avgpool1d"] = (_g([("x", [2, 3, 7])],
                         [("y", "avg_pool", ["x"], dict(kernel=[3], stride=[2], pad=[1], dilation=[1]))],
                         "y", [2, 3, 4]), False)
    G["unary_chain"] = (_g([("x", [2, 3])],
                           [("a", "exp", ["x"], {}), ("b", "tanh", ["a"], {}), ("c", "sigmoid", ["b"], {}),
                            ("d", "square", ["c"], {}), ("e", "gelu", ["d"], {}), ("y", "neg", ["e"], {})],
                           "y", [2, 3]), False)
    G["binary_bcast"] = (_g([("x", [2, 1, 3]), ("z", [4, 1])],
                            [("a", "add", ["x", "z"], {}), ("b", "mul", ["a", "z"], {}), ("c", "sub", ["b", "x"], {}),
                             ("y", "div", ["c", "x"], {})],
                            "y", [2, 4, 3]), False)
    G["self_product"] = (_g([("x", [3, 2]), ("w", [2])],
                            [("a", "mul", ["x", "x"], {}), ("b", "add", ["a", "x"], {}), ("y", "mul", ["b", "w"], {})],
                            "y", [3, 2]), False)
    G["maxmin"] = (_g([("x", [3, 4]), ("z", [4]), ("u", [3, 1])],
                      [("a", "maximum", ["x", "z"], {}), ("y", "minimum", ["a", "u"], {})],
                      "y", [3, 4]), True)
    # min(max(x, z), x) == x: z is read (syntactic footprint) but cannot
    # change the value (semantic footprint); perturbation must give a subset.
    G["select_absorb"] = (_g([("x", [2, 3]), ("z", [3])],
                             [("a", "maximum", ["x", "z"], {}), ("y", "minimum", ["a", "x"], {})],
                             "y", [2, 3]), True)
    G["reductions"] = (_g([("x", [2, 3, 4])],
                          [("a", "sum", ["x"], dict(dims=[0, 2], keepdim=1)), ("b", "mul", ["a", "x"], {}),
                           ("c", "mean", ["b"], dict(dims=[1], keepdim=0)), ("y", "prod", ["c"], dict(dims=[-1], keepdim=1))],
                          "y", [2, 1]), False)
    G["amax_full"] = (_g([("x", [2, 3]), ("z", [2, 3])],
                         [("a", "add", ["x", "z"], {}), ("y", "amax", ["a"], dict(dims=[0, 1], keepdim=0))],
                         "y", [1]), True)
    G["softmax"] = (_g([("x", [2, 3, 4])], [("y", "softmax", ["x"], dict(dim=1))], "y", [2, 3, 4]), False)
    G["log_softmax"] = (_g([("x", [3, 5])], [("y", "log_softmax", ["x"], dict(dim=-1))], "y", [3, 5]), False)
    G["group_norm"] = (_g([("x", [2, 4, 3]), ("g", [4]), ("b", [4])],
                          [("y", "group_norm", ["x", "g", "b"], dict(groups=2))], "y", [2, 4, 3]), False)
    G["group_norm_plain"] = (_g([("x", [1, 6, 2, 2])],
                                [("y", "group_norm", ["x"], dict(groups=3))], "y", [1, 6, 2, 2]), False)
    G["batch_norm"] = (_g([("x", [3, 2, 2]), ("g", [2]), ("b", [2])],
                          [("y", "batch_norm", ["x", "g", "b"], {})], "y", [3, 2, 2]), False)
    G["layer_norm"] = (_g([("x", [2, 3, 2]), ("g", [3, 2]), ("b", [3, 2])],
                          [("y", "layer_norm", ["x", "g", "b"], dict(ndims=2))], "y", [2, 3, 2]), False)
    G["channel_affine"] = (_g([("x", [2, 3, 2]), ("s", [3]), ("t", [3])],
                              [("y", "channel_affine", ["x", "s", "t"], {})], "y", [2, 3, 2]), False)
    G["views"] = (_g([("x", [2, 3, 4]), ("z", [4, 1])],
                     [("a", "slice", ["x"], dict(dim=2, start=1, end=4, step=2)),
                      ("b", "permute", ["a"], dict(dims=[2, 0, 1])),
                      ("c", "reshape", ["b"], dict(shape=[4, 3])),
                      ("d", "expand", ["z"], dict(shape=[2, 4, 3])),
                      ("y", "add", ["c", "d"], {})],
                     "y", [2, 4, 3]), False)
    G["convT2d_groups"] = (_g([("x", [1, 6, 3, 4]), ("W", [6, 2, 3, 2]), ("b", [6])],
                              [("y", "conv_transpose", ["x", "W", "b"],
                                dict(stride=[2, 1], pad=[1, 0], output_padding=[1, 0], dilation=[1, 2], groups=3))],
                              "y", [1, 6, 6, 6]), False)
    G["convT3d_groups"] = (_g([("x", [1, 4, 2, 3, 2]), ("W", [4, 1, 2, 3, 2])],
                              [("t", "conv_transpose", ["x", "W"],
                                dict(stride=[2, 2, 1], pad=[0, 1, 0], output_padding=[1, 1, 0], dilation=[1, 1, 1],
                                     groups=2)),
                               ("y", "relu", ["t"], {})],
                              "y", [1, 2, 5, 6, 3]), True)
    # conv -> flatten of the spatial dims -> softmax over them: the merged
    # output couples the conv's two spatial dims, so its input and weight
    # are viewed with merged spatial dims too.
    G["conv_flatten_softmax"] = (_g([("x", [1, 2, 4, 5]), ("W", [3, 2, 3, 2]), ("b", [3])],
                                    [("t", "conv", ["x", "W", "b"],
                                      dict(stride=[1, 2], pad=[1, 1], dilation=[1, 1], groups=1)),
                                     ("f", "reshape", ["t"], dict(shape=[1, 3, 12])),
                                     ("y", "softmax", ["f"], dict(dim=2))],
                                    "y", [1, 3, 12]), False)
    # Dims (2, 3) merged into 6 and 4 split into (2, 2) by one reshape.
    G["reshape_split_merge"] = (_g([("x", [2, 3, 4]), ("s", [6, 1, 2])],
                                   [("e", "exp", ["x"], {}),
                                    ("r", "reshape", ["e"], dict(shape=[6, 2, 2])),
                                    ("m", "mul", ["r", "s"], {}),
                                    ("y", "sum", ["m"], dict(dims=[1], keepdim=0))],
                                   "y", [6, 2]), False)
    # [6, 4] -> [3, 8]: both sides have two dims; strides 1 | 4 | 8 | 24 refine both.
    G["reshape_refine"] = (_g([("x", [6, 4]), ("z", [3, 1])],
                              [("r", "reshape", ["x"], dict(shape=[3, 8])), ("y", "add", ["r", "z"], {})],
                              "y", [3, 8]), False)
    G["unflatten_linear"] = (_g([("x", [2, 5]), ("W", [12, 5]), ("b", [12])],
                                [("h", "linear", ["x", "W", "b"], {}),
                                 ("u", "reshape", ["h"], dict(shape=[2, 3, 4])),
                                 ("p", "permute", ["u"], dict(dims=[0, 2, 1])),
                                 ("y", "layer_norm", ["p"], dict(ndims=1))],
                                "y", [2, 4, 3]), False)
    G["convT1d"] = (_g([("x", [2, 3, 5]), ("W", [3, 2, 4]), ("b", [2])],
                       [("y", "conv_transpose", ["x", "W", "b"],
                         dict(stride=[3], pad=[2], output_padding=[1], dilation=[1], groups=1))],
                       "y", [2, 2, 13]), False)
    G["views_sep"] = (_g([("x", [2, 3, 4]), ("z", [4, 1])],
                         [("a", "slice", ["x"], dict(dim=2, start=1, end=4, step=2)),
                          ("b", "permute", ["a"], dict(dims=[2, 0, 1])),
                          ("c", "reshape", ["b"], dict(shape=[2, 1, 2, 3])),
                          ("d", "expand", ["z"], dict(shape=[2, 4, 3])),
                          ("e", "reshape", ["d"], dict(shape=[2, 4, 1, 3])),
                          ("y", "add", ["c", "e"], {})],
                         "y", [2, 4, 2, 3]), False)
    G["gather_exact_div"] = (_g([("x", [2, 4]), ("w", [3])],
                                [("y", "affine_gather", ["x", "w"],
                                  dict(shape=[2, 8], window=[3], idx0=["o0", "(o1+1-w0)/2"], idx1=["w0"], mult=[1, 1]))],
                                "y", [2, 8]), False)
    G["gather_floor_flat"] = (_g([("x", [3, 5]), ("v", [2, 3])],
                                 [("y", "affine_gather", ["x", "v"],
                                   dict(shape=[4, 3], window=[2, 3], flat=[1, 5],
                                        idx0=["(o0+w0)//2", "2*o1-w1+1"], idx1=["w0", "w1"], mult=[2, 1]))],
                                 "y", [4, 3]), False)
    G["diamond"] = (_g([("x", [2, 3]), ("W", [3, 3])],
                       [("t", "matmul", ["x", "W"], {}), ("a", "tanh", ["t"], {}), ("b", "sigmoid", ["t"], {}),
                        ("c", "add", ["a", "b"], {}), ("d", "softmax", ["c"], dict(dim=1)), ("y", "mul", ["d", "t"], {})],
                       "y", [2, 3]), False)
    # Shrunken workloads.
    G["c1"] = (_g([("A", [8, 16]), ("B", [16, 8])],
                  [("C", "matmul", ["A", "B"], {}), ("R", "relu", ["C"], {}), ("y", "sum", ["R"], dict(dims=[1], keepdim=0))],
                  "y", [8]), True)
    G["c2_small"] = (_g([("x", [2, 3, 6, 6]), ("W", [4, 3, 3, 3]), ("conv_b", [4]), ("bias", [4, 1, 1])],
                        [("t1", "conv", ["x", "W", "conv_b"], dict(stride=[1, 1], pad=[1, 1], dilation=[1, 1], groups=1)),
                         ("t2", "add", ["t1", "bias"], {}), ("t3", "gelu", ["t2"], {}),
                         ("y", "max_pool", ["t3"], dict(kernel=[2, 2], stride=[2, 2], pad=[0, 0], dilation=[1, 1]))],
                        "y", [2, 4, 3, 3]), True)
    G["c3_small"] = (_g([("x", [1, 2, 3, 3, 4]), ("W", [2, 3, 3, 3, 3]), ("b", [3])],
                        [("t1", "conv_transpose", ["x", "W", "b"],
                          dict(stride=[2, 2, 2], pad=[1, 1, 1], output_padding=[1, 1, 1], dilation=[1, 1, 1], groups=1)),
                         ("t2", "mean", ["t1"], dict(dims=[1], keepdim=0)), ("y", "softmax", ["t2"], dict(dim=3))],
                        "y", [1, 6, 6, 8]), False)
    G["c4_small"] = (_g([("x", [3, 8]), ("W", [8, 6]), ("bias", [6]), ("gamma", [6]), ("beta", [6])],
                        [("h", "matmul", ["x", "W"], {}), ("h2", "add", ["h", "bias"], {}),
                         ("gn", "group_norm", ["h2", "gamma", "beta"], dict(groups=2)), ("ht", "hardtanh", ["gn"], {}),
                         ("xs", "slice", ["x"], dict(dim=1, start=0, end=6, step=1)), ("y", "add", ["ht", "xs"], {})],
                        "y", [3, 6]), True)
    G["c5_small_ref"] = (c5_reference_text(n=1, c=2, hw=3, co=2), True)
    G["c5_small_var"] = (c5_variant_text(n=1, c=2, hw=3, co=2, splits=3), True)
    G["paper_ref_small"] = (paper_reference_text(N=2, C=3, H=4, W=2), True)
    G["paper_kernel_small"] = (paper_kernel_text(N=2, C=3, H=4, W=2, h_limit=2), True)
    return G


def dag_catalogue():
    """Graphs for the expression-DAG path beyond the catalogue: index
    functions coupling two window variables (taken point by point), a list
    variable whose table is too large for the per-variable path, reads that
    leave the operand at the boundary, and coupled reads of a non-leaf
    tensor."""
    G = {}
    G["gather_coupled"] = _g([("x", [6, 10])],
                             [("y", "affine_gather", ["x"],
                               dict(shape=[6, 5], window=[3, 4], idx0=["o0", "o1+w0+w1-2"], mult=[1]))],
                             "y", [6, 5])
    G["gather_coupled_nonleaf"] = _g([("x", [4, 9]), ("v", [3])],
                                     [("r", "relu", ["x"], {}),
                                      ("y", "affine_gather", ["r", "v"],
                                       dict(shape=[4, 4], window=[3, 2, 2], idx0=["(o0+w1)/2", "2*o1+w0-w2"],
                                            idx1=["w0"], mult=[1, 2]))],
                                     "y", [4, 4])
    G["gather_big_list"] = _g([("x", [600]), ("w", [1100])],
                              [("y", "affine_gather", ["x", "w"],
                                dict(shape=[5], window=[1100], idx0=["(o0+w0)/2"], idx1=["w0"], mult=[1, 3]))],
                              "y", [5])
    # Stride and dilation both 2: the tap coefficient shares the divisor, so
    # every tap or none reaches an output element (the exact division's
    # progression has step 1 and a divisibility condition of its own).
    G["convT_stride_dilation"] = _g([("x", [1, 2, 4]), ("W", [2, 2, 3])],
                                    [("y", "conv_transpose", ["x", "W"],
                                      dict(stride=[2], pad=[1], output_padding=[0], dilation=[2], groups=1))],
                                    "y", [1, 2, 9])
    # A transposed convolution with a bias, averaged: the mean's node reads
    # 216 conv nodes whose windows hold 16 to 128 points (1 to 8 taps of 16
    # input channels), so a wave's batch holds nodes above and below half a
    # wave of points, each followed by its bias edge.
    G["convT3d_bias_mean"] = _g([("x", [1, 16, 3, 3, 3]), ("W", [16, 2, 3, 3, 3]), ("b", [2])],
                                [("t", "conv_transpose", ["x", "W", "b"],
                                  dict(stride=[2, 2, 2], pad=[1, 1, 1], output_padding=[1, 1, 1], dilation=[1, 1, 1],
                                       groups=1)),
                                 ("y", "mean", ["t"], dict(dims=[2, 3, 4], keepdim=0))],
                                "y", [1, 2])
    G["gather_shift"] = _g([("x", [2, 5]), ("z", [2, 5])],
                           [("t", "exp", ["x"], {}),
                            ("y", "affine_gather", ["t", "z"],
                             dict(shape=[2, 5], window=[1], idx0=["o0", "o1-1"], idx1=["o0", "o1+1+w0"], mult=[1, 1]))],
                           "y", [2, 5])
    return G


def nested_layer_norms(n):
    """Three layer norms in a row over n elements: path counts near
    n^5 (past 2^32 from n = 1024 on)."""
    return _g([("x", [1, n])],
               [("a", "layer_norm", ["x"], dict(ndims=1)), ("b", "layer_norm", ["a"], dict(ndims=1)),
                ("y", "layer_norm", ["b"], dict(ndims=1))], "y", [1, n])


def large_count_norms(shape, variant=None):
    """Three layer norms over the last two dims of x: the static count bound
    of [1, 6, 12] is 2,101,864,255, just below 2^32 and reached.  variant
    "permuted": x goes through two transposes that undo each other (same
    rows, other plan); "mid_1d": the middle norm is over the last dim only
    (same footprint, other counts)."""
    ops, src = [], "x"
    if variant == "permuted":
        ops += [("p", "permute", ["x"], dict(dims=[0, 2, 1])), ("q", "permute", ["p"], dict(dims=[0, 2, 1]))]
        src = "q"
    mid = 1 if variant == "mid_1d" else 2
    ops += [("a", "layer_norm", [src], dict(ndims=2)), ("b", "layer_norm", ["a"], dict(ndims=mid)),
            ("y", "layer_norm", ["b"], dict(ndims=2))]
    return _g([("x", list(shape))], ops, "y", list(shape))


def nested_layer_norm_counts(n, loc):
    """Closed form of three nested layer norms (no affine) over n elements.
    One norm reaches x[s] n + 2 times through its statistics and x[l] once
    more, so its path-count matrix is M = a J + I with a = n + 2 and J the
    all-ones matrix; path counts compose as matrix products and J^2 = n J
    gives M^3 = c J + I with c = (a^2 n + 2a)(a n + 1) + a."""
    a = n + 2
    c = (a * a * n + 2 * a) * (a * n + 1) + a
    return [c + (1 if s == loc else 0) for s in range(n)]


# Shapes whose element counts wrap 64-bit arithmetic or pass 2^62: a leaf
# (3 x 1431655766^3 is about 8.8e27) and a broadcast result of two leaves
# that each fit ((2^31 - 1)^3 elements).
OVERFLOWING_SHAPES = [
    "dgir 1\nleaf x 3,1431655766,1431655766,1431655766\nleaf y 4\nop z relu y\noutput z 4\n",
    "dgir 1\nleaf a 2147483647,1,1\nleaf b 1,2147483647,2147483647\nop y add a b\n"
    "output y 2147483647,2147483647,2147483647\n",
]


def merged_view_pairs():
    """Pairs over the same leaves where one graph reads a leaf through
    merged dims and the other does not (the comparison then views both
    over the joined dims): (name, text a, text b)."""
    A = _g([("x", [2, 3]), ("v", [4, 3])],
           [("a", "sum", ["x"], dict(dims=[0, 1], keepdim=0)), ("b", "sum", ["v"], dict(dims=[0], keepdim=0)),
            ("y", "mul", ["a", "b"], {})], "y", [3])
    B = _g([("x", [2, 3]), ("v", [4, 3])],
           [("f", "reshape", ["x"], dict(shape=[6])), ("a", "sum", ["f"], dict(dims=[0], keepdim=1)),
            ("b", "sum", ["v"], dict(dims=[0], keepdim=0)), ("y", "mul", ["a", "b"], {})], "y", [3])
    C = _g([("x", [2, 3]), ("v", [4, 3])],
           [("f", "reshape", ["x"], dict(shape=[6])), ("s", "slice", ["f"], dict(dim=0, start=1, end=6, step=1)),
            ("a", "sum", ["s"], dict(dims=[0], keepdim=1)), ("b", "sum", ["v"], dict(dims=[0], keepdim=0)),
            ("y", "mul", ["a", "b"], {})], "y", [3])
    D = _g([("x", [2, 3]), ("v", [4, 3])],
           [("f", "reshape", ["x"], dict(shape=[6])), ("a", "sum", ["f"], dict(dims=[0], keepdim=1)),
            ("g", "reshape", ["v"], dict(shape=[2, 6])), ("h", "sum", ["g"], dict(dims=[0], keepdim=0)),
            ("k", "reshape", ["h"], dict(shape=[2, 3])), ("k2", "mul", ["k", "k"], {}),
            ("b", "sum", ["k2"], dict(dims=[0], keepdim=0)), ("y", "mul", ["a", "b"], {})], "y", [3])
    return [("same_footprint", A, B), ("sliced", A, C), ("both_merge", B, D), ("counts", A, D)]


def factored_compare_pairs():
    """Pairs of graphs over the same leaves whose leaves are single terms
    (the comparison then checks factor by factor): (name, a, b, status at
    interior locations)."""
    def g(ops, out_shape):
        return _g([("x", [4, 7]), ("v", [7])], ops, "y", out_shape)
    win3 = ("a", "affine_gather", ["x"], dict(shape=[4, 7], window=[3], idx0=["o0", "o1+w0-1"], mult=[1]))
    win2 = ("a", "affine_gather", ["x"], dict(shape=[4, 7], window=[2], idx0=["o0", "o1+w0-1"], mult=[1]))
    mid = ("c", "affine_gather", ["x"], dict(shape=[4, 7], window=[1], idx0=["o0", "o1"], mult=[1]))
    scale_v = ("y", "mul", ["b", "v"], {})
    A = g([win3, ("b", "relu", ["a"], {}), scale_v], [4, 7])                        # x taps 1,1,1
    B = g([win3, mid, ("b", "add", ["a", "c"], {}), scale_v], [4, 7])               # x taps 1,2,1
    C = g([win2, ("b", "relu", ["a"], {}), scale_v], [4, 7])                        # x taps 1,1
    D = g([win3, ("b", "add", ["a", "a"], {}), scale_v], [4, 7])                    # x taps 2,2,2
    E = g([win3, ("b", "relu", ["a"], {}), ("v2", "mul", ["v", "v"], {}), ("y", "mul", ["b", "v2"], {})], [4, 7])
    return [("same", A, A, 0), ("middle_tap_doubled", A, B, 2), ("one_tap_fewer", A, C, 1),
            ("all_doubled", A, D, 2), ("other_leaf_doubled", A, E, 2)]
