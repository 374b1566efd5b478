"""Seeded synthetic inputs: dgir graph texts, location lists and fault variants.

This module is the one place that both the GPU path and the CPU oracle take
their inputs from.  It holds none of the enumeration arithmetic: it only
writes op lists (the shapes and attributes of the workloads), draws output
locations with SplitMix64 and draws the fault variants of the pair check.

The workloads stand in for the paper's corpus of KernelBench level-2
programs (Sec. 5, "Setup": 3-6 Torch operators per program), which is not
available here.  Values never matter: footprints are data independent
(Sec. 2; Sec. 3.4, "Flipping the quantifiers"), so only shapes are given.

dgir v1 text format (one statement per line, '#' starts a comment)::

    dgir 1
    leaf <name> <d0,d1,...>
    op <name> <kind> <operand> [<operand> ...] [; key=value ...]
    output <name> <d0,d1,...>

Attribute values are comma-separated integers, except the ``idxN``
attributes of ``affine_gather``, which are comma-separated index
expressions (one per dimension of operand N) such as ``o1+w0-1`` or
``(o2+1-w1)/2`` (exact division).
"""

from __future__ import annotations

import math

MASK64 = (1 << 64) - 1


# --------------------------------------------------------------------------
# SplitMix64 (Steele, Lea, Flood: "Fast splittable pseudorandom number
# generators", OOPSLA 2014), written from its published definition.
# --------------------------------------------------------------------------
class SplitMix64:
    GAMMA = 0x9E3779B97F4A7C15

    def __init__(self, seed: int):
        self.state = seed & MASK64

    def next(self) -> int:
        self.state = (self.state + self.GAMMA) & MASK64
        z = self.state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
        return z ^ (z >> 31)

    def below(self, n: int) -> int:
        """Uniform draw in [0, n): top bits for powers of two, else Lemire's
        multiply-shift on the high 32 bits (n < 2**32)."""
        if n <= 0:
            raise ValueError("n must be positive")
        z = self.next()
        if n & (n - 1) == 0:
            bits = n.bit_length() - 1
            return z >> (64 - bits) if bits else 0
        if n >= 1 << 32:
            raise ValueError("n too large for multiply-shift")
        return ((z >> 32) * n) >> 32


def sample_locations(numel: int, count: int, seed: int) -> list[int]:
    """``count`` distinct flat output locations in [0, numel), drawn with
    SplitMix64(seed) (duplicates rejected), returned sorted ascending.
    ``count >= numel`` returns every location."""
    if count >= numel:
        return list(range(numel))
    rng = SplitMix64(seed)
    seen: set[int] = set()
    while len(seen) < count:
        seen.add(rng.below(numel))
    return sorted(seen)


def _csv(xs) -> str:
    return ",".join(str(int(v)) for v in xs)


class GraphText:
    """Tiny writer for dgir v1 text."""

    def __init__(self):
        self.lines = ["dgir 1"]

    def leaf(self, name: str, shape) -> str:
        self.lines.append(f"leaf {name} {_csv(shape)}")
        return name

    def op(self, name: str, kind: str, *operands: str, **attrs) -> str:
        line = f"op {name} {kind} " + " ".join(operands)
        if attrs:
            parts = []
            for k, v in attrs.items():
                if isinstance(v, (list, tuple)):
                    parts.append(f"{k}={','.join(str(x) for x in v)}")
                else:
                    parts.append(f"{k}={v}")
            line += " ; " + " ".join(parts)
        self.lines.append(line)
        return name

    def output(self, name: str, shape) -> None:
        self.lines.append(f"output {name} {_csv(shape)}")

    def text(self) -> str:
        return "\n".join(self.lines) + "\n"


# --------------------------------------------------------------------------
# The five workload configurations
# --------------------------------------------------------------------------
def c1_text() -> str:
    """Tiny: C = relu(A[8,16] @ B[16,8]), then the sum over its 8 columns."""
    g = GraphText()
    g.leaf("A", [8, 16])
    g.leaf("B", [16, 8])
    g.op("C", "matmul", "A", "B")
    g.op("R", "relu", "C")
    g.op("y", "sum", "R", dims=1, keepdim=0)
    g.output("y", [8])
    return g.text()


def c2_text() -> str:
    """Conv2d(16x3x32x32 -> 16 ch, k3 s1 p1) + per-channel bias + GELU +
    MaxPool2d(2, 2)."""
    g = GraphText()
    g.leaf("x", [16, 3, 32, 32])
    g.leaf("W", [16, 3, 3, 3])
    g.leaf("conv_b", [16])
    g.leaf("bias", [16, 1, 1])
    g.op("t1", "conv", "x", "W", "conv_b", stride=[1, 1], pad=[1, 1], dilation=[1, 1], groups=1)
    g.op("t2", "add", "t1", "bias")
    g.op("t3", "gelu", "t2")
    g.op("y", "max_pool", "t3", kernel=[2, 2], stride=[2, 2], pad=[0, 0], dilation=[1, 1])
    g.output("y", [16, 16, 16, 16])
    return g.text()


def c3_text() -> str:
    """ConvTranspose3d(8x32x16x32x32 -> 64 ch, k3 s2 p1 output_padding 1),
    mean over channels, softmax over W."""
    g = GraphText()
    g.leaf("x", [8, 32, 16, 32, 32])
    g.leaf("W", [32, 64, 3, 3, 3])
    g.leaf("b", [64])
    g.op("t1", "conv_transpose", "x", "W", "b", stride=[2, 2, 2], pad=[1, 1, 1],
         output_padding=[1, 1, 1], dilation=[1, 1, 1], groups=1)
    g.op("t2", "mean", "t1", dims=1, keepdim=0)
    g.op("y", "softmax", "t2", dim=3)
    g.output("y", [8, 32, 64, 64])
    return g.text()


def c4_text() -> str:
    """GEMM x[128,1024] @ W[1024,512] + bias, GroupNorm(8 groups over 512
    features), Hardtanh, residual add of x[:, :512]."""
    g = GraphText()
    g.leaf("x", [128, 1024])
    g.leaf("W", [1024, 512])
    g.leaf("bias", [512])
    g.leaf("gamma", [512])
    g.leaf("beta", [512])
    g.op("h", "matmul", "x", "W")
    g.op("h2", "add", "h", "bias")
    g.op("gn", "group_norm", "h2", "gamma", "beta", groups=8)
    g.op("ht", "hardtanh", "gn")
    g.op("xs", "slice", "x", dim=1, start=0, end=512, step=1)
    g.op("y", "add", "ht", "xs")
    g.output("y", [128, 512])
    return g.text()


def c5_reference_text(n=64, c=64, hw=64, co=128) -> str:
    """Conv2d(NCHW, k3 p1) + per-channel affine (batch-norm inference form) +
    ReLU."""
    g = GraphText()
    g.leaf("x", [n, c, hw, hw])
    g.leaf("W", [co, c, 3, 3])
    g.leaf("conv_b", [co])
    g.leaf("scale", [co])
    g.leaf("shift", [co])
    g.op("t1", "conv", "x", "W", "conv_b", stride=[1, 1], pad=[1, 1], dilation=[1, 1], groups=1)
    g.op("t2", "channel_affine", "t1", "scale", "shift")
    g.op("y", "relu", "t2")
    g.output("y", [n, co, hw, hw])
    return g.text()


# Index expressions of the channels-last split-K variant.  Dimension order of
# the partial sums is (n, h, w, co); the window is (kh, kw, ci), so the
# reduction index K = (kh*3 + kw)*C + ci runs in row-major window order.
_C5_XC = ["o0", "o1+w0-1", "o2+w1-1", "w2"]
_C5_WC = ["o3", "w0", "w1", "w2"]

C5_FAULT_DIMS = ("xc-h", "xc-w", "Wc-kh", "Wc-kw")
C5_FAULT_KINDS = ("offset+1", "offset-1", "stride*2")
C5_SPLITS = 4


def _fault_expr(expr: str, kind: str) -> str:
    """Apply one index-map fault to an expression of the form
    ``[o<a>][+w<b>][+/-c]``: shift the constant by +-1, or double the
    coefficient of the output variable (of the window variable if there is
    no output variable)."""
    terms = _split_terms(expr)
    if kind == "offset+1" or kind == "offset-1":
        delta = 1 if kind == "offset+1" else -1
        const = sum(c for c, v in terms if v is None) + delta
        terms = [(c, v) for c, v in terms if v is not None] + ([(const, None)] if const else [])
    elif kind == "stride*2":
        target = next((v for c, v in terms if v is not None and v[0] == "o"), None)
        if target is None:
            target = next(v for c, v in terms if v is not None)
        terms = [(c * 2 if v == target else c, v) for c, v in terms]
    else:
        raise ValueError(kind)
    return _join_terms(terms)


def _split_terms(expr: str):
    out = []
    i = 0
    s = expr.replace(" ", "")
    while i < len(s):
        sign = 1
        if s[i] in "+-":
            sign = -1 if s[i] == "-" else 1
            i += 1
        j = i
        while j < len(s) and s[j] not in "+-":
            j += 1
        tok = s[i:j]
        i = j
        if "*" in tok:
            c, v = tok.split("*")
            out.append((sign * int(c), v))
        elif tok[0] in "ow":
            out.append((sign, tok))
        else:
            out.append((sign * int(tok), None))
    return out


def _join_terms(terms) -> str:
    s = ""
    for c, v in terms:
        if v is None:
            piece = str(abs(c))
        else:
            piece = v if abs(c) == 1 else f"{abs(c)}*{v}"
        if not s:
            s = ("-" if c < 0 else "") + piece
        else:
            s += ("-" if c < 0 else "+") + piece
    return s or "0"


def c5_faults(seed: int = 5, count: int = 16):
    """Draw ``count`` single-fault descriptors (split, dim, kind) without
    replacement from {split 0..3} x {xc-h, xc-w, Wc-kh, Wc-kw} x
    {offset+1, offset-1, stride*2}, in draw order."""
    space = [(s, d, k) for s in range(C5_SPLITS) for d in C5_FAULT_DIMS for k in C5_FAULT_KINDS]
    rng = SplitMix64(seed)
    picked: list[int] = []
    while len(picked) < count:
        i = rng.below(len(space))
        if i not in picked:
            picked.append(i)
    return [space[i] for i in picked]


# Sparse faults of the split-K variant: one index map of split 0 changed so
# that only boundary locations of the output read differently (the
# low-prevalence bugs the boundary tiers of the order target), 1/64 of the
# output each.
#   "last-row": x's row index o1+w0-1 becomes ((H+1)o1 + H w0 - (H-1)) // H,
#     equal to it except at the last output row (o1 = H-1), where it is one
#     more;
#   "last-col": the same for the column index o2+w1-1 and the last output
#     column (o2 = W-1).
# (A fault confined to the last row and column together needs one index map
# over both output coordinates, which couples the h and w dims; its merged
# view outgrows the LDS of one location.)
C5_SPARSE_FAULTS = ("last-row", "last-col")


def _sparse_index(kind: str, hw: int) -> tuple[int, str]:
    """(position in x's index maps, the faulty expression) of a sparse fault."""
    if kind == "last-row":
        return 1, f"({hw + 1}*o1+{hw}*w0-{hw - 1})//{hw}"
    if kind == "last-col":
        return 2, f"({hw + 1}*o2+{hw}*w1-{hw - 1})//{hw}"
    raise ValueError(kind)


def c5_variant_text(fault=None, n=64, c=64, hw=64, co=128, splits=C5_SPLITS) -> str:
    """The channels-last, split-K form of the C5 reference program: x and W
    are permuted to NHWC / (O, kh, kw, I), the K = 9*C reduction is split into
    ``splits`` contiguous flat ranges computed by separate gather kernels,
    then summed, biased, scaled and shifted in NHWC, and permuted back.
    ``fault`` = (split, dim, kind) perturbs one index map of one split; a
    name from C5_SPARSE_FAULTS applies that sparse fault to split 0."""
    k_total = 9 * c
    if k_total % splits:
        raise ValueError("K must split evenly")
    chunk = k_total // splits
    g = GraphText()
    g.leaf("x", [n, c, hw, hw])
    g.leaf("W", [co, c, 3, 3])
    g.leaf("conv_b", [co])
    g.leaf("scale", [co])
    g.leaf("shift", [co])
    g.op("xc", "permute", "x", dims=[0, 2, 3, 1])
    g.op("Wc", "permute", "W", dims=[0, 2, 3, 1])
    parts = []
    for s in range(splits):
        xc = list(_C5_XC)
        wc = list(_C5_WC)
        if isinstance(fault, str):
            if s == 0:
                pos, expr = _sparse_index(fault, hw)
                xc[pos] = expr
        elif fault is not None and fault[0] == s:
            _, dim, kind = fault
            if dim == "xc-h":
                xc[1] = _fault_expr(xc[1], kind)
            elif dim == "xc-w":
                xc[2] = _fault_expr(xc[2], kind)
            elif dim == "Wc-kh":
                wc[1] = _fault_expr(wc[1], kind)
            elif dim == "Wc-kw":
                wc[2] = _fault_expr(wc[2], kind)
            else:
                raise ValueError(dim)
        name = f"p{s}"
        g.op(name, "affine_gather", "xc", "Wc", shape=[n, hw, hw, co], window=[3, 3, c],
             flat=[s * chunk, (s + 1) * chunk], idx0=xc, idx1=wc, mult=[1, 1])
        parts.append(name)
    acc = parts[0]
    for i, p in enumerate(parts[1:]):
        acc = g.op(f"s{i + 1}", "add", acc, p)
    g.op("cb", "add", acc, "conv_b")
    g.op("sc", "mul", "cb", "scale")
    g.op("sh", "add", "sc", "shift")
    g.op("r", "relu", "sh")
    g.op("y", "permute", "r", dims=[0, 3, 1, 2])
    g.output("y", [n, co, hw, hw])
    return g.text()


# --------------------------------------------------------------------------
# The running example of the paper (Sec. 2 and the CHECK illustration):
# Y[n,c,w] = gelu(sum_{h<H} min_{c'} M[n,c',h,w]) + b[c] with M the
# post-convolution tensor [128,16,64,64].  The reference sums all H = 64 rows;
# the optimized kernel's loop bug leaves only h < 32.
# --------------------------------------------------------------------------
def paper_reference_text(N=128, C=16, H=64, W=64) -> str:
    g = GraphText()
    g.leaf("M", [N, C, H, W])
    g.leaf("b", [C, 1])
    g.op("R", "amin", "M", dims=1, keepdim=0)
    g.op("S", "sum", "R", dims=1, keepdim=1)
    g.op("G", "gelu", "S")
    g.op("Y", "add", "G", "b")
    g.output("Y", [N, C, W])
    return g.text()


def paper_kernel_text(N=128, C=16, H=64, W=64, h_limit=32) -> str:
    """The optimized program: the fused min/sum kernel as an affine gather.
    Block (bx, by) writes S[bx, 0, by] from the window (c', h) with h below
    ``h_limit``; the buggy loop gives ``h_limit = H/2``."""
    g = GraphText()
    g.leaf("M", [N, C, H, W])
    g.leaf("b", [C, 1])
    g.op("S", "affine_gather", "M", shape=[N, 1, W], window=[C, h_limit],
         idx0=["o0", "w0", "w1", "o2"], mult=[1])
    g.op("G", "gelu", "S")
    g.op("Y", "add", "G", "b")
    g.output("Y", [N, C, W])
    return g.text()


def paper_program_text(kernel: bool, N=128, Cin=3, C=16, H=64, W=64, h_limit=32) -> str:
    """The running example as the two whole programs that MERGE receives
    (Sec. 3.2, the trace-merge illustration): both start with the same
    convolution, whose result M is then reduced by the reference ops or by
    the fused kernel (``paper_reference_text`` / ``paper_kernel_text`` from M
    on).  The kernel program names and orders its inputs differently, so
    that its inputs are matched by shape."""
    g = GraphText()
    conv = dict(stride=[1, 1], pad=[1, 1], dilation=[1, 1], groups=1)
    if not kernel:
        g.leaf("x", [N, Cin, H, W])
        g.leaf("Wt", [C, Cin, 3, 3])
        g.leaf("conv_b", [C])
        g.leaf("b", [C, 1])
        g.op("M", "conv", "x", "Wt", "conv_b", **conv)
        g.op("R", "amin", "M", dims=1, keepdim=0)
        g.op("S", "sum", "R", dims=1, keepdim=1)
        g.op("G", "gelu", "S")
        g.op("Y", "add", "G", "b")
    else:
        g.leaf("wgt", [C, Cin, 3, 3])
        g.leaf("inp", [N, Cin, H, W])
        g.leaf("bias", [C, 1])
        g.leaf("cb", [C])
        g.op("conv_out", "conv", "inp", "wgt", "cb", **conv)
        g.op("S", "affine_gather", "conv_out", shape=[N, 1, W], window=[C, h_limit],
             idx0=["o0", "w0", "w1", "o2"], mult=[1])
        g.op("G", "gelu", "S")
        g.op("Y", "add", "G", "bias")
    g.output("Y", [N, C, W])
    return g.text()


CONFIGS = {
    "c1": dict(text=c1_text, numel=8, n_locs=8, seed=None,
               desc="matmul A[8x16]@B[16x8] -> relu -> row-sum"),
    "c2": dict(text=c2_text, numel=16 * 16 * 16 * 16, n_locs=4096, seed=2,
               desc="conv2d(16x3x32x32, 16ch k3 p1) + bias + gelu + maxpool2x2"),
    "c3": dict(text=c3_text, numel=8 * 32 * 64 * 64, n_locs=65536, seed=3,
               desc="conv_transpose3d(8x32x16x32x32, 64ch k3 s2 p1 op1) -> mean(C) -> softmax(W)"),
    "c4": dict(text=c4_text, numel=128 * 512, n_locs=65536, seed=None,
               desc="x[128x1024]@W[1024x512]+bias -> group_norm(8) -> hardtanh -> +x[:, :512]"),
    "c5": dict(text=c5_reference_text, numel=64 * 128 * 64 * 64, n_locs=1048576, seed=5,
               desc="pair check: conv2d(64x64x64x64, 128ch k3 p1)+affine+relu vs NHWC split-K=4 variant"),
}


def config_locations(name: str) -> list[int]:
    cfg = CONFIGS[name]
    if cfg["seed"] is None:
        return list(range(cfg["numel"]))
    return sample_locations(cfg["numel"], cfg["n_locs"], cfg["seed"])


def numel(shape) -> int:
    return math.prod(int(s) for s in shape)
