"""Seeded random dgir graphs over the whole op vocabulary, for fuzzing the
library against the oracle.

random_graph(seed) draws a chain of 1 to 4 ops starting from a small leaf:
each op takes the current tensor (and, for binary ops and ops with weights,
new leaves of drawn shapes or an earlier tensor), with drawn shapes, strides,
pads, dilations, output paddings, groups, reduction dims, slices,
permutations, reshapes (always with a common refinement of the two shapes),
expands and affine gathers (exact and floor divisions, flat window ranges).
Every tensor stays at most MAX_NUMEL elements so that the oracle and the host
emulation finish every output location in milliseconds.

The generator holds no enumeration arithmetic: it writes op lists only.
"""

from __future__ import annotations

import numpy as np

from paper_2609_19611_amd.workloads import GraphText

MAX_NUMEL = 192
UNARY = ["relu", "gelu", "gelu_tanh", "hardtanh", "clamp", "sigmoid", "tanh", "exp", "log", "log1p", "square",
         "sqrt", "rsqrt", "neg", "abs", "identity", "contiguous", "silu", "softplus", "erf", "scale", "leaky_relu",
         "elu", "reciprocal"]
BINARY = ["add", "sub", "mul", "div", "maximum", "minimum", "pow"]
REDUCE = ["sum", "mean", "amax", "amin", "prod", "max", "min"]


def numel(s):
    return int(np.prod(s)) if len(s) else 1


class _Gen:
    def __init__(self, seed):
        self.rng = np.random.default_rng(seed)
        self.g = GraphText()
        self.ops = []
        self.shapes = {}
        self.n = 0

    def r(self, lo, hi):
        """Integer in [lo, hi]."""
        return int(self.rng.integers(lo, hi + 1))

    def pick(self, xs):
        return xs[int(self.rng.integers(0, len(xs)))]

    def leaf(self, shape):
        # dgir lists every leaf before the first op: leaves go to the
        # writer at once, ops are kept and written after them.
        name = f"l{self.n}"
        self.n += 1
        self.g.leaf(name, list(shape))
        self.shapes[name] = list(shape)
        return name

    def op(self, kind, operands, out_shape, /, **attrs):
        name = f"t{self.n}"
        self.n += 1
        self.ops.append((name, kind, operands, attrs))
        self.shapes[name] = list(out_shape)
        return name

    # ---- ops: each returns the new tensor's name or None if it does not apply
    def unary(self, t):
        return self.op(self.pick(UNARY), [t], self.shapes[t])

    def binary(self, t):
        s = self.shapes[t]
        if self.rng.random() < 0.25:
            other = t  # a tensor with itself: every element read twice
        elif self.rng.random() < 0.3 and len(s) > 1:
            other = self.leaf(s[1:])  # fewer leading dims
        else:
            other = self.leaf([d if self.rng.random() < 0.6 else 1 for d in s])
        a, b = (t, other) if self.rng.random() < 0.5 else (other, t)
        return self.op(self.pick(BINARY), [a, b], s)

    def matmul(self, t):
        s = self.shapes[t]
        if len(s) < 2:
            return None
        N = self.r(1, 4)
        if self.rng.random() < 0.5:
            w = self.leaf([s[-1], N])
        else:
            w = self.leaf(s[:-2] + [s[-1], N])
        out = s[:-1] + [N]
        return self.op("matmul", [t, w], out) if numel(out) <= MAX_NUMEL else None

    def linear(self, t):
        s = self.shapes[t]
        N = self.r(1, 4)
        out = s[:-1] + [N]
        if numel(out) > MAX_NUMEL:
            return None
        ops = [t, self.leaf([N, s[-1]])]
        if self.rng.random() < 0.6:
            ops.append(self.leaf([N]))
        return self.op("linear", ops, out)

    def conv(self, t, transpose):
        s = self.shapes[t]
        nsp = len(s) - 2
        if nsp < 1 or nsp > 3:
            return None
        C = s[1]
        groups = self.pick([g for g in range(1, C + 1) if C % g == 0])
        k = [self.r(1, 3) for _ in range(nsp)]
        st = [self.r(1, 3 if transpose else 2) for _ in range(nsp)]
        dl = [self.r(1, 2) for _ in range(nsp)]
        pd = [self.r(0, dl[i] * (k[i] - 1)) for i in range(nsp)]
        if transpose:
            cog = self.r(1, 2)
            opd = [self.r(0, max(st[i], dl[i]) - 1) for i in range(nsp)]
            out_sp = [(s[2 + i] - 1) * st[i] - 2 * pd[i] + dl[i] * (k[i] - 1) + opd[i] + 1 for i in range(nsp)]
            w_shape = [C, cog] + k
            cout = cog * groups
        else:
            cout = groups * self.r(1, 2)
            out_sp = [(s[2 + i] + 2 * pd[i] - dl[i] * (k[i] - 1) - 1) // st[i] + 1 for i in range(nsp)]
            w_shape = [cout, C // groups] + k
            opd = None
        if min(out_sp) < 1:
            return None
        out = [s[0], cout] + out_sp
        if numel(out) > MAX_NUMEL:
            return None
        ops = [t, self.leaf(w_shape)]
        if self.rng.random() < 0.5:
            ops.append(self.leaf([cout]))
        attrs = dict(stride=st, pad=pd, dilation=dl, groups=groups)
        if transpose:
            attrs["output_padding"] = opd
        return self.op("conv_transpose" if transpose else "conv", ops, out, **attrs)

    def pool(self, t):
        s = self.shapes[t]
        nsp = self.r(1, min(3, len(s)))
        k = [self.r(1, 3) for _ in range(nsp)]
        st = [self.r(1, 2) for _ in range(nsp)]
        dl = [self.r(1, 2) for _ in range(nsp)]
        pd = [self.r(0, k[i] // 2) for i in range(nsp)]
        lead = len(s) - nsp
        out_sp = [(s[lead + i] + 2 * pd[i] - dl[i] * (k[i] - 1) - 1) // st[i] + 1 for i in range(nsp)]
        if min(out_sp) < 1 or numel(s[:lead] + out_sp) > MAX_NUMEL:
            return None
        return self.op(self.pick(["max_pool", "avg_pool"]), [t], s[:lead] + out_sp, kernel=k, stride=st, pad=pd,
                       dilation=dl)

    def reduce(self, t):
        s = self.shapes[t]
        dims = sorted(set(int(d) for d in self.rng.choice(len(s), self.r(1, len(s)), replace=False)))
        keep = self.r(0, 1)
        out = [1 if d in dims else s[d] for d in range(len(s))] if keep else [s[d] for d in range(len(s))
                                                                             if d not in dims]
        if not out:
            out = [1]
        neg = [d - len(s) if self.rng.random() < 0.3 else d for d in dims]
        return self.op(self.pick(REDUCE), [t], out, dims=neg, keepdim=keep)

    def softmax(self, t):
        s = self.shapes[t]
        d = self.r(0, len(s) - 1)
        return self.op(self.pick(["softmax", "log_softmax"]), [t], s, dim=d - len(s) if self.rng.random() < 0.3 else d)

    def norm(self, t):
        s = self.shapes[t]
        kind = self.pick(["group_norm", "batch_norm", "layer_norm"])
        if kind != "layer_norm" and len(s) < 2:
            kind = "layer_norm"
        affine = self.rng.random() < 0.5
        if kind == "group_norm":
            attrs = dict(groups=self.pick([g for g in range(1, s[1] + 1) if s[1] % g == 0]))
            aff = [s[1]]
        elif kind == "batch_norm":
            attrs, aff = {}, [s[1]]
        else:
            nd = self.r(1, len(s))
            attrs, aff = dict(ndims=nd), s[len(s) - nd:]
        ops = [t] + ([self.leaf(aff), self.leaf(aff)] if affine else [])
        return self.op(kind, ops, s, **attrs)

    def channel_affine(self, t):
        s = self.shapes[t]
        if len(s) < 2:
            return None
        return self.op("channel_affine", [t, self.leaf([s[1]]), self.leaf([s[1]])], s)

    def slice(self, t):
        s = self.shapes[t]
        d = self.r(0, len(s) - 1)
        n = s[d]
        start = self.r(0, n - 1)
        end = self.r(start + 1, n)
        step = self.r(1, 3)
        out = list(s)
        out[d] = (end - start + step - 1) // step
        return self.op("slice", [t], out, dim=d, start=start, end=end, step=step)

    def permute(self, t):
        s = self.shapes[t]
        p = [int(x) for x in self.rng.permutation(len(s))]
        return self.op("permute", [t], [s[i] for i in p], dims=p)

    def reshape(self, t):
        s = self.shapes[t]
        n = numel(s)
        for _ in range(20):
            out = _random_factorisation(n, self.rng)
            if _refinable(s, out):
                return self.op("reshape", [t], out, shape=out)
        return None

    def expand(self, t):
        s = self.shapes[t]
        out = list(s)
        ones = [d for d in range(len(s)) if s[d] == 1]
        if ones and self.rng.random() < 0.6:
            out[self.pick(ones)] = self.r(2, 3)
        elif len(s) < 4:
            out = [self.r(2, 3)] + out
        if numel(out) > MAX_NUMEL:
            return None
        return self.op("expand", [t], out, shape=out)

    def gather(self, t):
        s = self.shapes[t]
        R = self.r(1, 3)
        out = [self.r(1, 5) for _ in range(R)]
        Q = self.r(0, 2)
        win = [self.r(1, 3) for _ in range(Q)]
        idx = []
        for d in range(len(s)):
            parts = []
            if self.rng.random() < 0.8:
                parts.append(f"{self.pick([1, 1, 2, -1])}*o{self.r(0, R - 1)}")
            if Q and self.rng.random() < 0.6:
                parts.append(f"{self.pick([1, -1, 2])}*w{self.r(0, Q - 1)}")
            parts.append(str(self.r(-1, 2)))
            e = "+".join(parts).replace("+-", "-")
            mode = self.rng.random()
            if mode < 0.15:
                e = f"({e})/{self.r(2, 3)}"
            elif mode < 0.3:
                e = f"({e})//{self.r(2, 3)}"
            idx.append(e)
        attrs = dict(shape=out, idx0=idx, mult=[self.r(1, 3)])
        if Q:
            attrs["window"] = win
            wn = numel(win)
            if self.rng.random() < 0.4:
                lo = self.r(0, wn - 1)
                attrs["flat"] = [lo, self.r(lo, wn)]
        return self.op("affine_gather", [t], out, **attrs)


def _random_factorisation(n, rng):
    """A shape of 1 to 4 dims with product n (unit dims sometimes)."""
    fs = []
    m = n
    p = 2
    while p * p <= m:
        while m % p == 0:
            fs.append(p)
            m //= p
        p += 1
    if m > 1:
        fs.append(m)
    rng.shuffle(fs)
    k = int(rng.integers(1, 5))
    dims = [1] * k
    for f in fs:
        dims[int(rng.integers(0, k))] *= f
    if rng.random() < 0.2:
        dims.insert(int(rng.integers(0, k + 1)), 1)
    return dims[:4] if len(dims) > 4 and dims[4:] == [1] * (len(dims) - 4) else dims


def _refinable(a, b):
    """Whether the strides of the non-unit dims of a and b form one
    divisibility chain (a common refinement of the two factorisations)."""
    def strides(s):
        out, st = [], 1
        for d in reversed([d for d in s if d != 1]):
            out.append(st)
            st *= d
        return out, st
    sa, n = strides(a)
    sb, _ = strides(b)
    chain = sorted(set(sa + sb + [1, n]))
    return all(chain[i] % chain[i - 1] == 0 for i in range(1, len(chain)))


def random_graph(seed: int) -> str:
    """dgir text of one random graph (see the module docstring)."""
    G = _Gen(seed)
    rank = G.r(1, 4)
    shape = [G.r(1, 4) for _ in range(rank)]
    if rank >= 3 and G.rng.random() < 0.7:
        shape[1] = G.pick([2, 3, 4])  # a channel dim worth grouping
    t = G.leaf(shape)
    steps = G.r(1, 4)
    kinds = ["unary", "binary", "matmul", "linear", "conv", "conv_t", "pool", "reduce", "softmax", "norm",
             "channel_affine", "slice", "permute", "reshape", "expand", "gather"]
    done = 0
    tries = 0
    while done < steps and tries < 40:
        tries += 1
        k = G.pick(kinds)
        f = {"conv": lambda x: G.conv(x, False), "conv_t": lambda x: G.conv(x, True)}.get(k) or getattr(G, k)
        nt = f(t)
        if nt is None or numel(G.shapes[nt]) > MAX_NUMEL:
            continue
        t = nt
        done += 1
    for name, kind, operands, attrs in G.ops:
        G.g.op(name, kind, *operands, **attrs)
    G.g.output(t, G.shapes[t])
    return G.g.text()


# What the library may refuse (DG_E_UNSUPPORTED_OP) among these graphs: a
# merged index with more than four terms, a reshape whose two shapes have no
# common refinement.
REFUSALS = ("more than 4 terms", "no common refinement")


def squared_variant(text: str) -> str:
    """The same graph with its output multiplied by itself: same footprint,
    every count doubled."""
    lines = text.strip().split("\n")
    _, name, shape = lines[-1].split()
    return "\n".join(lines[:-1] + [f"op zz mul {name} {name}", f"output zz {shape}"]) + "\n"
