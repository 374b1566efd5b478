"""Evaluate dgir graphs with real PyTorch CPU ops (float64).

Two evaluators, both independent of the oracle's read loops:

* ``evaluate(text, leaves)`` runs the program itself with PyTorch's own
  operators, so perturbing one leaf element and watching which outputs move
  gives the semantic footprint (a subset of the syntactic one).
* ``linearised(text, leaves)`` replaces every op by the sum of the elements
  it reads (each read once per occurrence), built from PyTorch ops that carry
  PyTorch's own index semantics (stride, padding, dilation, output padding,
  groups, broadcasting).  The result is linear in the leaves and the gradient
  of output element l with respect to leaf element i is the number of
  occurrences of i in res(y[l]) (Sec. 3.4, "Back-projection").  Softmax and
  the normalisations are linearised through their primitive decompositions
  (exp / sum / div; mean / sub / square / mean / rsqrt / mul / add), so their
  multiplicities are derived here rather than restated.
"""

from __future__ import annotations

import itertools
import math
import re

import torch
import torch.nn.functional as F


def parse(text: str):
    leaves, ops, output = [], [], None
    for raw in text.splitlines():
        line = raw.split("#")[0].strip()
        if not line or line.startswith("dgir"):
            continue
        toks = line.split()
        if toks[0] == "leaf":
            leaves.append((toks[1], [int(v) for v in toks[2].split(",")]))
        elif toks[0] == "op":
            name, kind = toks[1], toks[2]
            rest = toks[3:]
            operands, attrs = [], {}
            if ";" in rest:
                i = rest.index(";")
                operands, kv = rest[:i], rest[i + 1:]
            else:
                operands, kv = rest, []
            for item in kv:
                k, v = item.split("=", 1)
                attrs[k] = v.split(",")
            ops.append((name, kind, operands, attrs))
        elif toks[0] == "output":
            output = toks[1]
    return leaves, ops, output


def _ints(attrs, key, default=None):
    if key not in attrs:
        return default
    return [int(v) for v in attrs[key]]


def _int(attrs, key, default=None):
    v = _ints(attrs, key)
    return default if v is None else v[0]


_UNARY = {
    "relu": torch.relu, "gelu": F.gelu, "gelu_tanh": lambda x: F.gelu(x, approximate="tanh"),
    "hardtanh": F.hardtanh, "clamp": lambda x: torch.clamp(x, -1.0, 1.0), "sigmoid": torch.sigmoid,
    "tanh": torch.tanh, "exp": torch.exp, "log": lambda x: torch.log(x.abs() + 1.0),
    "log1p": lambda x: torch.log1p(x.abs()), "square": torch.square, "sqrt": lambda x: torch.sqrt(x.abs() + 1.0),
    "rsqrt": lambda x: torch.rsqrt(x.abs() + 1.0), "neg": torch.neg, "abs": torch.abs,
    "identity": lambda x: x, "contiguous": lambda x: x.contiguous(), "silu": F.silu,
    "softplus": F.softplus, "erf": torch.erf, "scale": lambda x: 0.5 * x, "leaky_relu": F.leaky_relu,
    "elu": F.elu, "reciprocal": lambda x: 1.0 / (x.abs() + 1.0),
}
_BINARY = {
    "add": torch.add, "sub": torch.sub, "mul": torch.mul,
    "div": lambda a, b: a / (b.abs() + 1.0) * torch.sign(b + 1e-300),
    "maximum": torch.maximum, "minimum": torch.minimum,
    "pow": lambda a, b: (a.abs() + 1.0) ** b,
}


# ---- affine_gather: forward simulation of the custom kernel -------------
_TERM = re.compile(r"([+-]?)(?:(\d+)\*)?(o\d+|w\d+|\d+)")


def _parse_expr(s: str):
    div, mode = 1, 0
    m = re.fullmatch(r"\((.*)\)(//|/)(\d+)", s)
    if m:
        s, mode, div = m.group(1), (2 if m.group(2) == "//" else 1), int(m.group(3))
    terms, const = [], 0
    pos = 0
    while pos < len(s):
        mm = _TERM.match(s, pos)
        if not mm or mm.end() == pos:
            raise ValueError(f"bad expression {s!r}")
        sign = -1 if mm.group(1) == "-" else 1
        coef = int(mm.group(2)) if mm.group(2) else 1
        tok = mm.group(3)
        if tok[0] in "ow":
            terms.append((tok[0], int(tok[1:]), sign * coef))
        else:
            const += sign * int(tok)
        pos = mm.end()
    return terms, const, mode, div


def _gather(ins, attrs, linear: bool):
    shape = _ints(attrs, "shape")
    window = _ints(attrs, "window", [])
    wn = math.prod(window) if window else 1
    lo, hi = _ints(attrs, "flat", [0, wn])
    mult = _ints(attrs, "mult", [1] * len(ins))
    exprs = [[_parse_expr(e) for e in attrs[f"idx{j}"]] for j in range(len(ins))]
    out = torch.zeros(shape, dtype=torch.float64)
    # Index grids over (output, window-flat) pairs.
    o_grid = torch.stack(torch.meshgrid(*[torch.arange(s) for s in shape], indexing="ij"), dim=-1).reshape(-1, len(shape))
    wflat = torch.arange(lo, hi)
    wcoords = []
    rem = wflat.clone()
    for e in reversed(window):
        wcoords.append(rem % e)
        rem = rem // e
    wcoords = list(reversed(wcoords))
    P = o_grid.shape[0]
    Q = len(wflat)
    acc = torch.zeros(P, dtype=torch.float64) if not linear else torch.zeros(P, dtype=torch.float64)
    valid = torch.ones(P, Q, dtype=torch.bool)
    flats = []
    for j, x in enumerate(ins):
        flat = torch.zeros(P, Q, dtype=torch.int64)
        for d, (terms, const, mode, div) in enumerate(exprs[j]):
            v = torch.full((P, Q), const, dtype=torch.int64)
            for var, k, c in terms:
                if var == "o":
                    v = v + c * o_grid[:, k].unsqueeze(1)
                else:
                    v = v + c * wcoords[k].unsqueeze(0)
            if mode == 1:
                valid &= (v % div) == 0
                v = torch.div(v, div, rounding_mode="floor")
            elif mode == 2:
                v = torch.div(v, div, rounding_mode="floor")
            valid &= (v >= 0) & (v < x.shape[d])
            flat = flat * x.shape[d] + v.clamp(0, x.shape[d] - 1)
        flats.append(flat)
    if linear:
        for j, x in enumerate(ins):
            vals = x.reshape(-1)[flats[j]]
            acc = acc + (mult[j] * vals * valid).sum(dim=1)
    else:
        prod = torch.ones(P, Q, dtype=torch.float64)
        for j, x in enumerate(ins):
            prod = prod * x.reshape(-1)[flats[j]] ** mult[j]
        acc = (prod * valid).sum(dim=1)
    return acc.reshape(shape)


def _conv_fn(nsp, transpose):
    if transpose:
        return {1: F.conv_transpose1d, 2: F.conv_transpose2d, 3: F.conv_transpose3d}[nsp]
    return {1: F.conv1d, 2: F.conv2d, 3: F.conv3d}[nsp]


def _sum_pool(x, ks, st, pd, dl):
    nsp = len(ks)
    lead = x.shape[: x.dim() - nsp]
    C = math.prod(lead[1:]) if len(lead) > 1 else 1
    N = lead[0] if lead else 1
    xr = x.reshape(N, C, *x.shape[x.dim() - nsp:])
    w = torch.ones(C, 1, *ks, dtype=x.dtype)
    y = _conv_fn(nsp, False)(xr, w, None, stride=st, padding=pd, dilation=dl, groups=C)
    return y.reshape(*lead, *y.shape[2:])


def _norm_sets(kind, attrs, x):
    """Returns (sum_S(t) broadcast back to t's shape) as a function, and the
    per-element affine index view of gamma/beta."""
    if kind == "group_norm":
        G = _int(attrs, "groups")
        N = x.shape[0]

        def sum_s(t):
            r = t.reshape(N, G, -1).sum(-1, keepdim=True)
            return r.expand(N, G, t.numel() // (N * G)).reshape(t.shape)

        def aff(p):
            return p.reshape(1, -1, *([1] * (x.dim() - 2)))
    elif kind == "batch_norm":
        dims = [0] + list(range(2, x.dim()))

        def sum_s(t):
            return t.sum(dim=dims, keepdim=True).expand(t.shape)

        def aff(p):
            return p.reshape(1, -1, *([1] * (x.dim() - 2)))
    else:
        k = _int(attrs, "ndims", 1)
        dims = list(range(x.dim() - k, x.dim()))

        def sum_s(t):
            return t.sum(dim=dims, keepdim=True).expand(t.shape)

        def aff(p):
            return p
    return sum_s, aff


def _run(text: str, leaves: dict, linear: bool, every: bool = False):
    _, ops, output = parse(text)
    env = dict(leaves)
    for name, kind, operands, attrs in ops:
        ins = [env[o] for o in operands]
        x = ins[0]
        if kind in _UNARY:
            y = x if linear else _UNARY[kind](x)
        elif kind in _BINARY:
            y = ins[0] + ins[1] if linear else _BINARY[kind](ins[0], ins[1])
        elif kind == "matmul":
            a, b = ins
            y = a @ torch.ones_like(b) + torch.ones_like(a) @ b if linear else a @ b
        elif kind == "linear":
            w = ins[1]
            b = ins[2] if len(ins) == 3 else None
            if linear:
                y = F.linear(x, torch.ones_like(w)) + F.linear(torch.ones_like(x), w)
                if b is not None:
                    y = y + b
            else:
                y = F.linear(x, w, b)
        elif kind in ("conv", "conv_transpose"):
            w = ins[1]
            b = ins[2] if len(ins) == 3 else None
            nsp = x.dim() - 2
            kw = dict(stride=_ints(attrs, "stride", [1] * nsp), padding=_ints(attrs, "pad", [0] * nsp),
                      dilation=_ints(attrs, "dilation", [1] * nsp), groups=_int(attrs, "groups", 1))
            if kind == "conv_transpose":
                kw["output_padding"] = _ints(attrs, "output_padding", [0] * nsp)
            fn = _conv_fn(nsp, kind == "conv_transpose")
            if linear:
                y = fn(x, torch.ones_like(w), None, **kw) + fn(torch.ones_like(x), w, None, **kw)
                if b is not None:
                    y = y + b.reshape(1, -1, *([1] * nsp))
            else:
                y = fn(x, w, b, **kw)
        elif kind in ("max_pool", "avg_pool"):
            ks = _ints(attrs, "kernel")
            st = _ints(attrs, "stride", ks)
            pd = _ints(attrs, "pad", [0] * len(ks))
            dl = _ints(attrs, "dilation", [1] * len(ks))
            if linear:
                y = _sum_pool(x, ks, st, pd, dl)
            elif kind == "max_pool":
                nsp = len(ks)
                fn = {1: F.max_pool1d, 2: F.max_pool2d, 3: F.max_pool3d}[nsp]
                y = fn(x, ks, st, pd, dl)
            else:
                # Mean over the in-range window elements (padding excluded).
                y = _sum_pool(x, ks, st, pd, dl) / _sum_pool(torch.ones_like(x), ks, st, pd, dl)
        elif kind in ("sum", "mean", "amax", "amin", "prod", "max", "min"):
            dims = _ints(attrs, "dims")
            keep = bool(_int(attrs, "keepdim", 0))
            if linear or kind == "sum":
                y = x.sum(dim=dims, keepdim=keep)
            elif kind == "mean":
                y = x.mean(dim=dims, keepdim=keep)
            elif kind in ("amax", "max"):
                y = x.amax(dim=dims, keepdim=keep)
            elif kind in ("amin", "min"):
                y = x.amin(dim=dims, keepdim=keep)
            else:
                y = x
                for d in sorted([d % x.dim() for d in dims], reverse=True):
                    y = y.prod(dim=d, keepdim=keep)
            if y.dim() == 0:
                y = y.reshape(1)
        elif kind in ("softmax", "log_softmax"):
            dim = _int(attrs, "dim")
            if linear:
                e = x                                   # exp(x): reads x
                s = e.sum(dim=dim, keepdim=True)        # sum over the slice
                y = e + s                               # exp(x) / sum: reads both
            else:
                y = torch.softmax(x, dim) if kind == "softmax" else torch.log_softmax(x, dim)
        elif kind in ("group_norm", "batch_norm", "layer_norm"):
            g = ins[1] if len(ins) == 3 else None
            b = ins[2] if len(ins) == 3 else None
            if linear:
                sum_s, aff = _norm_sets(kind, attrs, x)
                mu = sum_s(x)              # mean_S(x)
                d = x + mu                 # x - mu
                sq = d                     # square(d)
                v = sum_s(sq)              # mean_S(square(d))
                r = v                      # rsqrt(v + eps)
                y = d + r                  # d * r
                if g is not None:
                    y = y + aff(g)         # * gamma
                    y = y + aff(b)         # + beta
            elif kind == "group_norm":
                y = F.group_norm(x, _int(attrs, "groups"), g, b)
            elif kind == "batch_norm":
                y = F.batch_norm(x, None, None, g, b, training=True)
            else:
                k = _int(attrs, "ndims", 1)
                y = F.layer_norm(x, list(x.shape[x.dim() - k:]), g, b)
        elif kind == "channel_affine":
            s, t = ins[1], ins[2]
            shp = (1, -1) + (1,) * (x.dim() - 2)
            y = x + s.reshape(shp) + t.reshape(shp) if linear else x * s.reshape(shp) + t.reshape(shp)
        elif kind == "slice":
            dim = _int(attrs, "dim")
            n = x.shape[dim]
            start = _int(attrs, "start", 0)
            end = _int(attrs, "end", n)
            step = _int(attrs, "step", 1)
            sl = [slice(None)] * x.dim()
            sl[dim] = slice(start, end, step)
            y = x[tuple(sl)]
        elif kind == "permute":
            y = x.permute(*_ints(attrs, "dims"))
        elif kind == "reshape":
            y = x.reshape(_ints(attrs, "shape"))
        elif kind == "expand":
            y = x.expand(*_ints(attrs, "shape"))
        elif kind == "affine_gather":
            y = _gather(ins, attrs, linear)
        else:
            raise NotImplementedError(kind)
        env[name] = y
    return env if every else env[output]


def evaluate(text: str, leaves: dict) -> torch.Tensor:
    return _run(text, leaves, linear=False)


def evaluate_all(text: str, leaves: dict) -> dict:
    """Every tensor of the program (leaves and op outputs) by name."""
    return _run(text, leaves, linear=False, every=True)


def linearised(text: str, leaves: dict) -> torch.Tensor:
    return _run(text, leaves, linear=True)


def leaf_shapes(text: str):
    return parse(text)[0]


def path_counts(text: str, locs):
    """{loc: {global id: count}} from autograd of the linearised graph."""
    shapes = leaf_shapes(text)
    leaves = {n: torch.ones(s, dtype=torch.float64, requires_grad=True) for n, s in shapes}
    y = linearised(text, leaves).reshape(-1)
    out = {}
    for loc in locs:
        grads = torch.autograd.grad(y[loc], [leaves[n] for n, _ in shapes], retain_graph=True, allow_unused=True)
        row = {}
        base = 0
        for (n, s), g in zip(shapes, grads):
            if g is not None:
                flat = g.reshape(-1)
                nz = torch.nonzero(flat).reshape(-1)
                for i in nz.tolist():
                    v = flat[i].item()
                    assert v == round(v) and v > 0
                    row[base + i] = int(round(v))
            base += math.prod(s)
        out[loc] = row
    return out


def perturbation_footprints(text: str, draws: int = 3, deltas=(0.5, -0.5, 10.0, -10.0), seed: int = 0):
    """{loc: set of global ids} whose perturbation moves output l in at least
    one (draw, delta) pair: the semantic footprint."""
    shapes = leaf_shapes(text)
    gen = torch.Generator().manual_seed(seed)
    touched = None
    for _ in range(draws):
        base_vals = {n: torch.randn(s, dtype=torch.float64, generator=gen) for n, s in shapes}
        y0 = evaluate(text, base_vals).reshape(-1)
        if touched is None:
            touched = [set() for _ in range(y0.numel())]
        gid = 0
        for n, s in shapes:
            flat = base_vals[n].reshape(-1)
            for i in range(flat.numel()):
                for dlt in deltas:
                    pert = dict(base_vals)
                    t = flat.clone()
                    t[i] += dlt
                    pert[n] = t.reshape(s)
                    y = evaluate(text, pert).reshape(-1)
                    moved = (y - y0).abs() > 1e-9 * (1.0 + y0.abs())
                    for loc in torch.nonzero(moved).reshape(-1).tolist():
                        touched[loc].add(gid + i)
            gid += flat.numel()
    return {loc: s for loc, s in enumerate(touched)}
