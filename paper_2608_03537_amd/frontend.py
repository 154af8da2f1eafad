"""Frontend: lowers a PyTorch GEMM + epilogue function to the fused node list.

The compilation stack of Sec. V, for this library's compiled vocabulary:

  capture   The function (one matrix product followed by memory-bound work)
            is traced to an ATen graph with LayerNorm, RMSNorm and softmax
            decomposed into their reductions and element-wise parts
            (torch.fx make_fx).
  Phi       (Sec. V-B) A top-down walk from the matrix-product node builds the
            Fusion Spec IR S = <N, E, tau, A, C>: the product becomes the
            accumulator entry, Python constants scalar broadcasts, 1-D
            placeholders row-vector broadcasts registered as runtime
            parameters (2-D ones full-tile operands), arithmetic binaries and
            unary functions compute nodes, and row reductions reduction nodes.
            Every reduction splits the graph (Sec. V-C): the nodes after it
            form a nested spec entered through the reduction's statistic and
            the pass-through tensor it reduced.  Anything else is outside the
            domain of Phi and is reported, never dropped.
  lower     The place of Psi (Sec. V-D).  There is no template renderer here:
            the kernels are compiled ahead of time, so the spec is matched,
            from its terminal node inwards, against the node grammar of
            cf_gemm_subgraph ([SCALE] [BIAS] [RESIDUAL] [LAYERNORM | RMSNORM]
            [GELU | GELU_TANH | RELU | SOFTCAP] [SOFTMAX] STORE
            [ROWAMAX_QUANT]).  A spec that matches nothing is reported as
            unsupported.

A function returns the stored tensor z, or a tuple holding z and the row
quantisation tail of the LN -> GELU -> amax chain: the scale
s = amax(|z|, -1, keepdim) / qmax and/or the codes (z / s).to(float8_e4m3fn)
(ROWAMAX_QUANT, Sec. III-B).  The amax is taken over the fp32 z before its
rounding to the output dtype, and a row whose amax is 0 gets s = 0 and codes
0, where eager PyTorch would divide by zero.

`compile_epilogue(fn)` returns a callable that runs the fused kernel.  A
function outside the domain raises `UnsupportedEpilogue` with the reason; only
with `fallback=True` does it return an explicitly marked (`fused` is False)
callable that runs the function eagerly in PyTorch, which is the standard
compilation pathway the paper falls back to.
"""
from __future__ import annotations

import math
import operator
import warnings
from dataclasses import dataclass, field

from . import comfuse as cf


class UnsupportedEpilogue(ValueError):
    """The function is outside the domain of the frontend (reason in args[0])."""


# ---------------------------------------------------------------------------
# Fusion Spec IR
# ---------------------------------------------------------------------------
@dataclass
class SpecNode:
    """One node of the Fusion Spec IR.

    kind: "acc" (the matrix product), "const" (scalar broadcast), "row"
    (row-vector broadcast of a 1-D runtime parameter), "tile" (a full M x N
    runtime parameter), "compute" (element-wise op) or "reduce" (row
    reduction; op "sum", "mean", "amax" or "var_mean", the last with two
    results read through "item").
    """
    idx: int
    kind: str
    op: str = ""
    inputs: tuple = ()
    value: float = 0.0
    param: str = ""
    attrs: dict = field(default_factory=dict)


@dataclass
class FusionSpec:
    """S = <N, E, tau, A, C> of Sec. V-B.

    nodes     N, topologically ordered (inputs before users).
    edges     E, (producer, consumer) index pairs.
    terminal  tau, the index of the node whose value is stored.
    params    A, runtime parameter name -> (role, argument position); roles
              "row" (1-D, broadcast over rows) and "tile" (M x N).
    nested    C, one entry per reduction: the nested spec it roots, as
              {"reduce": index, "stat": index of the statistic node(s),
               "passthrough": index of the reduced tensor,
               "nodes": indices of the nodes that depend on the statistic}.
    w_layout  layout of the weight operand (cf.CF_LAYOUT_NK or _KN);
    x_arg, w_arg: argument positions of the product's operands;
    outputs   the function's results in order (one entry: the terminal).
    """
    nodes: list
    edges: list
    terminal: int
    params: dict
    nested: list
    w_layout: int
    x_arg: int
    w_arg: int
    outputs: list = field(default_factory=list)


# ---------------------------------------------------------------------------
# Capture
# ---------------------------------------------------------------------------
def _aten():
    import torch
    return torch.ops.aten


def capture(fn, example_args):
    """ATen graph of fn(*example_args) with the row operators decomposed."""
    import torch
    from torch._decomp import get_decompositions
    from torch.fx.experimental.proxy_tensor import make_fx
    aten = torch.ops.aten
    table = get_decompositions([aten.native_layer_norm, aten.layer_norm, aten._softmax, aten.softmax,
                                aten.rms_norm, aten._fused_rms_norm, aten.linear, aten.t, aten.addmm,
                                aten.matmul])
    return make_fx(fn, decomposition_table=table)(*example_args)


# ---------------------------------------------------------------------------
# Phi: graph -> FusionSpec
# ---------------------------------------------------------------------------
def _is_last_dim(dims, ndim=2):
    dims = list(dims) if isinstance(dims, (list, tuple)) else [dims]
    return len(dims) == 1 and dims[0] in (-1, ndim - 1)


def phi(gm) -> FusionSpec:
    aten = _aten()
    graph = gm.graph
    placeholders = [n for n in graph.nodes if n.op == "placeholder"]
    pos = {n: i for i, n in enumerate(placeholders)}

    def meta_rank(n):
        v = n.meta.get("val")
        return None if v is None else v.dim()

    mms = [n for n in graph.nodes if n.op == "call_function" and n.target in (aten.mm.default, aten.addmm.default)]
    if len(mms) != 1:
        raise UnsupportedEpilogue(f"expected one matrix product, found {len(mms)}")
    mm = mms[0]
    if mm.target == aten.addmm.default:
        bias_node, a, b = mm.args[0], mm.args[1], mm.args[2]
    else:
        bias_node, (a, b) = None, mm.args[:2]
    if a.op != "placeholder" or meta_rank(a) != 2:
        raise UnsupportedEpilogue("the product's left operand must be a 2-D function argument")
    if b.op == "placeholder":
        w_layout, w = cf.CF_LAYOUT_KN, b
    elif (b.op == "call_function" and b.target in (aten.t.default, aten.transpose.int, aten.permute.default)
          and b.args[0].op == "placeholder"):
        if b.target == aten.transpose.int and sorted(b.args[1:3]) not in ([0, 1], [-2, -1], [-1, 0]):
            raise UnsupportedEpilogue("the weight transpose must swap its two dimensions")
        if b.target == aten.permute.default and list(b.args[1]) != [1, 0]:
            raise UnsupportedEpilogue("the weight permutation must swap its two dimensions")
        w_layout, w = cf.CF_LAYOUT_NK, b.args[0]
    else:
        raise UnsupportedEpilogue("the product's right operand must be a function argument or its transpose")

    nodes, ids = [], {}

    def new(kind, **kw):
        sn = SpecNode(idx=len(nodes), kind=kind, **kw)
        nodes.append(sn)
        return sn.idx

    params = {}

    def operand(v):
        """Spec index of an argument value: a derived node, a constant or a parameter."""
        if isinstance(v, (int, float)) and not isinstance(v, bool):
            return new("const", value=float(v))
        if hasattr(v, "op"):
            if v in ids:
                return ids[v]
            if v.op == "placeholder":
                r = meta_rank(v)
                role = "row" if r == 1 else "tile" if r == 2 else None
                if role is None:
                    raise UnsupportedEpilogue(f"argument {v.target} has rank {r}; only 1-D and 2-D operands broadcast")
                params[v.target] = (role, pos[v])
                ids[v] = new(role, param=v.target)
                return ids[v]
        raise UnsupportedEpilogue(f"operand {v!r} is neither a constant, an argument nor a derived value")

    acc = new("acc")
    ids[mm] = acc
    if bias_node is not None:   # addmm: the product plus a broadcast row vector
        bidx = operand(bias_node)
        if nodes[bidx].kind != "row":
            raise UnsupportedEpilogue("the fused bias of a linear layer must be a 1-D argument")
        ids[mm] = new("compute", op="add", inputs=(acc, bidx))

    binary = {aten.add.Tensor: "add", aten.add_.Tensor: "add", aten.add.Scalar: "add", aten.add_.Scalar: "add",
              aten.sub.Tensor: "sub", aten.sub.Scalar: "sub", aten.mul.Tensor: "mul", aten.mul.Scalar: "mul",
              aten.mul_.Tensor: "mul", aten.div.Tensor: "div", aten.div.Scalar: "div"}
    unary = {aten.tanh.default: "tanh", aten.exp.default: "exp", aten.relu.default: "relu",
             aten.rsqrt.default: "rsqrt", aten.sqrt.default: "sqrt", aten.neg.default: "neg",
             aten.gelu.default: "gelu", aten.reciprocal.default: "reciprocal", aten.abs.default: "abs"}
    import torch
    fp8 = getattr(torch, "float8_e4m3fn", None)
    output = None
    for n in graph.nodes:
        if n.op == "output":
            output = n.args[0]
            continue
        if n.op != "call_function" or n is mm or n is w or n in ids:
            continue
        if n is b and w_layout == cf.CF_LAYOUT_NK:
            continue
        t = n.target
        if t in binary:
            x, y = n.args[0], n.args[1]
            alpha = n.kwargs.get("alpha", 1)
            if alpha != 1:
                raise UnsupportedEpilogue("add/sub with alpha is outside the pattern set")
            op = binary[t]
            unit = 1.0 if op in ("mul", "div") else 0.0   # x * 1, x / 1, x + 0, x - 0 are x
            if isinstance(y, (int, float)) and float(y) == unit:
                ids[n] = operand(x)
            elif op in ("mul", "add") and isinstance(x, (int, float)) and float(x) == unit:
                ids[n] = operand(y)
            else:
                ids[n] = new("compute", op=op, inputs=(operand(x), operand(y)))
        elif t == aten.pow.Tensor_Scalar and n.args[1] == 2:
            xi = operand(n.args[0])
            ids[n] = new("compute", op="mul", inputs=(xi, xi))
        elif t in unary:
            attrs = {}
            if t == aten.gelu.default:
                attrs["approximate"] = n.kwargs.get("approximate", "none")
            ids[n] = new("compute", op=unary[t], inputs=(operand(n.args[0]),), attrs=attrs)
        elif t in (aten.sum.dim_IntList, aten.mean.dim, aten.amax.default):
            dims = n.args[1] if len(n.args) > 1 else n.kwargs.get("dim")
            keep = n.args[2] if len(n.args) > 2 else n.kwargs.get("keepdim", False)
            if not _is_last_dim(dims) or not keep:
                raise UnsupportedEpilogue(f"{t} must reduce the last dimension with keepdim")
            op = {aten.sum.dim_IntList: "sum", aten.mean.dim: "mean", aten.amax.default: "amax"}[t]
            ids[n] = new("reduce", op=op, inputs=(operand(n.args[0]),))
        elif t == aten.var_mean.correction:
            dims = n.args[1] if len(n.args) > 1 else n.kwargs.get("dim")
            if not _is_last_dim(dims) or not n.kwargs.get("keepdim", False) or n.kwargs.get("correction", 1) != 0:
                raise UnsupportedEpilogue("var_mean must be the biased variance over the last dimension")
            ids[n] = new("reduce", op="var_mean", inputs=(operand(n.args[0]),))
        elif t == operator.getitem and n.args[0] in ids and nodes[ids[n.args[0]]].op == "var_mean":
            ids[n] = new("compute", op="item", inputs=(ids[n.args[0]],), attrs={"i": n.args[1]})
        elif t in (aten.detach.default, aten.clone.default, aten.alias.default):
            ids[n] = operand(n.args[0])
        elif t == aten._to_copy.default and set(n.kwargs) <= {"dtype", "layout", "device"}:
            # dtype conversions of derived values: the epilogue computes in fp32
            # and rounds once at the store
            if not (hasattr(n.args[0], "op") and n.args[0] in ids):
                raise UnsupportedEpilogue("only derived values may be converted")
            if fp8 is not None and n.kwargs.get("dtype") == fp8:
                ids[n] = new("compute", op="e4m3", inputs=(ids[n.args[0]],))   # E4M3 codes
            else:
                ids[n] = ids[n.args[0]]
        else:
            raise UnsupportedEpilogue(f"{t} is outside the pattern set")
    outs = list(output) if isinstance(output, (tuple, list)) else [output]
    if not outs or any(not hasattr(o, "op") or o not in ids for o in outs):
        raise UnsupportedEpilogue("the function must return tensors derived from the product")
    # the stored value: the one result that is neither codes nor a row statistic
    main = [o for o in outs if nodes[ids[o]].op != "e4m3" and
            not (o.meta.get("val") is not None and o.meta["val"].dim() == 2 and o.meta["val"].shape[-1] == 1
                 and meta_rank(o) == 2 and len(outs) > 1)]
    if len(main) != 1:
        raise UnsupportedEpilogue("the function must return one stored tensor (plus, optionally, its row "
                                  "quantisation scale and codes)")
    output = main[0]
    edges = [(i, sn.idx) for sn in nodes for i in sn.inputs]
    users = {}
    for p_, c_ in edges:
        users.setdefault(p_, set()).add(c_)
    nested = []
    for sn in nodes:
        if sn.kind != "reduce":
            continue
        stat = [sn.idx] + [u for u in users.get(sn.idx, ()) if nodes[u].op == "item"]
        seen, todo = set(), list(stat)
        while todo:
            k = todo.pop()
            for u in users.get(k, ()):
                if u not in seen:
                    seen.add(u)
                    todo.append(u)
        nested.append({"reduce": sn.idx, "stat": stat, "passthrough": sn.inputs[0], "nodes": sorted(seen)})
    return FusionSpec(nodes=nodes, edges=edges, terminal=ids[output], params=params, nested=nested,
                      w_layout=w_layout, x_arg=pos[a], w_arg=pos[w], outputs=[ids[o] for o in outs])


# ---------------------------------------------------------------------------
# Lowering: FusionSpec -> node-list template
# ---------------------------------------------------------------------------
@dataclass
class NodeTemplate:
    """A cf_node with runtime parameters still named (bound at call time)."""
    kind: int
    f0: float = 0.0
    v0: str = ""      # parameter names
    v1: str = ""
    inp: str = ""


def _close(a, b, rtol=1e-6):
    return abs(a - b) <= rtol * max(abs(a), abs(b))


class _Matcher:
    def __init__(self, spec: FusionSpec):
        self.s = spec
        self.n = spec.nodes

    def node(self, i):
        return self.n[i]

    def is_op(self, i, op):
        return self.n[i].kind == "compute" and self.n[i].op == op

    def const(self, i):
        return self.n[i].value if self.n[i].kind == "const" else None

    def role(self, i):
        return self.n[i].kind if self.n[i].kind in ("row", "tile") else None

    def scaled(self, i):
        """(x, c) if node i is x * c, c * x or x / c with a constant c, else None."""
        nd = self.n[i]
        if nd.kind != "compute" or nd.op not in ("mul", "div"):
            return None
        a, b = nd.inputs
        if nd.op == "mul":
            if self.const(b) is not None:
                return a, self.const(b)
            if self.const(a) is not None:
                return b, self.const(a)
        elif self.const(b) is not None and self.const(b) != 0.0:
            return a, 1.0 / self.const(b)
        return None

    def commuted(self, i, op):
        """The two inputs of an op node, in both orders."""
        if not self.is_op(i, op):
            return []
        a, b = self.n[i].inputs
        return [(a, b), (b, a)] if op in ("add", "mul") else [(a, b)]

    # -- softmax: exp(x - amax(x)) / sum(exp(x - amax(x)))
    def softmax(self, t):
        for e, s in self.commuted(t, "div"):
            if not (self.is_op(e, "exp") and self.n[s].kind == "reduce" and self.n[s].op == "sum"
                    and self.n[s].inputs[0] == e):
                continue
            d = self.n[e].inputs[0]
            if not self.is_op(d, "sub"):
                continue
            x, m = self.n[d].inputs
            if self.n[m].kind == "reduce" and self.n[m].op == "amax" and self.n[m].inputs[0] == x:
                return x
        return None

    # -- activations
    def activation(self, t):
        nd = self.n[t]
        if self.is_op(t, "relu"):
            return nd.inputs[0], NodeTemplate(cf.CF_N_RELU)
        if self.is_op(t, "gelu"):
            kind = cf.CF_N_GELU if nd.attrs.get("approximate", "none") == "none" else cf.CF_N_GELU_TANH
            return nd.inputs[0], NodeTemplate(kind)
        sc = self.scaled(t)   # cap * tanh(x / cap)
        if sc is not None and self.is_op(sc[0], "tanh"):
            inner = self.scaled(self.n[sc[0]].inputs[0])
            cap = sc[1]
            if inner is not None and cap > 0 and math.isfinite(cap) and _close(inner[1], 1.0 / cap):
                return inner[0], NodeTemplate(cf.CF_N_SOFTCAP, f0=cap)
        return None

    def rsqrt_eps(self, i):
        """(v, eps) if node i is rsqrt(v + eps) or 1 / sqrt(v + eps), else None."""
        if self.is_op(i, "rsqrt"):
            arg = self.n[i].inputs[0]
        elif self.is_op(i, "reciprocal") and self.is_op(self.n[i].inputs[0], "sqrt"):
            arg = self.n[self.n[i].inputs[0]].inputs[0]
        else:
            return None
        for v, e in self.commuted(arg, "add"):
            if self.const(e) is not None and self.const(e) >= 0:
                return v, self.const(e)
        return None

    def ln_stats(self, var_node, mean_node):
        """x if (var_node, mean_node) are the biased variance and the mean of x."""
        vn, mn = self.n[var_node], self.n[mean_node]
        if vn.op == "item" and mn.op == "item" and vn.inputs == mn.inputs and vn.attrs["i"] == 0 \
                and mn.attrs["i"] == 1:
            return self.n[vn.inputs[0]].inputs[0]
        # explicit: mean(x); var = mean((x - mean(x))^2)
        if mn.kind == "reduce" and mn.op == "mean" and vn.kind == "reduce" and vn.op == "mean":
            x = mn.inputs[0]
            sq = vn.inputs[0]
            if self.is_op(sq, "mul"):
                a, b = self.n[sq].inputs
                if a == b and self.is_op(a, "sub") and self.n[a].inputs == (x, mean_node):
                    return x
        return None

    # -- LayerNorm core: (x - mean) * rsqrt(var + eps), or (x - mean) / sqrt(var + eps)
    def ln_core(self, t):
        cands = [(d, r) for d, r in self.commuted(t, "mul")]
        if self.is_op(t, "div"):
            d, s = self.n[t].inputs
            if self.is_op(s, "sqrt"):
                for v, e in self.commuted(self.n[s].inputs[0], "add"):
                    if self.const(e) is not None and self.is_op(d, "sub"):
                        x, m = self.n[d].inputs
                        if self.ln_stats(v, m) == x:
                            return x, self.const(e)
        for d, r in cands:
            if not self.is_op(d, "sub"):
                continue
            re = self.rsqrt_eps(r)
            if re is None:
                continue
            x, m = self.n[d].inputs
            if self.ln_stats(re[0], m) == x:
                return x, re[1]
        return None

    # -- RMSNorm core: x * rsqrt(mean(x * x) + eps)
    def rms_core(self, t):
        for x, r in self.commuted(t, "mul"):
            re = self.rsqrt_eps(r)
            if re is None:
                continue
            ms = self.n[re[0]]
            if ms.kind == "reduce" and ms.op == "mean" and self.is_op(ms.inputs[0], "mul") \
                    and self.n[ms.inputs[0]].inputs == (x, x):
                return x, re[1]
        return None

    def norm(self, t):
        """(x, template) if node t is LayerNorm / RMSNorm of x with optional row affine."""
        beta, g, core = "", "", t
        for c, b in self.commuted(t, "add"):
            if self.role(b) == "row":
                beta, core = self.n[b].param, c
                break
        for c, gg in self.commuted(core, "mul"):
            if self.role(gg) == "row":
                g, core2 = self.n[gg].param, c
                ln = self.ln_core(core2)
                rms = self.rms_core(core2)
                if ln or rms:
                    core = core2
                    break
                g = ""
        ln = self.ln_core(core)
        if ln is not None:
            return ln[0], NodeTemplate(cf.CF_N_LAYERNORM, f0=ln[1], v0=g, v1=beta)
        rms = self.rms_core(core)
        if rms is not None and not beta:
            return rms[0], NodeTemplate(cf.CF_N_RMSNORM, f0=rms[1], v0=g)
        return None


def quant_tail(spec: FusionSpec):
    """(qmax, roles) for the results beside the stored tensor, or None when
    the function returns only it.  roles[i] is "z", "s" or "q" for result i:
    s = amax(|z|) / qmax (row statistic), q = e4m3(z / s)."""
    outs = spec.outputs or [spec.terminal]
    if len(outs) == 1:
        return None
    m = _Matcher(spec)
    z = spec.terminal

    def scale_of(i):   # qmax if node i is amax(|z|) / qmax (or * 1/qmax)
        sc = m.scaled(i)
        if sc is None or not (sc[1] > 0 and math.isfinite(sc[1])):
            return None
        r = m.node(sc[0])
        if r.kind == "reduce" and r.op == "amax" and m.is_op(r.inputs[0], "abs") and m.node(r.inputs[0]).inputs[0] == z:
            return 1.0 / sc[1]
        return None

    roles, qmax, s_node = [], None, None
    for o in outs:
        if o == z:
            roles.append("z")
            continue
        if m.is_op(o, "e4m3"):
            d = m.node(o).inputs[0]
            q_s = None
            if m.is_op(d, "div") and m.node(d).inputs[0] == z:
                q_s = m.node(d).inputs[1]
            elif m.is_op(d, "mul"):
                for zz, rcp in m.commuted(d, "mul"):
                    if zz == z and m.is_op(rcp, "reciprocal"):
                        q_s = m.node(rcp).inputs[0]
            if q_s is None or scale_of(q_s) is None:
                raise UnsupportedEpilogue("codes must be (z / s).to(float8_e4m3fn) with s = amax(|z|) / qmax")
            if s_node is not None and s_node != q_s:
                raise UnsupportedEpilogue("the codes and the returned scale use different scales")
            s_node, qmax = q_s, scale_of(q_s)
            roles.append("q")
            continue
        if scale_of(o) is not None:
            if s_node is not None and s_node != o:
                raise UnsupportedEpilogue("the codes and the returned scale use different scales")
            s_node, qmax = o, scale_of(o)
            roles.append("s")
            continue
        raise UnsupportedEpilogue("a second result must be the row scale amax(|z|) / qmax or the E4M3 codes")
    if roles.count("z") != 1 or roles.count("s") > 1 or roles.count("q") > 1:
        raise UnsupportedEpilogue("results: the stored tensor once, the scale and the codes at most once each")
    return qmax, roles


def lower(spec: FusionSpec) -> list:
    """Node-list template for spec (without the STORE; a row quantisation tail
    comes last, after the place of the STORE), or UnsupportedEpilogue."""
    tail = quant_tail(spec)
    out = _lower_main(spec)
    if tail is not None:
        out.append(NodeTemplate(cf.CF_N_ROWAMAX_QUANT, f0=tail[0]))
    return out


def _lower_main(spec: FusionSpec) -> list:
    m = _Matcher(spec)
    out = []
    t = spec.terminal
    sm = m.softmax(t)
    if sm is not None:
        out.append(NodeTemplate(cf.CF_N_SOFTMAX))
        t = sm
    act = m.activation(t)
    if act is not None:
        out.append(act[1])
        t = act[0]
    nrm = m.norm(t)
    if nrm is not None:
        if sm is not None:
            raise UnsupportedEpilogue("a normalisation followed by softmax is outside the node grammar")
        out.append(nrm[1])
        t = nrm[0]
    seen = set()
    while True:   # additive broadcasts in any order: bias (row) and residual (tile), once each
        step = None
        for x, p in m.commuted(t, "add"):
            r = m.role(p)
            if r in ("row", "tile") and r not in seen:
                step = (x, r, m.node(p).param)
                break
        if step is None:
            break
        seen.add(step[1])
        out.append(NodeTemplate(cf.CF_N_BIAS, v0=step[2]) if step[1] == "row"
                   else NodeTemplate(cf.CF_N_RESIDUAL, inp=step[2]))
        t = step[0]
    sc = m.scaled(t)
    if sc is not None:
        out.append(NodeTemplate(cf.CF_N_SCALE, f0=sc[1]))
        t = sc[0]
    if m.node(t).kind != "acc":
        nd = m.node(t)
        raise UnsupportedEpilogue(f"no rule of the node grammar matches the subgraph at node {t} "
                                  f"({nd.kind} {nd.op})")
    rank = {cf.CF_N_SCALE: 0, cf.CF_N_BIAS: 1, cf.CF_N_RESIDUAL: 2}
    out.reverse()
    out.sort(key=lambda n: rank.get(n.kind, 10))   # stable: only the additive pair can swap
    return out


# ---------------------------------------------------------------------------
# Compiled epilogue
# ---------------------------------------------------------------------------
class FusedGemmEpilogue:
    """fn(*args) as one fused GEMM + row-subgraph launch.

    `spec` is the Fusion Spec IR, `templates` the lowered node list, `fused`
    is True.  Arguments are the function's own; the output is bf16 for bf16
    operands and fp32 for fp32 ones (out_dtype overrides).
    """
    fused = True

    def __init__(self, spec, templates, out_dtype=None, path=cf.PATH_AUTO):
        self.spec, self.templates, self.out_dtype, self.path = spec, templates, out_dtype, path
        tail = quant_tail(spec)
        self.roles = tail[1] if tail is not None else None

    def node_kinds(self):
        k = [t.kind for t in self.templates if t.kind != cf.CF_N_ROWAMAX_QUANT] + [cf.CF_N_STORE]
        return k + [t.kind for t in self.templates if t.kind == cf.CF_N_ROWAMAX_QUANT]

    def __call__(self, *args, out=None, ws=None, stream=None):
        torch = cf._torch()
        X, W = args[self.spec.x_arg], args[self.spec.w_arg]
        M = X.shape[0]
        N = W.shape[0] if self.spec.w_layout == cf.CF_LAYOUT_NK else W.shape[1]
        names = {name: args[p] for name, (_, p) in self.spec.params.items()}
        Y = out if out is not None else torch.empty((M, N), dtype=self.out_dtype or X.dtype, device=X.device)
        spec, quant = [], None
        for t in self.templates:
            if t.kind == cf.CF_N_ROWAMAX_QUANT:
                quant = t
                continue
            d = dict(kind=t.kind, f0=t.f0)
            if t.v0:
                d["v0"] = names[t.v0]
            if t.v1:
                d["v1"] = names[t.v1]
            if t.inp:
                r = names[t.inp]
                if r.dtype != X.dtype:
                    raise UnsupportedEpilogue("the residual operand must have the product's input dtype")
                d.update({"in": r, "ld": cf._ld(r), "dtype": cf._dt(r)})
            for k in ("v0", "v1"):
                if k in d and (d[k].dtype != torch.float32 or d[k].dim() != 1 or d[k].shape[0] != N):
                    raise UnsupportedEpilogue("row-vector operands must be fp32 [N]")
            spec.append(d)
        spec.append(dict(kind=cf.CF_N_STORE, out=Y, ld=cf._ld(Y), dtype=cf._dt(Y)))
        if quant is None:
            cf.gemm_subgraph(X, W, spec, w_layout=self.spec.w_layout, path=self.path, ws=ws, stream=stream)
            return Y
        # the row scale (fp32 [M], returned as [M, 1]) and the codes (bytes,
        # returned as float8_e4m3fn)
        s = torch.empty(M, dtype=torch.float32, device=X.device)
        Q = torch.empty((M, N), dtype=torch.uint8, device=X.device) if "q" in self.roles else None
        spec.append(dict(kind=cf.CF_N_ROWAMAX_QUANT, out=s, out2=Q, ld=N if Q is not None else 0, f0=quant.f0))
        cf.gemm_subgraph(X, W, spec, w_layout=self.spec.w_layout, path=self.path, ws=ws, stream=stream)
        res = {"z": Y, "s": s.view(M, 1), "q": Q.view(torch.float8_e4m3fn) if Q is not None else None}
        return tuple(res[r] for r in self.roles)


class EagerEpilogue:
    """The fallback pathway: fn run eagerly by PyTorch (`fused` is False)."""
    fused = False

    def __init__(self, fn, reason):
        self.fn, self.reason = fn, reason

    def __call__(self, *args, **kw):
        return self.fn(*args)


def compile_epilogue(fn, example_args, *, fallback=False, out_dtype=None, path=cf.PATH_AUTO):
    """Capture fn on example_args (any device, small shapes suffice: only the
    ranks and the graph matter), map it to the Fusion Spec IR and lower it.

    Returns FusedGemmEpilogue, or with fallback=True an EagerEpilogue when the
    function is outside the domain (a warning names the reason); raises
    UnsupportedEpilogue otherwise.
    """
    try:
        spec = phi(capture(fn, example_args))
        return FusedGemmEpilogue(spec, lower(spec), out_dtype=out_dtype, path=path)
    except UnsupportedEpilogue as e:
        if not fallback:
            raise
        warnings.warn(f"epilogue not fused, running it eagerly: {e}", RuntimeWarning, stacklevel=2)
        return EagerEpilogue(fn, str(e))
