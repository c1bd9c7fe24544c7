"""Front end: Logical SDQLite programs over one sparse matrix, differentiated
and lowered to the library's kernels.

Pipeline (Sections 3-5 of the paper, without equality saturation):
  1. parse the program (the Logical SDQLite grammar of Section 3);
  2. normalize it into sums of products of reals: every term is
     "sum over index variables of coef * product of tensor entries", with
     tensor-valued products expanded into explicit loops (the multiplication
     normalization rules of Section 5) and the iteration domain of a sparse
     loop kept as a mask (the stored keys it runs over);  `let`-bound tensors
     stay named intermediates, and a `let` of a real inside loops becomes a
     tensor over the loop indices it depends on (an ANF-style binding,
     Section 5.1);
  3. differentiate with the tensorized forward-mode rules (Section 4.2): the
     tangent of a product is the sum over its factors (product rule), the
     tangent of a lookup is the lookup of the tangent, a `let` binds its
     tangent beside it, and the gradient API seeds the input of interest with
     its one-hot tensor and every other input with zero (Section 4.3);
  4. propagate sparsity: products with a zero tangent vanish, sums with zero
     drop it, and equal terms merge (the first group of transformations of
     Section 5.2);
  5. lower each remaining term to one kernel of the library: SpMM / SpMV,
     the transposed product, SDDMM on the matrix's pattern, a dense dot
     product, or an axpby; the terms of one result accumulate in place.

All arithmetic runs in the library's kernels; this module only builds and
dispatches the calls.  Programs outside this class (two sparse iterations in
one term, `if`, `op`, products of tensors laid out differently) raise
`NotLowerable` with the reason.
"""
from __future__ import annotations

import itertools
import re
from dataclasses import dataclass, field, replace

# ------------------------------------------------------------------ errors


class SdqlError(Exception):
    """Malformed program (syntax, names, types or shapes)."""


class NotLowerable(SdqlError):
    """Well-formed program that the kernels here do not cover."""


# ------------------------------------------------------------ declarations


@dataclass(frozen=True)
class Sparse:
    """A sparse matrix input (CSR; its stored keys are the iteration domain)."""

    nrows: int
    ncols: int

    @property
    def shape(self):
        return (self.nrows, self.ncols)


@dataclass(frozen=True)
class SparseVec:
    """A sparse vector input (its stored keys are its iteration domain)."""

    n: int

    @property
    def shape(self):
        return (self.n,)


@dataclass(frozen=True)
class Dense:
    """A dense input: a real (no shape), a vector or a matrix (row-major)."""

    shape: tuple

    def __init__(self, *shape):
        object.__setattr__(self, "shape", tuple(int(s) for s in shape))


# ------------------------------------------------------------------ syntax


@dataclass(frozen=True)
class Num:
    value: float


@dataclass(frozen=True)
class Name:
    name: str


@dataclass(frozen=True)
class SumE:
    key: str
    val: str
    src: object
    body: object


@dataclass(frozen=True)
class Single:
    key: object
    val: object


@dataclass(frozen=True)
class EmptyE:
    pass


@dataclass(frozen=True)
class Lookup:
    dict: object
    key: object


@dataclass(frozen=True)
class LetE:
    name: str
    bound: object
    body: object


@dataclass(frozen=True)
class AddE:
    left: object
    right: object


@dataclass(frozen=True)
class MulE:
    left: object
    right: object


@dataclass(frozen=True)
class Other:
    """`if`, `not`, `=`, `true`/`false` and real unary operations: parsed,
    outside the sum-of-products class."""

    what: str
    args: tuple


_LEX = re.compile(r"\s+|(?P<num>\d*\.\d+(?:[eE][-+]?\d+)?|\d+\.?(?:[eE][-+]?\d+)?)"
                  r"|(?P<id>[A-Za-z_][\w']*)|(?P<op>->|[-+*=(){}<>,])")
_RESERVED = ("sum", "in", "let", "if", "then", "not", "true", "false")
_UNARY_OPS = ("exp", "log", "sin", "cos", "sqrt")


def _lex(text):
    toks, pos = [], 0
    while pos < len(text):
        m = _LEX.match(text, pos)
        if m is None:
            raise SdqlError(f"unexpected character {text[pos]!r} at offset {pos}")
        pos = m.end()
        if m.lastgroup == "num":
            toks.append(("num", m.group("num")))
        elif m.lastgroup == "id":
            w = m.group("id")
            toks.append((w if w in _RESERVED else "id", w))
        elif m.lastgroup == "op":
            toks.append((m.group("op"), m.group("op")))
    toks.append(("eof", ""))
    return toks


class _Reader:
    # Binding strength, loosest first: the greedy forms (sum, let, if),
    # equality, +, *, prefix (not, unary minus), postfix lookup, atoms.
    def __init__(self, text):
        self.toks = _lex(text)
        self.pos = 0

    def kind(self, off=0):
        return self.toks[self.pos + off][0]

    def eat(self, kind):
        k, v = self.toks[self.pos]
        if k != kind:
            raise SdqlError(f"expected {kind!r} but found {v or k!r} at token {self.pos}")
        self.pos += 1
        return v

    def parse(self):
        e = self.greedy()
        self.eat("eof")
        return e

    def greedy(self):
        k = self.kind()
        if k == "sum":
            self.eat("sum")
            self.eat("(")
            self.eat("<")
            key = self.eat("id")
            self.eat(",")
            val = self.eat("id")
            self.eat(">")
            self.eat("in")
            src = self.greedy()
            self.eat(")")
            return SumE(key, val, src, self.greedy())
        if k == "let":
            self.eat("let")
            name = self.eat("id")
            self.eat("=")
            bound = self.greedy()
            self.eat("in")
            return LetE(name, bound, self.greedy())
        if k == "if":
            self.eat("if")
            cond = self.greedy()
            self.eat("then")
            return Other("if", (cond, self.greedy()))
        return self.equality()

    def equality(self):
        e = self.plus()
        while self.kind() == "=":
            self.eat("=")
            e = Other("eq", (e, self.plus()))
        return e

    def plus(self):
        e = self.times()
        while self.kind() == "+":
            self.eat("+")
            e = AddE(e, self.times())
        return e

    def times(self):
        e = self.prefix()
        while self.kind() == "*":
            self.eat("*")
            e = MulE(e, self.prefix())
        return e

    def prefix(self):
        k = self.kind()
        if k in ("sum", "let", "if"):
            return self.greedy()
        if k == "not":
            self.eat("not")
            return Other("not", (self.prefix(),))
        if k == "-":
            self.eat("-")
            return MulE(Num(-1.0), self.prefix())
        return self.postfix()

    def postfix(self):
        e = self.atom()
        while self.kind() == "(":
            self.eat("(")
            key = self.greedy()
            self.eat(")")
            e = Lookup(e, key)
        return e

    def atom(self):
        k = self.kind()
        if k == "num":
            return Num(float(self.eat("num")))
        if k in ("true", "false"):
            self.eat(k)
            return Other(k, ())
        if k == "id":
            name = self.eat("id")
            if name in _UNARY_OPS and self.kind() == "(":
                self.eat("(")
                arg = self.greedy()
                self.eat(")")
                return Other(name, (arg,))
            return Name(name)
        if k == "(":
            self.eat("(")
            e = self.greedy()
            self.eat(")")
            return e
        if k == "{":
            self.eat("{")
            if self.kind() == "}":
                self.eat("}")
                return EmptyE()
            key = self.greedy()
            self.eat("->")
            val = self.greedy()
            self.eat("}")
            return Single(key, val)
        raise SdqlError(f"unexpected {self.toks[self.pos][1] or k!r} at token {self.pos}")


def parse(text: str):
    """Syntax tree of a Logical SDQLite program."""
    return _Reader(text).parse()


# ----------------------------------------------------------- sum-of-products


@dataclass(frozen=True)
class Fac:
    """Entry `tensor[idx]` of a named tensor, idx a tuple of index variables."""

    tensor: str
    idx: tuple


@dataclass(frozen=True)
class Term:
    """coef * sum over `loops` of the product of `facs`, restricted to the
    stored keys named by `masks`, as the entry at `keys` (output position p
    is the index variable keys[p])."""

    coef: float
    keys: tuple
    loops: frozenset
    facs: tuple
    masks: tuple = ()

    def variables(self):
        vs = set(self.keys) | set(self.loops)
        for f in self.facs + self.masks:
            vs.update(f.idx)
        return vs

    def rename(self, sub):
        def r(v):
            return sub.get(v, v)

        return Term(self.coef, tuple(r(v) for v in self.keys),
                    frozenset(r(v) for v in self.loops),
                    tuple(Fac(f.tensor, tuple(r(v) for v in f.idx)) for f in self.facs),
                    tuple(Fac(m.tensor, tuple(r(v) for v in m.idx)) for m in self.masks))


@dataclass
class Terms:
    """A tensor of the given order as a sum of terms."""

    order: int | None
    terms: list


@dataclass(frozen=True)
class Access:
    """A named tensor looked up at a prefix of its keys."""

    tensor: str
    idx: tuple


@dataclass
class TensorInfo:
    name: str
    kind: str            # "sparse" (input), "dense", "patterned" (on the sparse input's keys), "scalar"
    shape: tuple
    pattern: str | None = None
    definition: Terms | None = None   # intermediates only
    deps: tuple = ()                  # enclosing loop variables a hoisted let depends on

    @property
    def order(self):
        return len(self.shape)

    @property
    def input(self):
        return self.definition is None


@dataclass
class _Bind:
    kind: str            # "index", "access", "terms"
    value: object


class Program:
    """A compiled program: its value as terms, its intermediates, and the
    gradients of the gradient API on request."""

    def __init__(self, text: str, decls: dict):
        self.text = text
        self.tensors: dict[str, TensorInfo] = {}
        self.extent: dict[str, int] = {}
        self._counter = itertools.count()
        self._tangents: dict = {}
        sparse = [n for n, d in decls.items() if isinstance(d, Sparse)]
        if len(sparse) > 1:
            raise NotLowerable(f"one sparse matrix per program, got {sparse}")
        for name, d in decls.items():
            if isinstance(d, (Sparse, SparseVec)):
                self.tensors[name] = TensorInfo(name, "sparse", d.shape, pattern=name)
            elif isinstance(d, Dense):
                if len(d.shape) > 2:
                    raise NotLowerable(f"dense input {name} must have order 0, 1 or 2")
                self.tensors[name] = TensorInfo(name, "dense" if d.shape else "scalar", d.shape)
            else:
                raise SdqlError(f"declaration of {name} must be Sparse, SparseVec or Dense")
        self.sparse = sparse[0] if sparse else None
        self.inputs = dict(decls)
        env = {n: _Bind("access", Access(n, ())) for n in decls}
        self.value = self._as_terms(self._extract(parse(text), env, ()))
        self.value.terms = _simplify(self.value.terms, self.tensors)

    # -- naming
    def _fresh(self, base):
        return f"{base}#{next(self._counter)}"

    def _set_extent(self, var, n, where):
        old = self.extent.get(var)
        if old is not None and old != n:
            raise SdqlError(f"index {var.split('#')[0]} ranges over {old} and {n} ({where})")
        self.extent[var] = n

    def _is_sparse(self, tensor):
        return self.tensors[tensor].kind in ("sparse", "patterned")

    # -- step 2: normalization into sums of products
    def _as_terms(self, x):
        if isinstance(x, Terms):
            return x
        info = self.tensors[x.tensor]
        rest = []
        for pos in range(len(x.idx), info.order):
            v = self._fresh("k")
            self._set_extent(v, info.shape[pos], f"{x.tensor} at position {pos}")
            rest.append(v)
        idx = x.idx + tuple(rest)
        masks = (Fac(info.pattern, idx),) if self._is_sparse(x.tensor) else ()
        if info.kind == "scalar":
            return Terms(0, [Term(1.0, (), frozenset(), (Fac(x.tensor, ()),))])
        return Terms(len(rest), [Term(1.0, tuple(rest), frozenset(), (Fac(x.tensor, idx),),
                                      masks)])

    def _extract(self, e, env, loops):
        """Access or Terms for expression e; `loops` lists the enclosing
        sparse/dense iterations as (variable, tensor, prefix) triples."""
        if isinstance(e, Num):
            return Terms(0, [Term(float(e.value), (), frozenset(), ())])
        if isinstance(e, Name):
            b = env.get(e.name)
            if b is None:
                raise SdqlError(f"unbound name {e.name}")
            if b.kind == "index":
                raise NotLowerable(f"index {e.name} used as a real")
            if b.kind == "access":
                return b.value
            return Terms(b.value.order, [_fresh_loops(t, self) for t in b.value.terms])
        if isinstance(e, Lookup):
            d = self._extract(e.dict, env, loops)
            if not isinstance(d, Access):
                raise NotLowerable("lookup into a computed expression; bind it with let first")
            info = self.tensors[d.tensor]
            if len(d.idx) >= info.order:
                raise SdqlError(f"too many lookups into {d.tensor}")
            var = self._index(e.key, env)
            self._set_extent(var, info.shape[len(d.idx)], f"lookup into {d.tensor}")
            return Access(d.tensor, d.idx + (var,))
        if isinstance(e, Single):
            var = self._index(e.key, env)
            v = self._as_terms(self._extract(e.val, env, loops))
            return Terms(v.order + 1 if v.order is not None else None,
                         [replace(t, keys=(var,) + t.keys) for t in v.terms])
        if isinstance(e, EmptyE):
            return Terms(None, [])
        if isinstance(e, AddE):
            a = self._as_terms(self._extract(e.left, env, loops))
            b = self._as_terms(self._extract(e.right, env, loops))
            if a.order is not None and b.order is not None and a.order != b.order:
                raise SdqlError(f"adding tensors of orders {a.order} and {b.order}")
            return Terms(a.order if a.order is not None else b.order, a.terms + b.terms)
        if isinstance(e, MulE):
            a = self._as_terms(self._extract(e.left, env, loops))
            b = self._as_terms(self._extract(e.right, env, loops))
            out = []
            for s in a.terms:
                for t in b.terms:
                    t = _fresh_loops(t, self)
                    out.append(Term(s.coef * t.coef, s.keys + t.keys, s.loops | t.loops,
                                    s.facs + t.facs, s.masks + t.masks))
            order = None if a.order is None or b.order is None else a.order + b.order
            return Terms(order, out)
        if isinstance(e, SumE):
            src = self._extract(e.src, env, loops)
            if not isinstance(src, Access):
                raise NotLowerable("sum over a computed expression; bind it with let first")
            info = self.tensors[src.tensor]
            level = len(src.idx)
            if level >= info.order:
                raise SdqlError(f"sum over a real ({src.tensor} fully looked up)")
            var = self._fresh(e.key)
            self._set_extent(var, info.shape[level], f"sum over {src.tensor}")
            inner = dict(env)
            inner[e.key] = _Bind("index", var)
            inner[e.val] = _Bind("access", Access(src.tensor, src.idx + (var,)))
            body = self._as_terms(self._extract(e.body, inner, loops + ((var, src),)))
            mask = (Fac(info.pattern, src.idx + (var,)),) if self._is_sparse(src.tensor) else ()
            out = [Term(t.coef, t.keys, t.loops if var in t.keys else t.loops | {var}, t.facs,
                        t.masks + mask) for t in body.terms]
            return Terms(body.order, out)
        if isinstance(e, LetE):
            bound = self._extract(e.bound, env, loops)
            inner = dict(env)
            if isinstance(bound, Access):
                inner[e.name] = _Bind("access", bound)
            elif all(not t.facs and not t.keys and not t.masks and not t.loops
                     for t in bound.terms):
                inner[e.name] = _Bind("terms", bound)      # a constant: substituted
            else:
                inner[e.name] = _Bind("access", self._hoist(e.name, bound, loops))
            return self._extract(e.body, inner, loops)
        if isinstance(e, Other):
            raise NotLowerable(f"`{e.what}` is outside the sum-of-products class")
        raise SdqlError(f"unknown expression {e!r}")

    def _index(self, e, env):
        if not isinstance(e, Name) or e.name not in env or env[e.name].kind != "index":
            raise NotLowerable("dictionary keys and lookups must be loop indices")
        return env[e.name].value

    def _hoist(self, name, bound: Terms, loops):
        """Named intermediate for `let name = bound`: a tensor over the
        enclosing loop variables the bound expression uses, then its own keys."""
        used = set()
        for t in bound.terms:
            used |= t.variables() - set(t.loops) - set(t.keys)
        deps = tuple(v for v, _ in loops if v in used)
        terms = []
        for t in bound.terms:
            masks = t.masks
            # the domain of the enclosing sparse iteration, when the
            # intermediate spans all of that iteration's keys
            for v, src in loops:
                info = self.tensors[src.tensor]
                full = src.idx + (v,)
                if (self._is_sparse(src.tensor) and len(full) == info.order
                        and all(u in deps for u in full)):
                    masks = masks + (Fac(info.pattern, full),)
            terms.append(Term(t.coef, deps + t.keys, t.loops, t.facs, masks))
        keys_order = len(deps) + (bound.order or 0)
        inter = self._fresh(name).replace("#", "%")
        shape = tuple(self.extent[v] for v in deps)
        if bound.terms:
            shape = shape + tuple(self.extent[v] for v in bound.terms[0].keys)
        terms = _simplify(terms, self.tensors)
        kind, pattern = "dense", None
        if keys_order == 0:
            kind = "scalar"
        else:
            # on the stored keys of one sparse input: a value array aligned with them
            for P in self.inputs:
                pinfo = self.tensors[P]
                if pinfo.kind == "sparse" and pinfo.order == keys_order and terms and all(
                        any(m.tensor == P and m.idx == t.keys for m in t.masks)
                        for t in terms):
                    kind, pattern = "patterned", P
                    break
        self.tensors[inter] = TensorInfo(inter, kind, shape, pattern=pattern,
                                         definition=Terms(keys_order, terms), deps=deps)
        return Access(inter, deps)

    # -- step 3: tensorized forward mode with the gradient API's seeds
    def depends(self, tensor, x):
        info = self.tensors[tensor]
        if tensor == x:
            return True
        if info.input:
            return False
        return any(self.depends(f.tensor, x) for t in info.definition.terms for f in t.facs)

    def tangent(self, T: Terms, x: str, seed: str | None = None) -> Terms:
        """Tangent of T when the input x is seeded and every other input gets
        the zero tangent.  With seed None, x's tangent is its one-hot tensor
        (the gradient API of Section 4.3): the result has order T.order +
        order(x), x's keys after T's, and for a tensor-valued T it is the
        Jacobian.  With seed the name of a tangent input of x's layout (from
        seed_of), the result is the directional derivative along it, of T's
        order (the forward mode of Section 4.1)."""
        xinfo = self.tensors[x]
        out = []
        for t in T.terms:
            for p, f in enumerate(t.facs):
                rest = t.facs[:p] + t.facs[p + 1:]
                if f.tensor == x:
                    if seed is not None:
                        out.append(Term(t.coef, t.keys, t.loops, rest + (Fac(seed, f.idx),),
                                        t.masks))
                        continue
                    # x'(idx) is the one-hot tensor: 1 at the key idx, on x's
                    # stored keys only
                    masks = t.masks + ((Fac(xinfo.pattern, f.idx),)
                                       if self._is_sparse(x) else ())
                    out.append(Term(t.coef, t.keys + f.idx, t.loops - set(f.idx), rest, masks))
                elif not self.tensors[f.tensor].input and self.depends(f.tensor, x):
                    info = self.tensors[f.tensor]
                    dT = self._tangent_of(f.tensor, x, seed)
                    for s in dT.terms:
                        s = _fresh_all(s, self)
                        sub = {}
                        for kv, iv in zip(s.keys[:info.order], f.idx):
                            if sub.get(kv, iv) != iv:
                                raise NotLowerable(f"diagonal use of {info.name}")
                            sub[kv] = iv
                        s = s.rename(sub)
                        gkeys = s.keys[info.order:]
                        out.append(Term(t.coef * s.coef, t.keys + gkeys,
                                        (t.loops | s.loops) - set(gkeys), rest + s.facs,
                                        t.masks + s.masks))
        order = None if T.order is None else T.order + (0 if seed else xinfo.order)
        return Terms(order, _simplify(out, self.tensors))

    def _tangent_of(self, tensor, x, seed=None):
        key = (tensor, x, seed)
        if key not in self._tangents:
            self._tangents[key] = self.tangent(self.tensors[tensor].definition, x, seed)
        return self._tangents[key]

    def gradient(self, x: str) -> Terms:
        """`gradient e x` of the gradient API (Section 4.3): the program's
        derivative w.r.t. input x, as terms over x's keys; for a
        tensor-valued program, its Jacobian (the output's keys, then x's)."""
        if x not in self.inputs:
            raise SdqlError(f"{x} is not an input")
        return self.tangent(self.value, x)

    def seed_of(self, x: str) -> str:
        """Name of the tangent input of x: a tensor of x's layout (a value
        array on x's stored keys when x is sparse)."""
        if x not in self.inputs:
            raise SdqlError(f"{x} is not an input")
        name = x + "'"
        if name not in self.tensors:
            info = self.tensors[x]
            kind = {"sparse": "patterned"}.get(info.kind, info.kind)
            self.tensors[name] = TensorInfo(name, kind, info.shape, pattern=info.pattern)
        return name

    def jvp_terms(self, wrt) -> Terms:
        """The value's tangent along the tangents of the inputs in `wrt` (each
        the input seed_of(x)), summed over them: the total derivative along
        one direction, J v; a batch of directions is J V (Section 4.2)."""
        out = []
        for x in wrt:
            out += self.tangent(self.value, x, self.seed_of(x)).terms
        return Terms(self.value.order, _simplify(out, self.tensors))

    # -- step 5: lowering
    def plan(self, grads=(), value=True, fuse=True):
        """Kernel calls computing the value (when asked) and the gradients:
        one fused loss kernel when the whole program is one of the fused
        losses (and fuse is set), else one kernel per term."""
        if fuse:
            fused = _fused_plan(self, tuple(grads), value)
            if fused is not None:
                return fused
        return _Lowering(self).run(value, tuple(grads))

    def run(self, inputs: dict, grads=(), value=True, stream=None, fuse=True):
        """Executes the plan on device tensors: inputs maps a sparse matrix's
        name to a DeviceCsr, a sparse vector's to a DeviceSparseVec, a
        dense input's to a float32 tensor of its shape and a real's to a
        one-element float64 tensor.  Returns {"value": ..., "d<name>": ...};
        a result on an input's stored keys is a value array aligned with
        them (Plan.layout tells which keys)."""
        return self.plan(grads, value, fuse).execute(inputs, stream)

    def jvp_plan(self, wrt, fuse=True):
        """Kernel calls for the tangent along the inputs in `wrt` (see
        jvp_terms): one call for the whole batch when the program is a
        matrix product the batched tangent kernel covers (and fuse is set),
        else one pass of the term-by-term lowering per tangent."""
        wrt = tuple(wrt)
        for x in wrt:
            if x not in self.inputs:
                raise SdqlError(f"{x} is not an input")
        if fuse:
            fused = _fused_jvp_plan(self, wrt)
            if fused is not None:
                return fused
        plan = _Lowering(self).run_tangent(wrt)
        plan.per_tangent = True
        return plan

    def jvp(self, inputs: dict, tangents: dict, value=True, stream=None, fuse=True):
        """J V for a batch of m tangents: tangents maps input names to device
        tensors [m, *layout of the input] (a sparse input's tangent on its
        stored keys: [m, nnz]; a real's: [m] float64).  Returns {"value": ...
        (when asked), "tangent": [m, *layout of the value]}."""
        return _execute_jvp(self.jvp_plan(tuple(tangents), fuse), inputs, tangents, value,
                            stream)


def compile(text: str, **decls) -> Program:   # noqa: A001 - the natural name
    """Compiles a program; decls give each input as Sparse(...) or Dense(...)."""
    return Program(text, decls)


def _renamed(t: Term, prog, vs) -> Term:
    sub = {}
    for v in sorted(vs):
        sub[v] = prog._fresh(v.split("#")[0])
        prog.extent[sub[v]] = prog.extent[v]
    return t.rename(sub)


def _fresh_loops(t: Term, prog) -> Term:
    return _renamed(t, prog, t.loops)


def _fresh_all(t: Term, prog) -> Term:
    return _renamed(t, prog, t.variables())


# -------------------------------------------------- step 4: simplification


def _canonical(t: Term, tensors):
    """Term with masks completed and deduplicated, and a hashable form with
    its index variables renamed canonically, so that equal terms compare equal."""
    masks = list(dict.fromkeys(t.masks))
    for f in t.facs:   # a stored-keys-only factor is zero off its pattern
        info = tensors.get(f.tensor)
        if info and info.kind in ("sparse", "patterned") and len(f.idx) == info.order:
            m = Fac(info.pattern, f.idx)
            if m not in masks:
                masks.append(m)
    full = [m for m in masks if len(m.idx) == tensors[m.tensor].order]
    masks = [m for m in masks if m in full or not any(
        f.tensor == m.tensor and f.idx[:len(m.idx)] == m.idx for f in full)]
    t = Term(t.coef, t.keys, t.loops, t.facs, tuple(masks))
    names = {}
    for v in t.keys:
        names.setdefault(v, f"k{len(names)}")

    def sig(f):
        return (f.tensor, tuple(names.get(v, "?") for v in f.idx))

    for _ in range(2):
        for f in sorted(t.facs + t.masks, key=sig):
            for v in f.idx:
                names.setdefault(v, f"l{len(names)}")
    for v in sorted(t.loops):
        names.setdefault(v, f"l{len(names)}")
    c = t.rename(names)
    form = (c.keys, tuple(sorted(c.loops)), tuple(sorted((f.tensor, f.idx) for f in c.facs)),
            tuple(sorted((m.tensor, m.idx) for m in c.masks)))
    return t, form


def _simplify(terms, tensors):
    merged = {}
    for t in terms:
        if t.coef == 0.0:
            continue
        t, form = _canonical(t, tensors)
        if form in merged:
            old = merged[form]
            merged[form] = replace(old, coef=old.coef + t.coef)
        else:
            merged[form] = t
    return [t for t in merged.values() if t.coef != 0.0]


# ------------------------------------------------------------------ lowering


@dataclass
class Buf:
    """A device buffer of the plan: "input" (caller's), "out", "inter" or "temp".
    Layout "scalar" (one double), "pattern" (a float per stored key of the
    sparse input `pattern`; output key position p is that key's coordinate
    keymap[p]) or "dense" (float32 of `shape`)."""

    name: str
    role: str
    layout: str
    shape: tuple = ()
    pattern: str | None = None
    keymap: tuple = ()


@dataclass
class Call:
    kernel: str
    args: dict
    out: str


@dataclass
class Plan:
    prog: Program
    bufs: dict = field(default_factory=dict)
    calls: list = field(default_factory=list)
    results: dict = field(default_factory=dict)
    per_tangent: bool = False   # a tangent plan run once per tangent of a batch

    def kernels(self):
        return [c.kernel for c in self.calls]

    def layout(self, name):
        """(layout, pattern, keymap, shape) of a result."""
        b = self.bufs[name]
        return b.layout, b.pattern, b.keymap, b.shape

    def execute(self, inputs: dict, stream=None):
        return _execute(self, inputs, stream)


def _identity_map(n):
    return tuple(range(n))


class _Lowering:
    def __init__(self, prog: Program):
        self.p = prog
        self.plan = Plan(prog)
        self.done = set()
        self.ntemp = itertools.count()

    def _inputs(self):
        p = self.p
        for name, d in p.inputs.items():
            info = p.tensors[name]
            if info.kind == "sparse":
                self.plan.bufs[name] = Buf(name, "input", "pattern", d.shape, name,
                                           _identity_map(info.order))
            elif info.kind == "scalar":
                self.plan.bufs[name] = Buf(name, "input", "scalar")
            else:
                self.plan.bufs[name] = Buf(name, "input", "dense", d.shape)

    def run(self, value, grads):
        p = self.p
        self._inputs()
        if value:
            self._result("value", p.value, self._layout(p.value))
        for x in grads:
            g = p.gradient(x)
            info = p.tensors[x]
            if (p.value.order or 0) == 0:
                # the gradient of a real has x's own layout
                if info.kind == "sparse":
                    b = Buf("", "out", "pattern", info.shape, info.pattern,
                            _identity_map(info.order))
                elif info.kind == "scalar":
                    b = Buf("", "out", "scalar")
                else:
                    b = Buf("", "out", "dense", info.shape)
            else:
                b = self._layout(g, jacobian_of=x)
            self._result("d" + x, g, b)
        return self.plan

    def run_tangent(self, wrt):
        """The tangent along the inputs in wrt, for one tangent of each."""
        p = self.p
        self._inputs()
        T = p.jvp_terms(wrt)
        for x in wrt:
            s = p.seed_of(x)
            info = p.tensors[s]
            layout = {"patterned": "pattern", "scalar": "scalar"}.get(info.kind, "dense")
            self.plan.bufs[s] = Buf(s, "input", layout, info.shape, info.pattern,
                                    _identity_map(info.order) if info.pattern else ())
        # a tangent has the value's type, so the value's layout
        self._result("tangent", T, self._layout(p.value))
        return self.plan

    # -- result layouts
    def _layout(self, T, jacobian_of=None):
        """Layout of a result: on the stored keys of one sparse input when
        every term lies on them with the same key map (the Jacobians of the
        vector kernels, matrix-valued programs on a matrix's keys), a real
        for order 0, else dense."""
        p = self.p
        if not T.terms:
            if (T.order or 0) == 0:
                return Buf("", "out", "scalar")
            raise NotLowerable("a tensor-valued result with no terms (an empty Jacobian)")
        found = []
        for t in T.terms:
            full = [m for m in t.masks if len(m.idx) == p.tensors[m.tensor].order]
            on = None
            if len(full) == 1 and t.keys:
                m = full[0]
                if set(t.keys) == set(m.idx) and not set(t.keys) & set(t.loops):
                    if len(set(m.idx)) == len(m.idx):
                        on = (m.tensor, tuple(m.idx.index(v) for v in t.keys))
                    elif t.keys == m.idx:
                        # the diagonal keys (i, i) of a matrix, as its keys
                        on = (m.tensor, _identity_map(len(m.idx)))
            found.append(on)
        if all(f is not None and f == found[0] for f in found):
            P, keymap = found[0]
            shape = tuple(p.tensors[P].shape[i] for i in keymap)
            return Buf("", "out", "pattern", shape, P, keymap)
        keys = T.terms[0].keys
        if not keys:
            return Buf("", "out", "scalar")
        if len(keys) > 2:
            what = f"the Jacobian w.r.t. {jacobian_of}" if jacobian_of else "a result"
            raise NotLowerable(f"{what} has order {len(keys)} and is not on one input's "
                               "stored keys (its products with tangents are: jvp)")
        return Buf("", "out", "dense", tuple(p.extent[v] for v in keys))

    def _result(self, name, T, b: Buf):
        self.plan.bufs[name] = replace(b, name=name, role="out")
        self._emit_terms(T, name)
        self.plan.results[name] = name

    def _need(self, tensor):
        """Computes an intermediate (and what it needs) before its first use."""
        info = self.p.tensors[tensor]
        if info.input or tensor in self.done:
            return
        self.done.add(tensor)
        if info.kind == "scalar":
            self.plan.bufs[tensor] = Buf(tensor, "inter", "scalar")
        elif info.kind == "patterned":
            self.plan.bufs[tensor] = Buf(tensor, "inter", "pattern", info.shape, info.pattern,
                                         _identity_map(info.order))
        else:
            self.plan.bufs[tensor] = Buf(tensor, "inter", "dense", info.shape)
        self._emit_terms(info.definition, tensor)

    def _temp(self, like: Buf):
        name = f"tmp{next(self.ntemp)}"
        self.plan.bufs[name] = Buf(name, "temp", like.layout, like.shape, like.pattern,
                                   like.keymap)
        return name

    def _pattern_temp(self, P):
        info = self.p.tensors[P]
        return self._temp(Buf("", "temp", "pattern", info.shape, P, _identity_map(info.order)))

    def _emit_terms(self, T: Terms, out):
        for t in T.terms:
            for f in t.facs:
                self._need(f.tensor)
        if not T.terms:
            self._zero(out)
            return
        for n, t in enumerate(T.terms):
            self._emit_term(t, out, accumulate=n > 0)

    def _zero(self, out):
        b = self.plan.bufs[out]
        if b.layout == "scalar":
            self.plan.calls.append(Call("dot", dict(x=None, y=None, n=0, alpha=0.0,
                                                    acc=False), out))
        else:
            self.plan.calls.append(Call("axpby", dict(alpha=0.0, x=None, beta=0.0), out))

    def _emit_term(self, t: Term, out, accumulate):
        p = self.p
        masks = [m for m in t.masks]
        for m in masks:
            if len(m.idx) != p.tensors[m.tensor].order:
                raise NotLowerable("iteration over the rows of a sparse matrix without "
                                   "their entries")
        if len(set(masks)) > 1:
            raise NotLowerable("two sparse iterations in one term")
        # reals (inputs or computed) scale the rest of the term
        reals = tuple(f.tensor for f in t.facs if p.tensors[f.tensor].kind == "scalar")
        if len(reals) > 2:
            raise NotLowerable("more than two real factors in one term")
        t = replace(t, facs=tuple(f for f in t.facs if p.tensors[f.tensor].kind != "scalar"))
        self._emit_plain(t, out, accumulate, reals)

    def _emit_plain(self, t, out, accumulate, reals):
        p = self.p
        ob = self.plan.bufs[out]
        if not t.masks:
            self._emit_dense(t, out, ob, accumulate, reals)
            return
        m = t.masks[0]
        if p.tensors[m.tensor].order == 1:
            self._emit_vector(t, m, out, ob, accumulate, reals)
        elif m.idx[0] == m.idx[1]:
            self._emit_diagonal(t, m.idx[0], out, ob, accumulate, reals)
        else:
            self._emit_sparse(t, m, out, ob, accumulate, reals)

    def _via_temp(self, t, out, ob, accumulate, reals):
        """The term without its reals into a temporary, then scaled by them."""
        tmp = self._temp(ob)
        self._emit_plain(t, tmp, False, ())
        self._scale_into(out, ob, tmp, reals, accumulate)

    def _scale_into(self, out, ob, x, reals, accumulate, alpha=1.0):
        s1, s2 = (tuple(reals) + (None, None))[:2]
        beta = 1.0 if accumulate else 0.0
        if ob.layout == "scalar":
            self.plan.calls.append(Call("scale_real", dict(alpha=alpha, s1=s1, s2=s2, x=x,
                                                           beta=beta), out))
        else:
            self.plan.calls.append(Call("scale", dict(n=None, alpha=alpha, s1=s1, s2=s2, x1=x,
                                                      x2=None, x2_idx=None, beta=beta,
                                                      y_idx=None), out))

    def _product(self, ops, out, P, coef, reals, beta, y_idx=None):
        """out = coef * reals * (product of ops) (+ beta * out) key by key over
        the stored keys of P.  An op is ("v", name) for a value array aligned
        with P's keys or ("g", name, index) for a dense vector read at each
        key's row, column or index; one nsd_scale per pair beyond two."""
        calls = self.plan.calls
        ops = list(ops)

        def pair(a, b):
            if a is not None and a[0] == "g":
                a, b = b, a
            x1 = a[1] if a is not None else None
            if a is not None and a[0] == "g":
                raise AssertionError("two gathered operands in one call")
            x2, idx = (b[1], b[2] if b[0] == "g" else None) if b is not None else (None, None)
            return x1, x2, idx

        while len(ops) > 2 or (len(ops) == 2 and ops[0][0] == "g" and ops[1][0] == "g"):
            a, b = ops[0], ops[1]
            if a[0] == "g" and b[0] == "g":
                b = None   # materialise one gathered operand on its own
            tmp = self._pattern_temp(P)
            x1, x2, idx = pair(a, b)
            calls.append(Call("scale", dict(n=("nnz", P), alpha=1.0, s1=None, s2=None, x1=x1,
                                            x2=x2, x2_idx=idx, beta=0.0, y_idx=None), tmp))
            ops = [("v", tmp)] + ops[1 if b is None else 2:]
        a = ops[0] if ops else None
        b = ops[1] if len(ops) > 1 else None
        x1, x2, idx = pair(a, b)
        s1, s2 = (tuple(reals) + (None, None))[:2]
        calls.append(Call("scale", dict(n=("nnz", P), alpha=coef, s1=s1, s2=s2, x1=x1, x2=x2,
                                        x2_idx=idx, beta=beta, y_idx=y_idx), out))

    # terms over the stored keys (r, c) of the sparse matrix
    def _emit_sparse(self, t, mask, out, ob, accumulate, reals):
        p = self.p
        P = mask.tensor
        r, c = mask.idx
        W = [f for f in t.facs if p.tensors[f.tensor].kind in ("sparse", "patterned")]
        D = [f for f in t.facs if p.tensors[f.tensor].kind == "dense"]
        for f in W:
            if f.idx != (r, c) or p.tensors[f.tensor].pattern != P:
                raise NotLowerable(f"{f.tensor} is read off the iterated key")
        keys = t.keys
        calls = self.plan.calls
        if set(keys) == {r, c} and r not in t.loops and c not in t.loops:
            # a result on the matrix's keys
            if ob.layout != "pattern" or ob.pattern != P:
                raise NotLowerable("a result on the matrix's keys must have its layout")
            if ob.keymap != tuple(0 if v == r else 1 for v in keys):
                raise NotLowerable("terms of one result on different keys")
            summed = [f for f in D if any(v in t.loops for v in f.idx)]
            if not reals and not W and D and self._is_sampled(D, r, c, t.loops):
                X, Y, k = self._sampled(D, r, c, t.loops)
                dst = self._temp(ob) if accumulate else out
                calls.append(Call("sddmm", dict(X=X, Y=Y, k=k, alpha=t.coef), dst))
                if accumulate:
                    calls.append(Call("axpby", dict(alpha=1.0, x=dst, beta=1.0), out))
                return
            if not reals and not D and len(W) <= 1:
                x = self._vals(W[0].tensor) if W else None
                calls.append(Call("axpby", dict(alpha=t.coef, x=x, beta=1.0
                                                if accumulate else 0.0), out))
                return
            ops = [("v", self._vals(f.tensor)) for f in W]
            if summed:
                X, Y, k = self._sampled(summed, r, c, t.loops)
                tmp = self._pattern_temp(P)
                calls.append(Call("sddmm", dict(X=X, Y=Y, k=k, alpha=1.0), tmp))
                ops.append(("v", tmp))
            for f in D:
                if f in summed:
                    continue
                if f.idx == (r,):
                    ops.append(("g", f.tensor, ("rows", P)))
                elif f.idx == (c,):
                    ops.append(("g", f.tensor, ("cols", P)))
                else:
                    raise NotLowerable("a dense factor read at both coordinates of the "
                                       "matrix's key (outside SDDMM)")
            self._product(ops, out, P, t.coef, reals, 1.0 if accumulate else 0.0)
            return
        if reals:
            self._via_temp(t, out, ob, accumulate, reals)
            return
        # the product runs into a temporary when it must be added to `out`
        dst = self._temp(ob) if accumulate else out

        def finish(scale_done):
            if accumulate:
                calls.append(Call("axpby", dict(alpha=1.0 if scale_done else t.coef, x=dst,
                                                beta=1.0), out))
            elif not scale_done and t.coef != 1.0:
                calls.append(Call("axpby", dict(alpha=t.coef, x=out, beta=0.0), out))

        if len(W) > 1 and keys:
            raise NotLowerable("elementwise product of values on the pattern")
        vals = self._vals(W[0].tensor) if W else None
        if vals is None and keys:
            vals = self._ones_pattern()
        if keys and keys[0] == r and all(v != c for v in keys):
            # out[r, z] = sum_c W[r, c] D[c, z]  (SpMM / SpMV)
            if len(D) > 1 or (D and D[0].idx[0] != c) or (D and D[0].idx[1:] != keys[1:]):
                raise NotLowerable("row-indexed product outside SpMM")
            if len(keys) > 2:
                raise NotLowerable("results of order above 2")
            if D:
                dense, k = D[0].tensor, (p.extent[keys[1]] if len(keys) == 2 else 1)
            else:
                if len(keys) != 1:
                    raise NotLowerable("row-indexed product outside SpMM")
                dense, k = self._ones_dense(p.tensors[p.sparse].shape[1]), 1
            calls.append(Call("spmm", dict(vals=vals, B=dense, k=k), dst))
            finish(False)
            return
        if keys and keys[0] == c and all(v != r for v in keys):
            # out[c, z] = sum_r W[r, c] G[r, z]  (transposed product)
            if len(D) > 1 or (D and D[0].idx[0] != r) or (D and D[0].idx[1:] != keys[1:]):
                raise NotLowerable("column-indexed product outside the transposed product")
            if len(keys) > 2 or (not D and len(keys) != 1):
                raise NotLowerable("column-indexed product outside the transposed product")
            k = p.extent[keys[1]] if len(keys) == 2 else 1
            calls.append(Call("spmm_t", dict(vals=vals, G=D[0].tensor if D else None, k=k,
                                             alpha=t.coef), dst))
            finish(True)
            return
        if not keys:
            if ob.layout != "scalar":
                raise NotLowerable("a real result needs a scalar output")
            if D:
                if len(W) > 1:
                    raise NotLowerable("elementwise product of values on the pattern")
                X, Y, k = self._sampled(D, r, c, t.loops)
                tmp = self._pattern_temp(P)
                calls.append(Call("sddmm", dict(X=X, Y=Y, k=k, alpha=1.0), tmp))
                calls.append(Call("dot", dict(x=tmp, y=self._vals(W[0].tensor) if W else None,
                                              alpha=t.coef, acc=accumulate), out))
                return
            x = self._vals(W[0].tensor) if W else self._ones_pattern()
            y = self._vals(W[1].tensor) if len(W) > 1 else None
            if len(W) > 2:
                raise NotLowerable("elementwise product of values on the pattern")
            calls.append(Call("dot", dict(x=x, y=y, alpha=t.coef, acc=accumulate), out))
            return
        raise NotLowerable(f"result keys {keys} over the pattern ({r}, {c})")

    # terms over the stored diagonal keys (i, i) of the sparse matrix: the
    # trace and its gradient (Section 4.3, Example 3)
    def _emit_diagonal(self, t, i, out, ob, accumulate, reals):
        p = self.p
        if reals:
            self._via_temp(t, out, ob, accumulate, reals)
            return
        calls = self.plan.calls
        W = [f for f in t.facs if p.tensors[f.tensor].kind in ("sparse", "patterned")]
        if len(W) != len(t.facs) or len(W) > 1 or any(f.idx != (i, i) for f in W):
            raise NotLowerable("factors other than the matrix's values on its diagonal keys")
        shape = p.tensors[p.sparse].shape
        if t.keys == (i, i):
            # a result on the matrix's keys: coef on the stored diagonal keys
            if ob.layout != "pattern" or ob.pattern != p.sparse:
                raise NotLowerable("a result on the matrix's keys must have its layout")
            if W:
                raise NotLowerable("values times the diagonal indicator on the pattern")
            if not accumulate:
                calls.append(Call("diag", dict(alpha=t.coef), out))
            else:
                tmp = self._pattern_temp(p.sparse)
                calls.append(Call("diag", dict(alpha=t.coef), tmp))
                calls.append(Call("axpby", dict(alpha=1.0, x=tmp, beta=1.0), out))
            return
        if not t.keys:
            # a real: coef * sum of the values (or ones) on the stored diagonal keys
            if ob.layout != "scalar":
                raise NotLowerable("a real result needs a scalar output")
            tmp = self._temp(Buf("", "temp", "pattern", shape, p.sparse, (0, 1)))
            calls.append(Call("diag", dict(alpha=1.0), tmp))
            calls.append(Call("dot", dict(x=tmp, y=self._vals(W[0].tensor) if W else None,
                                          alpha=t.coef, acc=accumulate), out))
            return
        raise NotLowerable(f"result keys {t.keys} over the diagonal keys ({i}, {i})")

    # terms over the stored keys k of a sparse vector (the vector kernels of
    # Section 7.1)
    def _emit_vector(self, t, mask, out, ob, accumulate, reals):
        p = self.p
        P = mask.tensor
        (k,) = mask.idx
        calls = self.plan.calls
        ops = []
        for f in t.facs:
            info = p.tensors[f.tensor]
            if info.kind in ("sparse", "patterned"):
                if f.idx != (k,) or info.pattern != P:
                    raise NotLowerable(f"{f.tensor} is read off the iterated key")
                ops.append(("v", self._vals(f.tensor)))
            elif f.idx == (k,):
                ops.append(("g", f.tensor, ("keys", P)))
            else:
                raise NotLowerable(f"dense factor {f.tensor} of a sparse vector's term read "
                                   "at other than its key")
        keys = t.keys
        if keys and all(v == k for v in keys) and k not in t.loops:
            if ob.layout == "pattern" and ob.pattern == P:
                if ob.keymap != (0,) * len(keys):
                    raise NotLowerable("terms of one result on different keys")
                self._product(ops, out, P, t.coef, reals, 1.0 if accumulate else 0.0)
                return
            if ob.layout == "dense" and len(keys) == 1:
                # scattered into a dense vector (the keys are distinct)
                if not accumulate:
                    self._zero(out)
                self._product(ops, out, P, t.coef, reals, 1.0, y_idx=("keys", P))
                return
            raise NotLowerable(f"result keys {keys} over the sparse vector {P}'s keys")
        if not keys:
            if ob.layout != "scalar":
                raise NotLowerable("a real result needs a scalar output")
            dst = self._temp(ob) if reals else out
            if len(ops) <= 2 and all(o[0] == "v" for o in ops):
                x = ops[0][1] if ops else None
                y = ops[1][1] if len(ops) > 1 else None
            else:
                x, y = self._pattern_temp(P), None
                self._product(ops, x, P, 1.0, (), 0.0)
            calls.append(Call("dot", dict(x=x, y=y, n=("nnz", P), alpha=t.coef,
                                          acc=accumulate and not reals), dst))
            if reals:
                self._scale_into(out, ob, dst, reals, accumulate)
            return
        raise NotLowerable(f"result keys {keys} over the sparse vector {P}'s keys")

    def _is_sampled(self, D, r, c, loops):
        try:
            self._sampled(D, r, c, loops)
            return True
        except NotLowerable:
            return False

    def _sampled(self, D, r, c, loops):
        """X[r, z], Y[c, z] (or vectors X[r], Y[c]) of an SDDMM."""
        X = [f for f in D if f.idx and f.idx[0] == r]
        Y = [f for f in D if f.idx and f.idx[0] == c]
        if len(X) > 1 or len(Y) != 1 or len(X) + len(Y) != len(D):
            raise NotLowerable("sampled product outside SDDMM (one factor per side)")
        zx = X[0].idx[1:] if X else None
        zy = Y[0].idx[1:]
        if len(zy) > 1 or (X and zx != zy) or (zy and zy[0] not in loops):
            raise NotLowerable("sampled product outside SDDMM (one shared summed index)")
        k = self.p.extent[zy[0]] if zy else 1
        return (X[0].tensor if X else None), Y[0].tensor, k

    def _vals(self, tensor):
        if tensor is None:
            return None
        self._need(tensor)
        return tensor

    def _ones_pattern(self):
        name = "ones_nnz"
        if name not in self.plan.bufs:
            self.plan.bufs[name] = Buf(name, "temp", "pattern", self.p.tensors[self.p.sparse].shape,
                                       self.p.sparse, (0, 1))
            self.plan.calls.append(Call("axpby", dict(alpha=1.0, x=None, beta=0.0), name))
        return name

    def _ones_dense(self, n):
        name = f"ones_{n}"
        if name not in self.plan.bufs:
            self.plan.bufs[name] = Buf(name, "temp", "dense", (n,))
            self.plan.calls.append(Call("axpby", dict(alpha=1.0, x=None, beta=0.0), name))
        return name

    # terms over dense tensors only
    def _emit_dense(self, t, out, ob, accumulate, reals):
        calls = self.plan.calls
        if not t.facs and not t.keys:
            # a constant: coef times the number of points of its loops
            mult = 1
            for v in t.loops:
                mult *= self.p.extent[v]
            if ob.layout != "scalar":
                raise NotLowerable("a real result needs a scalar output")
            calls.append(Call("scale_real", dict(alpha=t.coef * mult, s1=(reals + (None,))[0],
                                                 s2=(reals + (None, None))[1], x=None,
                                                 beta=1.0 if accumulate else 0.0), out))
            return
        if not t.keys:
            if reals:
                self._via_temp(t, out, ob, accumulate, reals)
                return
            if ob.layout != "scalar":
                raise NotLowerable("a real result needs a scalar output")
            if not t.facs or len(t.facs) > 2 or any(f.idx != t.facs[0].idx for f in t.facs) \
                    or len(set(t.facs[0].idx)) != len(t.facs[0].idx):
                raise NotLowerable("dense contraction other than a dot product")
            shape = self.p.tensors[t.facs[0].tensor].shape
            for f in t.facs:
                if self.p.tensors[f.tensor].shape != shape:
                    raise NotLowerable("dot product of tensors of different shapes")
            calls.append(Call("dot", dict(x=t.facs[0].tensor,
                                          y=t.facs[1].tensor if len(t.facs) > 1 else None,
                                          alpha=t.coef, acc=accumulate), out))
            return
        if len(t.facs) <= 1 and (not t.facs or t.facs[0].idx == t.keys) and not t.loops \
                and len(set(t.keys)) == len(t.keys) and ob.layout == "dense":
            x = t.facs[0].tensor if t.facs else None
            if reals:
                s1, s2 = (reals + (None, None))[:2]
                calls.append(Call("scale", dict(n=None, alpha=t.coef, s1=s1, s2=s2, x1=x,
                                                x2=None, x2_idx=None,
                                                beta=1.0 if accumulate else 0.0, y_idx=None),
                                  out))
            else:
                calls.append(Call("axpby", dict(alpha=t.coef, x=x,
                                                beta=1.0 if accumulate else 0.0), out))
            return
        raise NotLowerable("dense term other than a copy or a dot product")


# ------------------------------------------------ whole-program fusion


def _only(terms):
    return terms[0] if len(terms) == 1 else None


def _facs_by_tensor(t):
    out = {}
    for f in t.facs:
        out.setdefault(f.tensor, []).append(f.idx)
    return out


def _sparse_mask(p, t):
    """(r, c) of the term's one full mask on the sparse matrix, else None."""
    if len(t.masks) != 1 or t.masks[0].tensor != p.sparse:
        return None
    r, c = t.masks[0].idx
    return None if r == c else (r, c)


def _dense(p, name, shape):
    info = p.tensors.get(name)
    return info is not None and info.input and info.kind == "dense" and info.shape == shape


def _fused_plan(p: Program, grads, value):
    """The whole program as one fused loss kernel of the library, when it is
    exactly one of them (the matrix's values entering linearly as written):
      sum_{(i,j) in A} A_ij x_j                     -> nsd_loss_sum_spmv
      0.5 * sum (C * C) with C = A B                -> nsd_loss_frob_spmm
      sum_{(i,j) in A} A_ij <G_i, H_j>              -> nsd_loss_bilinear
      sum_{(i,j) in A} R_ij R_ij, R = A - U V^T on A's keys -> nsd_loss_mf
    Else None (the program is lowered term by term)."""
    if p.sparse is None or p.value.order not in (0, None):
        return None
    t = _only(p.value.terms)
    if t is None or t.keys:
        return None
    nr, nc = p.tensors[p.sparse].shape
    A = p.sparse
    facs = _facs_by_tensor(t)
    mask = _sparse_mask(p, t)
    low = _Lowering(p)
    low._inputs()
    plan = low.plan

    def out(name, layout, shape, wanted):
        """A result buffer, or a temporary when the kernel writes an output
        nobody asked for."""
        key = name if wanted else f"unused_{name}"
        on = (A, (0, 1)) if layout == "pattern" else (None, ())
        plan.bufs[key] = Buf(key, "out" if wanted else "temp", layout, shape, *on)
        if wanted:
            plan.results[key] = key
        return key

    def want(x):
        return x in grads

    # SMVM
    if mask and t.coef == 1.0 and len(t.facs) == 2 and A in facs and len(facs) == 2:
        (x,) = [n for n in facs if n != A]
        r, c = mask
        if facs[A] == [(r, c)] and facs[x] == [(c,)] and _dense(p, x, (nc,)) \
                and set(grads) <= {A, x}:
            args = dict(x=x, loss=out("value", "scalar", (), value),
                        dA=out("d" + A, "pattern", (nr, nc), want(A)),
                        dx=out("d" + x, "dense", (nc,), want(x)))
            plan.calls.append(Call("loss_sum_spmv", args, args["loss"]))
            return plan
    # bilinear
    if mask and t.coef == 1.0 and len(t.facs) == 3 and len(facs) == 3 and A in facs:
        r, c = mask
        others = [n for n in facs if n != A]
        H = [n for n in others if facs[n][0][0] == c]
        G = [n for n in others if facs[n][0][0] == r]
        if len(H) == 1 and len(G) == 1 and facs[A] == [(r, c)]:
            H, G = H[0], G[0]
            hz, gz = facs[H][0], facs[G][0]
            if len(hz) == 2 and len(gz) == 2 and hz[1] == gz[1] and hz[1] in t.loops:
                k = p.extent[hz[1]]
                if _dense(p, H, (nc, k)) and _dense(p, G, (nr, k)) and set(grads) <= {A, H, G}:
                    args = dict(H=H, G=G, k=k, loss=out("value", "scalar", (), value),
                                dA=out("d" + A, "pattern", (nr, nc), want(A)),
                                dH=out("d" + H, "dense", (nc, k), want(H)))
                    plan.calls.append(Call("loss_bilinear", args, args["loss"]))
                    if want(G):   # dG = A H, not part of the fused kernel
                        dG = out("d" + G, "dense", (nr, k), True)
                        plan.calls.append(Call("spmm", dict(vals=A, B=H, k=k), dG))
                    return plan
    # 1/2 ||A B||^2
    if not t.masks and t.coef == 0.5 and len(t.facs) == 2 and len(facs) == 1:
        (Cn,) = facs
        info = p.tensors[Cn]
        if not info.input and info.kind == "dense" and facs[Cn][0] == facs[Cn][1]:
            d = _only(info.definition.terms)
            dm = d and _sparse_mask(p, d)
            if dm and d.coef == 1.0 and len(d.facs) == 2:
                r, c = dm
                df = _facs_by_tensor(d)
                Bn = [n for n in df if n != A]
                if A in df and len(Bn) == 1 and df[A] == [(r, c)]:
                    Bn = Bn[0]
                    bz = df[Bn][0]
                    if len(bz) == 2 and bz[0] == c and d.keys == (r, bz[1]):
                        k = p.extent[bz[1]]
                        if _dense(p, Bn, (nc, k)) and set(grads) <= {A, Bn}:
                            plan.bufs[Cn] = Buf(Cn, "inter", "dense", (nr, k))
                            args = dict(B=Bn, k=k, C=Cn, loss=out("value", "scalar", (), value),
                                        dA=out("d" + A, "pattern", (nr, nc), want(A)),
                                        dB=out("d" + Bn, "dense", (nc, k), want(Bn)))
                            plan.calls.append(Call("loss_frob_spmm", args, args["loss"]))
                            return plan
    # matrix factorisation
    if mask and t.coef == 1.0 and len(t.facs) == 2 and len(facs) == 1:
        (Rn,) = facs
        info = p.tensors[Rn]
        r, c = mask
        if not info.input and info.kind == "patterned" and facs[Rn] == [(r, c), (r, c)] \
                and len(info.definition.terms) == 2:
            a_term = [u for u in info.definition.terms if len(u.facs) == 1]
            uv_term = [u for u in info.definition.terms if len(u.facs) == 2]
            if len(a_term) == 1 and len(uv_term) == 1:
                at, ut = a_term[0], uv_term[0]
                ok = at.coef == 1.0 and at.facs[0].tensor == A and at.facs[0].idx == at.keys
                uf = _facs_by_tensor(ut)
                ri, ci = ut.keys
                Un = [n for n in uf if uf[n][0][0] == ri]
                Vn = [n for n in uf if uf[n][0][0] == ci]
                if ok and ut.coef == -1.0 and len(Un) == 1 and len(Vn) == 1:
                    Un, Vn = Un[0], Vn[0]
                    uz, vz = uf[Un][0], uf[Vn][0]
                    if len(uz) == 2 and uz[1] == vz[1] and uz[1] in ut.loops:
                        k = p.extent[uz[1]]
                        if _dense(p, Un, (nr, k)) and _dense(p, Vn, (nc, k)) \
                                and set(grads) <= {Un, Vn}:
                            args = dict(U=Un, V=Vn, k=k, loss=out("value", "scalar", (), value),
                                        dU=out("d" + Un, "dense", (nr, k), want(Un)),
                                        dV=out("d" + Vn, "dense", (nc, k), want(Vn)))
                            plan.calls.append(Call("loss_mf", args, args["loss"]))
                            return plan
    return None


def _fused_jvp_plan(p: Program, wrt):
    """The tangent of C = A B (or y = A x) along tangents of A and/or B, for
    a whole batch in one nsd_spmm_jvp_batch call; else None."""
    if p.sparse is None or not set(wrt) <= set(p.inputs):
        return None
    t = _only(p.value.terms)
    mask = t and _sparse_mask(p, t)
    if not mask or t.coef != 1.0 or len(t.facs) != 2:
        return None
    A = p.sparse
    r, c = mask
    nr, nc = p.tensors[A].shape
    facs = _facs_by_tensor(t)
    Bn = [n for n in facs if n != A]
    if facs.get(A) != [(r, c)] or len(Bn) != 1 or len(facs[Bn[0]]) != 1:
        return None
    Bn = Bn[0]
    bz = facs[Bn][0]
    if bz[0] != c or c not in t.loops or t.keys != (r,) + bz[1:] or len(bz) > 2:
        return None
    k = p.extent[bz[1]] if len(bz) == 2 else 1
    if not _dense(p, Bn, (nc, k) if len(bz) == 2 else (nc,)) or not set(wrt) <= {A, Bn}:
        return None
    low = _Lowering(p)
    low._inputs()
    plan = low.plan
    for x in wrt:
        s = p.seed_of(x)
        layout = "pattern" if x == A else "dense"
        plan.bufs[s] = Buf(s, "input", layout, p.tensors[x].shape, A if x == A else None,
                           (0, 1) if x == A else ())
    shape = (nr, k) if len(bz) == 2 else (nr,)
    plan.bufs["tangent"] = Buf("tangent", "out", "dense", shape)
    plan.results["tangent"] = "tangent"
    args = dict(B=Bn, k=k, dA=p.seed_of(A) if A in wrt else None,
                dB=p.seed_of(Bn) if Bn in wrt else None)
    plan.calls.append(Call("spmm_jvp_batch", args, "tangent"))
    return plan


# ------------------------------------------------------------------ execution


def _execute(plan: Plan, inputs: dict, stream=None, outputs=None, m=1):
    """Runs a plan's calls.  outputs: preallocated device tensors for some
    results.  m: the batch of a fused tangent plan (its tangent inputs and
    output carry a leading batch dimension)."""
    import torch

    from . import nsd

    prog = plan.prog
    pats = {}
    dev = None
    for name, d in prog.inputs.items():
        v = inputs.get(name)
        if v is None:
            raise SdqlError(f"missing input {name}")
        if isinstance(d, Sparse):
            if (v.nrows, v.ncols) != d.shape:
                raise SdqlError(f"{name} is {v.nrows}x{v.ncols}, declared {d.shape}")
            pats[name] = v
            dev = v.val.device
        elif isinstance(d, SparseVec):
            if getattr(v, "n", None) != d.n or not hasattr(v, "keys"):
                raise SdqlError(f"{name} must be a DeviceSparseVec of length {d.n}")
            pats[name] = v
            dev = v.val.device
        elif not d.shape:
            if v.dtype != torch.float64 or v.numel() != 1:
                raise SdqlError(f"{name} must be a one-element float64 tensor (a real)")
            dev = v.device
        else:
            if tuple(v.shape) != d.shape or v.dtype != torch.float32 or not v.is_contiguous():
                raise SdqlError(f"{name} must be a contiguous float32 tensor of shape {d.shape}")
            dev = v.device
    A = pats.get(prog.sparse) if prog.sparse else None

    def nnz(P):
        return pats[P].nnz

    mem = {}
    for name, b in plan.bufs.items():
        if outputs and name in outputs:
            mem[name] = outputs[name]
        elif b.role == "input":
            if name in pats:
                mem[name] = pats[name].val
            else:
                v = inputs.get(name)
                if v is None:
                    raise SdqlError(f"missing input {name}")
                mem[name] = v
        elif b.layout == "scalar":
            mem[name] = torch.empty(1, dtype=torch.float64, device=dev)
        elif b.layout == "pattern":
            n = nnz(b.pattern)
            mem[name] = torch.empty(max(n, 1), dtype=torch.float32, device=dev)[:n]
        else:
            mem[name] = torch.empty(b.shape, dtype=torch.float32, device=dev)
    kmax = max([c.args.get("k", 1) for c in plan.calls] + [1])
    need = 16384
    if A is not None:
        need = max(need, nsd.nsd_workspace_size(A.desc, A.csc, kmax))
        if any(c.kernel == "spmm_jvp_batch" for c in plan.calls):
            need = max(need, nsd.nsd_spmm_jvp_batch_workspace_size(A.desc, kmax))
    ws = torch.empty(need, dtype=torch.uint8, device=dev)

    def desc(vals):
        d = nsd.csr_desc(A.nrows, A.ncols, A.rowptr, A.rowidx, A.colind, mem[vals])
        d.plan = A.row_plan
        return d

    def m_(name):
        return None if name is None else mem[name]

    def index(ix):
        if ix is None:
            return None
        what, P = ix
        return {"rows": lambda: pats[P].rowidx, "cols": lambda: pats[P].colind,
                "keys": lambda: pats[P].keys}[what]()

    def count(n, out):
        if isinstance(n, tuple):
            return nnz(n[1])
        return out.numel() if n is None else n

    def csc():
        if A.csc is None:
            A.build_csc(stream)
        return A.csc

    for call in plan.calls:
        a, out = call.args, mem[call.out]
        if call.kernel == "axpby":
            nsd.nsd_axpby(out.numel(), a["alpha"], m_(a["x"]), a["beta"], out, stream)
        elif call.kernel == "scale":
            nsd.nsd_scale(count(a["n"], out), a["alpha"], m_(a["s1"]), m_(a["s2"]), m_(a["x1"]),
                          m_(a["x2"]), index(a["x2_idx"]), a["beta"], out, index(a["y_idx"]),
                          stream)
        elif call.kernel == "scale_real":
            nsd.nsd_scale_real(a["alpha"], m_(a["s1"]), m_(a["s2"]), m_(a["x"]), a["beta"], out,
                               stream)
        elif call.kernel == "dot":
            x = m_(a["x"])
            n = a.get("n")
            n = count(n, x) if n is not None else (x.numel() if x is not None else 0)
            nsd.nsd_dot(n, x, m_(a["y"]), a["alpha"], a["acc"], out, ws, stream)
        elif call.kernel == "sddmm":
            nsd.nsd_sddmm(A.desc, m_(a["X"]), m_(a["Y"]), a["k"], a["alpha"], out, stream)
        elif call.kernel == "diag":
            nsd.nsd_diag_keys(A.desc, a["alpha"], out, stream)
        elif call.kernel == "spmm":
            D = desc(a["vals"])
            if a["k"] == 1:
                nsd.nsd_spmv(D, m_(a["B"]), out, ws, stream)
            else:
                nsd.nsd_spmm(D, m_(a["B"]), a["k"], out, ws, stream)
        elif call.kernel == "spmm_t":
            nsd.nsd_spmm_t(desc(a["vals"]), csc(), m_(a["G"]), a["k"], a["alpha"], out, ws,
                           stream)
        elif call.kernel == "spmm_jvp_batch":
            nsd.nsd_spmm_jvp_batch(A.desc, m, m_(a["dA"]), m_(a["B"]), m_(a["dB"]), a["k"],
                                   (outputs or {}).get("value"), out, ws, stream)
        elif call.kernel == "loss_sum_spmv":
            nsd.nsd_loss_sum_spmv(A.desc, csc(), m_(a["x"]), 1.0, out, mem[a["dA"]],
                                  mem[a["dx"]], ws, stream)
        elif call.kernel == "loss_bilinear":
            nsd.nsd_loss_bilinear(A.desc, csc(), m_(a["H"]), m_(a["G"]), a["k"], 1.0, out,
                                  mem[a["dA"]], mem[a["dH"]], ws, stream)
        elif call.kernel == "loss_frob_spmm":
            nsd.nsd_loss_frob_spmm(A.desc, csc(), m_(a["B"]), a["k"], 1.0, mem[a["C"]], out,
                                   mem[a["dA"]], mem[a["dB"]], ws, stream)
        elif call.kernel == "loss_mf":
            nsd.nsd_loss_mf(A.desc, csc(), None, m_(a["U"]), m_(a["V"]), a["k"], 1.0, out,
                            mem[a["dU"]], mem[a["dV"]], ws, stream)
        else:
            raise SdqlError(f"unknown kernel {call.kernel}")
    return {name: mem[name] for name in plan.results}


def _execute_jvp(plan: Plan, inputs: dict, tangents: dict, value, stream):
    import torch

    prog = plan.prog
    if not tangents:
        raise SdqlError("jvp needs the tangents of at least one input")
    ms = {int(v.shape[0]) for v in tangents.values()}
    if len(ms) != 1:
        raise SdqlError(f"tangents of different batch sizes {sorted(ms)}")
    (m,) = ms
    seeded = dict(inputs)
    for x, v in tangents.items():
        b = plan.bufs[prog.seed_of(x)]
        want = (m,) + ((inputs[x].nnz,) if b.layout == "pattern" else b.shape)
        dtype = torch.float64 if b.layout == "scalar" else torch.float32
        if b.layout == "scalar":
            want = (m,)
        if tuple(v.shape) != want or v.dtype != dtype or not v.is_contiguous():
            raise SdqlError(f"the tangents of {x} must be a contiguous {dtype} tensor "
                            f"of shape {want}")
    ref = inputs[next(iter(tangents))] if tangents else None
    dev = ref.val.device if hasattr(ref, "val") else ref.device
    tb = plan.bufs["tangent"]
    if tb.layout == "pattern":
        rshape = (inputs[tb.pattern].nnz,)
    elif tb.layout == "scalar":
        rshape = ()
    else:
        rshape = tb.shape
    out = {}
    tan = torch.empty((m,) + rshape, dtype=torch.float64 if tb.layout == "scalar"
                      else torch.float32, device=dev)
    if not plan.per_tangent:
        outputs = {"tangent": tan}
        if value:
            out["value"] = outputs["value"] = torch.empty(rshape, dtype=torch.float32,
                                                          device=dev)
        for x, v in tangents.items():
            seeded[prog.seed_of(x)] = v
        _execute(plan, seeded, stream, outputs=outputs, m=m)
    else:
        for t in range(m):
            for x, v in tangents.items():
                seeded[prog.seed_of(x)] = v[t]
            _execute(plan, seeded, stream, outputs={"tangent": tan[t]})
        if value:
            out["value"] = prog.plan((), True).execute(inputs, stream)["value"]
    out["tangent"] = tan
    return out
