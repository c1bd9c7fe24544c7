"""Reference interpreter of Logical SDQLite, with scalar forward-mode AD.

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the CPU-baseline leg
of the benchmark may import this module; the library never does.  It shares
no code with the library's front end: its own tokenizer, parser, values and
evaluator, written from the paper's definitions.

Language (Section 3, the grammar of Logical SDQLite):
    sum(<k,v> in e) e | { e -> e } | {} | e(e) | let x = e in e | x
    | not e | if e then e | e + e | e * e | numbers | true | false
    | op(e) | e = e
Values (Section 2, semi-ring dictionaries):
  * a real is a Python float (or a Dual while differentiating);
  * an index is a Python int, a truth value a bool;
  * a tensor is a dict from int keys to values; a key that is not stored
    reads as the additive identity (`ZERO`), and building a sum inserts by
    adding to what a key already holds;
  * `e1 * e2` of tensors is the outer product: the left operand's values are
    multiplied by the right operand (Section 2, Example 2; typing rule of `*`);
  * `sum(<k,v> in d) f` folds the semi-ring addition over d's stored pairs.
Differentiation, two independent ways, tiny inputs only:
  * `gradient` (Section 4.1, scalar forward mode): every real carries a
    tangent; a tangent of 1 is seeded on one stored key of the chosen input
    at a time (the one-hot inputs of the gradient API, Section 4.3) and the
    result's tangent read, one evaluation per stored key;
  * `gradient_tensorized` (Sections 4.2 and 4.3, literally): the program is
    transformed by the tensorized forward-mode rules, the free variables are
    bound to their zero or one-hot tangent tensors, and the transformed
    program is evaluated once.
"""
from __future__ import annotations

import math
import re

# ---------------------------------------------------------------- values


class _Zero:
    """The additive identity of every semi-ring here; what an absent key
    holds, the value of `{}` and of a sum over nothing."""

    def __repr__(self):
        return "ZERO"


ZERO = _Zero()


class Dual:
    """A real with its tangent (Section 4.1)."""

    __slots__ = ("p", "t")

    def __init__(self, p, t=0.0):
        self.p = float(p)
        self.t = float(t)

    def __repr__(self):
        return f"Dual({self.p}, {self.t})"


def _is_real(x):
    return isinstance(x, (float, Dual)) or (isinstance(x, int) and not isinstance(x, bool))


def _primal(x):
    return x.p if isinstance(x, Dual) else x


def add(a, b):
    """Semi-ring addition: reals add, tensors add key-wise."""
    if a is ZERO:
        return b
    if b is ZERO:
        return a
    if isinstance(a, dict) and isinstance(b, dict):
        out = dict(a)
        for k, v in b.items():
            out[k] = add(out[k], v) if k in out else v
        return out
    if isinstance(a, bool) or isinstance(b, bool):
        return a or b
    if isinstance(a, Dual) or isinstance(b, Dual):
        a = a if isinstance(a, Dual) else Dual(a)
        b = b if isinstance(b, Dual) else Dual(b)
        return Dual(a.p + b.p, a.t + b.t)
    if _is_real(a) and _is_real(b):
        return a + b
    raise TypeError(f"cannot add {type(a).__name__} and {type(b).__name__}")


def mul(a, b):
    """Semi-ring multiplication; on tensors the outer product."""
    if a is ZERO or b is ZERO:
        return ZERO
    if isinstance(a, dict):
        return {k: mul(v, b) for k, v in a.items()}
    if isinstance(b, dict):
        return {k: mul(a, v) for k, v in b.items()}
    if isinstance(a, bool) or isinstance(b, bool):
        return a and b
    if isinstance(a, Dual) or isinstance(b, Dual):
        a = a if isinstance(a, Dual) else Dual(a)
        b = b if isinstance(b, Dual) else Dual(b)
        return Dual(a.p * b.p, a.p * b.t + a.t * b.p)
    return a * b


# real unary operations and their derivatives (the op / op' pairs of Section 4.1)
_OPS = {
    "exp": (math.exp, math.exp),
    "log": (math.log, lambda x: 1.0 / x),
    "sin": (math.sin, math.cos),
    "cos": (math.cos, lambda x: -math.sin(x)),
    "sqrt": (math.sqrt, lambda x: 0.5 / math.sqrt(x)),
}


def apply_op(name, x):
    f, df = _OPS[name]
    if x is ZERO:
        x = 0.0
    if isinstance(x, Dual):
        return Dual(f(x.p), df(x.p) * x.t)
    return f(float(x))


# ---------------------------------------------------------------- syntax

_TOKEN = re.compile(r"\s*(?:(\d+\.\d*(?:[eE][-+]?\d+)?|\d+(?:[eE][-+]?\d+)?|\.\d+)"
                    r"|([A-Za-z_][A-Za-z_0-9']*)|(->|[-(){}<>,*+=]))")
_KEYWORDS = {"sum", "in", "let", "if", "then", "not", "true", "false"}


def tokenize(text):
    out, pos = [], 0
    text = text.rstrip()
    while pos < len(text):
        m = _TOKEN.match(text, pos)
        if not m:
            raise SyntaxError(f"bad character at {pos}: {text[pos:pos + 10]!r}")
        num, name, sym = m.groups()
        if num is not None:
            out.append(("num", int(num) if num.isdigit() else float(num)))
        elif name is not None:
            out.append(("kw" if name in _KEYWORDS else "name", name))
        else:
            out.append(("sym", sym))
        pos = m.end()
    out.append(("end", None))
    return out


class _Parser:
    """Expressions as tuples: ("num", r) ("var", x) ("sum", k, v, e1, e2)
    ("single", e1, e2) ("empty",) ("get", e1, e2) ("let", x, e1, e2)
    ("add", e1, e2) ("mul", e1, e2) ("if", e1, e2) ("not", e) ("eq", e1, e2)
    ("op", name, e) ("bool", b).  The bodies of `sum`, `let` and `if`
    extend as far right as possible; `=` binds looser than `+`, `+` looser
    than `*`, and lookup binds tightest."""

    def __init__(self, text):
        self.toks = tokenize(text)
        self.i = 0

    def peek(self):
        return self.toks[self.i]

    def take(self, kind=None, val=None):
        t = self.toks[self.i]
        if (kind and t[0] != kind) or (val is not None and t[1] != val):
            raise SyntaxError(f"expected {val or kind}, found {t[1]!r} (token {self.i})")
        self.i += 1
        return t

    def at(self, kind, val=None):
        t = self.toks[self.i]
        return t[0] == kind and (val is None or t[1] == val)

    def program(self):
        e = self.expr()
        self.take("end")
        return e

    def expr(self):
        if self.at("kw", "let"):
            self.take()
            x = self.take("name")[1]
            self.take("sym", "=")
            e1 = self.expr()
            self.take("kw", "in")
            return ("let", x, e1, self.expr())
        if self.at("kw", "if"):
            self.take()
            c = self.expr()
            self.take("kw", "then")
            return ("if", c, self.expr())
        if self.at("kw", "sum"):
            self.take()
            self.take("sym", "(")
            self.take("sym", "<")
            k = self.take("name")[1]
            self.take("sym", ",")
            v = self.take("name")[1]
            self.take("sym", ">")
            self.take("kw", "in")
            src = self.expr()
            self.take("sym", ")")
            return ("sum", k, v, src, self.expr())
        return self.equality()

    def equality(self):
        e = self.additive()
        while self.at("sym", "="):
            self.take()
            e = ("eq", e, self.additive())
        return e

    def additive(self):
        e = self.product()
        while self.at("sym", "+"):
            self.take()
            e = ("add", e, self.product())
        return e

    def product(self):
        e = self.unary()
        while self.at("sym", "*"):
            self.take()
            e = ("mul", e, self.unary())
        return e

    def unary(self):
        if self.at("kw", "sum") or self.at("kw", "let") or self.at("kw", "if"):
            return self.expr()
        if self.at("kw", "not"):
            self.take()
            return ("not", self.unary())
        if self.at("sym", "-"):
            self.take()
            return ("mul", ("num", -1.0), self.unary())
        return self.postfix()

    def postfix(self):
        e = self.atom()
        while self.at("sym", "("):
            self.take()
            idx = self.expr()
            self.take("sym", ")")
            e = ("get", e, idx)
        return e

    def atom(self):
        t = self.peek()
        if t[0] == "num":
            self.take()
            return ("num", t[1])
        if t == ("kw", "true") or t == ("kw", "false"):
            self.take()
            return ("bool", t[1] == "true")
        if t[0] == "name":
            self.take()
            if t[1] in _OPS and self.at("sym", "("):
                self.take()
                e = self.expr()
                self.take("sym", ")")
                return ("op", t[1], e)
            return ("var", t[1])
        if t == ("sym", "("):
            self.take()
            e = self.expr()
            self.take("sym", ")")
            return e
        if t == ("sym", "{"):
            self.take()
            if self.at("sym", "}"):
                self.take()
                return ("empty",)
            k = self.expr()
            self.take("sym", "->")
            v = self.expr()
            self.take("sym", "}")
            return ("single", k, v)
        raise SyntaxError(f"unexpected {t[1]!r} (token {self.i})")


def parse(text):
    return _Parser(text).program()


# ------------------------------------------------------------ evaluation


def evaluate(e, env):
    """Value of expression `e` (a tuple tree or source text) in `env`."""
    if isinstance(e, str):
        e = parse(e)
    tag = e[0]
    if tag == "num":
        return e[1]
    if tag == "bool":
        return e[1]
    if tag == "var":
        if e[1] not in env:
            raise NameError(e[1])
        return env[e[1]]
    if tag == "empty":
        return ZERO
    if tag == "single":
        k = evaluate(e[1], env)
        if not isinstance(k, int) or isinstance(k, bool):
            raise TypeError(f"dictionary key must be an index, got {k!r}")
        return {k: evaluate(e[2], env)}
    if tag == "get":
        d = evaluate(e[1], env)
        k = evaluate(e[2], env)
        if d is ZERO:
            return ZERO
        if not isinstance(d, dict):
            raise TypeError("lookup into a non-dictionary")
        return d.get(k, ZERO)
    if tag == "let":
        inner = dict(env)
        inner[e[1]] = evaluate(e[2], env)
        return evaluate(e[3], inner)
    if tag == "sum":
        _, k, v, src, body = e
        d = evaluate(src, env)
        acc = ZERO
        if d is ZERO:
            return acc
        if not isinstance(d, dict):
            raise TypeError("sum over a non-dictionary")
        for key in sorted(d):
            inner = dict(env)
            inner[k] = key
            inner[v] = d[key]
            acc = add(acc, evaluate(body, inner))
        return acc
    if tag == "add":
        return add(evaluate(e[1], env), evaluate(e[2], env))
    if tag == "mul":
        return mul(evaluate(e[1], env), evaluate(e[2], env))
    if tag == "if":
        c = evaluate(e[1], env)
        return evaluate(e[2], env) if (c is not ZERO and c) else ZERO
    if tag == "not":
        c = evaluate(e[1], env)
        return not (c is not ZERO and c)
    if tag == "eq":
        a, b = evaluate(e[1], env), evaluate(e[2], env)
        a = 0 if a is ZERO else _primal(a)
        b = 0 if b is ZERO else _primal(b)
        return a == b
    if tag == "op":
        return apply_op(e[1], evaluate(e[2], env))
    if tag == "zero":
        return ZERO
    if tag == "dop":
        x = evaluate(e[2], env)
        return _OPS[e[1]][1](0.0 if x is ZERO else float(_primal(x)))
    if tag == "tmul":
        return tensor_mul(evaluate(e[1], env), evaluate(e[2], env), order(evaluate(e[3], env)))
    raise ValueError(f"unknown expression {tag}")


# ------------------------------------------------------- tensors <-> dicts


def dense_dict(a):
    """A dense numpy array (order 0..n) as a dictionary storing every key."""
    import numpy as np

    a = np.asarray(a, dtype=np.float64)
    if a.ndim == 0:
        return float(a)
    return {i: dense_dict(a[i]) for i in range(a.shape[0])}


def csr_dict(rowptr, colind, val):
    """A CSR matrix as a dictionary of its stored rows and entries (rows
    without entries are not stored)."""
    out = {}
    for i in range(len(rowptr) - 1):
        lo, hi = int(rowptr[i]), int(rowptr[i + 1])
        if hi > lo:
            out[i] = {int(colind[p]): float(val[p]) for p in range(lo, hi)}
    return out


def leaves(d, prefix=()):
    """(key tuple, value) of every stored real of a dictionary."""
    if isinstance(d, dict):
        for k in sorted(d):
            yield from leaves(d[k], prefix + (k,))
    else:
        yield prefix, d


def to_array(d, shape):
    """Dictionary -> dense fp64 array (absent keys 0)."""
    import numpy as np

    out = np.zeros(shape, dtype=np.float64)
    if d is ZERO:
        return out
    if not isinstance(d, dict):
        return np.asarray(_primal(d), dtype=np.float64).reshape(shape)
    for key, v in leaves(d):
        if v is not ZERO:
            out[key] = _primal(v)
    return out


def _replace_leaves(d, fn, prefix=()):
    if isinstance(d, dict):
        return {k: _replace_leaves(v, fn, prefix + (k,)) for k, v in d.items()}
    return fn(prefix, d)


def value(program, env):
    """Primal value of a program, tangents dropped."""
    out = evaluate(program, env)
    return _replace_leaves(out, lambda _, v: _primal(v)) if isinstance(out, dict) else (
        0.0 if out is ZERO else _primal(out))


def gradient(program, env, wrt):
    """Gradient of a real-valued program w.r.t. input `wrt` on its stored
    keys: {key tuple: d program / d wrt[key]}, by one forward-mode evaluation
    per stored key with that key's tangent seeded to 1 (Section 4.1; the
    one-hot seed of Section 4.3)."""
    e = parse(program) if isinstance(program, str) else program
    keys = [k for k, _ in leaves(env[wrt])]
    out = {}
    for target in keys:
        seeded = dict(env)
        seeded[wrt] = _replace_leaves(
            env[wrt], lambda key, v: Dual(v, 1.0 if key == target else 0.0))
        r = evaluate(e, seeded)
        if r is ZERO:
            out[target] = 0.0
        elif isinstance(r, Dual):
            out[target] = r.t
        elif _is_real(r):
            out[target] = 0.0
        else:
            raise TypeError("gradient of a program whose value is not a real")
    return out


def jacobian(program, env, wrt):
    """Jacobian of a program of any value (a real or a tensor) w.r.t. input
    `wrt` on its stored keys, by one forward-mode evaluation per stored key
    with that key's tangent seeded to 1 (Section 4.1): the column of the
    Jacobian for that key.  Returns {output key path + wrt key path: value}
    with the entries whose tangent is nonzero."""
    e = parse(program) if isinstance(program, str) else program
    out = {}
    for target, _ in leaves(env[wrt]):
        seeded = dict(env)
        seeded[wrt] = _replace_leaves(
            env[wrt], lambda key, v: Dual(v, 1.0 if key == target else 0.0))
        r = evaluate(e, seeded)
        for path, v in (leaves(r) if isinstance(r, dict) else [((), r)]):
            t = v.t if isinstance(v, Dual) else 0.0
            if t != 0.0:
                out[path + target] = t
    return out


# ------------------------------------------- tensorized forward mode (literal)


def order(v):
    """Number of dictionary levels of a value (a real, ZERO and {} count 0)."""
    if isinstance(v, dict):
        for x in v.values():
            return 1 + order(x)
    return 0


def tensor_mul(t, e2, m):
    """The product t *[tau] e2 of the tensorized rules: t has m primal levels
    followed by tau levels; the result keeps the m primal keys, then e2's
    keys, then the tau keys (each value v of t at depth m becomes e2 * v)."""
    if t is ZERO or e2 is ZERO:
        return ZERO
    if m == 0:
        return mul(e2, t)
    return {k: tensor_mul(v, e2, m - 1) for k, v in t.items()}


def tangent(e):
    """The tensorized forward-mode transformation of an expression (the rule
    for each construct of Section 4.2, applied to the syntax tree): the
    tangent of variable x is the variable x', constants and discrete values
    have a zero tangent, a product takes the product rule with the tau-aware
    product on its second term, a lookup looks up the tangent, and a sum over
    a dictionary binds the tangent of the current entry."""
    tag = e[0]
    if tag == "sum":
        _, k, v, src, body = e
        return ("sum", k, v, src,
                ("let", k + "'", ("zero",),
                 ("let", v + "'", ("get", tangent(src), ("var", k)), tangent(body))))
    if tag == "let":
        _, x, e1, e2 = e
        return ("let", x, e1, ("let", x + "'", tangent(e1), tangent(e2)))
    if tag == "if":
        return ("if", e[1], tangent(e[2]))
    if tag == "get":
        return ("get", tangent(e[1]), e[2])
    if tag == "single":
        return ("single", e[1], tangent(e[2]))
    if tag == "mul":
        return ("add", ("mul", e[1], tangent(e[2])), ("tmul", tangent(e[1]), e[2], e[1]))
    if tag == "add":
        return ("add", tangent(e[1]), tangent(e[2]))
    if tag == "op":
        return ("mul", ("dop", e[1], e[2]), tangent(e[2]))
    if tag == "var":
        return ("var", e[1] + "'")
    if tag in ("num", "bool", "empty", "not", "eq", "zero"):
        return ("zero",)
    raise ValueError(f"no tangent rule for {tag}")


def onehot(x):
    """The one-hot tensor of the gradient API for input x: for every stored
    key path p of x, the entry {p -> {p -> 1}} (order twice x's)."""
    out = {}
    for path, _ in leaves(x):
        inner = 1.0
        for k in reversed(path):
            inner = {k: inner}
        outer = inner
        for k in reversed(path):
            outer = {k: outer}
        out = add(out, outer) if out else outer
    return out if out else ZERO


def gradient_tensorized(program, env, wrt):
    """`gradient e x` of the gradient API evaluated literally: every free
    variable v gets v' = zero (v != x) or onehot x (v == x), then the
    tensorized tangent of the program is evaluated once.  For a real-valued
    program the result is a tensor over x's keys: {key path: value}."""
    e = parse(program) if isinstance(program, str) else program
    seeded = dict(env)
    for name in env:
        seeded[name + "'"] = onehot(env[name]) if name == wrt else ZERO
    r = evaluate(tangent(e), seeded)
    out = {p: 0.0 for p, _ in leaves(env[wrt])}
    if r is ZERO:
        return out
    if not isinstance(r, dict):
        raise TypeError("gradient of a program whose value is not a real")
    for p, v in leaves(r):
        if p not in out:
            raise KeyError(f"gradient key {p} is not a stored key of {wrt}")
        out[p] = 0.0 if v is ZERO else float(v)
    return out


def jacobian_tensorized(program, env, wrt):
    """`gradient e x` of a program of any value, evaluated literally as in
    gradient_tensorized: the tangent's output keys come first and x's keys
    after them (the tau levels of Section 4.2), so that for a tensor-valued
    program the result is its Jacobian.  Returns {output key path + wrt key
    path: value} for every entry the tangent stores (an output whose tangent
    is the zero value, such as a key only another input stores, has none)."""
    e = parse(program) if isinstance(program, str) else program
    seeded = dict(env)
    for name in env:
        seeded[name + "'"] = onehot(env[name]) if name == wrt else ZERO
    r = evaluate(tangent(e), seeded)
    if r is ZERO:
        return {}
    return {p: float(v) for p, v in (leaves(r) if isinstance(r, dict) else [((), r)])
            if v is not ZERO}


def jvp_tensorized(program, env, tangents):
    """The tensorized forward mode with a batch of tangents (Section 4.2: the
    tangent of an input may carry tau levels after its own keys; with tau a
    vector of m directions, one evaluation gives J V): every free variable v
    gets v' = tangents[v] (v's key paths followed by the batch key t) when
    given, else zero, and the tangent of the program is evaluated once.
    Returns {output key path + (t,): value} for every entry the tangent
    stores (t alone for a real-valued program)."""
    e = parse(program) if isinstance(program, str) else program
    seeded = dict(env)
    for name in env:
        seeded[name + "'"] = tangents.get(name, ZERO)
    r = evaluate(tangent(e), seeded)
    if r is ZERO:
        return {}
    return {p: float(v) for p, v in (leaves(r) if isinstance(r, dict) else [((), r)])
            if v is not ZERO}
