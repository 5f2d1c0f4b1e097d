"""Host-side derivation engine: from an operator's tensor algebra expression to the
derived program the library's kernels execute.

* Expressions (section 3): a scope is a traversal over iterators, a summation over
  iterators, and a product of tensor accesses whose indices are affine in the
  iterators; positions outside a tensor read its zero padding.  A scope's output
  tensor can be read by another scope (instantiation).  Guards restrict a summation
  to the points where an affine expression vanishes or is divisible by a constant.
* Intra-expression rules (section 4.2): summation splitting, variable substitution,
  traversal merging, boundary relaxing and tightening; plus the two forms of
  variable substitution the guided stage needs -- splitting one iterator into a block
  index and an offset (r = b*a + r') and eliminating a summation iterator that an
  equality guard determines.
* Instantiation (section 4.3): the iterator mapping table sorts a two-operand scope's
  iterators by the tensors they index; a scope whose groups and coefficients fit an
  operator (Matmul, Conv, G2BMM) is matched to it, every other scope becomes an
  eOperator.
* Hybrid derivation (section 5.2): breadth-first application of the rules up to a
  depth, pruned by expression fingerprints (section 5.3: iterators known by their
  range and traversal position, summations as a multiset, commutative operands
  sorted), with each state checked for a match.

The emitters turn derived programs into the geometry the C ABI takes (the GEMM shape
and operand layouts, the eOperator's tap map as stride / pad / dilation), so a test
can compare them with the formulas the kernels implement.  Nothing here runs on the
GPU; it is pure Python over small integer shapes.
"""
from __future__ import annotations

import hashlib
import itertools
from dataclasses import dataclass, field, replace
from typing import Dict, List, Optional, Sequence, Tuple


# ----------------------------------------------------------------------- expressions

@dataclass(frozen=True)
class Aff:
    """sum(coef * iterator) + const over integer iterators."""
    terms: Tuple[Tuple[str, int], ...] = ()
    const: int = 0

    @staticmethod
    def of(terms: Optional[Dict[str, int]] = None, const: int = 0) -> "Aff":
        t = tuple(sorted((k, v) for k, v in (terms or {}).items() if v != 0))
        return Aff(t, const)

    @staticmethod
    def var(name: str, coef: int = 1) -> "Aff":
        return Aff.of({name: coef})

    def coef(self, name: str) -> int:
        return dict(self.terms).get(name, 0)

    def iters(self) -> Tuple[str, ...]:
        return tuple(k for k, _ in self.terms)

    def __add__(self, o) -> "Aff":
        if isinstance(o, int):
            return Aff(self.terms, self.const + o)
        if isinstance(o, Quot):
            return o + self
        d = dict(self.terms)
        for k, v in o.terms:
            d[k] = d.get(k, 0) + v
        return Aff.of(d, self.const + o.const)

    def __sub__(self, o) -> "Aff":
        return self + (o * -1 if isinstance(o, Aff) else -o)

    def __mul__(self, c: int) -> "Aff":
        return Aff.of({k: v * c for k, v in self.terms}, self.const * c)

    def subs(self, name: str, e: "Aff") -> "Aff":
        c = self.coef(name)
        if c == 0:
            return self
        d = {k: v for k, v in self.terms if k != name}
        return Aff.of(d, self.const) + e * c

    def rename(self, m: Dict[str, str]) -> "Aff":
        return Aff.of({m.get(k, k): v for k, v in self.terms}, self.const)

    def eval(self, env: Dict[str, int]) -> int:
        return self.const + sum(v * env[k] for k, v in self.terms)

    def bounds(self, rng: Dict[str, Tuple[int, int]]) -> Tuple[int, int]:
        """[lo, hi) of the values over the iterators' ranges (a box)."""
        lo = hi = self.const
        for k, v in self.terms:
            a, b = rng[k]
            lo += min(v * a, v * (b - 1))
            hi += max(v * a, v * (b - 1))
        return lo, hi + 1

    def __str__(self):
        parts = [("%s" % k if v == 1 else "-%s" % k if v == -1 else "%d%s" % (v, k))
                 for k, v in self.terms]
        if self.const or not parts:
            parts.append(str(self.const))
        return "+".join(parts).replace("+-", "-")


@dataclass(frozen=True)
class Iter:
    name: str
    lo: int
    hi: int


@dataclass(frozen=True)
class Ref:
    """Access tensor[idx...]; the tensor is an input or another scope's output."""
    tensor: str
    idx: Tuple[Aff, ...]


@dataclass(frozen=True)
class Guard:
    """A summation point counts only if aff == 0 (mod == 0) or aff % mod == 0."""
    aff: Aff
    mod: int = 0


@dataclass(frozen=True)
class Scope:
    trav: Tuple[Iter, ...]
    sums: Tuple[Iter, ...]
    refs: Tuple[Ref, ...]
    guards: Tuple[Guard, ...] = ()

    def ranges(self) -> Dict[str, Tuple[int, int]]:
        return {i.name: (i.lo, i.hi) for i in self.trav + self.sums}

    def shape(self) -> Tuple[Tuple[int, int], ...]:
        return tuple((i.lo, i.hi) for i in self.trav)


@dataclass(frozen=True)
class Program:
    """Scopes by name; `out` is the result.  Inputs: name -> shape (zero outside)."""
    inputs: Tuple[Tuple[str, Tuple[int, ...]], ...]
    scopes: Tuple[Tuple[str, Scope], ...]
    out: str

    def scope(self, name: str) -> Scope:
        return dict(self.scopes)[name]

    def with_scopes(self, **kv) -> "Program":
        d = dict(self.scopes)
        d.update(kv)
        return replace(self, scopes=tuple(sorted(d.items())))

    def without(self, name: str) -> "Program":
        return replace(self, scopes=tuple((k, v) for k, v in self.scopes if k != name))

    def fresh(self, base: str = "S") -> str:
        names = {k for k, _ in self.scopes}
        i = 0
        while "%s%d" % (base, i) in names:
            i += 1
        return "%s%d" % (base, i)

    def parents(self, name: str) -> List[str]:
        return [k for k, s in self.scopes if any(r.tensor == name for r in s.refs)]


# -------------------------------------------------------------------- evaluation

def evaluate(prog: Program, tensors: Dict[str, "object"]):
    """Brute-force value of every scope over its traversal box (NumPy int64/float64),
    by the definition: a product of the accesses, summed over the summation box
    where the guards hold; accesses outside a tensor's box read 0.  Small shapes
    only (a test device for the rules)."""
    import numpy as np
    vals: Dict[str, Tuple["object", Tuple[int, ...]]] = {}
    for name, shp in prog.inputs:
        vals[name] = (np.asarray(tensors[name]), tuple(0 for _ in shp))
    done = set(vals)
    order: List[str] = []

    def visit(n):
        if n in done:
            return
        for r in prog.scope(n).refs:
            visit(r.tensor)
        done.add(n)
        order.append(n)
    visit(prog.out)
    for n in order:
        s = prog.scope(n)
        shape = tuple(i.hi - i.lo for i in s.trav)
        out = np.zeros(shape, dtype=np.float64)
        tn = [i.name for i in s.trav]
        sn = [i.name for i in s.sums]
        srng = [range(i.lo, i.hi) for i in s.sums]
        for tp in itertools.product(*[range(i.lo, i.hi) for i in s.trav]):
            env = dict(zip(tn, tp))
            acc = 0.0
            for sp in itertools.product(*srng):
                env.update(zip(sn, sp))
                if not all(_guard_ok(g, env) for g in s.guards):
                    continue
                p = 1.0
                for r in s.refs:
                    arr, org = vals[r.tensor]
                    ix = tuple(a.eval(env) - o for a, o in zip(r.idx, org))
                    if any(x < 0 or x >= d for x, d in zip(ix, arr.shape)):
                        p = 0.0
                        break
                    p *= float(arr[ix])
                acc += p
            out[tuple(v - i.lo for v, i in zip(tp, s.trav))] = acc
        vals[n] = (out, tuple(i.lo for i in s.trav))
    arr, org = vals[prog.out]
    return arr, org


def _guard_ok(g: Guard, env) -> bool:
    v = g.aff.eval(env)
    return v == 0 if g.mod == 0 else v % g.mod == 0


# ------------------------------------------------------------------------- rules
# Each rule returns the transformed program, or None where it does not apply.

def split_summation(prog: Program, name: str, inner: Sequence[str]) -> Optional[Program]:
    """Sum over (s1, s2) -> sum over s1 of an instantiated scope that sums over s2 =
    `inner` (section 4.2).  The new scope traverses the iterators its accesses use
    (among the traversal and s1) in their original order; guards stay outside."""
    s = prog.scope(name)
    sn = [i.name for i in s.sums]
    inner = list(inner)
    if not inner or len(inner) >= len(sn) or not set(inner) <= set(sn):
        return None
    if any(set(g.aff.iters()) & set(inner) for g in s.guards):
        return None
    used = {k for r in s.refs for a in r.idx for k in a.iters()}
    s1 = [i for i in s.sums if i.name not in inner]
    trav = tuple(i for i in s.trav + tuple(s1) if i.name in used)
    new = prog.fresh()
    inner_scope = Scope(trav, tuple(i for i in s.sums if i.name in inner), s.refs)
    outer = Scope(s.trav, tuple(s1), (Ref(new, tuple(Aff.var(i.name) for i in trav)),),
                  s.guards)
    return prog.with_scopes(**{name: outer, new: inner_scope})


def substitute(prog: Program, name: str, old: str, e: Aff, new: str) -> Optional[Program]:
    """Variable substitution on a traversal iterator of an instantiated scope: the
    iterators (old, rest) are replaced by (t = e, rest), where e has a non-zero
    coefficient on `old` and otherwise uses traversal iterators.  The map is
    injective, so the new scope holds every old value (its box over t is the range e
    takes: boundary relaxing, the extra points are computed and never read).  It
    applies when `old` appears in the body only inside indices of the form e + d with
    d free of `old`; readers index the scope with e at their indices (section 4.2)."""
    s = prog.scope(name)
    tn = [i.name for i in s.trav]
    if name == prog.out or old not in tn or e.coef(old) == 0 or new in s.ranges():
        return None
    if not set(e.iters()) <= set(tn) or any(g.aff.coef(old) for g in s.guards):
        return None
    refs = []
    for r in s.refs:
        idx = []
        for a in r.idx:
            if a.coef(old) == 0:
                idx.append(a)
                continue
            d = a - e
            if isinstance(a, Quot) or d.coef(old):
                return None                       # `old` outside e + (terms without it)
            idx.append(Aff.var(new) + d)
        refs.append(Ref(r.tensor, tuple(idx)))
    lo, hi = e.bounds(s.ranges())
    trav = tuple(Iter(new, lo, hi) if i.name == old else i for i in s.trav)
    out = {name: Scope(trav, s.sums, tuple(refs), s.guards)}
    pos = tn.index(old)
    for pn in prog.parents(name):
        ps = prog.scope(pn)
        prefs = []
        for r in ps.refs:
            if r.tensor == name:
                env = {tn[k]: r.idx[k] for k in range(len(tn))}
                val = Aff.of({}, e.const)
                for k, v in e.terms:
                    val = val + env[k] * v
                idx = list(r.idx)
                idx[pos] = val
                r = Ref(r.tensor, tuple(idx))
            prefs.append(r)
        out[pn] = replace(ps, refs=tuple(prefs))
    return prog.with_scopes(**out)


def permute(prog: Program, name: str, order: Sequence[str]) -> Optional[Program]:
    """Variable substitution by a permutation: an instantiated scope's traversal is
    reordered (its output layout changes) and its readers' indices follow."""
    s = prog.scope(name)
    tn = [i.name for i in s.trav]
    if name == prog.out or sorted(order) != sorted(tn):
        return None
    if list(order) == tn:
        return prog
    by = {i.name: i for i in s.trav}
    perm = [tn.index(k) for k in order]
    out = {name: replace(s, trav=tuple(by[k] for k in order))}
    for pn in prog.parents(name):
        ps = prog.scope(pn)
        out[pn] = replace(ps, refs=tuple(
            Ref(r.tensor, tuple(r.idx[k] for k in perm)) if r.tensor == name else r
            for r in ps.refs))
    return prog.with_scopes(**out)


def merge_traversal(prog: Program, name: str) -> Optional[Program]:
    """Traversal merging: a scope with no summation, read by one parent as its only
    operand, is folded into the parent (its iterators replaced by the parent's index
    expressions); the scope disappears (section 4.2)."""
    s = prog.scope(name)
    ps_names = prog.parents(name)
    if s.sums or s.guards or len(ps_names) != 1 or name == prog.out:
        return None
    pn = ps_names[0]
    ps = prog.scope(pn)
    if len(ps.refs) != 1:
        return None
    r = ps.refs[0]
    env = {i.name: r.idx[k] for k, i in enumerate(s.trav)}
    refs = []
    for q in s.refs:
        idx = []
        for a in q.idx:
            v = Aff.of({}, a.const)
            for k, c in a.terms:
                v = v + env[k] * c
            idx.append(v)
        refs.append(Ref(q.tensor, tuple(idx)))
    # the folded scope's box must cover what the parent reads, else it read padding
    rng = ps.ranges()
    for k, i in enumerate(s.trav):
        lo, hi = r.idx[k].bounds(rng)
        if lo < i.lo or hi > i.hi:
            return None
    return prog.without(name).with_scopes(**{pn: replace(ps, refs=tuple(refs))})


def tighten(prog: Program, name: str) -> Optional[Program]:
    """Boundary tightening: a traversal iterator t that indexes an input tensor as
    t + const (alone in that index) can only give non-zero products inside the
    tensor's box, so its range shrinks to it; readers outside read the padding."""
    s = prog.scope(name)
    shapes = dict(prog.inputs)
    trav = list(s.trav)
    changed = False
    for k, it in enumerate(trav):
        lo, hi = it.lo, it.hi
        for r in s.refs:
            if r.tensor not in shapes:
                continue
            for d, a in enumerate(r.idx):
                if a.iters() == (it.name,) and a.coef(it.name) == 1:
                    lo = max(lo, -a.const)
                    hi = min(hi, shapes[r.tensor][d] - a.const)
        if (lo, hi) != (it.lo, it.hi) and lo < hi:
            trav[k] = Iter(it.name, lo, hi)
            changed = True
    if not changed or name == prog.out:
        return None
    return prog.with_scopes(**{name: replace(s, trav=tuple(trav))})


def relax(prog: Program, name: str, it: str, hi: int) -> Optional[Program]:
    """Boundary relaxing on a summation iterator: extend its range to [lo, hi) when
    every added point reads the zero padding of some input (so it adds 0)."""
    s = prog.scope(name)
    shapes = dict(prog.inputs)
    for k, i in enumerate(s.sums):
        if i.name != it or hi <= i.hi:
            continue
        ok = False
        for r in s.refs:
            if r.tensor not in shapes:
                continue
            for d, a in enumerate(r.idx):
                if a.iters() == (it,) and a.coef(it) == 1 and a.const + i.hi >= shapes[r.tensor][d]:
                    ok = True
        if not ok:
            return None
        sums = list(s.sums)
        sums[k] = Iter(it, i.lo, hi)
        return prog.with_scopes(**{name: replace(s, sums=tuple(sums))})
    return None


def split_iter(prog: Program, name: str, it: str, block: int, a: str, b: str) -> Optional[Program]:
    """Variable substitution it = block*a + b on a summation iterator whose range is
    a whole number of blocks: a in [0, n/block), b in [0, block)."""
    s = prog.scope(name)
    for k, i in enumerate(s.sums):
        if i.name != it:
            continue
        if i.lo != 0 or i.hi % block or a in s.ranges() or b in s.ranges():
            return None
        e = Aff.of({a: block, b: 1})
        sums = s.sums[:k] + (Iter(a, 0, i.hi // block), Iter(b, 0, block)) + s.sums[k + 1:]
        refs = tuple(Ref(r.tensor, tuple(x.subs(it, e) for x in r.idx)) for r in s.refs)
        guards = tuple(Guard(g.aff.subs(it, e), g.mod) for g in s.guards)
        return prog.with_scopes(**{name: Scope(s.trav, sums, refs, guards)})
    return None


def residue_split(prog: Program, name: str, it: str, D: int, ip: str = "ip",
                  rho: str = "rho") -> Optional[Program]:
    """Variable substitution it = D*ip + rho (ip outer, rho inner) on a traversal
    iterator of range [0, n*D), with the data layout transformation that goes with it
    (section 5.2: T'[x'] = T[Phi(x')]).  Every operand index that uses `it` must read
    an input's dimension as it + D*e + c with e free of `it` and c a multiple of D;
    such an input is read through its residue view
        TR[.., rho, t', ..] = T[.., D*t' + rho, ..]
    (an identity eOperator: a strided view), where the index becomes ip + e + c/D.  The
    contraction moves to a new scope traversing (.., rho, ip, ..) with rho placed before
    the row, and the original scope, its traversal split in place as (.., ip, rho, ..)
    (the same memory layout), reads it back."""
    s = prog.scope(name)
    tn = [i.name for i in s.trav]
    if it not in tn or ip in s.ranges() or rho in s.ranges() or D < 2 or prog.parents(name):
        return None
    pos = tn.index(it)
    itr = s.trav[pos]
    if itr.lo != 0 or itr.hi % D:
        return None
    shapes = dict(prog.inputs)
    n = itr.hi // D
    views: Dict[str, Scope] = {}
    refs = []
    for r in s.refs:
        dims = [d for d, a in enumerate(r.idx) if a.coef(it)]
        if not dims:
            refs.append(r)
            continue
        if len(dims) != 1 or r.tensor not in shapes:
            return None
        d = dims[0]
        a = r.idx[d]
        if isinstance(a, Quot) or a.coef(it) != 1 or a.const % D:
            return None
        e = a - Aff.var(it) - a.const
        if any(c % D for _, c in e.terms):
            return None
        shp = shapes[r.tensor]
        if shp[d] % D:
            return None
        vname = r.tensor + "R"
        vit = ["v%d" % m for m in range(len(shp))]
        vtrav = tuple(Iter(vit[m], 0, shp[m]) for m in range(d)) + \
            (Iter("vr", 0, D), Iter("vq", 0, shp[d] // D)) + \
            tuple(Iter(vit[m], 0, shp[m]) for m in range(d + 1, len(shp)))
        vidx = tuple(Aff.var(vit[m]) for m in range(d)) + (Aff.of({"vq": D, "vr": 1}),) + \
            tuple(Aff.var(vit[m]) for m in range(d + 1, len(shp)))
        views[vname] = Scope(vtrav, (), (Ref(r.tensor, vidx),))
        e_div = Aff.of({k: c // D for k, c in e.terms}, a.const // D)
        idx = r.idx[:d] + (Aff.var(rho), Aff.var(ip) + e_div) + r.idx[d + 1:]
        refs.append(Ref(vname, idx))
    if not views or any(v in dict(prog.scopes) for v in views):
        return None
    gname = prog.fresh("G")
    gtrav = s.trav[:pos] + (Iter(rho, 0, D), Iter(ip, 0, n)) + s.trav[pos + 1:]
    g = Scope(gtrav, s.sums, tuple(refs), s.guards)
    otrav = s.trav[:pos] + (Iter(ip, 0, n), Iter(rho, 0, D)) + s.trav[pos + 1:]
    oidx = tuple(Aff.var(i.name) for i in gtrav)
    outer = Scope(otrav, (), (Ref(gname, oidx),))
    return prog.with_scopes(**{name: outer, gname: g}, **views)


def _box(prog: Program, tensor: str, dim: int) -> Tuple[int, int]:
    shapes = dict(prog.inputs)
    if tensor in shapes:
        return 0, shapes[tensor][dim]
    it = prog.scope(tensor).trav[dim]
    return it.lo, it.hi


def eliminate_guard(prog: Program, name: str, which: Optional[str] = None) -> Optional[Program]:
    """A summation iterator x with an equality guard  q*x + rest == 0  is determined
    by the others: x = -rest/q.  The sum over x collapses to that single point
    (variable substitution on the summation space), with  rest % q == 0  kept as a
    divisibility guard when |q| > 1.  Applies when x indexes tensors only as itself
    and each such tensor's box lies inside x's range, so that a solution outside the
    range reads the padding, as the dropped term would have been absent."""
    s = prog.scope(name)
    sums = {i.name: i for i in s.sums}
    for gi, g in enumerate(s.guards):
        if g.mod:
            continue
        for x, q in g.aff.terms:
            if x not in sums or (which is not None and x != which):
                continue
            it = sums[x]
            plain = True
            for r in s.refs:
                for d, a in enumerate(r.idx):
                    if a.coef(x) == 0:
                        continue
                    lo, hi = _box(prog, r.tensor, d)
                    if isinstance(a, Quot) or a != Aff.var(x) or lo < it.lo or hi > it.hi:
                        plain = False
            others = [h for k, h in enumerate(s.guards) if k != gi]
            if not plain or any(h.aff.coef(x) for h in others):
                continue
            num = (g.aff - Aff.var(x, q)) * (-1 if q > 0 else 1)   # x = num / |q|
            aq = abs(q)
            val = num if aq == 1 else Quot(num, aq)
            refs = tuple(Ref(r.tensor, tuple(val if a.coef(x) else a for a in r.idx))
                         for r in s.refs)
            guards = tuple(others) + ((Guard(num, aq),) if aq > 1 else ())
            new = Scope(s.trav, tuple(i for i in s.sums if i.name != x), refs, guards)
            return prog.with_scopes(**{name: new})
    return None


@dataclass(frozen=True)
class Quot(Aff):
    """(num / den) + const for a num that a guard makes divisible by den."""
    num: Aff = Aff()
    den: int = 1
    add: int = 0

    def __init__(self, num: Aff, den: int, add: int = 0):
        object.__setattr__(self, "terms", num.terms)
        object.__setattr__(self, "const", num.const)
        object.__setattr__(self, "num", num)
        object.__setattr__(self, "den", den)
        object.__setattr__(self, "add", add)

    def eval(self, env):
        v = self.num.eval(env)
        return v // self.den + self.add

    def iters(self):
        return self.num.iters()

    # Exact wherever a guard makes num divisible by den; any other combination would
    # lose the division, so it raises and the rule that asked declines.
    def __add__(self, o) -> "Quot":
        if isinstance(o, int):
            return Quot(self.num, self.den, self.add + o)
        if isinstance(o, Aff) and not isinstance(o, Quot) and not o.terms:
            return Quot(self.num, self.den, self.add + o.const)
        raise TypeError("a quotient index combines only with constants")

    def __sub__(self, o) -> "Quot":
        if isinstance(o, int):
            return self + (-o)
        raise TypeError("a quotient index combines only with constants")

    def __mul__(self, c: int) -> "Quot":
        return Quot(self.num * c, self.den, self.add * c)

    def subs(self, name: str, e: Aff) -> "Quot":
        if isinstance(e, Quot):
            raise TypeError("nested quotient")
        return Quot(self.num.subs(name, e), self.den, self.add)

    def rename(self, m: Dict[str, str]) -> "Quot":
        return Quot(self.num.rename(m), self.den, self.add)

    def bounds(self, rng):
        raise TypeError("no box for a quotient index")

    def __str__(self):
        return "(%s)/%d%s" % (self.num, self.den, "+%d" % self.add if self.add else "")


# ------------------------------------------------------------------ fingerprints

def fingerprint(prog: Program) -> str:
    """Hash of the program that ignores iterator names (a traversal iterator is known
    by its range and position, a summation iterator by its range, summations form a
    multiset), orders commutative operands, and knows an instantiated tensor by the
    fingerprint of the scope that produces it (section 5.3)."""
    memo: Dict[str, str] = {}

    def fp_scope(n: str) -> str:
        if n in memo:
            return memo[n]
        shapes = dict(prog.inputs)
        if n in shapes:
            memo[n] = "in:" + n
            return memo[n]
        s = prog.scope(n)
        canon = {}
        for k, i in enumerate(s.trav):
            canon[i.name] = "t%d[%d,%d)" % (k, i.lo, i.hi)
        # summation iterators: by range; equal ranges are told apart by where they
        # are used, so renaming them cannot change the hash
        for i in s.sums:
            uses = sorted("%s.%d:%d" % (fp_scope(r.tensor), d, a.coef(i.name))
                          for r in s.refs for d, a in enumerate(r.idx) if a.coef(i.name))
            canon[i.name] = "s[%d,%d){%s}" % (i.lo, i.hi, ",".join(uses))

        def fa(a):
            base = "+".join(sorted("%d*%s" % (c, canon[k]) for k, c in a.terms)) + "%+d" % a.const
            if isinstance(a, Quot):
                return "(%s)/%d%+d" % (base, a.den, a.add)
            return base
        refs = sorted("%s[%s]" % (fp_scope(r.tensor), ";".join(fa(a) for a in r.idx))
                      for r in s.refs)
        guards = sorted("%s|%d" % (fa(g.aff), g.mod) for g in s.guards)
        sums = sorted(canon[i.name] for i in s.sums)
        text = "L(%s)S(%s)*(%s)G(%s)" % (",".join(canon[i.name] for i in s.trav),
                                          ",".join(sums), "*".join(refs), ",".join(guards))
        memo[n] = hashlib.sha1(text.encode()).hexdigest()[:16]
        return memo[n]
    return fp_scope(prog.out)


# ------------------------------------------------- instantiation: the mapping table

@dataclass
class Match:
    op: str                       # "Matmul", "Conv", "G2BMM"
    scope: str
    groups: Dict[str, List[str]]  # group -> iterators, in traversal/summation order
    detail: Dict[str, object] = field(default_factory=dict)


def mapping_table(prog: Program, name: str):
    """Iterators of a two-operand scope sorted by the tensors that use them:
    'all' (input, weight, output), 'io' (input+output), 'wo' (weight+output),
    'iw' (input+weight), following the iterator mapping table (section 4.3)."""
    s = prog.scope(name)
    if len(s.refs) != 2 or s.guards:
        return None
    a, b = s.refs
    ua = {k for x in a.idx for k in x.iters()}
    ub = {k for x in b.idx for k in x.iters()}
    out = {i.name for i in s.trav}
    groups = {"all": [], "io": [], "wo": [], "iw": []}
    for i in s.trav + s.sums:
        n = i.name
        key = ("all" if n in ua and n in ub and n in out else
               "io" if n in ua and n in out else
               "wo" if n in ub and n in out else
               "iw" if n in ua and n in ub else None)
        if key is None:
            return None
        groups[key].append(n)
    return groups


def match_matmul(prog: Program, name: str) -> Optional[Match]:
    """Matmul: groups m = io, n = wo, k = iw (batch = all), every index a single
    iterator with coefficient 1 and each operand's dims ordered as its groups'
    flattening (row-major m then k, n then k): Eq. (3) and (4) of the layouts."""
    g = mapping_table(prog, name)
    if g is None or g["all"] or not g["io"] or not g["wo"] or not g["iw"]:
        return None
    s = prog.scope(name)
    a, b = s.refs
    rng = s.ranges()

    def simple(r):
        return all(len(x.terms) == 1 and x.terms[0][1] == 1 and x.const == 0 for x in r.idx)
    if not (simple(a) and simple(b)):
        return None
    ai = [x.iters()[0] for x in a.idx]
    bi = [x.iters()[0] for x in b.idx]
    shapes = dict(prog.inputs)
    # every dim of each operand is fully traversed from 0 (a reshape, not a slice)
    for r, its in ((a, ai), (b, bi)):
        if r.tensor in shapes:
            if tuple(rng[k][1] - rng[k][0] for k in its) != tuple(shapes[r.tensor]):
                return None
            if any(rng[k][0] != 0 for k in its):
                return None
    tm, tn = [k for k in ai if k in g["io"]], [k for k in bi if k in g["wo"]]
    km_a, km_b = [k for k in ai if k in g["iw"]], [k for k in bi if k in g["iw"]]
    if ai != tm + km_a or bi != tn + km_b or km_a != km_b:
        return None
    # the output layout must be m then n; a scope that still needs that reordering
    # reports it (the guided stage applies it as a permutation of its traversal)
    order = tm + tn
    ext = {k: rng[k][1] - rng[k][0] for k in rng}

    def prod(ks):
        p = 1
        for k in ks:
            p *= ext[k]
        return p
    return Match("Matmul", name, {"m": tm, "n": tn, "k": km_a},
                 {"M": prod(tm), "N": prod(tn), "K": prod(km_a), "A": a.tensor, "B": b.tensor,
                  "order": order, "reordered": [i.name for i in s.trav] != order})


def match_conv(prog: Program, name: str) -> Optional[Match]:
    """Conv: io = (n, h, w), wo = (f), iw = (c, r, s) with the input indexed
    [n, h + r - p, w + s - p, c] (h and r with equal coefficients, stride 1) and the
    weight [r, s, f, c]."""
    g = mapping_table(prog, name)
    if g is None or g["all"] or len(g["io"]) != 3 or len(g["wo"]) != 1 or len(g["iw"]) != 3:
        return None
    s = prog.scope(name)
    a, w = s.refs
    if len(a.idx) != 4 or len(w.idx) != 4:
        return None
    n_, h_, w_ = g["io"]
    f_ = g["wo"][0]
    c_ = [k for k in g["iw"] if a.idx[3].iters() == (k,)]
    if len(c_) != 1:
        return None
    c_ = c_[0]
    r_ = [k for k in a.idx[1].iters() if k != h_]
    s_ = [k for k in a.idx[2].iters() if k != w_]
    if len(r_) != 1 or len(s_) != 1:
        return None
    r_, s_ = r_[0], s_[0]
    ok = (a.idx[0] == Aff.var(n_) and a.idx[1].coef(h_) == 1 and a.idx[1].coef(r_) == 1 and
          a.idx[2].coef(w_) == 1 and a.idx[2].coef(s_) == 1 and
          a.idx[1].const == a.idx[2].const and
          [x.iters() for x in w.idx] == [(r_,), (s_,), (f_,), (c_,)])
    if not ok:
        return None
    rng = s.ranges()
    return Match("Conv", name, {"io": [n_, h_, w_], "wo": [f_], "iw": [c_, r_, s_]},
                 {"R": rng[r_][1] - rng[r_][0], "S": rng[s_][1] - rng[s_][0],
                  "pad": -a.idx[1].const, "K": rng[f_][1] - rng[f_][0],
                  "out_h": rng[h_], "out_w": rng[w_]})


def match_g2bmm(prog: Program, name: str) -> Optional[Match]:
    """G2BMM (Table 2): iterators in all three tensors (the batch iterators and the row
    i, last), the band offset j in weight+output, the contraction d in input+weight;
    input Q[batch.., i, d], weight K[batch.., i + D*(j - w), d]: a band of width 2w+1
    with dilation D (D = 1 is the non-dilated band)."""
    g = mapping_table(prog, name)
    if g is None or len(g["all"]) < 2 or len(g["wo"]) != 1 or len(g["iw"]) != 1 or g["io"]:
        return None
    s = prog.scope(name)
    q, k = s.refs
    batch, i_ = g["all"][:-1], g["all"][-1]
    j_, d_ = g["wo"][0], g["iw"][0]
    nb = len(batch)
    if [x.iters() for x in q.idx] != [(x,) for x in batch] + [(i_,), (d_,)]:
        return None
    if any(q.idx[m] != Aff.var(batch[m]) or k.idx[m] != Aff.var(batch[m]) for m in range(nb)):
        return None
    if len(k.idx) != nb + 2 or q.idx[nb] != Aff.var(i_) or q.idx[nb + 1] != Aff.var(d_):
        return None
    t = k.idx[nb]
    if isinstance(t, Quot):
        return None
    D = t.coef(j_)
    if t.coef(i_) != 1 or D <= 0 or set(t.iters()) != {i_, j_} or k.idx[nb + 1] != Aff.var(d_):
        return None
    rng = s.ranges()
    wj = rng[j_]
    if t.const + D * wj[0] > 0 or (-t.const) % D:
        return None
    return Match("G2BMM", name, {"all": list(g["all"]), "wo": [j_], "iw": [d_]},
                 {"dilation": D, "w": (-t.const) // D - wj[0], "band": wj[1] - wj[0],
                  "L": rng[i_][1] - rng[i_][0], "row": i_, "batch": list(batch)})


MATCHERS = {"Matmul": match_matmul, "Conv": match_conv, "G2BMM": match_g2bmm}


# ------------------------------------------------------------ hybrid derivation

def _try(rule, *args):
    """A rule application, or None where the rule would have to combine a quotient
    index non-exactly (it declines instead of miscomputing)."""
    try:
        return rule(*args)
    except TypeError:
        return None


def _moves(prog: Program):
    """Every rule application the explorative stage tries on a program."""
    return _moves_all(prog)


def _moves_all(prog: Program):
    for name, s in prog.scopes:
        sn = [i.name for i in s.sums]
        for k in range(1, len(sn)):
            for inner in itertools.combinations(sn, k):
                p = _try(split_summation, prog, name, inner)
                if p is not None:
                    yield ("split", name, inner), p
        p = _try(tighten, prog, name)
        if p is not None:
            yield ("tighten", name), p
        p = _try(merge_traversal, prog, name)
        if p is not None:
            yield ("merge", name), p
        for x in sorted({k for g in s.guards if not g.mod for k in g.aff.iters()}):
            p = _try(eliminate_guard, prog, name, x)
            if p is not None:
                yield ("eliminate", name, x), p
        # data layout changes: variable substitution by a transposition of two
        # neighbouring traversal iterators of an instantiated scope (the program's
        # result keeps its layout)
        if name != prog.out:
            tn_ = [i.name for i in s.trav]
            for k in range(len(tn_) - 1):
                order = tn_[:k] + [tn_[k + 1], tn_[k]] + tn_[k + 2:]
                p = _try(permute, prog, name, order)
                if p is not None:
                    yield ("swap", name, tn_[k], tn_[k + 1]), p
        # substitution candidates: a multi-iterator index expression over this
        # scope's traversal iterators becomes a new iterator
        tn = {i.name for i in s.trav}
        seen = set()
        for r in s.refs:
            for a in r.idx:
                if isinstance(a, Quot) or len(a.terms) < 2 or not set(a.iters()) <= tn:
                    continue
                if a in seen:
                    continue
                seen.add(a)
                taken = set(s.ranges())
                fresh = next("t%d" % k for k in itertools.count() if "t%d" % k not in taken)
                for old, c in a.terms:
                    p = _try(substitute, prog, name, old, a, fresh)
                    if p is not None:
                        yield ("subst", name, old, str(a)), p


@dataclass
class Derived:
    prog: Program
    steps: List[tuple]
    matches: List[Match]
    eops: List[str]
    guided: int = 0               # how many of the steps (the last ones) were guided


def _plain(a: Aff) -> Optional[str]:
    """The iterator of an index that is that iterator alone, else None."""
    if isinstance(a, Quot) or len(a.terms) != 1 or a.terms[0][1] != 1 or a.const:
        return None
    return a.terms[0][0]


def derived_match(prog: Program, target: str) -> Optional[Match]:
    """The program is a derived program for `target` when one scope is that operator in
    the exact form a kernel takes (Matmul: operand and output layouts of Eq. (3) and
    (4), read by an eOperator; G2BMM: a non-dilated band) and every other scope is an
    eOperator or a view.  Returns the operator's match."""
    for name, _ in prog.scopes:
        m = MATCHERS[target](prog, name)
        if m is None:
            continue
        if target == "Matmul" and (m.detail.get("reordered") or name == prog.out or
                                   len(prog.scopes) < 2):
            continue
        if target == "G2BMM" and m.detail["dilation"] != 1:
            continue
        return m
    return None


def select_rules(prog: Program, target: str) -> List[Tuple[tuple, Program]]:
    """The guided stage's choice of rules (section 5.2, Alg. 2 SelectRules): the
    mismatches between the iterator mapping table of each two-operand scope with a
    summation and the target's iterator groups (Table 2) decide what to apply, the
    first kind that applies per scope, in this order:
      * contraction-group mismatch: summation iterators other than the plain indices
        that both operands share (they also shift an input index, or a guard uses
        them) -- summation splitting keeps only the shared ones inside;
      * iterator-group mismatch: a traversal iterator coupled with another iterator in
        one index (the group needs single iterators) -- variable substitution merges
        the index into one new iterator; then boundary tightening shrinks the new
        iterator to the tensor's box;
      * a band whose weight index has dilation D > 1 (G2BMM): the row iterator is split
        by residue and the operands are read through residue views (a data layout
        transformation), which makes the band non-dilated;
      * data-layout mismatch (Matmul): the scope's traversal order differs from the
        target's (m, n) output layout -- a permutation of its traversal."""
    moves: List[Tuple[tuple, Program]] = []
    for name, s in prog.scopes:
        if len(s.refs) != 2 or not s.sums:
            continue
        a, b = s.refs
        shared = [i.name for i in s.sums
                  if any(_plain(x) == i.name for x in a.idx) and
                  any(_plain(x) == i.name for x in b.idx) and
                  not any(g.aff.coef(i.name) for g in s.guards)]
        if shared and len(shared) < len(s.sums):
            q = _try(split_summation, prog, name, shared)
            if q is not None:
                moves.append((("split", name, tuple(shared)), q))
                continue
        if s.guards:
            continue                              # a guarded scope stays an eOperator
        tn = [i.name for i in s.trav]
        found = False
        for r, other in ((a, b), (b, a)):
            used_other = {k for y in other.idx for k in y.iters()}
            for x in r.idx:
                if isinstance(x, Quot) or len(x.terms) < 2 or not set(x.iters()) <= set(tn):
                    continue
                olds = [k for k in x.iters() if k not in used_other]
                if len(olds) != 1:
                    continue
                taken = set(s.ranges())
                fresh = next("t%d" % k for k in itertools.count() if "t%d" % k not in taken)
                q = _try(substitute, prog, name, olds[0], x, fresh)
                if q is not None:
                    moves.append((("subst", name, olds[0], str(x)), q))
                    found = True
                    break
            if found:
                break
        if found:
            continue
        q = _try(tighten, prog, name)
        if q is not None:
            moves.append((("tighten", name), q))
            continue
        if target == "G2BMM":
            m = match_g2bmm(prog, name)
            if m is not None and m.detail["dilation"] > 1:
                q = _try(residue_split, prog, name, m.detail["row"], m.detail["dilation"])
                if q is not None:
                    moves.append((("residue", name, m.detail["row"], m.detail["dilation"]), q))
                    continue
        if target == "Matmul":
            m = match_matmul(prog, name)
            if m is not None and m.detail.get("reordered"):
                q = _try(permute, prog, name, m.detail["order"])
                if q is not None:
                    moves.append((("permute", name, tuple(m.detail["order"])), q))
    return moves


def guided_derive(prog: Program, target: str, steps: List[tuple], found: List[Derived],
                  found_fp: set, budget: int = 8, stats: Optional[Dict[str, int]] = None,
                  _seen: Optional[set] = None, _depth: int = 0):
    """Guided derivation of one program toward `target` (Alg. 2 GuidedDerive): a
    program that is derived (one target operator, the rest eOperators) is recorded;
    otherwise each rule select_rules picks is applied and the result derived further,
    up to `budget` guided steps."""
    seen = set() if _seen is None else _seen
    m = derived_match(prog, target)
    if m is not None:
        fp = fingerprint(prog)
        if fp not in found_fp:
            found_fp.add(fp)
            found.append(Derived(prog, steps, [m], [n for n, _ in prog.scopes if n != m.scope],
                                 _depth))
        return
    if budget <= 0:
        return
    for mv, q in select_rules(prog, target):
        fq = fingerprint(q)
        if fq in seen:
            continue
        seen.add(fq)
        if stats is not None:
            stats["guided"] = stats.get("guided", 0) + 1
        guided_derive(q, target, steps + [mv], found, found_fp, budget - 1, stats, seen,
                      _depth + 1)


def derive(prog: Program, targets: Sequence[str] = ("Matmul",), max_depth: int = 4,
           max_states: int = 20000, prune: bool = True,
           stats: Optional[Dict[str, int]] = None, guided: bool = True,
           guided_budget: int = 8) -> List[Derived]:
    """Hybrid derivation (section 5.2, Alg. 2): breadth-first explorative derivation
    (every rule on every state) up to `max_depth`, skipping programs whose fingerprint
    was seen (prune=False explores them again); from every explorative state, guided
    derivation toward each target (guided=False: the state itself is only checked for a
    derived program, i.e. explorative derivation alone).  `stats` receives the counts of
    explorative states, pruned states and guided rule applications.  Results are
    returned in the order found (shallowest explorative depth first)."""
    seen = set()
    queue = [(prog, [])]
    found: List[Derived] = []
    found_fp = set()
    states = 0
    while queue:
        nxt = []
        for p, steps in queue:
            fp = fingerprint(p)
            if prune and fp in seen:
                if stats is not None:
                    stats["pruned"] = stats.get("pruned", 0) + 1
                continue
            seen.add(fp)
            states += 1
            if stats is not None:
                stats["states"] = states
            if states > max_states:
                return found
            for t in targets:
                if guided:
                    guided_derive(p, t, steps, found, found_fp, guided_budget, stats)
                else:
                    m = derived_match(p, t)
                    if m is not None and fp not in found_fp:
                        found_fp.add(fp)
                        found.append(Derived(p, steps, [m],
                                             [n for n, _ in p.scopes if n != m.scope]))
            if len(steps) < max_depth:
                for mv, q in _moves(p):
                    nxt.append((q, steps + [mv]))
        queue = nxt
    return found


# ------------------------------------------------------------------- expressions

def conv2d_expr(n, c, h, w, k, r, s, stride=(1, 1), pad=(0, 0), dil=(1, 1)) -> Program:
    """E1 of section 4.2 with batch, stride, padding and dilation:
    out[n,ho,wo,f] = sum_{r,s,c} A[n, ho*sh - ph + r*dh, wo*sw - pw + s*dw, c] K[r,s,f,c]."""
    ho = (h + 2 * pad[0] - dil[0] * (r - 1) - 1) // stride[0] + 1
    wo = (w + 2 * pad[1] - dil[1] * (s - 1) - 1) // stride[1] + 1
    a = Ref("A", (Aff.var("n"), Aff.of({"ho": stride[0], "r": dil[0]}, -pad[0]),
                  Aff.of({"wo": stride[1], "s": dil[1]}, -pad[1]), Aff.var("c")))
    kk = Ref("K", (Aff.var("r"), Aff.var("s"), Aff.var("f"), Aff.var("c")))
    e = Scope((Iter("n", 0, n), Iter("ho", 0, ho), Iter("wo", 0, wo), Iter("f", 0, k)),
              (Iter("r", 0, r), Iter("s", 0, s), Iter("c", 0, c)), (a, kk))
    return Program((("A", (n, h, w, c)), ("K", (r, s, k, c))), (("E", e),), "E")


def conv_transpose2d_expr(n, c, h, w, k, r, s, stride=(1, 1), pad=(0, 0), dil=(1, 1),
                          out_pad=(0, 0)) -> Program:
    """The transposed convolution as the adjoint of conv2d, in scatter form: output
    (ho, wo) receives X[hi, wi] K[r, s] wherever ho = hi*sh - ph + r*dh (equality
    guards over the summation (hi, wi, r, s, c))."""
    ho = (h - 1) * stride[0] - 2 * pad[0] + dil[0] * (r - 1) + out_pad[0] + 1
    wo = (w - 1) * stride[1] - 2 * pad[1] + dil[1] * (s - 1) + out_pad[1] + 1
    x = Ref("X", (Aff.var("n"), Aff.var("hi"), Aff.var("wi"), Aff.var("c")))
    kk = Ref("K", (Aff.var("r"), Aff.var("s"), Aff.var("f"), Aff.var("c")))
    g1 = Guard(Aff.of({"hi": stride[0], "r": dil[0], "ho": -1}, -pad[0]))
    g2 = Guard(Aff.of({"wi": stride[1], "s": dil[1], "wo": -1}, -pad[1]))
    e = Scope((Iter("n", 0, n), Iter("ho", 0, ho), Iter("wo", 0, wo), Iter("f", 0, k)),
              (Iter("hi", 0, h), Iter("wi", 0, w), Iter("r", 0, r), Iter("s", 0, s),
               Iter("c", 0, c)), (x, kk), (g1, g2))
    return Program((("X", (n, h, w, c)), ("K", (r, s, k, c))), (("E", e),), "E")


def g2bmm_expr(b, l, d, w, dil) -> Program:
    """S[b,i,j] = sum_d Q[b,i,d] K[b, i + (j - w)*dil, d], j in [0, 2w]."""
    q = Ref("Q", (Aff.var("b"), Aff.var("i"), Aff.var("d")))
    k = Ref("K", (Aff.var("b"), Aff.of({"i": 1, "j": dil}, -w * dil), Aff.var("d")))
    e = Scope((Iter("b", 0, b), Iter("i", 0, l), Iter("j", 0, 2 * w + 1)),
              (Iter("d", 0, d),), (q, k))
    return Program((("Q", (b, l, d)), ("K", (b, l, d))), (("E", e),), "E")


# ---------------------------------------------------------------------- emitters

@dataclass
class ConvPlan:
    """A derived convolution program as the library runs it: the GEMM stage
    Y[m][n] = sum_k A'[m][k] B[n][k] and the eOperator's tap map."""
    M: int
    N: int
    K: int
    a_rows: List[str]          # input iterators flattened into m (row-major)
    b_rows: List[str]          # weight iterators flattened into n
    k_iters: List[str]
    transposed: bool
    stride: Tuple[int, int]
    pad: Tuple[int, int]
    dil: Tuple[int, int]


def _axis(idx: Aff, o: str, r: str, transposed: bool) -> Tuple[int, int, int]:
    """(stride, pad, dilation) of one axis from the eOperator's Y row index:
    forward  hi = stride*o - pad + dil*r;  transposed  hi = (o + pad - dil*r) / stride
    (a plain affine index when the stride is 1)."""
    if not transposed:
        if isinstance(idx, Quot) or set(idx.iters()) - {o, r}:
            raise ValueError(idx)
        return idx.coef(o), -idx.const, idx.coef(r)
    num, den = (idx.num, idx.den) if isinstance(idx, Quot) else (idx, 1)
    if num.coef(o) != 1 or set(num.iters()) - {o, r}:
        raise ValueError(idx)
    return den, num.const, -num.coef(r)


def _gather_form(prog: Program, eop: str, pixel: Sequence[str]) -> Tuple[Program, List[tuple]]:
    """The eOperator in the form its kernel evaluates (the eOperator generation of
    section 4.3.2): each summation iterator that reads a pixel coordinate of the scope
    (`pixel`) and that an equality guard determines is eliminated, so the kernel sums
    over the taps and gathers the partials that land on an output instead of searching
    the input space for them (the selective add)."""
    steps = []
    for x in pixel:
        if x not in {i.name for i in prog.scope(eop).sums}:
            continue
        q = _try(eliminate_guard, prog, eop, x)
        if q is None:
            continue
        steps.append(("eliminate", eop, x))
        prog = q
    return prog, steps


def derive_conv(prog: Program, transposed: bool = False,
                max_depth: int = 0) -> Tuple[ConvPlan, Derived]:
    """Derive a convolution-family expression to Matmul + eOperator by hybrid
    derivation (explorative up to `max_depth`, guided from every state), bring the
    eOperator to its gather form, and read its tap map off the derived expression."""
    res = derive(prog, ("Matmul",), max_depth=max_depth)
    for dv in res:
        m = dv.matches[0]
        outer_names = [n for n, _ in dv.prog.scopes if n != m.scope]
        if len(outer_names) != 1:
            continue
        ref = [r for r in dv.prog.scope(outer_names[0]).refs if r.tensor == m.scope]
        if len(ref) != 1:
            continue
        tpos = {i.name: k for k, i in enumerate(dv.prog.scope(m.scope).trav)}
        pixel = [x for k in m.groups["m"] for x in ref[0].idx[tpos[k]].iters()]
        p, more = _gather_form(dv.prog, outer_names[0], pixel)
        eop = p.scope(outer_names[0])
        # the eOperator reads Y once per tap; Y is the only operand
        if len(eop.refs) != 1 or eop.refs[0].tensor != m.scope:
            continue
        y = eop.refs[0]
        inner = p.scope(m.scope)
        pos = {i.name: k for k, i in enumerate(inner.trav)}
        if len(m.groups["m"]) != 3 or eop.sums and len(eop.sums) != 2:
            continue
        tr = transposed
        try:
            sh, ph, dh = _axis(y.idx[pos[m.groups["m"][1]]], "ho", "r", tr)
            sw, pw, dw = _axis(y.idx[pos[m.groups["m"][2]]], "wo", "s", tr)
        except ValueError:
            continue
        plan = ConvPlan(m.detail["M"], m.detail["N"], m.detail["K"], m.groups["m"],
                        m.groups["n"], m.groups["k"], tr, (sh, sw), (ph, pw), (dh, dw))
        return plan, Derived(p, dv.steps + more, dv.matches, dv.eops, dv.guided)
    raise ValueError("no Matmul + eOperator program within depth %d" % max_depth)


@dataclass
class BandPlan:
    """The dilated band as per-residue non-dilated bands: residue rho's rows are the
    strided view rho, rho + D, ... of length ceil((L - rho) / D)."""
    dilation: int
    w: int
    residues: List[Tuple[int, int, int]]    # (start, stride, length)


def derive_band(b: int, l: int, d: int, w: int, dil: int) -> Tuple[BandPlan, Match, Match]:
    """The dilated G2BMM matches the G2BMM pattern with dilation D.  Hybrid derivation
    toward the non-dilated G2BMM splits the row iterator by residue, i = D*i' + rho,
    and reads Q and K through residue views, turning every residue into a band of
    dilation 1 over the strided subsequence (the dilated-to-non-dilated rewrite of
    section 6.4).  The residue split needs a whole number of rows per residue, so the
    derivation runs on the l rounded up to a multiple of D (rows past l read the zero
    padding and are never stored); the plan's residue lengths are those of l itself."""
    m0 = match_g2bmm(g2bmm_expr(b, l, d, w, dil), "E")
    if m0 is None:
        raise ValueError("not a G2BMM")
    lr = -(-l // dil) * dil
    res = derive(g2bmm_expr(b, lr, d, w, dil), ("G2BMM",), max_depth=0)
    if not res:
        raise ValueError("no non-dilated band derived")
    m1 = res[0].matches[0]
    if m1.detail["dilation"] != 1 or m1.detail["w"] != w:
        raise ValueError("the derived band is not the non-dilated band of half-width w")
    D = 1
    for st in res[0].steps:
        if st[0] == "residue":
            D = st[3]
    residues = [(rho, D, (l - rho + D - 1) // D) for rho in range(D) if l - rho > 0]
    return BandPlan(D, w, residues), m0, m1


def derive_band_program(b: int, l: int, d: int, w: int, dil: int) -> Derived:
    """The hybrid derivation's program for the band (l a multiple of dil): the
    non-dilated G2BMM over residue views, read back by the output in its own layout."""
    res = derive(g2bmm_expr(b, l, d, w, dil), ("G2BMM",), max_depth=0)
    if not res:
        raise ValueError("no non-dilated band derived")
    return res[0]


def _residue_band(b, l, d, w, dil, rho, n) -> Program:
    """Rows i = dil*i' + rho of the dilated band: K's row i + (j - w)*dil becomes
    dil*(i' + j - w) + rho, i.e. row i' + j - w of the residue view KR[b, i', d] =
    K[b, dil*i' + rho, d] -- a band of dilation 1 (variable substitution on i)."""
    q = Ref("QR", (Aff.var("b"), Aff.var("i"), Aff.var("d")))
    k = Ref("KR", (Aff.var("b"), Aff.of({"i": 1, "j": 1}, -w), Aff.var("d")))
    e = Scope((Iter("b", 0, b), Iter("i", 0, n), Iter("j", 0, 2 * w + 1)),
              (Iter("d", 0, d),), (q, k))
    return Program((("QR", (b, n, d)), ("KR", (b, n, d))), (("E", e),), "E")


@dataclass
class Split3Plan:
    """R x S -> 3x3: blocks (nbr, nbs), the 3x3 stage's padding, the block OffsetAdd's
    offsets (er + 3a, es + 3b)."""
    nbr: int
    nbs: int
    pad3: Tuple[int, int]
    offsets: List[Tuple[int, int]]
    conv: Match


def derive_split3x3(n, c, h, w, k, r, s, pad) -> Tuple[Split3Plan, Program]:
    """Boundary relaxing (r, s up to whole 3-blocks), iterator splitting r = 3a + r',
    s = 3b + s', summation splitting of (r', s', c) into an inner scope, variable
    substitution of the inner scope's input rows, and boundary tightening; the inner
    scope then matches Conv with R = S = 3."""
    p = conv2d_expr(n, c, h, w, k, r, s, (1, 1), pad, (1, 1))
    nbr, nbs = -(-r // 3), -(-s // 3)
    p = relax(p, "E", "r", 3 * nbr) if 3 * nbr > r else p
    p = relax(p, "E", "s", 3 * nbs) if 3 * nbs > s else p
    if p is None:
        raise ValueError("kernel relaxing failed")
    p = split_iter(p, "E", "r", 3, "a", "rr")
    p = split_iter(p, "E", "s", 3, "bb", "ss")
    p = split_summation(p, "E", ("rr", "ss", "c"))
    inner = [nm for nm, _ in p.scopes if nm != "E"][0]
    # the inner scope reads A[n, ho + 3a - ph + rr, ...]: its row becomes
    # i = ho + er + 3a, read as A[n, i + rr - (ph + er), ...] (a 3x3 stage padded by
    # ph + er, whose row ho + er + 3a the block OffsetAdd reads)
    er, es = 3 * nbr - r, 3 * nbs - s
    p = substitute(p, inner, "ho", Aff.of({"ho": 1, "a": 3}, er), "i")
    p = substitute(p, inner, "wo", Aff.of({"wo": 1, "bb": 3}, es), "j")
    s_in = p.scope(inner)
    # the weight blocks (a, bb) become output channels: (a, bb, f) traversed as one
    # group -- the order the split weight lays them out
    m = _match_block_conv(p, inner)
    if m is None:
        raise ValueError("the inner scope is not a 3x3 convolution")
    offs = [(er + 3 * a, es + 3 * b) for a in range(nbr) for b in range(nbs)]
    return Split3Plan(nbr, nbs, (pad[0] + er, pad[1] + es), offs, m), p


def _match_block_conv(p: Program, name: str) -> Optional[Match]:
    """The inner scope of the split form: A[n, i + rr - ph', j + ss - pw', c] *
    K[3a + rr, 3bb + ss, f, c] over (rr, ss, c), traversing (n, a, bb, i, j, f) -- a
    3x3 Conv whose output channels are (a, bb, f) once the weight is re-laid as
    W3[rr][ss][(a, bb, f)][c]."""
    s = p.scope(name)
    a, w = s.refs
    tn = [i.name for i in s.trav]
    if not {"n", "i", "j", "f", "a", "bb"} <= set(tn):
        return None
    if [x.iters() for x in w.idx][2:] != [("f",), ("c",)]:
        return None
    if w.idx[0] != Aff.of({"a": 3, "rr": 1}) or w.idx[1] != Aff.of({"bb": 3, "ss": 1}):
        return None
    hi, wi = a.idx[1], a.idx[2]
    if set(hi.iters()) != {"i", "rr"} or set(wi.iters()) != {"j", "ss"}:
        return None
    rng = s.ranges()
    if rng["rr"] != (0, 3) or rng["ss"] != (0, 3):
        return None
    return Match("Conv", name, {"io": ["n", "i", "j"], "wo": ["a", "bb", "f"],
                                "iw": ["c", "rr", "ss"]},
                 {"R": 3, "S": 3, "pad": (-hi.const, -wi.const),
                  "K": (rng["a"][1] * rng["bb"][1] * (rng["f"][1] - rng["f"][0]))})


def conv_desc_fields(plan: ConvPlan, n: int, c: int, h: int, w: int, k: int, r: int,
                     s: int) -> Dict[str, int]:
    """The C ABI descriptor (ollie_conv_desc) fields of a derived convolution plan:
    the GEMM shape it implies (m = n*h*w rows of X, r*s*k columns of Wt, c deep) must
    be the one the library runs, and the tap map's stride / pad / dilation are the
    descriptor's."""
    if plan.M != n * h * w or plan.N != r * s * k or plan.K != c:
        raise ValueError("plan does not match the operator's GEMM shape")
    return {"n": n, "c": c, "h": h, "w": w, "k": k, "r": r, "s": s,
            "stride_h": plan.stride[0], "stride_w": plan.stride[1],
            "pad_h": plan.pad[0], "pad_w": plan.pad[1],
            "dil_h": plan.dil[0], "dil_w": plan.dil[1]}


def conv_entry(plan: ConvPlan) -> str:
    """The C ABI entry point that runs a derived convolution plan."""
    if plan.transposed:
        return "derived_conv_transpose2d"
    return "derived_conv2d" if plan.dil == (1, 1) else "derived_dilated_conv2d"


def split3_workspace_bytes(plan: Split3Plan, n: int, c: int, h: int, w: int, k: int,
                           in_bytes: int, fused_stage: bool, y_bytes: int = 4) -> int:
    """Workspace of the split form as the plan lays it out: the split weights
    W3 [3][3][nbr*nbs*K][c], then (256-byte aligned) either the 3x3 stage's output Z
    (fp32, extent h + 2*pad3 - 2) when that stage is the fused kernel, or its scope
    Y [n*h*w][9*nbr*nbs*K] when its two eOperators run fused over Y."""
    k3 = plan.nbr * plan.nbs * k
    w3 = (9 * k3 * c * in_bytes + 255) // 256 * 256
    if fused_stage:
        hz, wz = h + 2 * plan.pad3[0] - 2, w + 2 * plan.pad3[1] - 2
        return w3 + n * hz * wz * k3 * 4
    return w3 + n * h * w * 9 * k3 * y_bytes

