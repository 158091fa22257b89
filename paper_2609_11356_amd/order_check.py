"""Static equivalence of reduction orders from gfx950 assembly (Sec. 6).

Two compiled kernels are bitwise equivalent when every output element they
store is the same floating-point expression over the same loaded elements, up
to the commutativity of the combines (Sec. 6, "The algorithm").  This module
reads the AMDGCN text that hipcc writes for a kernel built here, walks one
entry function in program order over one wave, and reduces the expression
reaching each global store to a canonical tree and then to a signature.

The walk (Sec. 6, "The algorithm" and "Implementation"):

* A register maps to the node that stands for its contents, per lane.  Each
  instruction is a transfer function on that map: it looks its operands up
  and writes a node into its destination.
* A global load becomes a data node keyed on the address the lane read, so
  two kernels that reach one element through different index arithmetic
  share the leaf.  Addresses are affine forms over the kernel's symbols (its
  pointer arguments and the workgroup id) with a per-lane constant part.
* A floating-point combine becomes an arithmetic node over the nodes its
  operands hold.  Cross-lane moves (DPP lane permutations, ds_swizzle,
  ds_bpermute) move nodes between lanes and combine nothing.
* The nodes reaching a global store are the roots, one per stored element.
* Canonicalisation sorts the operands of each commutative node (add, max,
  min, mul), nothing else: floating-point addition does not associate, so a
  regrouped sum is a different tree.  A bottom-up hash gives the signature.

What differs from the paper's checker, by design of this slice: the lanes are
concrete (one wave of 64 lanes with its real lane ids), so masks, shifts and
compares on lane-derived integers evaluate exactly and branches on them are
followed; only the floating-point values and the pointer and workgroup
symbols stay symbolic.  A branch on anything else, a loop whose trip count is
not fixed by lane-derived values, or more than a fixed number of steps raises
Unsupported.  An instruction the walk does not model writes an opaque node
that carries its own text, which equals only an identical text (Sec. 6:
opaque syntax keeps the answer sound).  The balanced-tree collapse of Sec. 6
is not applied: two trees are equal only when their logical structure is, so
the answer errs towards splitting classes, never merging them.
"""
from __future__ import annotations

import hashlib
import os
import re
import subprocess
import tempfile

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
WAVE = 64
MAX_STEPS = 200000


class Unsupported(Exception):
    """The walk cannot follow this kernel (data-dependent control flow, an
    unmodelled branch, or too many steps)."""


# ------------------------------------------------------------------ values

class Aff:
    """An integer: const + sum coeff * symbol (symbols: pointer arguments,
    32-bit arguments, workgroup ids).  A purely constant Aff is concrete."""
    __slots__ = ("c", "t")

    def __init__(self, c=0, t=None):
        self.c = c
        self.t = {k: v for k, v in (t or {}).items() if v}

    def concrete(self):
        return not self.t

    def __add__(self, o):
        t = dict(self.t)
        for k, v in o.t.items():
            t[k] = t.get(k, 0) + v
        return Aff(self.c + o.c, t)

    def neg(self):
        return Aff(-self.c, {k: -v for k, v in self.t.items()})

    def scale(self, m):
        return Aff(self.c * m, {k: v * m for k, v in self.t.items()})

    def key(self):
        return (self.c, tuple(sorted(self.t.items())))

    def __repr__(self):
        return "+".join(["%s*%d" % (k, v) for k, v in sorted(self.t.items())] + [str(self.c)])


class HiWord:
    """The high word of a 64-bit address whose low word carries the affine
    form (set by a pointer argument's high word or a carry step)."""
    __slots__ = ()


class Node:
    """A floating-point value: op with children (leaf: the address read)."""
    __slots__ = ("op", "kids", "leaf", "_canon")

    def __init__(self, op, kids=(), leaf=None):
        self.op, self.kids, self.leaf, self._canon = op, tuple(kids), leaf, None


COMMUTATIVE = {"add", "max", "min", "mul", "prod"}


def canon(n: Node) -> str:
    """The canonical text of a tree: commutative operands sorted."""
    if n._canon is None:
        if n.op == "load":
            n._canon = "L(%r)" % (n.leaf,)
        elif n.op == "const":
            n._canon = "const(%s)" % n.leaf
        elif n.op == "opaque":
            n._canon = "opaque[%s](%s)" % (n.leaf, ",".join(canon(k) for k in n.kids))
        else:
            kids = [canon(k) for k in n.kids]
            if n.op in COMMUTATIVE:
                kids.sort()
            elif n.op == "fma":                 # a * b + c: the product commutes
                kids = sorted(kids[:2]) + kids[2:]
            elif n.op == "chunk":               # acc, then a set of exact products
                kids = kids[:1] + sorted(kids[1:])
            n._canon = "%s(%s)" % (n.op, ",".join(kids))
    return n._canon


# ------------------------------------------------------------------ parsing

def _tokens(rest: str):
    """Split an operand field at top-level spaces (brackets and parentheses
    kept together)."""
    out, cur, depth = [], "", 0
    for ch in rest:
        if ch in "[(":
            depth += 1
        elif ch in "])":
            depth -= 1
        if ch.isspace() and depth == 0:
            if cur:
                out.append(cur)
            cur = ""
        else:
            cur += ch
    if cur:
        out.append(cur)
    return out


def parse_line(line: str):
    line = line.split(";")[0].strip()
    if not line or line.startswith(".") or line.endswith(":"):
        return None
    op, _, rest = line.partition(" ")
    toks = _tokens(rest)
    ops, mods, i = [], [], 0
    while i < len(toks):
        t = toks[i]
        if t.endswith(","):
            ops.append(t[:-1])
            i += 1
            continue
        ops.append(t)
        mods = toks[i + 1:]
        break
    return op, ops, mods


def functions(asm: str) -> dict[str, list[str]]:
    """The body lines of each entry function in the assembly text."""
    out, cur, name = {}, None, None
    for line in asm.splitlines():
        m = re.match(r"^([A-Za-z_.$][\w.$]*):", line)
        if m and not line.startswith(".L") and not m.group(1).startswith(".L"):
            name, cur = m.group(1), []
            out[name] = cur
            continue
        if cur is not None:
            if line.startswith(".Lfunc_end") or "\t.section" in line and name in out and out[name]:
                cur = None
                continue
            cur.append(line)
    names = set(re.findall(r"\.type\s+([\w.$]+),@function", asm))
    return {k: v for k, v in out.items() if k in names}


def _kernel_meta(asm: str, name: str) -> dict:
    i = asm.find(".amdhsa_kernel " + name + "\n")
    meta = {}
    if i >= 0:
        j = asm.find(".end_amdhsa_kernel", i)
        for m in re.finditer(r"\.(amdhsa_\w+)\s+(\d+)", asm[i:j]):
            meta[m.group(1)] = int(m.group(2))
    return meta


# ------------------------------------------------------------------ the walk

def _reg(tok):
    """('v'|'s'|'a', first, count) for a register operand, else None."""
    m = re.fullmatch(r"([vsa])(\d+)", tok)
    if m:
        return m.group(1), int(m.group(2)), 1
    m = re.fullmatch(r"([vsa])\[(\d+):(\d+)\]", tok)
    if m:
        a, b = int(m.group(2)), int(m.group(3))
        return m.group(1), a, b - a + 1
    return None


def _imm(tok):
    try:
        return int(tok, 0)
    except ValueError:
        return None


def _dpp_src(mods, lane):
    """Source lane of a DPP move for this lane, or None (invalid source)."""
    row = lane & ~15
    for m in mods:
        if m.startswith("quad_perm:"):
            p = [int(x) for x in m[len("quad_perm:["):-1].split(",")]
            return (lane & ~3) | p[lane & 3]
        if m == "row_mirror":
            return row + 15 - (lane & 15)
        if m == "row_half_mirror":
            return (lane & ~7) + 7 - (lane & 7)
        for kind in ("row_shl:", "row_shr:", "row_ror:"):
            if m.startswith(kind):
                n = int(m[len(kind):], 0)
                i = lane & 15
                if kind == "row_shl:":
                    return row + i + n if i + n < 16 else None
                if kind == "row_shr:":
                    return row + i - n if i - n >= 0 else None
                return row + ((i - n) % 16)
        if m == "row_bcast:15":
            return row - 1 if row > 0 else None
        if m == "row_bcast:31":
            return 31 if lane >= 32 else None
    raise Unsupported("DPP control " + " ".join(mods))


def _dpp_writes(mods, lane):
    rm = bm = 0xF
    for m in mods:
        if m.startswith("row_mask:"):
            rm = int(m[len("row_mask:"):], 0)
        if m.startswith("bank_mask:"):
            bm = int(m[len("bank_mask:"):], 0)
    return bool((rm >> (lane >> 4)) & 1) and bool((bm >> ((lane & 15) >> 2)) & 1)


def _swizzle_src(mods, lane):
    for m in mods:
        if not m.startswith("offset:"):
            continue
        v = m[len("offset:"):]
        g = re.fullmatch(r"swizzle\((\w+),?(.*)\)", v)
        if g:
            mode, arg = g.group(1), g.group(2)
            if mode == "SWAP":
                return lane ^ int(arg, 0) if int(arg, 0) < 32 else None
            if mode == "REVERSE":
                n = int(arg, 0)
                return (lane & ~(n - 1)) | ((n - 1) - (lane & (n - 1)))
            if mode == "BROADCAST":
                n, k = [int(x, 0) for x in arg.split(",")]
                return (lane & ~(n - 1)) | k
            if mode == "QDMODE_PERM":
                p = [int(x, 0) for x in arg.split(",")]
                return (lane & ~3) | p[lane & 3]
            raise Unsupported("swizzle mode " + mode)
        off = int(v, 0)
        if off & 0x8000:
            return (lane & ~3) | ((off >> (2 * (lane & 3))) & 3)
        a, o, x = off & 0x1F, (off >> 5) & 0x1F, (off >> 10) & 0x1F
        return (lane & 0x20) | ((((lane & 0x1F) & a) | o) ^ x)
    raise Unsupported("ds_swizzle without an offset")


class Walk:
    """One entry function walked over one wave."""

    def __init__(self, asm: str, name: str, block=(64, 1, 1), args=None):
        """block: the workgroup shape; args: {kernel-argument byte offset:
        value} for 32-bit integer arguments bound to a configuration (loops
        whose trip count they fix are then walked exactly)."""
        self.args = dict(args or {})
        fns = functions(asm)
        if name not in fns:
            raise KeyError(name)
        self.name, self.lines = name, fns[name]
        self.meta = _kernel_meta(asm, name)
        self.stores = {}              # address key -> (Aff, Node)
        self.lds = {}                 # LDS byte address (4-byte words) -> value
        self._leaves = {}
        self._addr_of = {}
        self.opaque = []
        nthreads = block[0] * block[1] * block[2]
        # one state per wave of the workgroup: registers, exec, vcc, scc
        self.waves = []
        for w in range((nthreads + WAVE - 1) // WAVE):
            t0 = WAVE * w
            n = min(WAVE, nthreads - t0)
            # v0: work-item ids (x in bits 0-9, y and z above when present)
            tid = [t0 + l for l in range(WAVE)]
            V = {0: [Aff((t % block[0]) | ((t // block[0] % block[1]) << 10) | ((t // (block[0] * block[1])) << 20))
                     for t in tid]}
            # s[0:1]: the kernel-argument pointer; after the user SGPRs, the workgroup ids
            S = {0: ("kernarg", 0)}
            k = self.meta.get("amdhsa_user_sgpr_count", 2)
            for d in "xyz":
                if self.meta.get("amdhsa_system_sgpr_workgroup_id_" + d, 1 if d == "x" else 0):
                    S[k] = Aff(0, {"wg_" + d: 1})
                    k += 1
            self.waves.append(dict(V=V, S=S, exec=(1 << n) - 1, vcc=0, scc=0, pc=0, done=False))
        self._run()

    def _enter(self, w):
        st = self.waves[w]
        self.V, self.S, self.exec, self.vcc, self.scc = st["V"], st["S"], st["exec"], st["vcc"], st["scc"]

    def _leave(self, w):
        st = self.waves[w]
        st["V"], st["S"], st["exec"], st["vcc"], st["scc"] = self.V, self.S, self.exec, self.vcc, self.scc

    # --- registers
    def v(self, tok, lane):
        r = _reg(tok)
        if r and r[0] in "va":
            return self.V.get((r[1] if r[0] == "v" else 1000 + r[1]), [None] * WAVE)[lane]
        if r and r[0] == "s":
            x = self.S.get(r[1])
            if isinstance(x, tuple) and x[0] == "arg":
                return Aff(0, {"arg%d" % x[1]: 1})        # a pointer's low word (or a 32-bit argument)
            if isinstance(x, tuple) and x[0] == "arghi":
                return HiWord()                          # a pointer's high word
            return x
        i = _imm(tok)
        if i is not None:
            return Aff(i)
        if tok in ("vcc", "vcc_lo"):
            return Aff((self.vcc >> lane) & 1)
        f = self._fconst(tok)
        if f is not None:
            return f
        raise Unsupported("operand " + tok)

    def fval(self, tok, lane):
        """A floating-point operand: a register's node, or a literal constant."""
        if _reg(tok) is None and (_imm(tok) is not None or self._fconst(tok) is not None):
            return Node("const", leaf=tok)
        return self.v(tok, lane)

    def _fconst(self, tok):
        try:
            float(tok)
        except ValueError:
            return None
        return Node("const", leaf=tok)

    def setv(self, tok, lane, val, k=0):
        r = _reg(tok)
        if not r or r[0] not in "va":
            raise Unsupported("vector destination " + tok)
        idx = (r[1] if r[0] == "v" else 1000 + r[1]) + k
        self.V.setdefault(idx, [None] * WAVE)[lane] = val

    def lanes(self):
        return [l for l in range(WAVE) if (self.exec >> l) & 1]

    def mask(self, tok):
        if tok in ("vcc", "vcc_lo"):
            return self.vcc
        if tok == "exec":
            return self.exec
        r = _reg(tok)
        if r and r[0] == "s":
            m = self.S.get(r[1])
            if isinstance(m, tuple) and m[0] == "mask":
                return m[1]
            h = self.S.get(r[1] + 1)
            if isinstance(m, Aff) and m.concrete() and isinstance(h, Aff) and h.concrete():
                return ((m.c & 0xFFFFFFFF) | ((h.c & 0xFFFFFFFF) << 32)) & ((1 << WAVE) - 1)
        if _imm(tok) is not None:
            return _imm(tok) & ((1 << WAVE) - 1)
        raise Unsupported("mask operand " + tok)

    def setmask(self, tok, m):
        if tok in ("vcc", "vcc_lo"):
            self.vcc = m
        elif tok == "exec":
            self.exec = m
        else:
            r = _reg(tok)
            if not r or r[0] != "s":
                raise Unsupported("mask destination " + tok)
            self.S[r[1]] = ("mask", m)

    def _ptr(self, tok):
        r = _reg(tok)
        if not r or r[0] != "s":
            raise Unsupported("address base " + tok)
        p = self.S.get(r[1])
        if isinstance(p, tuple) and p[0] == "arg":
            return Aff(0, {"arg%d" % p[1]: 1})
        if isinstance(p, Aff) and (isinstance(self.S.get(r[1] + 1), tuple) and self.S.get(r[1] + 1)[0] == "arghi"
                                   or isinstance(self.S.get(r[1] + 1), HiWord)):
            return p
        raise Unsupported("address base " + tok)

    def leaf(self, addr: Aff):
        k = addr.key()
        if k not in self._leaves:
            self._leaves[k] = Node("load", leaf=repr(addr))
            self._addr_of[id(self._leaves[k])] = addr
        return self._leaves[k]

    def half(self, word, h):
        """Element h (0 low, 1 high) of a word holding two 16-bit values: a
        leaf at its own byte address when the word was loaded."""
        a = self._addr_of.get(id(word)) if isinstance(word, Node) else None
        if a is not None:
            return self.leaf(a + Aff(2 * h))
        if not isinstance(word, Node):
            word = Node("const", leaf=repr(word))
        return Node("half%d" % h, [word])

    def _mfma16(self, ops):
        """v_mfma_f32_16x16x32 (bf16 or f16): for output (i, j) in lane
        j + 16 (i / 4), register i % 4, the 32 k fold as four chunks of 8 in
        increasing k, each updating the accumulator once (the chunk rule the
        probes measured on gfx950); chunk c's operands sit in lane group c:
        A row i in lane i + 16 c, B column j in lane j + 16 c, element e of
        the chunk in register e / 2, half e % 2."""
        d, ra, rb, c = _reg(ops[0]), _reg(ops[1]), _reg(ops[2]), ops[3]
        idx = lambda r, k: (r[1] if r[0] == "v" else 1000 + r[1]) + k
        rc = _reg(c)
        vals = {}
        for l in self.lanes():
            i0, j = 4 * (l >> 4), l & 15
            for q in range(4):
                i = i0 + q
                if rc is None:
                    acc = Node("const", leaf=c)
                else:
                    acc = self.V.get(idx(rc, q), [None] * WAVE)[l]
                    if isinstance(acc, Aff) and acc.concrete():
                        acc = Node("const", leaf=str(acc.c & 0xFFFFFFFF))    # bits written as an integer
                    if not isinstance(acc, Node):
                        raise Unsupported("MFMA accumulator not a value")
                for ch in range(4):
                    la, lb = i + 16 * ch, j + 16 * ch
                    if not ((self.exec >> la) & 1 and (self.exec >> lb) & 1):
                        raise Unsupported("MFMA with inactive lanes")
                    prods = [Node("prod", [self.half(self.V.get(idx(ra, e // 2), [None] * WAVE)[la], e % 2),
                                           self.half(self.V.get(idx(rb, e // 2), [None] * WAVE)[lb], e % 2)])
                             for e in range(8)]
                    acc = Node("chunk", [acc] + prods)
                vals[(l, q)] = acc
        for (l, q), x in vals.items():
            self.setv(ops[0], l, x, q)

    # --- the interpreter
    def _run(self):
        labels, prog = {}, []
        for line in self.lines:
            s = line.split(";")[0].strip()
            m = re.match(r"^(\.?L[\w.$]+):", s)
            if m:
                labels[m.group(1)] = len(prog)
                continue
            p = parse_line(line)
            if p:
                prog.append((p, s))
        # each wave runs to its next barrier (or its end), then the next wave:
        # an order every barrier-synchronised program allows
        steps = 0
        while not all(st["done"] for st in self.waves):
            for w, st in enumerate(self.waves):
                if st["done"]:
                    continue
                self._enter(w)
                pc = st["pc"]
                while True:
                    if pc >= len(prog):
                        st["done"] = True
                        break
                    steps += 1
                    if steps > MAX_STEPS:
                        raise Unsupported("step limit")
                    (op, ops, mods), text = prog[pc]
                    pc += 1
                    if op == "s_endpgm":
                        st["done"] = True
                        break
                    if op == "s_barrier":
                        break
                    jump = self._branch(op, ops)
                    if jump is not None:
                        if jump is True:
                            if ops[0] not in labels:
                                raise Unsupported("branch target " + ops[0])
                            pc = labels[ops[0]]
                        continue
                    self._step(op, ops, mods, text)
                st["pc"] = pc
                self._leave(w)

    def _branch(self, op, ops):
        if not op.startswith("s_branch") and not op.startswith("s_cbranch"):
            return None
        if op == "s_branch":
            return True
        if op == "s_cbranch_execz":
            return self.exec == 0
        if op == "s_cbranch_execnz":
            return self.exec != 0
        if op == "s_cbranch_vccz":
            return (self.vcc & self.exec) == 0
        if op == "s_cbranch_vccnz":
            return (self.vcc & self.exec) != 0
        if op in ("s_cbranch_scc0", "s_cbranch_scc1"):
            if not isinstance(self.scc, int):
                raise Unsupported("branch on a symbolic condition")
            return self.scc == (1 if op.endswith("1") else 0)
        raise Unsupported(op)

    def _step(self, op, ops, mods, text):
        base = re.sub(r"_e(32|64)$", "", op)
        if op.startswith("s_waitcnt") or op in ("s_nop", "s_setprio", "s_sleep") or \
                op.startswith("s_sched") or op == "s_setreg_imm32_b32" or op == "s_denorm_mode":
            return
        # scalar: argument loads, exec and mask logic
        if op.startswith("s_load_dword"):
            n = {"s_load_dword": 1, "s_load_dwordx2": 2, "s_load_dwordx4": 4, "s_load_dwordx8": 8, "s_load_dwordx16": 16}[op]
            src = self.S.get(_reg(ops[1])[1])
            off = _imm(ops[2])
            if off is None:
                raise Unsupported("scalar load with a register offset")
            d = _reg(ops[0])[1]
            if src == ("kernarg", 0):
                for k in range(n):
                    o = off + 4 * k
                    if o in self.args:
                        self.S[d + k] = Aff(self.args[o])
                    else:
                        self.S[d + k] = ("arg", o) if o % 8 == 0 else ("arghi", o - 4)
                return
            base = self._ptr(ops[1])              # data: one leaf per dword
            for k in range(n):
                self.S[d + k] = self.leaf(base + Aff(off + 4 * k))
            return
        if self._salu(op, ops):
            return
        if op in ("s_and_saveexec_b64", "s_or_saveexec_b64"):
            old = self.exec
            m = self.mask(ops[1])
            self.setmask(ops[0], old)
            self.exec = (old & m) if "and" in op else (old | m)
            self.scc = int(self.exec != 0)
            return
        if op in ("s_and_b64", "s_or_b64", "s_xor_b64", "s_andn2_b64", "s_orn2_b64", "s_mov_b64"):
            a = self.mask(ops[1])
            b = self.mask(ops[2]) if len(ops) > 2 else None
            full = (1 << WAVE) - 1
            r = {"s_and_b64": lambda: a & b, "s_or_b64": lambda: a | b, "s_xor_b64": lambda: a ^ b,
                 "s_andn2_b64": lambda: a & ~b & full, "s_orn2_b64": lambda: (a | ~b) & full,
                 "s_mov_b64": lambda: a}[op]()
            self.setmask(ops[0], r)
            self.scc = int(r != 0)
            return
        if base.startswith("v_cmp_") or base.startswith("v_cmpx_"):
            self._cmp(base, ops)
            return
        # vector integer arithmetic on lane-derived values
        ints = {"v_lshlrev_b32", "v_lshrrev_b32", "v_ashrrev_i32", "v_and_b32", "v_or_b32", "v_xor_b32",
                "v_add_u32", "v_add_nc_u32", "v_sub_u32", "v_subrev_u32", "v_mul_lo_u32", "v_mul_u32_u24",
                "v_mbcnt_lo_u32_b32", "v_mbcnt_hi_u32_b32", "v_cndmask_b32", "v_mov_b32", "v_lshl_add_u32",
                "v_add_lshl_u32", "v_lshl_or_b32", "v_and_or_b32", "v_or3_b32", "v_xad_u32"}
        if base in ints:
            for l in self.lanes():
                self.setv(ops[0], l, self._int_op(base, ops, l))
            return
        if base in ("v_addc_co_u32", "v_subbrev_co_u32", "v_subb_co_u32", "v_addc_u32"):
            for l in self.lanes():
                self.setv(ops[0], l, HiWord())
            return
        if base in ("v_sub_co_u32", "v_subrev_co_u32"):
            for l in self.lanes():
                name = "v_sub_u32" if base == "v_sub_co_u32" else "v_subrev_u32"
                self.setv(ops[0], l, self._int_op(name, [ops[0], ops[2], ops[3]], l))
            return
        if base in ("v_add_co_u32",):
            for l in self.lanes():
                self.setv(ops[0], l, self._int_op("v_add_u32", [ops[0], ops[2], ops[3]], l))
            return
        # floating-point combines (plain or with a DPP source)
        fops = {"v_add_f32": "add", "v_max_f32": "max", "v_min_f32": "min", "v_mul_f32": "mul",
                "v_sub_f32": "sub", "v_subrev_f32": "subrev", "v_fma_f32": "fma", "v_fmac_f32": "fmac"}
        dpp = op.endswith("_dpp")
        fb = op[:-4] if dpp else base
        if fb in fops:
            self._fop(fops[fb], ops, mods if dpp else None)
            return
        if op == "v_mov_b32_dpp":
            vals = {}
            for l in self.lanes():
                if _dpp_writes(mods, l):
                    s = _dpp_src(mods, l)
                    if s is None and not any(m.startswith("bound_ctrl") for m in mods):
                        continue
                    vals[l] = self.v(ops[1], s) if s is not None else Node("const", leaf="0")
            for l, x in vals.items():
                self.setv(ops[0], l, x)
            return
        if op in ("v_readlane_b32", "v_readfirstlane_b32"):
            if op == "v_readfirstlane_b32":
                ls = self.lanes()
                if not ls:
                    raise Unsupported("v_readfirstlane_b32 with no lane active")
                src = ls[0]
            else:
                src = self.v(ops[2], 0)
                if not isinstance(src, Aff) or not src.concrete():
                    raise Unsupported("v_readlane_b32 lane not fixed")
                src = src.c & (WAVE - 1)
            self.S[_reg(ops[0])[1]] = self.v(ops[1], src)
            return
        if op == "ds_swizzle_b32":
            vals = {l: self._src_lane(ops[1], _swizzle_src(mods, l)) for l in self.lanes()}
            for l, x in vals.items():
                self.setv(ops[0], l, x)
            return
        if op == "ds_bpermute_b32":
            off = 0
            for m in mods:
                if m.startswith("offset:"):
                    off = int(m[len("offset:"):], 0)
            vals = {}
            for l in self.lanes():
                a = self.v(ops[1], l)
                if not isinstance(a, Aff) or not a.concrete():
                    raise Unsupported("ds_bpermute address not lane-derived")
                vals[l] = self._src_lane(ops[2], ((a.c + off) >> 2) & (WAVE - 1))
            for l, x in vals.items():
                self.setv(ops[0], l, x)
            return
        if op in ("v_accvgpr_write_b32", "v_accvgpr_read_b32", "v_accvgpr_mov_b32"):
            vals = {l: self.v(ops[1], l) for l in self.lanes()}
            for l, x in vals.items():
                self.setv(ops[0], l, x)
            return
        if op == "v_mad_u64_u32":
            # D (64 bits) = a * b + c (64 bits): the low word needs only c's low
            # word; the high word is kept only when every part is concrete
            for l in self.lanes():
                a, b = self.v(ops[2], l), self.v(ops[3], l)
                rc = _reg(ops[4])
                clo = self.v("v%d" % rc[1], l) if rc and rc[0] == "v" else self.v(ops[4], l)
                chi = self.v("v%d" % (rc[1] + 1), l) if rc and rc[0] == "v" and rc[2] == 2 else Aff(0)
                if not (isinstance(a, Aff) and isinstance(b, Aff) and isinstance(clo, Aff)):
                    raise Unsupported("v_mad_u64_u32 operands")
                if a.concrete():
                    lo = b.scale(a.c) + clo
                elif b.concrete():
                    lo = a.scale(b.c) + clo
                else:
                    raise Unsupported("v_mad_u64_u32 of two symbols")
                if lo.concrete() and isinstance(chi, Aff) and chi.concrete():
                    full = (a.c & 0xFFFFFFFF) * (b.c & 0xFFFFFFFF) + (clo.c & 0xFFFFFFFF) + ((chi.c & 0xFFFFFFFF) << 32)
                    self.setv(ops[0], l, Aff(full & 0xFFFFFFFF), 0)
                    self.setv(ops[0], l, Aff((full >> 32) & 0xFFFFFFFF), 1)
                else:
                    self.setv(ops[0], l, lo if not lo.concrete() else Aff(lo.c & 0xFFFFFFFF), 0)
                    self.setv(ops[0], l, Node("const", leaf="unknown-high-word"), 1)
            return
        if op == "v_lshlrev_b64":
            for l in self.lanes():
                sh = self.v(ops[1], l)
                r = _reg(ops[2])
                lo, hi = self.v("v%d" % r[1], l), self.v("v%d" % (r[1] + 1), l)
                if not all(isinstance(x, Aff) and x.concrete() for x in (sh, lo, hi)):
                    raise Unsupported("v_lshlrev_b64 on symbolic values")
                full = (((hi.c & 0xFFFFFFFF) << 32) | (lo.c & 0xFFFFFFFF)) << (sh.c & 63)
                self.setv(ops[0], l, Aff(full & 0xFFFFFFFF), 0)
                self.setv(ops[0], l, Aff((full >> 32) & 0xFFFFFFFF), 1)
            return
        if op in ("v_mfma_f32_16x16x32_bf16", "v_mfma_f32_16x16x32_f16"):
            self._mfma16(ops)
            return
        if op == "v_lshl_add_u64":
            # 64-bit (a << shift) + b on register pairs: the low word carries the
            # affine value, the high word marks a pointer (or is a concrete 0)
            for l in self.lanes():
                (alo, ahi), sh, (blo, bhi) = self._pair(ops[1], l), self.v(ops[2], l), self._pair(ops[3], l)
                if not (isinstance(sh, Aff) and sh.concrete()):
                    raise Unsupported("v_lshl_add_u64 shift")
                aptr, bptr = isinstance(ahi, HiWord), isinstance(bhi, HiWord)
                if (aptr and sh.c) or (aptr and bptr):
                    raise Unsupported("v_lshl_add_u64 on two pointers or a shifted pointer")
                self.setv(ops[0], l, alo.scale(1 << sh.c) + blo, 0)
                self.setv(ops[0], l, HiWord() if (aptr or bptr) else Aff(0), 1)
            return
        if op.startswith("ds_write") or op.startswith("ds_read"):
            self._lds(op, ops, mods)
            return
        if op.startswith("global_load_dword"):
            n = {"global_load_dword": 1, "global_load_dwordx2": 2, "global_load_dwordx3": 3,
                 "global_load_dwordx4": 4}[op]
            for l in self.lanes():
                addr = self._gaddr(ops[1], ops[2], mods, l)
                for k in range(n):
                    self.setv(ops[0], l, self.leaf(addr + Aff(4 * k)), k)
            return
        if op.startswith("global_store_dword"):
            n = {"global_store_dword": 1, "global_store_dwordx2": 2, "global_store_dwordx3": 3,
                 "global_store_dwordx4": 4}[op]
            r = _reg(ops[1])
            base = r[1] if r[0] == "v" else 1000 + r[1]
            for l in self.lanes():
                addr = self._gaddr(ops[0], ops[2], mods, l)
                for k in range(n):
                    x = self.V.get(base + k, [None] * WAVE)[l]
                    if not isinstance(x, Node):
                        x = Node("opaque", leaf="int " + repr(x))
                    a = addr + Aff(4 * k)
                    self.stores[a.key()] = (a, x)
            return
        # anything else: an uninterpreted function of its operands, named by
        # its own text (equal only to the same instruction on the same inputs)
        self.opaque.append(text)
        if ops:
            r = _reg(ops[0])
            if r and r[0] in "va":
                vals = {l: Node("opaque", [self._as_node(t, l) for t in ops[1:]], leaf=" ".join([op] + mods))
                        for l in self.lanes()}
                for l, x in vals.items():
                    for k in range(r[2]):
                        self.setv(ops[0], l, x if r[2] == 1 else Node("part%d" % k, [x]), k)
            elif r and r[0] == "s":
                for k in range(r[2]):
                    self.S[r[1] + k] = ("opaque", text)

    def _pair(self, tok, l):
        """A 64-bit operand as (low word value, high word value)."""
        r = _reg(tok)
        if r and r[2] == 2:
            if r[0] == "s":
                lo, hi = self.v("s%d" % r[1], l), self.v("s%d" % (r[1] + 1), l)
            else:
                lo, hi = self.v("v%d" % r[1], l), self.v("v%d" % (r[1] + 1), l)
            if isinstance(lo, Aff) and (isinstance(hi, HiWord) or (isinstance(hi, Aff) and hi.concrete() and hi.c == 0)):
                return lo, hi
            raise Unsupported("64-bit operand " + tok)
        i = _imm(tok)
        if i is not None:
            return Aff(i), Aff(0)
        raise Unsupported("64-bit operand " + tok)

    def _sval(self, tok):
        x = self.v(tok, 0) if _reg(tok) is None or _reg(tok)[0] == "s" else None
        return x

    def _salu(self, op, ops):
        """Scalar integer work on concrete values and affine addresses; False
        if op is not one of these."""
        b32 = {"s_add_i32", "s_add_u32", "s_sub_i32", "s_sub_u32", "s_mul_i32", "s_lshl_b32", "s_lshr_b32",
               "s_ashr_i32", "s_and_b32", "s_or_b32", "s_xor_b32", "s_min_i32", "s_min_u32", "s_max_i32",
               "s_max_u32", "s_mov_b32", "s_cselect_b32", "s_addc_u32", "s_subb_u32", "s_lshl1_add_u32",
               "s_lshl2_add_u32", "s_lshl3_add_u32", "s_lshl4_add_u32", "s_bfe_u32", "s_mul_hi_u32", "s_movk_i32"}
        if op.startswith("s_cmp_"):
            g = re.fullmatch(r"s_cmp_(eq|lg|lt|le|gt|ge)_(i32|u32|u64)", op)
            if not g:
                raise Unsupported(op)
            a, b = self._sval(ops[0]), self._sval(ops[1])
            if not (isinstance(a, Aff) and isinstance(b, Aff)):
                raise Unsupported("scalar compare on " + str(ops))
            d = a + b.neg()
            if not d.concrete():
                if g.group(1) in ("eq", "lg") and a.t and b.t and a.t == b.t:
                    pass
                else:
                    raise Unsupported("scalar compare on symbolic values")
            if a.concrete() and b.concrete():
                x, y = a.c, b.c
                if g.group(2) == "i32":
                    x, y = [(z & 0xFFFFFFFF) - (1 << 32) if (z & 0xFFFFFFFF) >> 31 else z & 0xFFFFFFFF for z in (x, y)]
                elif g.group(2) == "u32":
                    x, y = x & 0xFFFFFFFF, y & 0xFFFFFFFF
            else:
                x, y = d.c, 0
            self.scc = int({"eq": x == y, "lg": x != y, "lt": x < y, "le": x <= y, "gt": x > y, "ge": x >= y}[g.group(1)])
            return True
        if op == "s_mov_b64" and ops[0] not in ("exec", "vcc"):
            r, q = _reg(ops[0]), _reg(ops[1])
            if r and q and r[0] == q[0] == "s":
                self.S[r[1]], self.S[r[1] + 1] = self.S.get(q[1]), self.S.get(q[1] + 1)
                return True
            if r and q is None and _imm(ops[1]) is not None:
                self.S[r[1]], self.S[r[1] + 1] = Aff(_imm(ops[1])), Aff(0)
                return True
            return False
        if op not in b32:
            return False
        d = _reg(ops[0])
        if op in ("s_addc_u32", "s_subb_u32"):
            self.S[d[1]] = ("arghi", -1)                 # the high word of a 64-bit address
            return True
        if op == "s_movk_i32":
            v = _imm(ops[1]) & 0xFFFF
            self.S[d[1]] = Aff(v - 0x10000 if v >> 15 else v)
            return True
        if op == "s_mov_b32":
            x = self.S.get(_reg(ops[1])[1]) if _reg(ops[1]) else Aff(_imm(ops[1]) or 0)
            self.S[d[1]] = x
            return True
        if op == "s_cselect_b32":
            self.S[d[1]] = self._sval(ops[1]) if self.scc else self._sval(ops[2])
            return True
        a = [self._sval(t) for t in ops[1:]]
        if not all(isinstance(x, Aff) for x in a):
            raise Unsupported("scalar op %s on %s" % (op, ops))
        if op in ("s_add_i32", "s_add_u32"):
            r = a[0] + a[1]
        elif op in ("s_sub_i32", "s_sub_u32"):
            r = a[0] + a[1].neg()
        elif op == "s_mul_i32" and (a[0].concrete() or a[1].concrete()):
            r = a[1].scale(a[0].c) if a[0].concrete() else a[0].scale(a[1].c)
        elif op == "s_lshl_b32" and a[1].concrete():
            r = a[0].scale(1 << (a[1].c & 31))
        elif op.startswith("s_lshl") and op.endswith("_add_u32"):
            r = a[0].scale(1 << int(op[6])) + a[1]
        elif all(x.concrete() for x in a):
            c = [x.c & 0xFFFFFFFF for x in a]
            sg = [(z - (1 << 32)) if z >> 31 else z for z in c]
            f = {"s_lshr_b32": lambda: c[0] >> (c[1] & 31), "s_ashr_i32": lambda: sg[0] >> (c[1] & 31),
                 "s_and_b32": lambda: c[0] & c[1], "s_or_b32": lambda: c[0] | c[1], "s_xor_b32": lambda: c[0] ^ c[1],
                 "s_min_i32": lambda: min(sg), "s_max_i32": lambda: max(sg), "s_min_u32": lambda: min(c),
                 "s_max_u32": lambda: max(c), "s_mul_i32": lambda: c[0] * c[1],
                 "s_bfe_u32": lambda: (c[0] >> (c[1] & 31)) & ((1 << ((c[1] >> 16) & 0x7F)) - 1),
                 "s_mul_hi_u32": lambda: (c[0] * c[1]) >> 32}
            if op not in f:
                raise Unsupported(op)
            r = Aff(f[op]() & 0xFFFFFFFF)
        else:
            raise Unsupported("scalar op %s on symbolic values" % op)
        self.S[d[1]] = r
        self.scc = int(r.concrete() and (r.c & 0xFFFFFFFF) != 0) if op not in ("s_add_u32", "s_sub_u32") else 0
        return True

    def _lds(self, op, ops, mods):
        """LDS words move values between the waves of the workgroup (Sec. 6:
        a store to shared memory, a barrier and a load are one cross-wave
        exchange that combines nothing)."""
        g = re.fullmatch(r"ds_(read|write)(2?)(st64)?_b(32|64|128)", op)
        if not g:
            raise Unsupported(op)
        rd, two, st64, bits = g.group(1) == "read", g.group(2) == "2", g.group(3) is not None, int(g.group(4))
        words = bits // 32
        opt = {}
        for m in mods:
            k, _, v = m.partition(":")
            opt[k] = int(v, 0)
        if two:
            unit = (bits // 8) * (64 if st64 else 1)
            offs = [opt.get("offset0", 0) * unit, opt.get("offset1", 0) * unit]
        else:
            offs = [opt.get("offset", 0)]
        addr_tok = ops[1] if rd else ops[0]
        data = [ops[0]] if rd else ops[1:]
        vals = {}
        for l in self.lanes():
            a = self.v(addr_tok, l)
            if not isinstance(a, Aff) or not a.concrete():
                raise Unsupported("LDS address not lane-derived")
            for j, off in enumerate(offs):
                for k in range(words):
                    byte = (a.c + off) & 0xFFFFFFFF
                    if rd:
                        vals[(l, j * words + k)] = self.lds.get(byte + 4 * k, Node("const", leaf="lds-uninit"))
                    else:
                        r = _reg(data[j] if two else data[0])
                        if not r or r[0] not in "va":
                            raise Unsupported("LDS store of " + str(data))
                        base = r[1] if r[0] == "v" else 1000 + r[1]
                        self.lds[byte + 4 * k] = self.V.get(base + k, [None] * WAVE)[l]
        if rd:
            for (l, k), x in vals.items():
                self.setv(ops[0], l, x, k)

    def _as_node(self, tok, l):
        try:
            x = self.v(tok, l)
        except Unsupported:
            return Node("const", leaf=tok)
        if isinstance(x, Node):
            return x
        return Node("const", leaf=repr(x) if isinstance(x, Aff) else str(x))

    def _src_lane(self, tok, s):
        if s is None or not (self.exec >> s) & 1:
            return Node("const", leaf="0")
        return self.v(tok, s)

    def _gaddr(self, vtok, stok, mods, l):
        off = 0
        for m in mods:
            if m.startswith("offset:"):
                off = int(m[len("offset:"):], 0)
        if stok == "off":
            r = _reg(vtok)
            if not r or r[0] != "v" or r[2] != 2:
                raise Unsupported("vector address " + vtok)
            lo, hi = self.V.get(r[1], [None] * WAVE)[l], self.V.get(r[1] + 1, [None] * WAVE)[l]
            if not isinstance(lo, Aff) or not isinstance(hi, HiWord):
                raise Unsupported("64-bit address not from a pointer")
            return lo + Aff(off)
        base = self._ptr(stok)
        v = self.v(vtok, l)
        if not isinstance(v, Aff):
            raise Unsupported("address from a float")
        return base + v + Aff(off)

    def _int_op(self, base, ops, l):
        def ival(tok):
            x = self.v(tok, l)
            if not isinstance(x, Aff):
                raise Unsupported("integer op on a float")
            return x
        if base == "v_mov_b32":
            return self.v(ops[1], l)
        if base == "v_cndmask_b32":
            m = self.mask(ops[3]) if len(ops) > 3 else self.vcc
            return self.v(ops[2], l) if (m >> l) & 1 else self.v(ops[1], l)
        if base == "v_mbcnt_lo_u32_b32":
            m, a = ival(ops[1]), ival(ops[2])
            return Aff(bin((m.c & 0xFFFFFFFF) & ((1 << min(l, 32)) - 1)).count("1")) + a
        if base == "v_mbcnt_hi_u32_b32":
            m, a = ival(ops[1]), ival(ops[2])
            return Aff(bin((m.c & 0xFFFFFFFF) & ((1 << max(l - 32, 0)) - 1)).count("1")) + a
        a = [ival(t) for t in ops[1:]]
        if base in ("v_add_u32", "v_add_nc_u32"):
            return a[0] + a[1]
        if base == "v_sub_u32":
            return a[0] + a[1].neg()
        if base == "v_subrev_u32":
            return a[1] + a[0].neg()
        if base == "v_lshlrev_b32" and a[0].concrete():
            return a[1].scale(1 << a[0].c)
        if base in ("v_mul_lo_u32", "v_mul_u32_u24"):
            if a[0].concrete():
                return a[1].scale(a[0].c)
            if a[1].concrete():
                return a[0].scale(a[1].c)
        if base == "v_lshl_add_u32" and a[1].concrete():
            return a[0].scale(1 << a[1].c) + a[2]
        if base == "v_add_lshl_u32" and a[2].concrete():
            return (a[0] + a[1]).scale(1 << a[2].c)
        if all(x.concrete() for x in a):
            c = [x.c & 0xFFFFFFFF for x in a]
            f = {"v_lshlrev_b32": lambda: c[1] << (c[0] & 31), "v_lshrrev_b32": lambda: c[1] >> (c[0] & 31),
                 "v_ashrrev_i32": lambda: (c[1] - (1 << 32) if c[1] >> 31 else c[1]) >> (c[0] & 31),
                 "v_and_b32": lambda: c[0] & c[1], "v_or_b32": lambda: c[0] | c[1], "v_xor_b32": lambda: c[0] ^ c[1],
                 "v_lshl_or_b32": lambda: (c[0] << (c[1] & 31)) | c[2], "v_and_or_b32": lambda: (c[0] & c[1]) | c[2],
                 "v_or3_b32": lambda: c[0] | c[1] | c[2], "v_xad_u32": lambda: (c[0] ^ c[1]) + c[2]}
            if base in f:
                return Aff(f[base]() & 0xFFFFFFFF)
        raise Unsupported("integer op %s on symbolic values" % base)

    def _cmp(self, base, ops):
        g = re.fullmatch(r"v_cmpx?_(\w+?)_([iuf]\d+)", base)
        if not g:
            raise Unsupported(base)
        rel, ty = g.group(1), g.group(2)
        if ty.startswith("f"):
            raise Unsupported("compare on floating-point data")
        dst, a_t, b_t = (ops[0], ops[1], ops[2]) if len(ops) == 3 else ("vcc", ops[0], ops[1])
        m = 0
        for l in self.lanes():
            a, b = self.v(a_t, l), self.v(b_t, l)
            if not (isinstance(a, Aff) and isinstance(b, Aff) and a.concrete() and b.concrete()):
                raise Unsupported("compare on symbolic values")
            x, y = a.c & 0xFFFFFFFF, b.c & 0xFFFFFFFF
            if ty.startswith("i"):
                x, y = (x - (1 << 32) if x >> 31 else x), (y - (1 << 32) if y >> 31 else y)
            r = {"lt": x < y, "le": x <= y, "gt": x > y, "ge": x >= y, "eq": x == y, "ne": x != y,
                 "lg": x != y}.get(rel)
            if r is None:
                raise Unsupported(base)
            m |= int(r) << l
        if base.startswith("v_cmpx_"):
            self.exec &= m
        self.setmask(dst, m)

    def _fop(self, name, ops, dppmods):
        vals = {}
        for l in self.lanes():
            if dppmods is not None and not _dpp_writes(dppmods, l):
                continue
            if dppmods is not None:
                s = _dpp_src(dppmods, l)
                if s is None and not any(m.startswith("bound_ctrl") for m in dppmods):
                    continue                      # an invalid source lane leaves the lane unwritten
                a0 = self.fval(ops[1], s) if s is not None else Node("const", leaf="0")
            else:
                a0 = self.fval(ops[1], l)
            rest = [self.fval(t, l) for t in ops[2:]]
            args = [a0] + rest
            for x in args:
                if not isinstance(x, Node):
                    raise Unsupported("floating-point op on an integer register")
            if name == "sub":
                vals[l] = Node("sub", args)
            elif name == "subrev":
                vals[l] = Node("sub", [args[1], args[0]])
            elif name == "fmac":
                vals[l] = Node("fma", [args[0], args[1], self.fval(ops[0], l)])
            else:
                vals[l] = Node(name, args)
        for l, x in vals.items():
            self.setv(ops[0], l, x)

    # --- results
    def roots(self, outputs=None):
        """(address, canonical tree) per stored element, in address order;
        outputs: a list of (pointer-argument byte offset, element byte
        offset) pairs to keep, None for every store."""
        items = sorted(self.stores.values(), key=lambda an: an[0].key())
        if outputs is not None:
            want = {Aff(o, {"arg%d" % p: 1}).key() for p, o in outputs}
            items = [an for an in items if an[0].key() in want]
        return [(repr(a), canon(n)) for a, n in items]

    def signature(self, outputs=None) -> str:
        h = hashlib.sha256()
        for a, t in self.roots(outputs):
            h.update(a.encode())
            h.update(b"=")
            h.update(hashlib.sha256(t.encode()).digest())
            h.update(b";")
        return h.hexdigest()


def compile_asm(source: str, include_dirs=(), extra=()) -> str:
    """gfx950 assembly of a HIP source file (device code only, -O3, the
    library's own floating-point flags)."""
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "k.s")
        cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-ffp-contract=off", "-fno-fast-math",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "--cuda-device-only", "-S",
               "-o", out, source] + ["-I" + i for i in include_dirs] + list(extra)
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError("hipcc failed:\n" + r.stderr[-2000:])
        return open(out).read()


def classes(signatures: dict) -> list[list]:
    """Configurations grouped by signature (Sec. 6: the pruning predicate
    keeps the class of a reference configuration)."""
    by = {}
    for k, s in signatures.items():
        by.setdefault(s, []).append(k)
    return sorted(by.values(), key=lambda g: str(g[0]))


def prune(signatures: dict, reference) -> list:
    """The configurations bitwise equivalent to the reference (Sec. 6: a
    search that benchmarks only these keeps the reference's bits); reference
    is a key of signatures or a signature."""
    ref = signatures.get(reference, reference)
    return [k for k, s in signatures.items() if s == ref]


def main(argv=None) -> int:
    """python -m paper_2609_11356_amd.order_check SOURCE.hip [KERNEL ...]
    [--block N] [--arg OFFSET=VALUE ...] [-I DIR ...]: the classes of the
    named kernels (every entry function of SOURCE when none is named)."""
    import argparse
    ap = argparse.ArgumentParser(prog="order_check", description=main.__doc__)
    ap.add_argument("source")
    ap.add_argument("kernels", nargs="*")
    ap.add_argument("--block", type=int, default=64, help="threads per workgroup (x only)")
    ap.add_argument("--arg", action="append", default=[], help="bind a 32-bit argument: byte offset=value")
    ap.add_argument("-I", dest="include", action="append", default=[])
    a = ap.parse_args(argv)
    asm = compile_asm(a.source, a.include)
    names = a.kernels or sorted(functions(asm))
    args = {int(k, 0): int(v, 0) for k, v in (x.split("=") for x in a.arg)}
    sigs = {}
    for n in names:
        try:
            sigs[n] = Walk(asm, n, block=(a.block, 1, 1), args=args).signature()
        except Unsupported as e:
            print("%s: not walked (%s)" % (n, e))
    for c in classes(sigs):
        print("%s  %s" % (sigs[c[0]][:16], " ".join(c)))
    return 0


if __name__ == "__main__":
    raise SystemExit(main())
