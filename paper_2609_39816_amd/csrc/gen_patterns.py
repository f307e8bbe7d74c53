"""Writes fm_patterns.inc: the nonzero structures (not the coefficient
values) of the scheme families the kernels are specialized for.

A formation or reconstruction kernel compiled for a pattern has every block
index as a compile-time constant, so the operand blocks live in registers
with static indices; only the coefficient values are read per gauge.  The
library matches each evaluated scheme against these patterns at run time and
falls back to a generic kernel when none matches.

Families: Strassen applied 1, 2 and 3 times (and any sign variant of them,
which keeps the nonzero structure, Sec. 2.1), Laderman 3x3x3, the dense
structures that random invertible gauges of Strassen and Laderman produce,
and the rank-1 plain product.

Run:  python gen_patterns.py  (from any directory)
"""
from __future__ import annotations

import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))
import schemes  # noqa: E402  (the package's own tables)


def kron_nz(a, b):
    """Nonzero structure of scheme b applied inside the blocks of scheme a
    (outer level a): r = ra*Rb + rb, i = ia*mb + ib, l = la*kb + lb, ..."""
    (Ua, Va, Wa, ma, ka, na), (Ub, Vb, Wb, mb, kb, nb) = a, b
    Ra, Rb = Ua.shape[0], Ub.shape[0]
    m, k, n = ma * mb, ka * kb, na * nb
    U = np.zeros((Ra * Rb, m * k), bool)
    V = np.zeros((Ra * Rb, k * n), bool)
    W = np.zeros((Ra * Rb, m * n), bool)
    for ra in range(Ra):
        for rb in range(Rb):
            r = ra * Rb + rb
            for ia in range(ma):
                for ib in range(mb):
                    for la in range(ka):
                        for lb in range(kb):
                            U[r, (ia * mb + ib) * k + la * kb + lb] = Ua[ra, ia * ka + la] and Ub[rb, ib * kb + lb]
            for la in range(ka):
                for lb in range(kb):
                    for ja in range(na):
                        for jb in range(nb):
                            V[r, (la * kb + lb) * n + ja * nb + jb] = Va[ra, la * na + ja] and Vb[rb, lb * nb + jb]
            for ia in range(ma):
                for ib in range(mb):
                    for ja in range(na):
                        for jb in range(nb):
                            W[r, (ia * mb + ib) * n + ja * nb + jb] = Wa[ra, ia * na + ja] and Wb[rb, ib * nb + jb]
    return U, V, W, m, k, n


def kron_vals(a, b):
    """Coefficient values of scheme b applied inside the blocks of scheme a
    (same index maps as kron_nz), float64."""
    (Ua, Va, Wa, ma, ka, na), (Ub, Vb, Wb, mb, kb, nb) = a, b
    Ra, Rb = Ua.shape[0], Ub.shape[0]
    m, k, n = ma * mb, ka * kb, na * nb
    U = np.zeros((Ra * Rb, m * k))
    V = np.zeros((Ra * Rb, k * n))
    for ra in range(Ra):
        for rb in range(Rb):
            r = ra * Rb + rb
            for ia in range(ma):
                for ib in range(mb):
                    for la in range(ka):
                        for lb in range(kb):
                            U[r, (ia * mb + ib) * k + la * kb + lb] = Ua[ra, ia * ka + la] * Ub[rb, ib * kb + lb]
            for la in range(ka):
                for lb in range(kb):
                    for ja in range(na):
                        for jb in range(nb):
                            V[r, (la * kb + lb) * n + ja * nb + jb] = Va[ra, la * na + ja] * Vb[rb, lb * nb + jb]
    return U, V, None, m, k, n


def power_vals(base, L):
    out = base
    for _ in range(L - 1):
        out = kron_vals(out, base)
    return out


def nz(base):
    U, V, W, m, k, n = base
    return U != 0, V != 0, W != 0, m, k, n


def power_nz(base, L):
    out = nz(base)
    for _ in range(L - 1):
        out = kron_nz(out, nz(base))
    return out


def dense(R, m, k, n):
    return (np.ones((R, m * k), bool), np.ones((R, k * n), bool), np.ones((R, m * n), bool), m, k, n)


# Coefficient values of the families whose block sums share prefixes: the
# base scheme flattened.  A sign variant multiplies every coefficient of a
# block by that block's sign, so its chains share the same prefixes; the
# library finds each gauge's block signs on the host and the kernels build
# the coefficients from them and these values.
VALUES = {
    "Strassen1": power_vals(schemes.strassen(), 1),
    "Strassen2": power_vals(schemes.strassen(), 2),
    "Strassen3": power_vals(schemes.strassen(), 3),
    "Laderman1": power_vals(schemes.laderman(), 1),
}

FAMILIES = [
    ("Classical1", nz(schemes.classical(1, 1, 1))),
    ("Strassen1", power_nz(schemes.strassen(), 1)),
    ("Strassen2", power_nz(schemes.strassen(), 2)),
    ("Strassen3", power_nz(schemes.strassen(), 3)),
    ("Laderman1", power_nz(schemes.laderman(), 1)),
    ("DenseR7G2", dense(7, 2, 2, 2)),
    ("DenseR23G3", dense(23, 3, 3, 3)),
]


def lists(U, V, W, m, k, n):
    """Per product: A blocks (i,l) row-major -> i*k + l; B blocks (l,j)
    row-major -> j*k + l (index into B^T's n x k grid); C blocks (i,j)
    row-major -> i*n + j."""
    R = U.shape[0]
    out = {}
    for side in "ABW":
        rowptr, idx = [0], []
        for r in range(R):
            if side == "A":
                idx += [i * k + l for i in range(m) for l in range(k) if U[r, i * k + l]]
            elif side == "B":
                idx += [j * k + l for l in range(k) for j in range(n) if V[r, l * n + j]]
            else:
                idx += [i * n + j for i in range(m) for j in range(n) if W[r, i * n + j]]
            rowptr.append(len(idx))
        out[side] = (rowptr, idx)
    return out


def trie(rowptr, idx, vals):
    """Prefix sharing of the block-sum chains of one side.

    Chain r is the list of (block idx[e], coefficient vals[e]) for e in
    [rowptr[r], rowptr[r + 1]), summed by fused multiply-adds in that order
    from +0.  Chains that start with the same (block, coefficient) entries
    compute the same partial sums, so the distinct prefixes form a trie:
    node = one entry appended to its parent's partial sum.  Returns the
    nodes in depth-first order (parent before children; a node's parent is
    the latest node one level up) as (depth, block, representative entry),
    the products completed at each node (CSR over the completion order),
    and the representative entry of every node (its coefficient is the
    node's)."""
    R = len(rowptr) - 1
    children, key = {}, {}
    nodes = []  # (parent, block, entry, depth)
    ends = {}
    for r in range(R):
        parent, prefix = -1, ()
        for pos, e in enumerate(range(rowptr[r], rowptr[r + 1])):
            prefix = prefix + ((idx[e], float(vals[e])),)
            if prefix not in key:
                key[prefix] = len(nodes)
                nodes.append((parent, idx[e], e, pos))
                children.setdefault(parent, []).append(key[prefix])
            parent = key[prefix]
        ends.setdefault(parent, []).append(r)
    order = []

    def dfs(n):
        order.append(n)
        for c in children.get(n, []):
            dfs(c)
    for c in children.get(-1, []):
        dfs(c)
    depth = [nodes[n][3] for n in order]
    blk = [nodes[n][1] for n in order]
    ent = [nodes[n][2] for n in order]
    endptr, endprod = [0], []
    for n in order:
        endprod += ends.get(n, [])
        endptr.append(len(endprod))
    return depth, blk, ent, endptr, endprod


def f32bits(v):
    """fp32 bit pattern of v (exactly representable) as a C literal."""
    b = np.float32(v)
    assert float(b) == float(v)
    return f"0x{int(b.view(np.uint32)):08x}u"


def arr(vals, per_line=24):
    s = [str(v) for v in vals]
    lines = [", ".join(s[i:i + per_line]) for i in range(0, len(s), per_line)]
    return "{\n      " + ",\n      ".join(lines) + "}"


def main():
    out = ["// Generated by gen_patterns.py -- nonzero structures of the scheme",
           "// families with specialized kernels.  Do not edit by hand.",
           "#pragma once", "#include <stdint.h>", "", "namespace fm {", "namespace pat {", ""]
    names = []
    for name, fam in FAMILIES:
        U, V, W, m, k, n = fam
        R = U.shape[0]
        L = lists(U, V, W, m, k, n)
        out.append(f"struct {name} {{")
        out.append(f"  static constexpr int gm = {m}, gk = {k}, gn = {n}, R = {R};")
        for side, nbk in (("A", m * k), ("B", n * k), ("W", m * n)):
            rowptr, idx = L[side]
            out.append(f"  struct {side} {{")
            out.append(f"    static constexpr int R = {R}, NB = {nbk}, NNZ = {len(idx)};")
            out.append(f"    static constexpr int16_t rowptr[{R + 1}] = {arr(rowptr)};")
            out.append(f"    static constexpr int16_t idx[{max(1, len(idx))}] = {arr(idx or [0])};")
            if side != "W" and name in VALUES:
                Uv, Vv = VALUES[name][0], VALUES[name][1]
                vals = []
                for r in range(R):
                    if side == "A":
                        vals += [Uv[r, i * k + l] for i in range(m) for l in range(k) if Uv[r, i * k + l]]
                    else:
                        vals += [Vv[r, l * n + j] for l in range(k) for j in range(n) if Vv[r, l * n + j]]
                assert len(vals) == len(idx)
                depth, blk, ent, endptr, endprod = trie(rowptr, idx, vals)
                out.append("    // prefix-shared chains (depth-first trie; see gen_patterns.trie) and the")
                out.append("    // base scheme's coefficients (fp32 bits) per node and per list entry")
                out.append(f"    static constexpr bool TRIE = true;")
                out.append(f"    static constexpr int NN = {len(depth)}, MAXD = {max(depth) + 1};")
                out.append(f"    static constexpr int16_t tdepth[{len(depth)}] = {arr(depth)};")
                out.append(f"    static constexpr int16_t tblk[{len(depth)}] = {arr(blk)};")
                out.append(f"    static constexpr int16_t tent[{len(depth)}] = {arr(ent)};")
                out.append(f"    static constexpr int16_t tendptr[{len(endptr)}] = {arr(endptr)};")
                out.append(f"    static constexpr int16_t tendprod[{len(endprod)}] = {arr(endprod)};")
                out.append(f"    static constexpr uint32_t tval[{len(depth)}] = "
                           f"{arr([f32bits(vals[e]) for e in ent], 8)};")
                out.append(f"    static constexpr uint32_t val[{len(vals)}] = {arr([f32bits(v) for v in vals], 8)};")
            else:
                out.append("    static constexpr bool TRIE = false;")
                out.append("    static constexpr int NN = 0, MAXD = 1;")
                out.append("    static constexpr int16_t tdepth[1] = {0}, tblk[1] = {0}, tent[1] = {0};")
                out.append("    static constexpr int16_t tendptr[2] = {0, 0}, tendprod[1] = {0};")
                out.append("    static constexpr uint32_t tval[1] = {0}, val[1] = {0};")
            out.append("  };")
        # where H_rs = <w_r, w_s> <u_r, u_s> of the joint rounding can be
        # nonzero: both products share a block of A and one of C (families of
        # at most 64 products only)
        hp, hi = [0], []
        if R <= 64:
            Ou = (U.astype(int) @ U.T.astype(int)) > 0
            Ow = (W.astype(int) @ W.T.astype(int)) > 0
            for r in range(R):
                hi += [t for t in range(R) if Ou[r, t] and Ow[r, t]]
                hp.append(len(hi))
        else:
            hp = [0] * (R + 1)
        out.append("  struct H {")
        out.append(f"    static constexpr bool JOINT = {'true' if R <= 64 else 'false'};")
        out.append(f"    static constexpr int R = {R}, NNZ = {len(hi)};")
        out.append(f"    static constexpr int16_t rowptr[{R + 1}] = {arr(hp)};")
        out.append(f"    static constexpr int16_t idx[{max(1, len(hi))}] = {arr(hi or [0])};")
        out.append("  };")
        out.append("};")
        out.append("")
        names.append(name)
    out.append("#define FM_PATTERN_FAMILIES(X) " + " ".join(f"X({n})" for n in names))
    out.append("")
    out.append("}  // namespace pat")
    out.append("}  // namespace fm")
    inc = os.path.join(HERE, "fm_patterns.inc")
    text = "\n".join(out) + "\n"
    if not os.path.exists(inc) or open(inc).read() != text:
        with open(inc, "w") as f:
            f.write(text)
    # one translation unit per family, so the unrolled kernels build in parallel
    for name in names:
        path = os.path.join(HERE, f"fm_fam_{name}.hip")
        text = ("// Generated by gen_patterns.py: the specialized kernels of the " + name + "\n"
                "// family.  Do not edit by hand.\n"
                '#include "fm_device.h"\n'
                '#include "fm_joint.h"\n\n'
                "namespace fm {\n"
                f"FM_DEFINE_FAMILY({name})\n"
                f"FM_DEFINE_JOINT({name})\n"
                "}  // namespace fm\n")
        old = open(path).read() if os.path.exists(path) else None
        if old != text:
            with open(path, "w") as f:
                f.write(text)


def family_names():
    return [name for name, _ in FAMILIES]


if __name__ == "__main__":
    main()
