"""Map the AES S-box circuit onto three-input lookup gates (gfx950 v_bitop3_b32).

    python paper_2410_15240_amd/csrc/gen_sbox_lut3.py > paper_2410_15240_amd/csrc/sbox_lut3.inc

(the body of bs::sbox in aes_bitslice.h).

Input: Boyar and Peralta's depth-16 S-box circuit of 128 two-input gates (J. Boyar
and R. Peralta, "A depth-16 circuit for the AES S-box", IFIP SEC 2012), written
below as a gate list. Output: C statements computing the same eight outputs with
gates of up to three inputs, each `lut3<TT>(a, b, c)` with TT the 8-bit truth table
indexed by a*4 + b*2 + c (the v_bitop3_b32 convention).

Method: standard cut-based technology mapping. Every node gets its 3-feasible
cuts (sets of at most three nodes from which it is computed); a cover is chosen
by area flow and refined by exact-area recovery passes, which trade duplicated
logic against shared nodes. The script checks the mapped network against the
gate list on all 256 inputs before it prints anything.
"""
import random
import sys

RESTARTS = 200

GATES = """
T1 = U0 ^ U3
T2 = U0 ^ U5
T3 = U0 ^ U6
T4 = U3 ^ U5
T5 = U4 ^ U6
T6 = T1 ^ T5
T7 = U1 ^ U2
T8 = U7 ^ T6
T9 = U7 ^ T7
T10 = T6 ^ T7
T11 = U1 ^ U5
T12 = U2 ^ U5
T13 = T3 ^ T4
T14 = T6 ^ T11
T15 = T5 ^ T11
T16 = T5 ^ T12
T17 = T9 ^ T16
T18 = U3 ^ U7
T19 = T7 ^ T18
T20 = T1 ^ T19
T21 = U6 ^ U7
T22 = T7 ^ T21
T23 = T2 ^ T22
T24 = T2 ^ T10
T25 = T20 ^ T17
T26 = T3 ^ T16
T27 = T1 ^ T12
M1 = T13 & T6
M2 = T23 & T8
M3 = T14 ^ M1
M4 = T19 & U7
M5 = M4 ^ M1
M6 = T3 & T16
M7 = T22 & T9
M8 = T26 ^ M6
M9 = T20 & T17
M10 = M9 ^ M6
M11 = T1 & T15
M12 = T4 & T27
M13 = M12 ^ M11
M14 = T2 & T10
M15 = M14 ^ M11
M16 = M3 ^ M2
M17 = M5 ^ T24
M18 = M8 ^ M7
M19 = M10 ^ M15
M20 = M16 ^ M13
M21 = M17 ^ M15
M22 = M18 ^ M13
M23 = M19 ^ T25
M24 = M22 ^ M23
M25 = M22 & M20
M26 = M21 ^ M25
M27 = M20 ^ M21
M28 = M23 ^ M25
M29 = M28 & M27
M30 = M26 & M24
M31 = M20 & M23
M32 = M27 & M31
M33 = M27 ^ M25
M34 = M21 & M22
M35 = M24 & M34
M36 = M24 ^ M25
M37 = M21 ^ M29
M38 = M32 ^ M33
M39 = M23 ^ M30
M40 = M35 ^ M36
M41 = M38 ^ M40
M42 = M37 ^ M39
M43 = M37 ^ M38
M44 = M39 ^ M40
M45 = M42 ^ M41
M46 = M44 & T6
M47 = M40 & T8
M48 = M39 & U7
M49 = M43 & T16
M50 = M38 & T9
M51 = M37 & T17
M52 = M42 & T15
M53 = M45 & T27
M54 = M41 & T10
M55 = M44 & T13
M56 = M40 & T23
M57 = M39 & T19
M58 = M43 & T3
M59 = M38 & T22
M60 = M37 & T20
M61 = M42 & T1
M62 = M45 & T4
M63 = M41 & T2
L0 = M61 ^ M62
L1 = M50 ^ M56
L2 = M46 ^ M48
L3 = M47 ^ M55
L4 = M54 ^ M58
L5 = M49 ^ M61
L6 = M62 ^ L5
L7 = M46 ^ L3
L8 = M51 ^ M59
L9 = M52 ^ M53
L10 = M53 ^ L4
L11 = M60 ^ L2
L12 = M48 ^ M51
L13 = M50 ^ L0
L14 = M52 ^ M61
L15 = M55 ^ L1
L16 = M56 ^ L0
L17 = M57 ^ L1
L18 = M58 ^ L8
L19 = M63 ^ L4
L20 = L0 ^ L1
L21 = L1 ^ L7
L22 = L3 ^ L12
L23 = L18 ^ L2
L24 = L15 ^ L9
L25 = L6 ^ L10
L26 = L7 ^ L9
L27 = L8 ^ L10
L28 = L11 ^ L14
L29 = L11 ^ L17
S0 = L6 ^ L24
S1 = L16 ~^ L26
S2 = L19 ~^ L28
S3 = L6 ^ L21
S4 = L20 ^ L22
S5 = L25 ^ L29
S6 = L13 ~^ L27
S7 = L6 ~^ L23
"""

INPUTS = ["U%d" % i for i in range(8)]
OUTPUTS = ["S%d" % i for i in range(8)]
OPS = {"^": lambda a, b: a ^ b, "&": lambda a, b: a & b, "~^": lambda a, b: 1 ^ a ^ b}


def parse():
    nodes = {}
    for line in GATES.strip().splitlines():
        name, expr = [x.strip() for x in line.split("=")]
        a, op, b = expr.split()
        nodes[name] = (op, a, b)
    return nodes


def evaluate(nodes, x):
    v = {"U%d" % i: (x >> (7 - i)) & 1 for i in range(8)}
    for name, (op, a, b) in nodes.items():
        v[name] = OPS[op](v[a], v[b])
    return v


def truth_table(nodes, root, leaves):
    """8-bit truth table of root over the ordered leaves (index a*4 + b*2 + c)."""
    leaves = list(leaves) + [None] * (3 - len(leaves))
    tt = 0
    for idx in range(8):
        assign = {leaves[0]: (idx >> 2) & 1, leaves[1]: (idx >> 1) & 1, leaves[2]: idx & 1}
        memo = {}

        def val(n):
            if n in assign:
                return assign[n]
            if n in memo:
                return memo[n]
            op, a, b = nodes[n]
            memo[n] = OPS[op](val(a), val(b))
            return memo[n]
        if val(root):
            tt |= 1 << idx
    return tt


def enumerate_cuts(nodes):
    cuts = {u: [frozenset([u])] for u in INPUTS}
    for name, (op, a, b) in nodes.items():
        cs = {frozenset([name])}
        for ca in cuts[a]:
            for cb in cuts[b]:
                u = ca | cb
                if len(u) <= 3:
                    cs.add(u)
        # drop dominated cuts (a superset of another cut of the same node)
        cs = [c for c in cs if not any(o < c for o in cs)]
        cuts[name] = cs
    return cuts


def select_cover(nodes, cuts, fanout_est):
    """Pick one cut per node by area flow, then cover from the outputs."""
    af, best = {u: 0.0 for u in INPUTS}, {}
    for name in nodes:
        cands = []
        for c in cuts[name]:
            if c == frozenset([name]):
                continue
            cands.append((1.0 + sum(af[l] / max(fanout_est.get(l, 1), 1) for l in c), len(c), sorted(c), c))
        cands.sort(key=lambda t: (t[0], t[1], t[2]))
        af[name], best[name] = cands[0][0], cands[0][3]
    chosen, stack = {}, list(OUTPUTS)
    while stack:
        n = stack.pop()
        if n in chosen or n in INPUTS:
            continue
        chosen[n] = best[n]
        stack.extend(best[n])
    return chosen


def cover_size(sel):
    need, stack = set(), list(OUTPUTS)
    while stack:
        n = stack.pop()
        if n in need or n in INPUTS:
            continue
        need.add(n)
        stack.extend(sel[n])
    return need


def exact_area(nodes, cuts, start, rng=None):
    """Area recovery: visit the nodes (in a random order when rng is given) and
    give each the cut that minimises the total number of gates of the cover,
    until no single change helps."""
    full = dict(start)
    for name in nodes:           # every node gets some cut, in case it becomes needed
        if name not in full:
            full[name] = min((c for c in cuts[name] if c != frozenset([name])), key=len)
    names = list(nodes)
    size = len(cover_size(full))
    improved = True
    while improved:
        improved = False
        if rng is not None:
            rng.shuffle(names)
        for name in names:
            for c in cuts[name]:
                if c == frozenset([name]) or c == full[name]:
                    continue
                trial = dict(full)
                trial[name] = c
                s = len(cover_size(trial))
                if s < size:
                    full, size, improved = trial, s, True
    return {n: full[n] for n in cover_size(full)}


def topo(nodes, chosen):
    order, seen = [], set(INPUTS)

    def visit(n):
        if n in seen:
            return
        for l in sorted(chosen[n]):
            visit(l)
        seen.add(n)
        order.append(n)
    for o in OUTPUTS:
        visit(o)
    return order


def main():
    nodes = parse()
    cuts = enumerate_cuts(nodes)
    fan = {}
    for op, a, b in nodes.values():
        fan[a] = fan.get(a, 0) + 1
        fan[b] = fan.get(b, 0) + 1
    chosen = select_cover(nodes, cuts, fan)
    for _ in range(3):      # refine the fanout estimate with the current cover
        fan2 = {}
        for n, c in chosen.items():
            for l in c:
                fan2[l] = fan2.get(l, 0) + 1
        chosen = select_cover(nodes, cuts, fan2)
    chosen = exact_area(nodes, cuts, chosen)
    # restarts from random covers (fixed seeds, so the output is reproducible)
    for seed in range(RESTARTS):
        rng = random.Random(seed)
        start = {n: rng.choice([c for c in cuts[n] if c != frozenset([n])]) for n in nodes}
        cand = exact_area(nodes, cuts, start, rng)
        if len(cand) < len(chosen):
            chosen = cand
    order = topo(nodes, chosen)
    gates = []
    for n in order:
        leaves = sorted(chosen[n])
        gates.append((n, leaves, truth_table(nodes, n, leaves)))
    # check the mapped network on every input
    for x in range(256):
        ref = evaluate(nodes, x)
        v = {"U%d" % i: (x >> (7 - i)) & 1 for i in range(8)}
        for n, leaves, tt in gates:
            bits = [v[l] for l in leaves] + [0] * (3 - len(leaves))
            v[n] = (tt >> (bits[0] * 4 + bits[1] * 2 + bits[2])) & 1
        assert all(v[o] == ref[o] for o in OUTPUTS), x
    print("    // %d three-input gates (gen_sbox_lut3.py); inputs U0..U7 and outputs S0..S7 most"
          % len(gates))
    print("    // significant bit first")
    for i in range(8):
        print("    const uint32_t U%d = x[%d];" % (i, 7 - i))
    for n, leaves, tt in gates:
        args = leaves + ["0u"] * (3 - len(leaves))
        print("    const uint32_t %s = lut3<0x%02X>(%s);" % (n, tt, ", ".join(args)))
    for i in range(8):
        print("    x[%d] = S%d;" % (7 - i, i))
    return 0


if __name__ == "__main__":
    sys.exit(main())
