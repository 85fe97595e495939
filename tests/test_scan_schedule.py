"""Step model of the bf16 scan's LDS rings (gdn_scan_bf16.hip), on the CPU.

The kernel runs one barrier per 32-row sub-chunk step; ring slots are
reused as soon as the schedule allows, with no run-time check.  This model
replays that schedule for streams of 0-69 and 127-129 sub-chunks and checks,
step by step, that no two waves touch one slot in the same step when either
writes it, and that every read finds the sub-chunk it expects.  The ring
sizes and the DMA lookahead are read from the kernel source, so the model
follows the kernel; shrinking a ring must make it fail (the negative
controls below).

Who does what (one step = the work between two barriers):
- the prep wave on DMA duty at step n writes K(n + LK) and V(n + LV) by DMA;
  the writes may land until the barrier that ends step n + WAIT;
- the state waves at step n read the K, V, W, Tu and gate-vector slots of
  sub-chunk n + 1;
- prep wave p runs its sub-chunk pairs (m, m + 1), m = 2p (mod 8), over
  steps m - 9 .. m - 2: gate vectors, A, three solve steps, Tu and Tw, then
  W = Tw K for m (and for m + 1 one step later, with the next pair)."""
import itertools
import os
import re

SRC = os.path.join(os.path.dirname(__file__), "..", "paper_2609_33477_amd", "csrc", "gdn_scan_bf16.hip")
S0 = -9          # first step (pipeline fill)


def kernel_constants():
    s = open(SRC).read()
    num = lambda pat: int(re.search(pat, s).group(1))
    c = {"NK": num(r"int NK = (\d+);"), "NV": num(r"int NV = (\d+);"), "NTU": num(r"int NTU = (\d+);"),
         "NVEC": num(r"int NVEC = (\d+);"), "LK": num(r"kbuf\(nn \+ (\d+)\)"), "LV": num(r"vbuf\(nn \+ (\d+)\)"),
         "NW": 2 if "(m & 1) * CF::SZ_W" in s else None}
    # the prep barrier waits for the requests of step nn - 2
    c["WAIT"] = 2 if "dma_prev2" in s else 1
    return c


def simulate(nsc, c, NP=4):
    NK, NV, NW, NTU, NVEC = c["NK"], c["NV"], c["NW"], c["NTU"], c["NVEC"]
    events = {}
    barriers = {}

    def ev(n, w, op, buf, slot, tag):
        events.setdefault(n, []).append((w, op, buf, slot, tag))

    nb = 0
    for n in range(S0, nsc):
        if 0 <= n + c["LK"] < nsc:
            for dd in range(c["WAIT"] + 1):
                ev(n + dd, "D", "w", "K", (n + c["LK"]) % NK, ("K", n + c["LK"]))
        if 0 <= n + c["LV"] < nsc:
            for dd in range(c["WAIT"] + 1):
                ev(n + dd, "D", "w", "V", (n + c["LV"]) % NV, ("V", n + c["LV"]))
        j = n + 1
        if 0 <= j < nsc:
            for buf, sl in (("K", j % NK), ("V", j % NV), ("W", j % NW), ("TU", j % NTU), ("VEC", j % NVEC)):
                ev(n, "S", "r", buf, sl, (buf, j))
        nb += 1
    barriers["S"] = nb
    for p in range(NP):
        w = f"P{p}"
        n = S0
        nb = 0

        def make_w(n, mc, cc):
            ev(n, w, "r", ("PRIV", p), ("TW", cc), ("TW", mc))
            ev(n, w, "r", "K", mc % NK, ("K", mc))
            ev(n, w, "w", "W", mc % NW, ("W", mc))

        while n < 2 * p + S0 and n < nsc:
            n += 1
            nb += 1
        m = 2 * p
        while m < nsc:
            if m >= 8:
                make_w(n, m - 7, 1)
            n += 1
            nb += 1
            ev(n, w, "w", "VEC", m % NVEC, ("VEC", m))
            ev(n, w, "w", "VEC", (m + 1) % NVEC, ("VEC", m + 1))
            n += 1
            nb += 1
            ev(n, w, "w", ("PRIV", p), "A", ("A", m))
            n += 1
            nb += 1
            for _ in range(3):
                ev(n, w, "r", ("PRIV", p), "A", ("A", m))
                n += 1
                nb += 1
            ev(n, w, "w", "TU", m % NTU, ("TU", m))
            ev(n, w, "w", "TU", (m + 1) % NTU, ("TU", m + 1))
            ev(n, w, "w", ("PRIV", p), ("TW", 0), ("TW", m))
            ev(n, w, "w", ("PRIV", p), ("TW", 1), ("TW", m + 1))
            n += 1
            nb += 1
            make_w(n, m, 0)
            n += 1
            nb += 1
            m += 8
        if m >= 8 and m - 7 < nsc:
            make_w(n, m - 7, 1)
            n += 1
            nb += 1
        while n < nsc:
            n += 1
            nb += 1
        barriers[w] = nb
    errs = []
    if len(set(barriers.values())) != 1 or barriers["S"] != nsc - S0:
        errs.append(f"barrier counts differ: {barriers}")
    content = {}
    for n in range(S0, nsc + c["WAIT"] + 1):
        evs = events.get(n, [])
        for (w1, o1, b1, s1, _), (w2, o2, b2, s2, _) in itertools.combinations(evs, 2):
            if w1 != w2 and b1 == b2 and s1 == s2 and "w" in (o1, o2):
                errs.append(f"step {n}: {w1} {o1} / {w2} {o2} on {b1}[{s1}]")
        for (w, o, b, sl, tag) in evs:
            if o == "r" and content.get((b, sl)) != tag:
                errs.append(f"step {n}: {w} reads {b}[{sl}] expecting {tag}, finds {content.get((b, sl))}")
        for (w, o, b, sl, tag) in evs:
            if o == "w":
                content[(b, sl)] = tag
    return errs


LENGTHS = list(range(0, 70)) + [127, 128, 129]


def test_kernel_rings_have_no_conflicts():
    c = kernel_constants()
    assert c["NW"] == 2 and c["LK"] > c["LV"] >= 1
    for nsc in LENGTHS:
        assert simulate(nsc, c) == [], (nsc, simulate(nsc, c)[:3])


def test_smaller_rings_are_caught():
    c = kernel_constants()
    for key in ("NK", "NV", "NTU"):
        small = dict(c, **{key: c[key] - 1})
        assert any(simulate(nsc, small) for nsc in range(8, 40)), key
    # a DMA waited for one step later than the kernel does needs bigger rings
    late = dict(c, WAIT=c["WAIT"] + 1)
    assert any(simulate(nsc, late) for nsc in range(8, 40))
