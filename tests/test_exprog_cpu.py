"""Exchange programs (Section 5.2) on the CPU: the paper's example programs
are valid under Definition "Closure; validity" and stop being valid when an
action they need is removed; the preamble of Example "Generating a preamble"
needs a body, which the naive program provides; the native checker agrees
with the oracle's literal closure on random programs."""
import ctypes
import json
import re
import os

import numpy as np
import pytest

import oracle
from paper_2609_03905_amd import ea, exprog

with open(os.path.join(os.path.dirname(__file__), "golden", "exprog_examples.json")) as f:
    EX = json.load(f)


@pytest.mark.parametrize("name", ["swap", "doubling", "v100"])
def test_paper_examples_are_valid(name):
    assert exprog.check(EX[name]) == (True, "")


@pytest.mark.parametrize("name,drop", [("swap", "B @ 1 -> 0"), ("doubling", "C+D @ 2 -> 0"),
                                       ("v100", "E+F @ 4 -> 0")])
def test_removing_a_needed_action_invalidates(name, drop):
    text = EX[name]
    assert drop in text
    bad = text.replace(drop + ";", "").replace(drop, "")
    valid, why = exprog.check(bad)
    assert not valid and why


def test_v100_groups_must_follow_the_pillars():
    # with the partitions fixed to the machine's sockets instead, the body
    # (which aggregates across the 0-4, 1-5, 2-6, 3-7 pairs) is invalid; with
    # the groups the paper names it is valid
    sock = EX["v100"].replace("G1 {size 4} G2 {size 4}", "G1 {0, 1, 2, 3} G2 {4, 5, 6, 7}")
    assert not exprog.check(sock)[0]
    g1, g2 = EX["v100_groups"]
    named = EX["v100"].replace("G1 {size 4} G2 {size 4}",
                               "G1 {%s} G2 {%s}" % (", ".join(map(str, g1)), ", ".join(map(str, g2))))
    assert exprog.check(named) == (True, "")


def test_preamble_needs_a_body_and_the_naive_program_is_valid():
    valid, why = exprog.check(EX["preamble"])
    assert not valid and "X1+Y1" in why
    prog = exprog.naive(EX["preamble"])
    assert prog.startswith(EX["preamble"])
    assert exprog.check(prog) == (True, "")
    for name in ("swap", "doubling", "v100"):
        decl = EX[name].split("\n\n")[0] + "\n"
        assert exprog.check(exprog.naive(decl)) == (True, "")


def test_syntax_errors():
    for bad in ("IN: A @ 0\nOUT: B @ 0\n",            # unknown atom
                "GPUS: 0, 1\nIN: A @ 2\nOUT: A @ 0\n",  # site not among the GPUS
                "IN: A @ 0\nOUT: A @ G1\n",            # unknown partition
                "GPUS: 0, 1\nPARTITIONS: G1 {size 3}\nIN: A @ 0\nOUT: A @ G1\n"):  # partitions do not cover
        with pytest.raises(ea.EAError) as e:
            exprog.check(bad)
        assert e.value.code == -5


def _render(n_sites, ins, outs, actions):
    names = {a: f"A{a}" for a, _ in ins}
    agg = lambda xs: "+".join(names[a] for a in sorted(xs))
    text = "GPUS: " + ", ".join(map(str, range(n_sites))) + "\n"
    text += "IN: " + "; ".join(f"{names[a]} @ {s}" for a, s in ins) + "\n"
    text += "OUT: " + "; ".join(f"{agg(x)} @ " + ", ".join(map(str, ss)) for x, ss in outs) + "\n\n"
    for x, srcs, hops in actions:
        text += f"{agg(x)} @ " + ", ".join(map(str, srcs)) + "".join(" -> " + ", ".join(map(str, h)) for h in hops) + "\n"
    return text


@pytest.mark.parametrize("seed", range(40))
def test_checker_matches_the_literal_closure(seed):
    rng = np.random.default_rng(seed)
    n_sites, n_atoms = int(rng.integers(2, 5)), int(rng.integers(2, 6))
    ins = [(a, int(rng.integers(0, n_sites))) for a in range(n_atoms)]

    def rand_agg():
        k = int(rng.integers(1, n_atoms + 1))
        return frozenset(int(x) for x in rng.choice(n_atoms, k, replace=False))

    def rand_sites():
        return sorted(set(int(x) for x in rng.choice(n_sites, int(rng.integers(1, n_sites + 1)))))

    outs = [(rand_agg(), rand_sites()) for _ in range(int(rng.integers(1, 3)))]
    actions = []
    for _ in range(int(rng.integers(0, 8)) if seed % 3 else 0):  # seed % 3 == 0: the gather body alone
        hops = [rand_sites() for _ in range(int(rng.integers(0, 3)))]
        actions.append((rand_agg(), rand_sites(), hops))
    if seed % 3 != 2:  # a gather-everything body, valid on its own
        for x, ss in outs:
            for s in ss:
                for a in x:
                    src = dict(ins)[a]
                    if src != s:
                        actions.append((frozenset([a]), [src], [[s]]))
                if len(x) > 1:
                    actions.append((x, [s], []))
    text = _render(n_sites, ins, outs, actions)
    assert exprog.check(text)[0] == oracle.exprog_valid(ins, outs, actions), text


# ---- the full-mesh simulator: closed forms on links of L GB/s and memory of
# H GB/s, 1 GB atoms unless sized
L, H = 100.0, 1000.0


def _sim(text):
    return exprog.simulate(text, L, H)


def test_simulator_swap_and_doubling_closed_forms():
    # swap: both transfers on their own links (1/L), then an aggregation of two
    # parts at each GPU (read 2, write 1: 3/H)
    assert _sim(EX["swap"]) == pytest.approx(1 / L + 3 / H, rel=1e-9)
    # doubling: two rounds of (aggregate if needed, transfer), then the final
    # aggregation of two parts: 1/L + (3/H + 1/L) + 3/H
    assert _sim(EX["doubling"]) == pytest.approx(2 / L + 6 / H, rel=1e-9)


def test_simulator_links_multicast_relay_and_sizes():
    base = "IN: A @ 0; B @ 0 (size: 0.5 GB)\nOUT: A @ 1, 2, 3\n\n"
    # a multicast uses one link per destination on a full mesh
    assert _sim(base + "A @ 0 -> 1, 2, 3") == pytest.approx(1 / L, rel=1e-9)
    # two transfers on one directed link share it
    two = "IN: A @ 0; B @ 0\nOUT: A @ 1; B @ 1\n\nA @ 0 -> 1; B @ 0 -> 1"
    assert _sim(two) == pytest.approx(2 / L, rel=1e-9)
    # a relay is two transfers in a row; a half-size atom takes half the time
    assert _sim("IN: A @ 0\nOUT: A @ 2\n\nA @ 0 -> 1 -> 2") == pytest.approx(2 / L, rel=1e-9)
    assert _sim("IN: B @ 0 (size: 0.5 GB)\nOUT: B @ 1\n\nB @ 0 -> 1") == pytest.approx(0.5 / L, rel=1e-9)


def test_simulator_topology_changes_the_best_program():
    # on a full mesh every GPU gathers the other three atoms at once (1/L,
    # then 4 parts read + 1 written: 5/H), faster than recursive doubling's
    # two rounds
    decl = EX["doubling"].split("\n\n")[0] + "\n"
    gather = _sim(exprog.naive(decl))
    assert gather == pytest.approx(1 / L + 5 / H, rel=1e-9)
    assert gather < _sim(EX["doubling"])


def test_simulator_rejects_invalid_programs():
    with pytest.raises(ea.EAError) as e:
        _sim("IN: A @ 0\nOUT: A @ 1\n\n")
    assert e.value.code == -1


# ---- preamble generation (Section 5.3) ----------------------------------

def _norm(text):
    return " ".join(text.replace(";", " ; ").split())


def test_preamble_matches_the_paper_example():
    """Section 5.3, Example "Generating a preamble": the 256x256 product C of
    the matmul example, row-split in two with F11, F12, F21, F22 on GPUs
    0..3, consumed by a softmax over four 64-row blocks."""
    t = exprog.preamble([[0, 128, 256], [0, 256]], [(0, 0), (0, 1), (1, 2), (1, 3)],
                        [[0, 64, 128, 192, 256], [0, 256]], [0, 1, 2, 3], 4)
    assert _norm(t) == _norm(EX["preamble"])
    assert exprog.check(exprog.naive(t)) == (True, "")


def _parse_preamble(text):
    sec = {}
    for line in text.strip().splitlines():
        k, v = line.split(":", 1)
        sec[k.strip()] = v.strip()
    ins = {}
    for item in filter(None, (x.strip() for x in sec["IN"].split(";"))):
        name, rest = item.split("@")
        gpu = rest.split("(")[0].strip()
        size = float(rest.split("size:")[1].split("GB")[0]) if "size:" in rest else None
        ins[name.strip()] = (int(gpu), size)
    outs = {}
    for item in filter(None, (x.strip() for x in sec["OUT"].split(";"))):
        agg, dst = item.split("@")
        outs[frozenset(agg.strip().split("+"))] = sorted(int(s.strip()[1:]) for s in dst.split(","))
    return ins, outs


@pytest.mark.parametrize("seed", range(6))
def test_preamble_atoms_against_elementwise_grouping(seed):
    """Atoms are the nonempty intersections of a producer block with a
    consumer block; grouped element by element on a small 2-D tensor."""
    rng = np.random.default_rng(seed)
    shape = (int(rng.integers(3, 9)), int(rng.integers(3, 9)))

    def tiling():
        return [[0] + sorted(rng.choice(np.arange(1, n), int(rng.integers(0, min(3, n - 1) + 1)),
                                        replace=False).tolist()) + [n] for n in shape]

    pt, ct = tiling(), tiling()
    npb = (len(pt[0]) - 1) * (len(pt[1]) - 1)
    ncb = (len(ct[0]) - 1) * (len(ct[1]) - 1)
    cons = [b for b in range(ncb) for _ in range(int(rng.integers(1, 3)))]
    n_gpus = len(cons)
    prod = [(b, int(rng.integers(0, n_gpus))) for b in range(npb) for _ in range(int(rng.integers(1, 3)))]
    t = exprog.preamble(pt, prod, ct, cons, n_gpus, elem_bytes=4)
    ins, outs = _parse_preamble(t)

    # brute force: (producer block, consumer block) of every element
    def block_of(tl, i, j):
        bi = int(np.searchsorted(tl[0], i, side="right")) - 1
        bj = int(np.searchsorted(tl[1], j, side="right")) - 1
        return bi * (len(tl[1]) - 1) + bj

    groups = {}
    for i in range(shape[0]):
        for j in range(shape[1]):
            groups.setdefault((block_of(pt, i, j), block_of(ct, i, j)), []).append((i, j))
    assert len(outs) == len(groups)
    copies_of_block = {}
    for s, (b, g) in enumerate(prod):
        copies_of_block.setdefault(b, []).append((s, g))
    letters = "XYZWVU"
    expected_in = {}
    for (pb, cb), cells in groups.items():
        for c, (s, g) in enumerate(copies_of_block[pb]):
            expected_in.setdefault(letters[c], []).append((g, len(cells) * 4 / 1e9, pb, cb))
    # every OUT item aggregates all copies of one atom, delivered to its readers
    matched = set()
    for agg, dst in outs.items():
        letters_here = sorted(a[0] for a in agg)
        idx = {a[1:] for a in agg}
        assert len(idx) == 1
        atom = idx.pop()
        gpu_size = [ins[a] for a in agg]
        cand = [(pb, cb) for (pb, cb), cells in groups.items()
                if len(copies_of_block[pb]) == len(agg)
                and sorted(g for _, g in copies_of_block[pb]) == sorted(g for g, _ in gpu_size)
                and all(abs(sz - len(cells) * 4 / 1e9) < 1e-15 for _, sz in gpu_size)
                and dst == sorted(k + 1 for k, b in enumerate(cons) if b == cb)
                and (pb, cb) not in matched]
        assert cand, (agg, dst)
        matched.add(cand[0])
        assert letters_here == sorted(letters[:len(agg)])
    assert len(matched) == len(groups)
    # each copy of a producer block is cut into atoms that sum to the block
    for s, (b, g) in enumerate(prod):
        cells = sum(len(v) for (pb, _), v in groups.items() if pb == b)
        assert cells > 0
    assert sum(sz for _, sz in ins.values()) == pytest.approx(
        sum(len(v) * 4 / 1e9 * len(copies_of_block[pb]) for (pb, _), v in groups.items()), rel=1e-12)
    assert exprog.check(exprog.naive(t)) == (True, "")


def test_preamble_rejects_mismatched_tilings_and_bad_indices():
    with pytest.raises(ea.EAError):
        exprog.preamble([[0, 4]], [(0, 0)], [[0, 5]], [0], 1)
    with pytest.raises(ea.EAError):
        exprog.preamble([[0, 4]], [(1, 0)], [[0, 4]], [0], 1)
    with pytest.raises(ea.EAError):
        exprog.preamble([[0, 4]], [(0, 2)], [[0, 4]], [0], 2)
    with pytest.raises(ea.EAError):
        exprog.preamble([[0, 2, 2, 4]], [(0, 0)], [[0, 4]], [0], 1)
    with pytest.raises(ea.EAError):
        exprog.preamble([[0, 4]], [(0, 0)], [[0, 4]], [0], 2)


# ---- body synthesis (Section 5.4) ----------------------------------------

def _parse_concrete(text):
    """A synthesized program (memberships written out, concrete sites in the
    body) as the oracle's (ins, outs, actions)."""
    decl, body = text.split("\n\n", 1)
    sec = {}
    for line in decl.splitlines():
        k, v = line.split(":", 1)
        sec[k.strip()] = v
    parts = {}
    for name, members in re.findall(r"(\w+)\s*\{([^}]*)\}", sec.get("PARTITIONS", "")):
        parts[name] = [int(m) for m in members.split(",")]

    def sites(s):
        out = []
        for tok in s.split(","):
            tok = tok.strip()
            out += parts[tok] if tok in parts else [int(tok)]
        return out

    ins = [(a.split("@")[0].strip(), int(a.split("@")[1].split("(")[0])) for a in sec["IN"].split(";")]
    outs = [(tuple(o.split("@")[0].strip().split("+")), sites(o.split("@")[1])) for o in sec["OUT"].split(";")]
    acts = []
    for line in filter(None, (x.strip() for x in body.splitlines())):
        hops = line.split("->")
        agg, src = hops[0].split("@")
        acts.append((tuple(agg.strip().split("+")), sites(src), [sites(h) for h in hops[1:]]))
    return ins, outs, acts


def _synth_ok(decl, iters=1500, seed=0):
    prog, t = exprog.synthesize(decl, L, H, iters=iters, seed=seed)
    assert exprog.check(prog) == (True, "")
    assert oracle.exprog_valid(*_parse_concrete(prog))
    # the written program reproduces the reported time
    assert _sim(prog) == pytest.approx(t, rel=1e-12)
    return prog, t


def test_synthesis_relays_around_one_contended_link():
    """Four 1 GB atoms from GPU 0 to GPU 1 on a 4-GPU mesh.  The naive body
    shares link 0->1 (4/L).  GPU 1 has three incoming links for 4 GB, so some
    link carries 2 GB and 2/L is a lower bound; two relays reach it."""
    decl = "GPUS: 0, 1, 2, 3\nIN: A @ 0; B @ 0; C @ 0; D @ 0\nOUT: A @ 1; B @ 1; C @ 1; D @ 1\n"
    assert _sim(exprog.naive(decl)) == pytest.approx(4 / L, rel=1e-9)
    prog, t = _synth_ok(decl)
    assert t == pytest.approx(2 / L, rel=1e-9)
    assert any(line.count("->") == 2 for line in prog.splitlines())


def test_synthesis_pushes_aggregation_below_the_transfer():
    """X+Y required at GPU 1 with X and Y at GPU 0 and no relay: the naive
    body sends both (2/L) then aggregates (3/H).  GPU 1 must receive at least
    one aggregate-sized piece and somebody must aggregate, so 1/L + 3/H is a
    lower bound; aggregation pushdown reaches it."""
    decl = "GPUS: 0, 1\nIN: X @ 0; Y @ 0\nOUT: X+Y @ 1\n"
    assert _sim(exprog.naive(decl)) == pytest.approx(2 / L + 3 / H, rel=1e-9)
    prog, t = _synth_ok(decl)
    assert t == pytest.approx(1 / L + 3 / H, rel=1e-9)
    assert "X+Y @ 0 -> 1" in prog


def test_synthesis_chooses_the_memberships_of_the_paper_preamble():
    """Section 5.3's preamble: each S_j must sit at a GPU holding one copy of
    its atom (GPUs 0, 1 for atoms 1, 2; GPUs 2, 3 for atoms 3, 4), receive the
    other copy (1/L) and aggregate two parts (3/H), the lower bound."""
    prog, t = _synth_ok(EX["preamble"])
    assert t == pytest.approx(1 / L + 3 / H, rel=1e-9)
    members = dict(re.findall(r"(S\d)\s*\{(\d+)\}", prog))
    assert {members["S1"], members["S2"]} == {"0", "1"}
    assert {members["S3"], members["S4"]} == {"2", "3"}


@pytest.mark.parametrize("name", ["swap", "doubling", "v100"])
def test_synthesis_never_worse_than_naive_on_the_paper_examples(name):
    decl = EX[name].split("\n\n")[0] + "\n"
    _, t = _synth_ok(decl)
    assert t <= _sim(exprog.naive(decl)) * (1 + 1e-12)
    # deterministic for a seed
    assert exprog.synthesize(decl, L, H, iters=300, seed=7) == exprog.synthesize(decl, L, H, iters=300, seed=7)


@pytest.mark.parametrize("seed", range(8))
def test_synthesis_on_random_preambles(seed):
    """Random exchange problems (atoms of random sizes at random GPUs,
    aggregates required at random sites): every program the search returns is
    valid under the oracle's literal closure and no slower than the naive
    body under the same memberships."""
    rng = np.random.default_rng(100 + seed)
    n_gpus = int(rng.integers(2, 6))
    n_atoms = int(rng.integers(1, 6))
    ins = [(f"A{i}", int(rng.integers(0, n_gpus)), float(rng.choice([0.25, 0.5, 1.0, 2.0]))) for i in range(n_atoms)]
    outs = []
    for _ in range(int(rng.integers(1, 4))):
        k = int(rng.integers(1, n_atoms + 1))
        atoms = sorted(rng.choice(n_atoms, k, replace=False).tolist())
        dst = sorted(rng.choice(n_gpus, int(rng.integers(1, n_gpus + 1)), replace=False).tolist())
        outs.append(("+".join(f"A{a}" for a in atoms), dst))
    decl = ("GPUS: " + ", ".join(map(str, range(n_gpus))) + "\nIN: "
            + "; ".join(f"{a} @ {g} (size: {s} GB)" for a, g, s in ins) + "\nOUT: "
            + "; ".join(f"{x} @ " + ", ".join(map(str, d)) for x, d in outs) + "\n")
    prog, t = _synth_ok(decl, iters=800, seed=seed)
    assert t <= _sim(exprog.naive(decl)) * (1 + 1e-12)


def test_synthesis_argument_and_capacity_errors():
    decl = "GPUS: 0, 1\nIN: A @ 0\nOUT: A @ 1\n"
    with pytest.raises(ea.EAError) as e:
        exprog.synthesize(decl, 0.0, H)
    assert e.value.code == -1
    with pytest.raises(ea.EAError) as e:
        exprog.synthesize(decl, L, H, iters=-1)
    assert e.value.code == -1
    with pytest.raises(ea.EAError) as e:
        exprog.synthesize("GPUS: 0, 1\nIN: A @ 0\nOUT: A @ 7\n", L, H)
    assert e.value.code == -5  # site 7 is not among the GPUS
    # zero iterations return the naive program under the best membership
    prog, t = exprog.synthesize(decl, L, H, iters=0)
    assert t == pytest.approx(1 / L, rel=1e-9) and "A @ 0 -> 1" in prog
    # the capacity error still reports the needed length
    n = ctypes.c_int64()
    sec = ctypes.c_double()
    rc = ea.lib().ea_exprog_synthesize(decl.encode(), L, H, 0, 0, None, 0, ctypes.byref(n), ctypes.byref(sec))
    assert rc == -4 and n.value == len(prog) and sec.value == pytest.approx(t)
