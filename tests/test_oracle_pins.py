"""Pins for the FP64 oracle: checks against what the paper and the
mathematics fix (worked example, closed forms, invariants, exact rational
arithmetic, brute force on tiny inputs).  CPU only."""
import itertools
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import mol_oracle as mo

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_example.txt")


# ---------------------------------------------------------------- helpers
def unit(v):
    return v / np.linalg.norm(v, axis=-1, keepdims=True)


def make_problem(rng, B, N, Pq, Px, d, H, scale=0.1, zero_gating=False):
    """Small float32 problem with unit-norm components."""
    P = Pq * Px
    Q = unit(rng.normal(size=(B, Pq, d))).astype(np.float32)
    X = unit(rng.normal(size=(Px, N, d))).astype(np.float32)
    g = (lambda *s: np.zeros(s, np.float32)) if zero_gating else \
        (lambda *s: (scale * rng.normal(size=s)).astype(np.float32))
    return mo.Problem(Q, X, g(B, P), g(N, P), g(H, P), g(H), g(P, H), g(P), "f32")


def frac_dot(a, b):
    return sum(Fraction(float(x)) * Fraction(float(y)) for x, y in zip(a, b))


def read_golden():
    rows, expect = {}, {}
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line:
                continue
            if line.startswith("#"):
                body = line[1:].strip()
                for key in ("exact top-2", "TopKPerEmbedding(K'=2) candidates",
                            "Algorithm 1 S_min", "Algorithm 1 second-pass set G'",
                            "Theorem 2 S_K", "Theorem 2 S ", "Theorem 2 bound S - S_K",
                            "Definition 2 gap (tight)", "looser bound from retrieved items"):
                    if body.startswith(key):
                        expect[key.strip()] = body[len(key):].split()
                continue
            name, *vals = line.split()
            rows[name] = [float(v) for v in vals]
    return rows, expect


def worked_example_problem():
    """The example table realised through the MoL definition: one query with
    f = e1 (P_q = 1), two item components g_p(x) = dot_p(x) e1 (P_x = 2), no
    MLP contribution, and per-item gating logits a_x that give the table's
    weights: (0, 0) for pi = (1/2, 1/2) and (+20, -20) for pi ~ (1, 0)."""
    rows, expect = read_golden()
    names = sorted(rows)
    N, d = len(names), 2
    Q = np.zeros((1, 1, d), np.float32)
    Q[0, 0, 0] = 1.0
    X = np.zeros((2, N, d), np.float32)
    a_x = np.zeros((N, 2), np.float32)
    for n, name in enumerate(names):
        dot1, dot2, pi1, pi2, _ = rows[name]
        X[0, n, 0], X[1, n, 0] = dot1, dot2
        if pi1 != pi2:
            a_x[n] = (20.0, -20.0) if pi1 > pi2 else (-20.0, 20.0)
    z = lambda *s: np.zeros(s, np.float32)
    prob = mo.Problem(Q, X, z(1, 2), a_x, z(1, 2), z(1), z(2, 1), z(2), "f32")
    return prob, names, rows, expect


# ---------------------------------------------------------- storage format
def test_bf16_decode_known_bit_patterns():
    bits = np.array([0x3F80, 0xC000, 0x3F81, 0x0000, 0x8000, 0x7F7F, 0x0001], np.uint16)
    got = mo.decode(bits, "bf16")
    want = [1.0, -2.0, 1.0078125, 0.0, -0.0, (2 - 2 ** -7) * 2.0 ** 127, 2.0 ** -133]
    assert got.tolist() == want


def test_bf16_rounding_ties_to_even():
    # bf16 has 8 significant bits: the ulp at 1.0 is 2^-7, halfway is 2^-8
    x = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 1 + 2 ** -8 + 2 ** -30,
                  2.0 ** -133 * 1.5, 0.0])
    want = np.array([0x3F80, 0x3F82, 0xBF80, 0x3F81, 0x0002, 0x0000], np.uint16)
    assert mo.round_to_storage(x, "bf16").tolist() == want.tolist()


def test_bf16_rounding_matches_torch_on_float32_values():
    rng = np.random.default_rng(1)
    x = (rng.normal(size=20000) * np.exp(rng.uniform(-30, 30, size=20000))).astype(np.float32)
    ours = mo.round_to_storage(x.astype(np.float64), "bf16")
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


# ------------------------------------------------------------ dot products
def test_component_dots_equal_exact_rational_dots_in_p_order():
    rng = np.random.default_rng(2)
    prob = make_problem(rng, B=2, N=5, Pq=2, Px=3, d=7, H=4)
    for b in range(2):
        s = mo.component_dots(prob.Q[b], prob.items(slice(0, 5)))
        for n in range(5):
            for pq in range(2):
                for px in range(3):
                    exact = frac_dot(prob.Q[b, pq], prob.X[px, n])
                    assert abs(s[n, pq * 3 + px] - float(exact)) <= 1e-15


def test_single_component_score_is_the_dot_product():
    """Lemma 1: with one component the weight is identically 1 and MoL is
    the dot product; top-k is then plain maximum inner product search."""
    rng = np.random.default_rng(3)
    prob = make_problem(rng, B=3, N=300, Pq=1, Px=1, d=16, H=8, scale=0.5)
    phi = mo.mol_scores(prob, [0, 1, 2])
    for b in range(3):
        s = mo.component_dots(prob.Q[b], prob.items(slice(None)))[:, 0]
        assert np.array_equal(phi[b], s)
        exact = [frac_dot(prob.Q[b, 0], prob.X[0, n]) for n in range(prob.N)]
        order = sorted(range(prob.N), key=lambda n: (-exact[n], n))[:25]
        _, ids = mo.exact_topk(prob, [b], 25)
        assert ids[0].tolist() == order


# ------------------------------------------------------------------ gating
def test_gating_weights_sum_to_one_and_phi_is_convex_combination():
    rng = np.random.default_rng(4)
    prob = make_problem(rng, B=4, N=500, Pq=4, Px=4, d=32, H=16, scale=1.0)
    for b in range(4):
        s, pi, phi = mo.mol_terms(prob, b, slice(None))
        assert np.all(pi >= 0) and np.all(pi <= 1)
        assert np.max(np.abs(pi.sum(axis=1) - 1)) < 1e-12
        assert np.all(phi <= s.max(axis=1) + 1e-15)
        assert np.all(phi >= s.min(axis=1) - 1e-15)


def test_softmax_is_invariant_to_a_common_logit_shift():
    rng = np.random.default_rng(5)
    prob = make_problem(rng, B=2, N=200, Pq=2, Px=4, d=16, H=8, scale=0.5)
    _, pi0, phi0 = mo.mol_terms(prob, 1, slice(None))
    prob.b2 = prob.b2 + 7.25
    _, pi1, phi1 = mo.mol_terms(prob, 1, slice(None))
    assert np.max(np.abs(pi0 - pi1)) < 1e-12
    assert np.max(np.abs(phi0 - phi1)) < 1e-12


def test_uniform_gating_gives_mean_and_topk_avg_is_exact():
    """With uniform weights phi is the mean dot product, and TopKAvg returns
    the exact top-k (Section 3.2, top-K average heuristic)."""
    rng = np.random.default_rng(6)
    prob = make_problem(rng, B=2, N=400, Pq=2, Px=4, d=16, H=8, zero_gating=True)
    for b in range(2):
        s, pi, phi = mo.mol_terms(prob, b, slice(None))
        assert np.max(np.abs(pi - 1.0 / prob.P)) < 1e-15
        # closed form: mean of dots = <sum_pq f, sum_px g> / P, in rationals
        for n in range(0, 400, 37):
            fs = [sum(Fraction(float(v)) for v in prob.Q[b, :, t]) for t in range(16)]
            gs = [sum(Fraction(float(v)) for v in prob.X[:, n, t]) for t in range(16)]
            exact = sum(a * c for a, c in zip(fs, gs)) / prob.P
            assert abs(phi[n] - float(exact)) < 1e-15
        _, want = mo.topk_desc(phi, 20)
        avg = mo.averaged_problem(prob)          # float32-rounded sums
        gap20 = np.sort(phi)[::-1][19] - np.sort(phi)[::-1][20]
        assert gap20 > 1e-5                       # rounding cannot reorder
        _, got = mo.topk_avg(prob, b, 20, avg)
        assert set(got.tolist()) == set(want.tolist())


@pytest.mark.parametrize("where", ["a_x", "a_q", "b2"])
def test_one_hot_gating_logit_selects_that_component(where):
    """A dominant logit on component p* makes pi ~ e_{p*}, so phi equals
    <f_{pq*}, g_{px*}> with p* = pq* P_x + px* (the p order of Eq. 2)."""
    rng = np.random.default_rng(7)
    Pq, Px = 2, 3
    prob = make_problem(rng, B=2, N=6, Pq=Pq, Px=Px, d=5, H=3, zero_gating=True)
    for pstar in range(Pq * Px):
        prob.a_x[:] = 0
        prob.a_q[:] = 0
        prob.b2[:] = 0
        getattr(prob, where)[..., pstar] = 40.0
        _, _, phi = mo.mol_terms(prob, 1, slice(None))
        pq, px = divmod(pstar, Px)
        for n in range(6):
            assert abs(phi[n] - float(frac_dot(prob.Q[1, pq], prob.X[px, n]))) < 1e-15


def test_gating_mlp_closed_form():
    """Two hidden units with pre-activation ln 3, where sigmoid = 3/4, so
    SiLU = (3/4) ln 3 exactly.  W2 = [[1, 1/2], [-1, 1/4]] then gives
    l_1 - l_2 = 2.25 c with c = (3/4) ln 3, hence
    pi_1 = 1 / (1 + 3^(-2.25 * 0.75))."""
    rng = np.random.default_rng(8)
    prob = make_problem(rng, B=1, N=4, Pq=1, Px=2, d=6, H=2, zero_gating=True)
    for n in range(4):
        s1 = float(frac_dot(prob.Q[0, 0], prob.X[1, n]))     # p = 1
        prob.W1[:] = 0
        prob.W1[0, 1] = 1.0                                  # u_0 = s_1 + b1_0
        prob.b1[:] = [math.log(3.0) - s1, math.log(3.0)]     # u_0 = u_1 = ln 3
        prob.W2[:] = [[1.0, 0.5], [-1.0, 0.25]]
        s, pi, phi = mo.mol_terms(prob, 0, np.array([n]))
        pi1 = 1.0 / (1.0 + 3.0 ** (-2.25 * 0.75))
        assert abs(pi[0, 0] - pi1) < 1e-12
        s0 = float(frac_dot(prob.Q[0, 0], prob.X[0, n]))
        assert abs(phi[0] - (pi1 * s0 + (1 - pi1) * s1)) < 1e-12


def test_silu_identities():
    u = np.linspace(-30, 30, 601)
    assert np.max(np.abs(mo.silu(-u) - (mo.silu(u) - u))) < 1e-12
    assert mo.silu(np.array([0.0]))[0] == 0.0
    assert abs(mo.silu(np.array([math.log(3.0)]))[0] - 0.75 * math.log(3.0)) < 1e-15
    assert mo.silu(np.array([-800.0]))[0] == 0.0


# ---------------------------------------------------------- worked example
def test_worked_example_scores_and_exact_topk():
    prob, names, rows, expect = worked_example_problem()
    s, pi, phi = mo.mol_terms(prob, 0, slice(None))
    for n, name in enumerate(names):
        dot1, dot2, pi1, pi2, phi_t = rows[name]
        assert abs(s[n, 0] - dot1) < 1e-7 and abs(s[n, 1] - dot2) < 1e-7
        assert abs(pi[n, 0] - pi1) < 1e-12 and abs(pi[n, 1] - pi2) < 1e-12
        assert abs(phi[n] - phi_t) < 1e-7
    _, ids = mo.exact_topk(prob, [0], 2)
    assert [names[i] for i in ids[0]] == expect["exact top-2"]


def test_worked_example_per_embedding_candidates_and_gap_bound():
    prob, names, rows, expect = worked_example_problem()
    res = mo.approx_topk(prob, 0, k=2, kprime=2)
    cand = mo.union_dedup([res["cand"]])
    assert [names[i] for i in cand] == expect["TopKPerEmbedding(K'=2) candidates"]
    bnd = mo.gap_bound_per_embd(prob, 0, k=2, kprime=2)
    assert abs(bnd["S_K"] - float(expect["Theorem 2 S_K"][0])) < 1e-7
    assert abs(bnd["S"] - float(expect["Theorem 2 S"][0])) < 1e-7
    assert abs(bnd["bound"] - float(expect["Theorem 2 bound S - S_K"][0])) < 1e-7
    assert abs(bnd["looser"] - float(expect["looser bound from retrieved items"][0])) < 1e-7
    phi = mo.mol_scores(prob, [0])[0]
    g = mo.gap(phi, res["ids"], 2)
    assert abs(g - float(expect["Definition 2 gap (tight)"][0])) < 1e-7


def test_worked_example_two_pass_exact():
    prob, names, rows, expect = worked_example_problem()
    s = mo.all_dots(prob, 0)
    G = mo.union_dedup([mo.topk_desc(s[:, p], 2)[1] for p in range(2)])
    _, _, phiG = mo.mol_terms(prob, 0, G)
    assert abs(phiG.min() - float(expect["Algorithm 1 S_min"][0])) < 1e-7
    G2 = np.nonzero((s >= phiG.min()).any(axis=1))[0]
    assert [names[i] for i in G2] == expect["Algorithm 1 second-pass set G'"]
    _, ids = mo.exact_two_pass(prob, 0, 2)
    assert [names[i] for i in ids] == expect["exact top-2"]


# --------------------------------------------------------------- selection
def test_topk_matches_brute_force_over_all_subsets_with_ties():
    rng = np.random.default_rng(9)
    for trial in range(30):
        n, k = 8, 3
        v = rng.integers(0, 5, size=n).astype(np.float64)   # many ties
        got_v, got_i = mo.topk_desc(v, k)
        # the answer is the k-subset with the largest value sum, ties broken
        # by the lexicographically smallest sorted id tuple
        best = max(itertools.combinations(range(n), k),
                   key=lambda c: (sum(v[list(c)]), [-i for i in sorted(c)]))
        assert sorted(got_i.tolist()) == sorted(best)
        # and the output order is (value desc, id asc)
        assert all((got_v[i] > got_v[i + 1]) or
                   (got_v[i] == got_v[i + 1] and got_i[i] < got_i[i + 1])
                   for i in range(k - 1))


def test_two_pass_equals_brute_force_on_random_instances():
    """Algorithm 1 is exact (Section 3.1): its result equals brute force."""
    rng = np.random.default_rng(10)
    for seed in range(4):
        prob = make_problem(rng, B=2, N=600, Pq=2, Px=3, d=8, H=8, scale=2.0)
        for b in range(2):
            want_v, want_i = mo.exact_topk(prob, [b], 10)
            got_v, got_i = mo.exact_two_pass(prob, b, 10)
            assert got_i.tolist() == want_i[0].tolist()
            assert np.array_equal(got_v, want_v[0])


def test_two_pass_kth_threshold_is_exact_and_tighter():
    """Algorithm 1 with the k-th largest MoL score over G as threshold: the
    result is still the brute-force top-k, the threshold is at least S_min and
    at most the corpus-wide k-th score, and its second-pass set is a subset
    of the S_min one."""
    rng = np.random.default_rng(21)
    for seed in range(3):
        prob = make_problem(rng, B=2, N=500, Pq=2, Px=3, d=8, H=8, scale=2.0)
        for b in range(2):
            phi = mo.mol_scores(prob, [b])[0]
            want_v, want_i = mo.topk_desc(phi, 10)
            t_min = mo.two_pass_threshold(prob, b, 10, "min")
            t_kth = mo.two_pass_threshold(prob, b, 10, "kth")
            assert t_min <= t_kth <= mo.kth_largest(phi, 10)
            got_v, got_i = mo.exact_two_pass(prob, b, 10, "kth")
            assert got_i.tolist() == want_i.tolist() and np.array_equal(got_v, want_v)
            s = mo.all_dots(prob, b)
            assert np.all((s >= t_kth).any(axis=1) <= (s >= t_min).any(axis=1))


def test_bounded_topk_filters_by_max_component_dot():
    """The second pass on its own, against a filter written out item by item
    from exact rational dot products: only items with some s_p >= bound are
    ranked; a bound at or below the k-th score gives the exact top-k, a bound
    above every s_p gives an all-padding row."""
    rng = np.random.default_rng(22)
    prob = make_problem(rng, B=1, N=90, Pq=2, Px=2, d=4, H=4, scale=2.0)
    phi = mo.mol_scores(prob, [0])[0]
    m = [max(frac_dot(prob.Q[0, pq], prob.X[px, n]) for pq in range(2) for px in range(2))
         for n in range(prob.N)]
    kth = mo.kth_largest(phi, 6)
    mid = float(sorted(m)[prob.N // 2])           # half the items qualify
    for bound in (-math.inf, kth, mid, float(max(m)) + 1.0):
        keep = [n for n in range(prob.N) if float(m[n]) >= bound]
        order = sorted(keep, key=lambda n: (-phi[n], n))[:6]
        v, i = mo.exact_topk_bounded(prob, 0, 6, bound)
        assert i[:len(order)].tolist() == order
        assert np.all(i[len(order):] == -1) and np.all(np.isneginf(v[len(order):]))
        assert np.array_equal(v[:len(order)], phi[order])
    # phi never exceeds the largest component dot (Eq. 1 is a convex combination)
    assert np.all(phi <= np.array([float(x) for x in m]) + 1e-15)


def test_max_dot_topk_against_rational_dots_and_per_component_lists():
    """Max approximation: ranking by m = max_p s_p written out from exact
    rational dot products; the top-k by m lies in the union of the
    per-component top-k lists (an item outside list p is beaten in s_p by k
    items, which then also beat it in m)."""
    rng = np.random.default_rng(23)
    prob = make_problem(rng, B=2, N=120, Pq=2, Px=3, d=4, H=4)
    for b in range(2):
        m = [max(frac_dot(prob.Q[b, pq], prob.X[px, n]) for pq in range(2) for px in range(3))
             for n in range(prob.N)]
        order = sorted(range(prob.N), key=lambda n: (-m[n], n))[:9]
        v, i = mo.max_dot_topk(prob, b, 9)
        assert i.tolist() == order
        assert np.allclose(v, [float(m[n]) for n in order], rtol=0, atol=1e-15)
        _, ids, _, _ = mo.topk_per_embedding(prob, b, 9)
        assert set(i.tolist()) <= set(mo.union_dedup([ids]).tolist())
    # with one component it is the dot-product top-k (Lemma 1's setting)
    one = make_problem(rng, B=1, N=200, Pq=1, Px=1, d=8, H=4)
    _, ids, _, _ = mo.topk_per_embedding(one, 0, 20)
    assert mo.max_dot_topk(one, 0, 20)[1].tolist() == ids[0].tolist()


def test_theorem2_non_candidates_score_at_most_S():
    rng = np.random.default_rng(11)
    prob = make_problem(rng, B=2, N=800, Pq=2, Px=4, d=8, H=8, scale=2.0)
    for b in range(2):
        _, ids, kth, nxt = mo.topk_per_embedding(prob, b, 5)
        cand = mo.union_dedup([ids])
        phi = mo.mol_scores(prob, [b])[0]
        rest = np.setdiff1d(np.arange(prob.N), cand)
        assert phi[rest].max() <= nxt.max() + 1e-15
        res = mo.approx_topk(prob, b, k=10, kprime=5)
        bnd = mo.gap_bound_per_embd(prob, b, 10, 5)
        assert mo.gap(phi, res["ids"], 10) <= bnd["bound"] + 1e-15


def test_theorem3_combined_gap_bound():
    rng = np.random.default_rng(12)
    prob = make_problem(rng, B=2, N=800, Pq=2, Px=4, d=8, H=8, scale=2.0)
    avg = mo.averaged_problem(prob)
    for b in range(2):
        res = mo.approx_topk(prob, b, k=10, kprime=3, k_avg=15, avg=avg)
        phi = mo.mol_scores(prob, [b])[0]
        bnd = mo.gap_bound_combined(prob, b, 10, 3, 15, avg)
        assert mo.gap(phi, res["ids"], 10) <= bnd["bound"] + 1e-15
        cand = mo.union_dedup([res["cand"]])
        rest = np.setdiff1d(np.arange(prob.N), cand)
        assert phi[rest].max() <= bnd["S"] + 1e-15


THEOREM3 = os.path.join(os.path.dirname(__file__), "golden", "theorem3_example.txt")
THEOREM3_KEYS = ("per-component lists (K'=1)", "TopKAvg (K_avg=1)", "candidates", "Theorem 3 S' ",
                 "Theorem 3 S_K", "Theorem 3 bound S' - S_K", "Definition 2 gap")


def theorem3_problem():
    """The hand-built Theorem 3 instance, realised like the Appendix B
    example: f = e1, g_p(x) = dot_p(x) e1, per-item gating logits only."""
    rows, expect = {}, {}
    with open(THEOREM3) as f:
        for line in f:
            line = line.strip()
            if not line:
                continue
            if line.startswith("#"):
                body = line[1:].strip()
                for key in THEOREM3_KEYS:
                    if body.startswith(key):
                        expect[key.strip()] = body[len(key):].split()
                continue
            name, *vals = line.split()
            rows[name] = [float(v) for v in vals]
    names = sorted(rows)
    N, d = len(names), 2
    Q = np.zeros((1, 1, d), np.float32)
    Q[0, 0, 0] = 1.0
    X = np.zeros((2, N, d), np.float32)
    a_x = np.zeros((N, 2), np.float32)
    for n, name in enumerate(names):
        dot1, dot2, pi1, pi2, _ = rows[name]
        X[0, n, 0], X[1, n, 0] = dot1, dot2
        if pi1 != pi2:
            a_x[n] = (20.0, -20.0) if pi1 > pi2 else (-20.0, 20.0)
    z = lambda *s: np.zeros(s, np.float32)
    prob = mo.Problem(Q, X, z(1, 2), a_x, z(1, 2), z(1), z(2, 1), z(2), "f32")
    return prob, names, rows, expect


def test_theorem3_value_pin_on_hand_built_instance():
    """S', S_K and the bound of Theorem 3 equal the hand-derived values.  The
    instance has an item in one component's list that carries the largest
    dot of the other component outside that component's own list and the
    TopKAvg set, so excluding the whole candidate union from every
    component (a plausible mistake) gives a different S'."""
    prob, names, rows, expect = theorem3_problem()
    s, pi, phi = mo.mol_terms(prob, 0, slice(None))
    for n, name in enumerate(names):
        assert abs(phi[n] - rows[name][4]) < 1e-12
    avg = mo.averaged_problem(prob)
    lists = [mo.topk_desc(s[:, p], 1)[1] for p in range(2)]
    assert [names[int(l[0])] for l in lists] == expect["per-component lists (K'=1)"]
    _, avg_ids = mo.topk_avg(prob, 0, 1, avg)
    assert [names[int(i)] for i in avg_ids] == expect["TopKAvg (K_avg=1)"]
    res = mo.approx_topk(prob, 0, k=3, kprime=1, k_avg=1, avg=avg)
    assert [names[int(i)] for i in mo.union_dedup([res["cand"]])] == expect["candidates"]
    bnd = mo.gap_bound_combined(prob, 0, 3, 1, 1, avg)
    assert bnd["S"] == float(expect["Theorem 3 S'"][0])
    assert abs(bnd["S_K"] - float(expect["Theorem 3 S_K"][0])) < 1e-12
    assert abs(bnd["bound"] - float(expect["Theorem 3 bound S' - S_K"][0])) < 1e-12
    g = mo.gap(phi, res["ids"], 3)
    assert abs(g - float(expect["Definition 2 gap"][0])) < 1e-12
    assert g <= bnd["bound"]


def test_union_dedup_is_set_union_and_rerank_pads():
    rng = np.random.default_rng(13)
    lists = [rng.integers(-1, 50, size=30) for _ in range(4)]
    want = sorted(set(int(x) for l in lists for x in l if x >= 0))
    assert mo.union_dedup(lists).tolist() == want
    prob = make_problem(rng, B=1, N=50, Pq=2, Px=2, d=8, H=4)
    cand = np.array([3, 3, 7, -1, 7, 11], np.int64)
    s, i, nu = mo.rerank(prob, 0, cand, 5)
    assert nu == 3 and i[3:].tolist() == [-1, -1] and np.all(np.isneginf(s[3:]))
    phi = mo.mol_scores(prob, [0])[0]
    order = sorted([3, 7, 11], key=lambda n: (-phi[n], n))
    assert i[:3].tolist() == order


def test_averaged_embeddings_round_the_exact_sum():
    """x' is the exact component sum rounded to bf16 (ties to even)."""
    rng = np.random.default_rng(14)
    # bf16 inputs in +-[0.5, 1): sums of four have <= 11 significant bits,
    # so float32 holds them exactly and torch's float32 -> bf16 rounding is
    # an independent reference for the final rounding.
    mant = rng.integers(128, 256, size=(4, 64, 16))
    sign = rng.choice([-1.0, 1.0], size=(4, 64, 16))
    X = (sign * mant / 256.0).astype(np.float32)
    Xb = torch.from_numpy(X).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    Q = Xb[:2, :3, :].transpose(1, 0, 2).copy()                 # [3][2][16]
    z = lambda *s: np.zeros(s, np.float32)
    one = torch.zeros(1, 1).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    prob = mo.Problem(Q, Xb, z(3, 8), z(64, 8), np.repeat(one, 8, 1), z(1),
                      np.repeat(one, 8, 0), z(8), "bf16")
    qbar, xbar = mo.averaged_embeddings(prob)
    ref = torch.from_numpy(X.sum(axis=0)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(xbar, ref)
    refq = torch.from_numpy(X[:2, :3, :].sum(axis=0)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(qbar, refq)


# ---------------------------------------------------------- tau rule helper
def test_tau_rule_accepts_exact_and_rejects_planted_mistakes():
    rng = np.random.default_rng(15)
    v = rng.normal(size=1000)
    _, ids = mo.topk_desc(v, 20)
    assert mo.valid_topk(v, ids, 20, 1e-4)[0]
    bad = ids.copy()
    bad[5] = np.argsort(v)[0]                     # swap in the worst item
    assert not mo.valid_topk(v, bad, 20, 1e-4)[0]
    dup = ids.copy()
    dup[3] = dup[4]
    assert not mo.valid_topk(v, dup, 20, 1e-4)[0]
    # a near tie at the boundary may go either way
    w = v.copy()
    w[ids[19]] = v[ids[19]]
    order = np.argsort(-w, kind="stable")
    w[order[20]] = w[order[19]] - 1e-6
    alt = order[:20].copy()
    alt[19] = order[20]
    assert mo.valid_topk(w, alt, 20, 1e-4)[0]
