"""Planted mistakes in a copy of the oracle (CPU only): each must fail at
least one of the pins, which shows the pins constrain every part of it.

Each mutant is the oracle source with one plausible slip, compiled to a
temporary library; the original file is never touched.
"""
import os
import subprocess

import numpy as np
import pytest

import oracle
from oracle.oracle import CXXFLAGS
from fstcheck import assert_same, brute_force, canon_of, label_matrices, path_weights
from paper_1805_06383_amd import workloads as W

SRC = os.path.join(os.path.dirname(oracle.__file__), "fst_oracle.cpp")

MUTANTS = {
    # output label taken from M2's input side instead of its output side
    "wrong_output_label": ("m1->ilabel[e1], m2->olabel[e2]}", "m1->ilabel[e1], m2->ilabel[e2]}"),
    # input label taken from M1's output side
    "wrong_input_label": ("m1->ilabel[e1], m2->olabel[e2]}", "m1->olabel[e1], m2->olabel[e2]}"),
    # join on M1's input symbol instead of its output (inner) symbol
    "join_on_input": ("const uint32_t b = m1->olabel[e1];", "const uint32_t b = m1->ilabel[e1];"),
    # one factor of the product dropped
    "dropped_factor": ("m1->weight[e1] * m2->weight[e2]", "m1->weight[e1] * 1.0f"),
    # duplicates overwrite instead of adding
    "no_merge_sum": ("+= (double)prod;", "= (double)prod;"),
    # target pair transposed
    "swapped_target": ("ArcKey{m1->dst[e1], m2->dst[e2]", "ArcKey{m2->dst[e2], m1->dst[e1]"),
    # accept test ignores M2
    "final_ignores_m2": ("&& m2->final[res.pairs[i].second]", "&& 1"),
    # level cap off by one
    "cap_off_by_one": ("res.depth[u] >= max_levels", "res.depth[u] > max_levels"),
    # new states not searched (no push on the frontier)
    "no_push": ("        A.push_back(vid);\n", "\n"),
}


# planted mistakes in the epsilon filter (compose_eps)
MUTANTS_EPS = {
    # M2 may move alone after M1 moved alone: two orders of the same moves
    "eps_both_orders": ("if (f == 0 || f == 1) {  // M2 alone", "if (true) {  // M2 alone"),
    # both moving on the empty label is never taken
    "eps_no_joint_move": ("if (b != eps || f == 0) {", "if (b != eps) {"),
    # both moving on the empty label allowed from every filter state
    "eps_joint_any_state": ("if (b != eps || f == 0) {", "if (true) {"),
    # M1 alone returns to filter state 0
    "eps_m1_alone_state": ("out.push_back({m1->dst[e1], q2, 2,", "out.push_back({m1->dst[e1], q2, 0,"),
    # M2 alone carries weight one instead of its arc's
    "eps_m2_alone_weight": ("m2->olabel[e2], m2->weight[e2]});", "m2->olabel[e2], 1.0f});"),
    # M1 alone writes its input symbol instead of the empty string
    "eps_m1_alone_label": ("m1->ilabel[e1], eps, m1->weight[e1]", "m1->ilabel[e1], m1->ilabel[e1], m1->weight[e1]"),
}


def _tiny(seed):
    rng = np.random.default_rng(seed)
    m1 = W.tiny_random(rng, 4, 2, 2, 12, final_frac=0.5)
    m2 = W.tiny_random(rng, 4, 2, 2, 12, final_frac=0.5)
    return m1, m2


def run_pins(lib):
    """Returns the names of the pins that fail for the library at ``lib``."""
    failed = set()
    for seed in range(12):
        m1, m2 = _tiny(seed)
        try:
            got = oracle.compose(m1, m2, lib_path=lib)
            assert_same(canon_of(got), canon_of(brute_force(m1, m2)), rtol=1e-6)
        except (AssertionError, IndexError, ValueError):
            failed.add("brute_force")
        try:
            got = oracle.compose(m1, m2, max_levels=2, lib_path=lib)
            assert_same(canon_of(got), canon_of(brute_force(m1, m2, max_levels=2)), rtol=1e-6)
        except (AssertionError, IndexError, ValueError):
            failed.add("brute_force_cap")
        try:
            r = oracle.compose(m1, m2, lib_path=lib)
            T1 = label_matrices(4, 0, 2, 2, m1.src, m1.dst, m1.ilabel, m1.olabel, m1.weight)
            T2 = label_matrices(4, 0, 2, 2, m2.src, m2.dst, m2.ilabel, m2.olabel, m2.weight)
            Tc = label_matrices(r.num_states, 0, 2, 2, r.src, r.dst, r.a, r.c, r.w)
            for ln in (1, 2, 3):
                W1 = path_weights(T1, m1.start, m1.final.astype(float), ln)
                W2 = path_weights(T2, m2.start, m2.final.astype(float), ln)
                Wc = path_weights(Tc, 0, r.final.astype(float), ln)
                np.testing.assert_allclose(Wc, W1 @ W2, rtol=1e-5, atol=1e-12)
        except (AssertionError, IndexError, ValueError):
            failed.add("path_sum")
    rng = np.random.default_rng(5)
    A = W.random_weights(rng, 12).reshape(3, 4)
    B = W.random_weights(rng, 8).reshape(4, 2)
    try:
        r = oracle.compose(W.one_state_dense(A), W.one_state_dense(B), lib_path=lib)
        P = A.astype(np.float64) @ B.astype(np.float64)
        np.testing.assert_allclose(r.w.astype(np.float64), P[r.a, r.c], rtol=1e-6)
        assert r.num_arcs == 6
    except (AssertionError, IndexError, ValueError):
        failed.add("matrix_product")
    return failed


@pytest.fixture(scope="module")
def mutant_dir(tmp_path_factory):
    return tmp_path_factory.mktemp("oracle_mutants")


def test_unmutated_copy_passes(mutant_dir):
    out = mutant_dir / "liboracle_clean.so"
    subprocess.run(["g++", *CXXFLAGS, "-o", str(out), SRC], check=True)
    assert run_pins(out) == set()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, mutant_dir):
    old, new = MUTANTS[name]
    text = open(SRC).read()
    assert text.count(old) >= 1, f"mutation site for {name} not found"
    src = mutant_dir / f"{name}.cpp"
    src.write_text(text.replace(old, new))
    out = mutant_dir / f"lib{name}.so"
    subprocess.run(["g++", *CXXFLAGS, "-o", str(out), str(src)], check=True)
    failed = run_pins(out)
    assert failed, f"planted mistake {name} passed every pin"


# Planted mistakes in the composition without reduction; caught by its own
# pins (brute force without merging, the one-state closed form).
MUTANTS_UNREDUCED = {
    # product with one factor dropped
    "unreduced_dropped_factor": ("m1->weight[e1] * m2->weight[e2]});",
                                 "m1->weight[e1] * 1.0f});"),
    # identical arcs merged after all
    "unreduced_merges": ("    if (!reduce) {", "    if (false) {"),
    # every arc points back at its source
    "unreduced_self_target": ("res.arcs.push_back({u, vid, j.a, j.c, j.w});",
                              "res.arcs.push_back({u, u, j.a, j.c, j.w});"),
    # output label from M2's input side
    "unreduced_wrong_output": ("m1->ilabel[e1], m2->olabel[e2],\n", "m1->ilabel[e1], m2->ilabel[e2],\n"),
}


def run_pins_unreduced(lib):
    from fstcheck import assert_same_multiset, brute_force_unreduced, multiset_of
    failed = set()
    for seed in range(12):
        m1, m2 = _tiny(seed)
        try:
            got = oracle.compose(m1, m2, lib_path=lib, reduce=False)
            assert_same_multiset(multiset_of(got), multiset_of(brute_force_unreduced(m1, m2)))
        except (AssertionError, IndexError, ValueError):
            failed.add("brute_force_unreduced")
    rng = np.random.default_rng(6)
    A = W.random_weights(rng, 12).reshape(3, 4)
    B = W.random_weights(rng, 8).reshape(4, 2)
    try:
        r = oracle.compose(W.one_state_dense(A), W.one_state_dense(B), lib_path=lib, reduce=False)
        assert r.num_arcs == 24
        a, b, c = np.meshgrid(np.arange(3), np.arange(4), np.arange(2), indexing="ij")
        want = np.stack([a.ravel(), c.ravel(), (A[a, b].astype(np.float32) * B[b, c].astype(
            np.float32)).ravel().view(np.uint32)], 1).astype(np.int64)
        have = np.stack([r.a, r.c, r.w.view(np.uint32)], 1).astype(np.int64)
        assert np.array_equal(have[np.lexsort(have.T[::-1])], want[np.lexsort(want.T[::-1])])
    except (AssertionError, IndexError, ValueError):
        failed.add("closed_form_unreduced")
    return failed


def test_unmutated_copy_passes_unreduced(mutant_dir):
    out = mutant_dir / "liboracle_clean_u.so"
    subprocess.run(["g++", *CXXFLAGS, "-o", str(out), SRC], check=True)
    assert run_pins_unreduced(out) == set()


@pytest.mark.parametrize("name", sorted(MUTANTS_UNREDUCED))
def test_unreduced_mutant_is_caught(name, mutant_dir):
    old, new = MUTANTS_UNREDUCED[name]
    text = open(SRC).read()
    assert text.count(old) >= 1, f"mutation site for {name} not found"
    src = mutant_dir / f"{name}.cpp"
    src.write_text(text.replace(old, new))
    out = mutant_dir / f"lib{name}.so"
    subprocess.run(["g++", *CXXFLAGS, "-o", str(out), str(src)], check=True)
    assert run_pins_unreduced(out), f"planted mistake {name} passed every pin"


# Planted mistakes in the per-source expansion (oracle_expand_pairs): its
# batch assembly is its own code, so each slip there must fail one of its
# pins (tests/test_oracle_expand.py's checks, run here on a few batches).
MUTANTS_EXPAND = {
    # the merge map survives from one source to the next
    "expand_map_not_reset": ("    std::map<ArcKey, double> acc;\n    r->premerge",
                             "    static std::map<ArcKey, double> acc;\n    r->premerge"),
    # arcs carry the next batch index
    "expand_src_off_by_one": ("r->arcs.push_back({(uint32_t)i, vid,",
                              "r->arcs.push_back({(uint32_t)(i + 1 < n ? i + 1 : i), vid,"),
    # targets numbered from 0, on top of the sources
    "expand_targets_from_zero": ("vid = (uint32_t)r->pairs.size();",
                                 "vid = (uint32_t)(r->pairs.size() - n);"),
    # a target pair seen before gets a new id again
    "expand_no_target_dedup": ("auto it = tid.find(v);", "auto it = tid.end();"),
    # accept flags ignore M2
    "expand_final_ignores_m2": ("&& m2->final[r->pairs[i].second]", "&& 1"),
    # the joined count keeps only the last source
    "expand_count_overwritten": ("r->premerge += expand_pair(", "r->premerge = expand_pair("),
}


def run_pins_expand(lib):
    from test_oracle_expand import check_batch
    failed = set()
    cases = []
    for seed in range(8):
        m1, m2 = _tiny(100 + seed)
        rng = np.random.default_rng(seed)
        k = 6
        cases.append((m1, m2, rng.integers(0, 4, k).astype(np.uint32),
                      rng.integers(0, 4, k).astype(np.uint32)))
    m1, m2 = W.config1(2)
    rng = np.random.default_rng(3)
    cases.append((m1, m2, rng.integers(0, 200, 30).astype(np.uint32),
                  rng.integers(0, 200, 30).astype(np.uint32)))
    for m1, m2, q1s, q2s in cases:
        try:
            check_batch(oracle.expand_pairs(m1, m2, q1s, q2s, lib_path=lib), m1, m2, q1s, q2s)
        except (AssertionError, IndexError, ValueError):
            failed.add("batch")
    return failed


def test_unmutated_copy_passes_expand(mutant_dir):
    out = mutant_dir / "liboracle_clean_e.so"
    subprocess.run(["g++", *CXXFLAGS, "-o", str(out), SRC], check=True)
    assert run_pins_expand(out) == set()


@pytest.mark.parametrize("name", sorted(MUTANTS_EXPAND))
def test_expand_mutant_is_caught(name, mutant_dir):
    old, new = MUTANTS_EXPAND[name]
    text = open(SRC).read()
    assert text.count(old) == 1, f"mutation site for {name} not found once"
    src = mutant_dir / f"{name}.cpp"
    src.write_text(text.replace(old, new))
    out = mutant_dir / f"lib{name}.so"
    subprocess.run(["g++", *CXXFLAGS, "-o", str(out), str(src)], check=True)
    assert run_pins_expand(out), f"planted mistake {name} passed every pin"


def run_pins_eps(lib):
    """Names of the epsilon-composition pins failing for the library at lib."""
    import test_oracle_eps as E
    failed = set()
    for seed in range(40):
        m1, m2 = E.acyclic_pair(seed) if seed < 25 else E.acyclic_pair(
            1000 + seed, eps_in=0.3, eps_inner=0.8, eps_out=0.3)
        try:
            r = oracle.compose_eps(m1, m2, E.EPS, lib_path=lib)
            E.assert_relations_equal(E.result_relation(r), E.composed_relation(m1, m2))
        except (AssertionError, IndexError, ValueError, KeyError):
            failed.add("relation")
    for name in ("test_one_output_eps_meets_one_input_eps", "test_two_output_eps_against_one_input_eps",
                 "test_epsilon_then_symbol", "test_both_sides_empty_everywhere"):
        fn = getattr(E, name)
        saved = E.oracle.compose_eps
        try:
            E.oracle.compose_eps = lambda *a, **k: saved(*a, lib_path=lib, **k)
            fn()
        except (AssertionError, IndexError, ValueError, KeyError):
            failed.add(name)
        finally:
            E.oracle.compose_eps = saved
    return failed


def test_eps_pins_pass_on_the_oracle():
    assert run_pins_eps(None) == set()


@pytest.mark.parametrize("name", sorted(MUTANTS_EPS))
def test_eps_mutant_is_caught(tmp_path, name):
    old, new = MUTANTS_EPS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site of {name} not unique"
    mut = tmp_path / f"{name}.cpp"
    mut.write_text(src.replace(old, new))
    lib = tmp_path / f"lib{name}.so"
    subprocess.run(["g++", *CXXFLAGS, "-o", str(lib), str(mut)], check=True)
    assert run_pins_eps(lib), f"mutant {name} passes every epsilon pin"
