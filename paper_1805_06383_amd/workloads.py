"""Seeded synthetic transducers shaped like the workloads of Argueta & Chiang,
"Composing Finite State Transducers on GPUs" (§3.1 Table 1, §4.1).

This module only draws inputs.  It holds none of the composition arithmetic and
is shared, unchanged, by the CPU oracle side and the HIP side, which otherwise
share no code.

A transducer is M = (Q, Sigma, Gamma, s, F, delta) (§2).  It is stored as a
coordinate list of arcs, one row per transition q -a:b/p-> r:

    src[k] = q,  dst[k] = r,  ilabel[k] = a,  olabel[k] = b,  weight[k] = p

with states 0..num_states-1, input symbols 0..num_isyms-1, output symbols
0..num_osyms-1 and start state ``start``.  ``final[q]`` is 1 for accept states.
There are no epsilon labels (§2): every label is an ordinary symbol.  Arcs form
a multiset: the same (src, dst, ilabel, olabel) may be listed more than once.

Weights are drawn as k / 2**24 with k uniform in 1..2**24, i.e. uniform on
(0, 1] at float32 resolution near 1, so every weight is an exact float32 and no
weight is zero.

Config numbering follows the five workload descriptions (tiny random pair,
medium sparse pair, lexicon trie pair, HMM-like dense inner alphabet, large
power-law pair).  Seeds: ``np.random.default_rng(1000 * config + seed)``.
"""
from __future__ import annotations

import hashlib
from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "FST", "random_weights", "tiny_random", "config1", "config2", "config3",
    "config4", "config5", "make_config", "identity", "one_state_dense",
    "CONFIG_NAMES", "PAPER_SHAPES", "lm_tm", "paper_pair",
]

CONFIG_NAMES = {
    1: "tiny random pair (|Q|=200, 2k arcs each)",
    2: "medium sparse pair (|Q|=10k, 200k arcs each, Zipf inner over 5k)",
    3: "lexicon trie pair (50k words, |Gamma|=50k, |Delta|=20k)",
    4: "HMM-like dense inner alphabet (|Q|=1k, m=64, 256 arcs/state)",
    5: "large power-law pair (|Q|=1M, 20M arcs each)",
}


@dataclass
class FST:
    """Coordinate-list weighted transducer (see module docstring)."""

    num_states: int
    start: int
    num_isyms: int
    num_osyms: int
    src: np.ndarray
    dst: np.ndarray
    ilabel: np.ndarray
    olabel: np.ndarray
    weight: np.ndarray
    final: np.ndarray
    name: str = ""
    meta: dict = field(default_factory=dict)

    def __post_init__(self):
        self.src = np.ascontiguousarray(self.src, dtype=np.uint32)
        self.dst = np.ascontiguousarray(self.dst, dtype=np.uint32)
        self.ilabel = np.ascontiguousarray(self.ilabel, dtype=np.uint32)
        self.olabel = np.ascontiguousarray(self.olabel, dtype=np.uint32)
        self.weight = np.ascontiguousarray(self.weight, dtype=np.float32)
        self.final = np.ascontiguousarray(self.final, dtype=np.uint8)
        n = len(self.src)
        assert len(self.dst) == n and len(self.ilabel) == n
        assert len(self.olabel) == n and len(self.weight) == n
        assert len(self.final) == self.num_states

    @property
    def num_arcs(self) -> int:
        return int(len(self.src))

    def digest(self) -> str:
        """SHA-256 over the header and every array, for run reports."""
        h = hashlib.sha256()
        h.update(np.array([self.num_states, self.start, self.num_isyms,
                           self.num_osyms, self.num_arcs], dtype=np.uint64).tobytes())
        for a in (self.src, self.dst, self.ilabel, self.olabel, self.weight, self.final):
            h.update(a.tobytes())
        return h.hexdigest()


def random_weights(rng: np.random.Generator, n: int) -> np.ndarray:
    """n weights uniform on (0, 1], each k/2**24 for integer k in [1, 2**24]."""
    k = rng.integers(1, 2**24 + 1, size=n, dtype=np.int64)
    return (k.astype(np.float64) / float(2**24)).astype(np.float32)


def _finals(rng: np.random.Generator, num_states: int, frac: float) -> np.ndarray:
    """Exactly round(frac * num_states) accept states, chosen without replacement."""
    f = np.zeros(num_states, dtype=np.uint8)
    k = int(round(frac * num_states))
    if k > 0:
        f[rng.choice(num_states, size=k, replace=False)] = 1
    return f


def _zipf(rng: np.random.Generator, n: int, s: float, size: int) -> np.ndarray:
    """Symbol ids 0..n-1 with P(id = k-1) proportional to k**-s (finite Zipf)."""
    p = np.arange(1, n + 1, dtype=np.float64) ** (-s)
    p /= p.sum()
    return rng.choice(n, size=size, p=p).astype(np.uint32)


def tiny_random(rng: np.random.Generator, nq: int, nin: int, nout: int,
                narcs: int, final_frac: float = 0.3, start: int = 0) -> FST:
    """Small FST with uniform src/dst/labels; used for brute-force checks."""
    return FST(
        num_states=nq, start=start, num_isyms=nin, num_osyms=nout,
        src=rng.integers(0, nq, narcs), dst=rng.integers(0, nq, narcs),
        ilabel=rng.integers(0, nin, narcs), olabel=rng.integers(0, nout, narcs),
        weight=random_weights(rng, narcs),
        final=(rng.random(nq) < final_frac).astype(np.uint8),
        name=f"tiny(q={nq},in={nin},out={nout},arcs={narcs})",
    )


def eps_random(rng: np.random.Generator, nq: int, nin: int, nout: int, narcs: int,
               eps_in: float, eps_out: float, final_frac: float = 0.3, acyclic: bool = False,
               eps: int = 0) -> FST:
    """Small FST whose labels are the empty-string label ``eps`` with
    probability eps_in (input tape) and eps_out (output tape), else uniform
    over the other symbols; with acyclic=True every arc goes from a lower to a
    higher state (its paths are finite)."""
    if acyclic:
        src = rng.integers(0, nq - 1, narcs)
        dst = src + 1 + (rng.random(narcs) * (nq - 1 - src)).astype(np.int64)
    else:
        src, dst = rng.integers(0, nq, narcs), rng.integers(0, nq, narcs)

    def labels(n, size, p):
        lab = rng.integers(0, size - 1, n)
        lab = lab + (lab >= eps)  # uniform over the symbols other than eps
        return np.where(rng.random(n) < p, eps, lab)

    return FST(num_states=nq, start=0, num_isyms=nin, num_osyms=nout, src=src, dst=dst,
               ilabel=labels(narcs, nin, eps_in), olabel=labels(narcs, nout, eps_out),
               weight=random_weights(rng, narcs),
               final=(rng.random(nq) < final_frac).astype(np.uint8),
               name=f"eps(q={nq},arcs={narcs},in={eps_in},out={eps_out})")


def eps_pair(seed: int = 0, nq: int = 200, narcs: int = 2000, nsym: int = 100,
             nouter: int = 50, eps_inner: float = 0.1, eps_outer: float = 0.05):
    """Config-1-shaped pair with the empty-string label 0 on every tape: M1's
    outputs and M2's inputs are label 0 with probability eps_inner, the outer
    tapes with probability eps_outer; other labels uniform."""
    rng = np.random.default_rng(7000 + seed)
    m1 = eps_random(rng, nq, nouter, nsym, narcs, eps_outer, eps_inner, final_frac=0.1)
    m2 = eps_random(rng, nq, nsym, nouter, narcs, eps_inner, eps_outer, final_frac=0.1)
    m1.name, m2.name = "eps.M1", "eps.M2"
    return m1, m2


def config1(seed: int = 0):
    """Tiny random pair: |Q|=200, |Sigma|=|Delta|=50, |Gamma|=100, 2,000 arcs
    each with uniform src, dst and labels, 10% accept states."""
    rng = np.random.default_rng(1000 * 1 + seed)
    nq, ns, ng, nd, na = 200, 50, 100, 50, 2000
    m1 = FST(nq, 0, ns, ng, rng.integers(0, nq, na), rng.integers(0, nq, na),
             rng.integers(0, ns, na), rng.integers(0, ng, na),
             random_weights(rng, na), _finals(rng, nq, 0.10), name="cfg1.M1")
    m2 = FST(nq, 0, ng, nd, rng.integers(0, nq, na), rng.integers(0, nq, na),
             rng.integers(0, ng, na), rng.integers(0, nd, na),
             random_weights(rng, na), _finals(rng, nq, 0.10), name="cfg1.M2")
    return m1, m2


def config2(seed: int = 0):
    """Medium sparse pair: |Q|=10,000, 200,000 arcs each (uniform sources, so
    out-degree is close to Poisson(20)), uniform targets, inner symbols
    Zipf(1.0) over 5,000, outer symbols uniform over 2,000, 5% accept."""
    rng = np.random.default_rng(1000 * 2 + seed)
    nq, na, ng, nouter = 10_000, 200_000, 5_000, 2_000

    def one(inner_is_output: bool, name: str) -> FST:
        src = rng.integers(0, nq, na)
        dst = rng.integers(0, nq, na)
        inner = _zipf(rng, ng, 1.0, na)
        outer = rng.integers(0, nouter, na)
        w = random_weights(rng, na)
        fin = _finals(rng, nq, 0.05)
        if inner_is_output:
            return FST(nq, 0, nouter, ng, src, dst, outer, inner, w, fin, name=name)
        return FST(nq, 0, ng, nouter, src, dst, inner, outer, w, fin, name=name)

    return one(True, "cfg2.M1"), one(False, "cfg2.M2")


def config3(seed: int = 0, num_words: int = 50_000, num_chars: int = 30,
            num_out: int = 20_000):
    """Lexicon trie pair.

    M1: prefix tree of ``num_words`` distinct random words (length uniform in
    3..12 over ``num_chars`` letters).  States are trie nodes (root = 0); each
    (word, position i) contributes one arc prefix_i -w[i]:wordid-> prefix_i+1,
    and word-end nodes accept.  M2: a single state (start and accept) with 1..5
    self-loops wordid:t per word, t drawn Zipf(1.1) over ``num_out`` ids.
    """
    rng = np.random.default_rng(1000 * 3 + seed)
    words: list[bytes] = []
    seen: set[bytes] = set()
    while len(words) < num_words:
        need = num_words - len(words)
        lens = rng.integers(3, 13, size=2 * need + 16)
        chars = rng.integers(0, num_chars, size=int(lens.sum()), dtype=np.uint8)
        pos = 0
        for ln in lens:
            w = chars[pos:pos + ln].tobytes()
            pos += ln
            if w not in seen:
                seen.add(w)
                words.append(w)
                if len(words) == num_words:
                    break
    node = {b"": 0}
    src, dst, il, ol = [], [], [], []
    for wid, w in enumerate(words):
        for i in range(len(w)):
            a = node[w[:i]]
            key = w[:i + 1]
            b = node.get(key)
            if b is None:
                b = len(node)
                node[key] = b
            src.append(a)
            dst.append(b)
            il.append(w[i])
            ol.append(wid)
    nq1 = len(node)
    fin1 = np.zeros(nq1, dtype=np.uint8)
    for w in words:
        fin1[node[w]] = 1
    n1 = len(src)
    m1 = FST(nq1, 0, num_chars, num_words, np.array(src), np.array(dst),
             np.array(il), np.array(ol), random_weights(rng, n1), fin1,
             name="cfg3.M1")
    k = rng.integers(1, 6, size=num_words)
    wid = np.repeat(np.arange(num_words), k)
    n2 = len(wid)
    t = _zipf(rng, num_out, 1.1, n2)
    m2 = FST(1, 0, num_words, num_out, np.zeros(n2), np.zeros(n2), wid, t,
             random_weights(rng, n2), np.ones(1, dtype=np.uint8), name="cfg3.M2")
    return m1, m2


def config4(seed: int = 0, nq: int = 1000, m: int = 64, nsym: int = 64,
            slots: int = 4, final_frac: float = 0.10):
    """HMM-like dense inner alphabet with heavy merging.

    Every state q owns ``slots`` fixed (outer symbol, target) pairs; for every
    inner symbol b in 0..m-1 and every slot there is one arc carrying that
    slot's outer symbol and target with its own weight, so each state has
    m * slots arcs and the composition repeats each (src, dst, in, out) key
    m times.  M1 reads outer symbols and writes inner ones; M2 the reverse.
    """
    rng = np.random.default_rng(1000 * 4 + seed)

    def one(inner_is_output: bool, name: str) -> FST:
        outer_slot = rng.integers(0, nsym, size=(nq, slots))
        tgt_slot = rng.integers(0, nq, size=(nq, slots))
        q = np.repeat(np.arange(nq), m * slots)
        b = np.tile(np.repeat(np.arange(m), slots), nq)
        k = np.tile(np.arange(slots), nq * m)
        outer = outer_slot[q, k]
        dst = tgt_slot[q, k]
        w = random_weights(rng, len(q))
        fin = _finals(rng, nq, final_frac)
        if inner_is_output:
            return FST(nq, 0, nsym, m, q, dst, outer, b, w, fin, name=name)
        return FST(nq, 0, m, nsym, q, dst, b, outer, w, fin, name=name)

    return one(True, "cfg4.M1"), one(False, "cfg4.M2")


def config5(seed: int = 0, nq: int = 1_000_000, na: int = 20_000_000,
            alpha: float = 2.1, dmin: int = 4, dmax: int = 10_000,
            ng: int = 100_000, nouter: int = 10_000, final_frac: float = 0.01,
            hub_start: bool = True):
    """Large pair: power-law out-degree P(d) ~ d**-alpha on [dmin, dmax],
    adjusted uniformly to exactly ``na`` arcs; uniform targets; inner symbols
    Zipf(1.0) over ``ng``; outer symbols uniform over ``nouter``; 1% accept.
    The start state 0 is a state of largest out-degree (its label is swapped
    with that state's), as the start of a language-model-like transducer is
    its busiest state; with a typical start the two start states would share
    no inner symbol and the composition would stop at one state.  With
    hub_start=False state 0 keeps its generated arcs."""
    rng = np.random.default_rng(1000 * 5 + seed)
    dvals = np.arange(dmin, dmax + 1, dtype=np.float64)
    pd = dvals ** (-alpha)
    pd /= pd.sum()

    def one(inner_is_output: bool, name: str) -> FST:
        deg = rng.choice(dvals.astype(np.int64), size=nq, p=pd)
        src = np.repeat(np.arange(nq, dtype=np.uint32), deg)
        if len(src) > na:
            keep = np.sort(rng.choice(len(src), size=na, replace=False))
            src = src[keep]
        elif len(src) < na:
            src = np.concatenate([src, rng.integers(0, nq, na - len(src)).astype(np.uint32)])
        perm = rng.permutation(na)
        src = src[perm]
        dst = rng.integers(0, nq, na)
        hub = int(np.argmax(np.bincount(src, minlength=nq)))
        if hub and hub_start:  # relabel: the busiest state becomes state 0
            relabel = np.arange(nq, dtype=np.int64)
            relabel[[0, hub]] = [hub, 0]
            src = relabel[src].astype(np.uint32)
            dst = relabel[dst]
        inner = _zipf(rng, ng, 1.0, na)
        outer = rng.integers(0, nouter, na)
        w = random_weights(rng, na)
        fin = _finals(rng, nq, final_frac)
        if inner_is_output:
            return FST(nq, 0, nouter, ng, src, dst, outer, inner, w, fin, name=name)
        return FST(nq, 0, ng, nouter, src, dst, inner, outer, w, fin, name=name)

    return one(True, "cfg5.M1"), one(False, "cfg5.M2")


# ---------------------------------------------------------------------------
# Transducers shaped like the paper's own (§4.1, Figure 3): a bigram language
# model over the output language pre-composed with a one-state translation
# model, so that a state is the last output word (plus a sentence-start
# state) and an arc e' -f:e-> e reads a source word f that translates to the
# output word e.  Sizes follow Table 1, reading its "Transitions" column as
# |Q|^2 (so |Q| = sqrt(Transitions)) and "Nonzero" as the number of arcs.
# The Europarl-trained models themselves are not available; every statistic
# below (Zipf word frequencies, successor counts, translation counts, weights)
# is drawn synthetically.
PAPER_SHAPES = {  # size -> language pair -> (states, arcs)
    "1k": {"de-en": (4658, 16_500), "en-de": (3507, 15_400), "en-es": (3536, 15_500),
           "en-it": (3619, 16_300)},
    "10k": {"de-en": (19849, 114_000), "en-de": (11747, 93_900), "en-es": (11619, 93_300),
            "en-it": (11958, 97_200)},
    "15k": {"de-en": (25179, 158_000), "en-de": (14177, 126_000), "en-es": (13964, 125_000),
            "en-it": (14457, 131_000)},
}


def lm_tm(rng: np.random.Generator, v_in: int, v_out: int, n_arcs: int,
          final_frac: float = 0.3, name: str = "") -> FST:
    """Bigram-LM x one-state-TM transducer from v_in source words to v_out
    output words with exactly n_arcs arcs.

    State 0 is the sentence start, state 1 + e the context "last output word
    was e".  Output words have Zipf(1.0) frequencies; each has 1 + Poisson(1)
    distinct translations drawn by Zipf(1.0) over the source words.  Each
    context has a successor set of output words (the sentence start a large
    one, a word context one growing with the word's frequency), drawn by
    frequency; every (context, successor e, translation f of e) is an arc
    context -f:e-> 1 + e with weight P(e | context) * P(f | e), both factors
    normalised random weights.  The arc list is then cut or topped up
    uniformly to exactly n_arcs."""
    nq = v_out + 1
    # translations of every output word
    ntr = 1 + rng.poisson(1.0, v_out)
    tr_word = np.repeat(np.arange(v_out), ntr)
    tr_src = _zipf(rng, v_in, 1.0, int(ntr.sum()))
    tr_p = random_weights(rng, len(tr_word)).astype(np.float64)
    tr_p /= np.bincount(tr_word, weights=tr_p, minlength=v_out)[tr_word]
    # successor sets: about n_arcs / mean(translations) (context, word) pairs
    n_bigrams = int(np.ceil(n_arcs / ntr.mean()))
    rank_w = 1.0 / np.arange(1, v_out + 1)  # Zipf(1.0) frequency of word ranks
    ctx_w = np.r_[0.05 * rank_w.sum(), rank_w]  # the sentence start: about 5% of contexts
    ctx = rng.choice(nq, size=n_bigrams, p=ctx_w / ctx_w.sum())
    nxt = _zipf(rng, v_out, 1.0, n_bigrams)
    bg = np.unique(np.stack([ctx, nxt], 1), axis=0)
    bg_p = random_weights(rng, len(bg)).astype(np.float64)
    bg_p /= np.bincount(bg[:, 0], weights=bg_p, minlength=nq)[bg[:, 0]]
    # arcs = bigram x translation of its word
    order = np.argsort(tr_word, kind="stable")
    first = np.r_[0, np.cumsum(ntr)]
    cnt = ntr[bg[:, 1]]
    rep = np.repeat(np.arange(len(bg)), cnt)
    k = np.arange(len(rep)) - np.repeat(np.cumsum(cnt) - cnt, cnt)  # translation index
    t = order[first[bg[rep, 1]] + k]
    src = bg[rep, 0]
    out = bg[rep, 1]
    w = (bg_p[rep] * tr_p[t]).astype(np.float32)
    inp = tr_src[t]
    if len(src) > n_arcs:
        keep = np.sort(rng.choice(len(src), size=n_arcs, replace=False))
        src, out, inp, w = src[keep], out[keep], inp[keep], w[keep]
    elif len(src) < n_arcs:
        extra = rng.integers(0, len(src), n_arcs - len(src))
        src, out, inp, w = (np.r_[src, src[extra]], np.r_[out, out[extra]],
                            np.r_[inp, inp[extra]], np.r_[w, w[extra]])
    return FST(nq, 0, v_in, v_out, src, 1 + out, inp, out, w, _finals(rng, nq, final_frac),
               name=name)


def paper_pair(size: str = "1k", target: str = "de", seed: int = 0):
    """(M1, M2) = (German-to-English, English-to-target) transducers of the
    paper's experiment at one of its three training sizes (Table 1), for the
    composition German -> target.  M1's output alphabet is M2's input
    alphabet (the English words)."""
    shapes = PAPER_SHAPES[size]
    q_en, arcs1 = shapes["de-en"]
    q_de = shapes["en-de"][0]
    q_t, arcs2 = shapes[f"en-{target}"]
    rng = np.random.default_rng(6000 + 100 * list(PAPER_SHAPES).index(size)
                                + 10 * ["de", "es", "it"].index(target) + seed)
    m1 = lm_tm(rng, q_de - 1, q_en - 1, arcs1, name=f"{size}.de-en")
    m2 = lm_tm(rng, q_en - 1, q_t - 1, arcs2, name=f"{size}.en-{target}")
    return m1, m2


def make_config(cfg: int, seed: int = 0):
    return {1: config1, 2: config2, 3: config3, 4: config4, 5: config5}[cfg](seed)


def identity(n: int, name: str = "Id") -> FST:
    """One-state identity transducer over n symbols: arcs b:b/1.0, start = accept."""
    b = np.arange(n)
    return FST(1, 0, n, n, np.zeros(n), np.zeros(n), b, b,
               np.ones(n, dtype=np.float32), np.ones(1, dtype=np.uint8), name=name)


def one_state_dense(W: np.ndarray, name: str = "dense") -> FST:
    """One-state transducer with an arc a:b/W[a, b] for every (a, b)."""
    W = np.asarray(W, dtype=np.float32)
    na, nb = W.shape
    a, b = np.meshgrid(np.arange(na), np.arange(nb), indexing="ij")
    a, b = a.ravel(), b.ravel()
    return FST(1, 0, na, nb, np.zeros(a.size), np.zeros(a.size), a, b,
               W[a, b], np.ones(1, dtype=np.uint8), name=name)


def wide_parts_pair(seed: int = 0, nq: int = 2000, hub_parts: int = 70_000,
                    small_arcs: int = 10, small_inner: int = 100, hub_dups: int = 5000):
    """A pair whose start states each have more than 2^16 distinct
    (target, outer symbol) pairs, so that a composed arc's two part ranks need
    more than 32 bits together.

    State 0 of M1 has ``hub_parts`` arcs k:k -> 1 + k mod (nq - 1) (outer
    symbol k, inner symbol k); state 0 of M2 has arcs k:k -> 1 + 7k mod
    (nq - 1).  The start pair joins them one to one.  Every other state has
    ``small_arcs`` arcs with uniform targets (state 0 included), inner symbols
    uniform over the first ``small_inner`` and outer symbols uniform, so that
    later levels mix sources of the hub states with small ones.  The first
    ``hub_dups`` hub arcs are listed twice (new weights), so that the start
    pair's composed arcs merge in pairs.  30% of states accept."""
    rng = np.random.default_rng(7000 + seed)
    ng = hub_parts  # inner alphabet: the hub's symbols

    def one(mult: int, inner_is_output: bool, name: str) -> FST:
        k = np.r_[np.arange(hub_parts), np.arange(hub_dups)]
        hsrc = np.zeros(len(k), np.int64)
        hdst = 1 + (mult * k) % (nq - 1)
        n = (nq - 1) * small_arcs
        ssrc = np.repeat(np.arange(1, nq), small_arcs)
        sdst = rng.integers(0, nq, n)
        sinner = rng.integers(0, small_inner, n)
        souter = rng.integers(0, hub_parts, n)
        src = np.r_[hsrc, ssrc]
        dst = np.r_[hdst, sdst]
        inner = np.r_[k, sinner]
        outer = np.r_[k, souter]
        w = random_weights(rng, len(src))
        fin = _finals(rng, nq, 0.3)
        if inner_is_output:
            return FST(nq, 0, hub_parts, ng, src, dst, outer, inner, w, fin, name=name)
        return FST(nq, 0, ng, hub_parts, src, dst, inner, outer, w, fin, name=name)

    return one(1, True, "wide.M1"), one(7, False, "wide.M2")


def hub_pair(seed: int = 0, nq: int = 8250, hub: int = 2900, ninner: int = 8):
    """A pair whose start states join on one inner symbol with ``hub`` arcs
    each (distinct targets 1..hub, outer symbols uniform over 64), so the start
    pair alone has hub^2 composed arcs to hub^2 distinct target pairs.  Every
    other state has one arc with a uniform target, inner symbol uniform over
    ``ninner`` and outer symbol uniform over 64.  With nq = 8250 the pair space
    (6.8e7) is above 2^26 and the start pair's 8.4M targets are enough to make
    the visited set's hash table outgrow a dense array of all pairs."""
    rng = np.random.default_rng(8000 + seed)

    def one(inner_is_output: bool, name: str) -> FST:
        hsrc = np.zeros(hub, np.int64)
        hdst = 1 + np.arange(hub)
        hin = np.zeros(hub, np.int64)
        ssrc = np.arange(1, nq)
        sdst = rng.integers(0, nq, nq - 1)
        sin = rng.integers(0, ninner, nq - 1)
        src, dst, inner = np.r_[hsrc, ssrc], np.r_[hdst, sdst], np.r_[hin, sin]
        outer = rng.integers(0, 64, len(src))
        w = random_weights(rng, len(src))
        fin = _finals(rng, nq, 0.2)
        if inner_is_output:
            return FST(nq, 0, 64, ninner, src, dst, outer, inner, w, fin, name=name)
        return FST(nq, 0, ninner, 64, src, dst, inner, outer, w, fin, name=name)

    return one(True, "hub.M1"), one(False, "hub.M2")
