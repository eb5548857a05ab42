"""Test-side checkers for composed transducers.

Nothing here is part of the oracle or of the HIP path: these are the
independent pins the oracle is checked against (brute force, path sums,
accessible part of a single transducer) and the canonical comparison used to
compare any two composition results.

A composition result, from either side, is described by
  q1, q2, final  -- per state id: its pair and accept flag
  src, dst, a, c, w -- per arc: source id, target id, input symbol, output
                       symbol, weight
"""
from __future__ import annotations

from collections import defaultdict, deque
from dataclasses import dataclass

import numpy as np


@dataclass
class Canon:
    """Result with state ids replaced by their (q1, q2) pairs, sorted."""

    states: np.ndarray   # (n, 2) uint64 rows (q1, q2), lexicographically sorted
    finals: np.ndarray   # (n,) accept flag aligned with ``states``
    keys: np.ndarray     # (m, 6) rows (src q1, src q2, dst q1, dst q2, a, c), sorted
    w: np.ndarray        # (m,) float32 weights aligned with ``keys``


def canon(q1, q2, final, src, dst, a, c, w) -> Canon:
    q1 = np.asarray(q1, np.uint64); q2 = np.asarray(q2, np.uint64)
    final = np.asarray(final).astype(np.uint8)
    src = np.asarray(src, np.int64); dst = np.asarray(dst, np.int64)
    st = np.stack([q1, q2], axis=1)
    order = np.lexsort((q2, q1))
    states = st[order]
    finals = final[order]
    keys = np.stack([q1[src], q2[src], q1[dst], q2[dst],
                     np.asarray(a, np.uint64), np.asarray(c, np.uint64)], axis=1)
    korder = np.lexsort(keys.T[::-1])
    return Canon(states, finals, keys[korder], np.asarray(w, np.float32)[korder])


def canon_of(res) -> Canon:
    """Canonical form of any object exposing q1, q2, final, src, dst, a, c, w."""
    return canon(res.q1, res.q2, res.final, res.src, res.dst, res.a, res.c, res.w)


def canon_eps(res) -> Canon:
    """Canonical form of a composition with epsilon transitions, whose states
    are triples (q1, q2, f): the pair column q2 carries 3 q2 + f."""
    q2f = np.asarray(res.q2, np.uint64) * 3 + np.asarray(res.f, np.uint64)
    return canon(res.q1, q2f, res.final, res.src, res.dst, res.a, res.c, res.w)


def unique_rows(x: np.ndarray) -> bool:
    if len(x) < 2:
        return True
    return bool(np.any(x[1:] != x[:-1], axis=1).all())


def assert_same(got: Canon, ref: Canon, rtol: float = 1e-5, what: str = ""):
    """Bit-exact states, accept flags and arc keys; weights within rtol."""
    assert unique_rows(got.states), f"{what}: duplicate states"
    assert unique_rows(got.keys), f"{what}: duplicate arc keys (unmerged arcs)"
    assert got.states.shape == ref.states.shape, \
        f"{what}: {len(got.states)} states vs {len(ref.states)}"
    assert np.array_equal(got.states, ref.states), f"{what}: state sets differ"
    assert np.array_equal(got.finals, ref.finals), f"{what}: accept flags differ"
    assert got.keys.shape == ref.keys.shape, f"{what}: {len(got.keys)} arcs vs {len(ref.keys)}"
    assert np.array_equal(got.keys, ref.keys), f"{what}: arc key sets differ"
    bad = ~weights_close(got.w, ref.w, rtol)
    if bad.any():
        i = int(np.argmax(bad))
        raise AssertionError(f"{what}: {int(bad.sum())} weights off, e.g. key {ref.keys[i]} "
                             f"got {float(got.w[i])!r} ref {float(ref.w[i])!r}")


def weights_close(got, ref, rtol, atol=0.0):
    """Per element: a NaN reference needs a NaN, an infinite reference the
    same infinity (sign included), a finite reference a finite weight within
    rtol * |ref| + atol of it.  rtol = inf leaves finite weights unchecked but
    still requires the NaN and infinity pattern to agree."""
    gw = np.asarray(got, np.float64)
    rw = np.asarray(ref, np.float64)
    gn, rn = np.isnan(gw), np.isnan(rw)
    gi, ri = np.isinf(gw), np.isinf(rw)
    ok = (gn == rn) & (gi == ri)
    ok &= ~ri | (gw == rw)
    fin = ~(rn | ri)
    if np.isinf(rtol):
        ok &= ~fin | np.isfinite(gw)
    else:
        with np.errstate(invalid="ignore"):
            within = np.abs(gw - rw) <= rtol * np.abs(rw) + atol
        ok &= ~fin | within
    return ok


# ---------------------------------------------------------------------------
# Pins independent of the oracle's structure
# ---------------------------------------------------------------------------

@dataclass
class Plain:
    q1: np.ndarray
    q2: np.ndarray
    final: np.ndarray
    src: np.ndarray
    dst: np.ndarray
    a: np.ndarray
    c: np.ndarray
    w: np.ndarray


def brute_force(m1, m2, max_levels: int = 0) -> Plain:
    """Naive composition over all of Q1 x Q2, then trimmed to reachable pairs.

    Every M1 arc is joined with every M2 arc that reads its output symbol
    (all-pairs, §2 / §3.1), identical (src, dst, in, out) arcs are summed, and
    a textbook BFS on the pair graph from (s1, s2) keeps the reachable pairs
    (at depth <= max_levels when capped) and the arcs of pairs that are
    expanded (depth < max_levels when capped).
    """
    by_in = defaultdict(list)
    for e2 in range(m2.num_arcs):
        by_in[int(m2.ilabel[e2])].append(e2)
    acc: dict[tuple, float] = {}
    for e1 in range(m1.num_arcs):
        for e2 in by_in.get(int(m1.olabel[e1]), ()):
            key = (int(m1.src[e1]), int(m2.src[e2]), int(m1.dst[e1]), int(m2.dst[e2]),
                   int(m1.ilabel[e1]), int(m2.olabel[e2]))
            p = np.float32(m1.weight[e1]) * np.float32(m2.weight[e2])
            acc[key] = acc.get(key, 0.0) + float(p)
    succ = defaultdict(set)
    for k in acc:
        succ[(k[0], k[1])].add((k[2], k[3]))
    s = (int(m1.start), int(m2.start))
    depth = {s: 0}
    dq = deque([s])
    while dq:
        u = dq.popleft()
        if max_levels and depth[u] >= max_levels:
            continue
        for v in sorted(succ.get(u, ())):
            if v not in depth:
                depth[v] = depth[u] + 1
                dq.append(v)
    states = sorted(depth)
    sid = {p: i for i, p in enumerate(states)}
    expanded = {p for p, d in depth.items() if not max_levels or d < max_levels}
    arcs = [(k, v) for k, v in acc.items() if (k[0], k[1]) in expanded]
    q1 = np.array([p[0] for p in states], np.uint32)
    q2 = np.array([p[1] for p in states], np.uint32)
    fin = np.array([int(m1.final[p[0]] and m2.final[p[1]]) for p in states], np.uint8)
    src = np.array([sid[(k[0], k[1])] for k, _ in arcs], np.int64)
    dst = np.array([sid[(k[2], k[3])] for k, _ in arcs], np.int64)
    a = np.array([k[4] for k, _ in arcs], np.uint32)
    c = np.array([k[5] for k, _ in arcs], np.uint32)
    w = np.array([v for _, v in arcs], np.float64).astype(np.float32)
    return Plain(q1, q2, fin, src, dst, a, c, w)


def accessible(m) -> list[int]:
    """States of a single transducer reachable from its start (BFS)."""
    succ = defaultdict(set)
    for e in range(m.num_arcs):
        succ[int(m.src[e])].add(int(m.dst[e]))
    seen = {int(m.start)}
    dq = deque([int(m.start)])
    while dq:
        u = dq.popleft()
        for v in succ.get(u, ()):
            if v not in seen:
                seen.add(v)
                dq.append(v)
    return sorted(seen)


def label_matrices(num_states, start, nin, nout, src, dst, a, c, w):
    """T[x, y] = num_states x num_states matrix of summed weights of arcs x:y (fp64)."""
    T = np.zeros((nin, nout, num_states, num_states), np.float64)
    np.add.at(T, (np.asarray(a, np.int64), np.asarray(c, np.int64),
                  np.asarray(src, np.int64), np.asarray(dst, np.int64)),
              np.asarray(w, np.float64))
    return T


def path_weights(T, start, end_vec, length):
    """W[x_1..x_l, y_1..y_l] = sum over paths from start with those labels of
    the product of arc weights, ending with weight end_vec[q] at state q.
    Returned as an array indexed by flattened label tuples (x, y)."""
    nin, nout, n, _ = T.shape
    # v[x-seq, y-seq, state], built one step at a time.
    v = np.zeros((1, 1, n))
    v[0, 0, start] = 1.0
    for _ in range(length):
        # v'[X*nin + x, Y*nout + y, r] = sum_q v[X, Y, q] T[x, y, q, r]
        nv = np.einsum("XYq,xyqr->XxYyr", v, T)
        v = nv.reshape(v.shape[0] * nin, v.shape[1] * nout, n)
    return v @ end_vec


# ---------------------------------------------------------------------------
# Composition without reduction (every joined arc pair is an arc)
# ---------------------------------------------------------------------------

def brute_force_unreduced(m1, m2, max_levels: int = 0) -> Plain:
    """All-pairs join over Q1 x Q2 without merging identical arcs, trimmed to
    the arcs of reachable, expanded pairs (textbook BFS on the pair graph).
    Each arc keeps its own float32 product."""
    by_in = defaultdict(list)
    for e2 in range(m2.num_arcs):
        by_in[int(m2.ilabel[e2])].append(e2)
    joined = []
    for e1 in range(m1.num_arcs):
        for e2 in by_in.get(int(m1.olabel[e1]), ()):
            joined.append(((int(m1.src[e1]), int(m2.src[e2])), (int(m1.dst[e1]), int(m2.dst[e2])),
                           int(m1.ilabel[e1]), int(m2.olabel[e2]),
                           np.float32(m1.weight[e1]) * np.float32(m2.weight[e2])))
    succ = defaultdict(set)
    for u, v, _, _, _ in joined:
        succ[u].add(v)
    s = (int(m1.start), int(m2.start))
    depth = {s: 0}
    dq = deque([s])
    while dq:
        u = dq.popleft()
        if max_levels and depth[u] >= max_levels:
            continue
        for v in sorted(succ.get(u, ())):
            if v not in depth:
                depth[v] = depth[u] + 1
                dq.append(v)
    states = sorted(depth)
    sid = {p: i for i, p in enumerate(states)}
    expanded = {p for p, d in depth.items() if not max_levels or d < max_levels}
    arcs = [j for j in joined if j[0] in expanded]
    q1 = np.array([p[0] for p in states], np.uint32)
    q2 = np.array([p[1] for p in states], np.uint32)
    fin = np.array([int(m1.final[p[0]] and m2.final[p[1]]) for p in states], np.uint8)
    return Plain(q1, q2, fin, np.array([sid[j[0]] for j in arcs], np.int64),
                 np.array([sid[j[1]] for j in arcs], np.int64),
                 np.array([j[2] for j in arcs], np.uint32), np.array([j[3] for j in arcs], np.uint32),
                 np.array([j[4] for j in arcs], np.float32))


@dataclass
class Multiset:
    states: np.ndarray   # [n, 2] sorted (q1, q2)
    finals: np.ndarray   # accept flag per sorted state
    rows: np.ndarray     # [m, 7] sorted (src q1, src q2, dst q1, dst q2, a, c, weight bits)


def multiset_of(res) -> Multiset:
    """Canonical form of a result whose arcs are a multiset: state ids replaced
    by their pairs, arcs (with their weight bits) in sorted order."""
    q1 = np.asarray(res.q1, np.int64)
    q2 = np.asarray(res.q2, np.int64)
    order = np.lexsort((q2, q1))
    states = np.stack([q1[order], q2[order]], 1)
    finals = np.asarray(res.final, np.uint8)[order]
    src = np.asarray(res.src, np.int64)
    dst = np.asarray(res.dst, np.int64)
    wbits = np.asarray(res.w, np.float32).view(np.uint32).astype(np.int64)
    rows = np.stack([q1[src], q2[src], q1[dst], q2[dst], np.asarray(res.a, np.int64),
                     np.asarray(res.c, np.int64), wbits], 1) if len(src) else np.zeros((0, 7), np.int64)
    rows = rows[np.lexsort(rows.T[::-1])] if len(rows) else rows
    return Multiset(states, finals, rows)


def multiset_eps(res) -> Multiset:
    """multiset_of for a composition with epsilon transitions (3 q2 + f in the
    q2 column)."""
    class _R:
        pass
    r = _R()
    r.q1, r.final, r.src, r.dst, r.a, r.c, r.w = res.q1, res.final, res.src, res.dst, res.a, res.c, res.w
    r.q2 = np.asarray(res.q2, np.int64) * 3 + np.asarray(res.f, np.int64)
    return multiset_of(r)


def assert_same_multiset(got: Multiset, ref: Multiset, what: str = ""):
    """Identical states, accept flags and arc multisets, weights bit for bit
    (each weight is one float32 product on both sides)."""
    assert np.array_equal(got.states, ref.states), f"{what}: state sets differ"
    assert np.array_equal(got.finals, ref.finals), f"{what}: accept flags differ"
    assert got.rows.shape == ref.rows.shape, f"{what}: {len(got.rows)} arcs vs {len(ref.rows)}"
    if not np.array_equal(got.rows, ref.rows):
        i = int(np.argmax(np.any(got.rows != ref.rows, axis=1)))
        raise AssertionError(f"{what}: arc multisets differ, first at sorted row {i}: "
                             f"{got.rows[i]} vs {ref.rows[i]}")


# ---------------------------------------------------------------------------
# Per-source expansion (no search): brute force over the arcs of two states
# ---------------------------------------------------------------------------

def brute_force_sources(m1, m2, q1s, q2s):
    """Merged out-arcs of each source pair (q1s[i], q2s[i]) on its own, from
    every pair of arcs leaving q1s[i] in M1 and q2s[i] in M2 that share the
    inner symbol (§2 arc rule), identical (target pair, a, c) summed in
    float64 over float32 products.  Numpy only.

    Returns (rows, w, joined): rows [k, 7] int64 (batch index, src q1, src q2,
    dst q1, dst q2, a, c) sorted, their weights (float32) and the number of
    arc pairs joined per source."""
    o1 = np.argsort(m1.src, kind="stable"); o2 = np.argsort(m2.src, kind="stable")
    b1 = np.searchsorted(m1.src[o1], np.arange(m1.num_states + 1))
    b2 = np.searchsorted(m2.src[o2], np.arange(m2.num_states + 1))
    rows, ws, joined = [], [], []
    for i, (q1, q2) in enumerate(zip(np.asarray(q1s, np.int64), np.asarray(q2s, np.int64))):
        e1 = o1[b1[q1]:b1[q1 + 1]]
        e2 = o2[b2[q2]:b2[q2 + 1]]
        hit = m1.olabel[e1][:, None] == m2.ilabel[e2][None, :]
        i1, i2 = np.nonzero(hit)
        e1, e2 = e1[i1], e2[i2]
        joined.append(len(e1))
        if not len(e1):
            continue
        key = np.stack([m1.dst[e1], m2.dst[e2], m1.ilabel[e1], m2.olabel[e2]], 1).astype(np.int64)
        prod = (m1.weight[e1] * m2.weight[e2]).astype(np.float32)
        uk, inv = np.unique(key, axis=0, return_inverse=True)
        acc = np.zeros(len(uk), np.float64)
        np.add.at(acc, inv.ravel(), prod.astype(np.float64))
        head = np.tile(np.array([i, q1, q2], np.int64), (len(uk), 1))
        rows.append(np.concatenate([head, uk], 1))
        ws.append(acc.astype(np.float32))
    if not rows:
        return np.zeros((0, 7), np.int64), np.zeros(0, np.float32), np.array(joined, np.int64)
    rows = np.concatenate(rows); w = np.concatenate(ws)
    order = np.lexsort(rows.T[::-1])
    return rows[order], w[order], np.array(joined, np.int64)


def source_rows(res, q1s, q2s):
    """Rows (batch index, src q1, src q2, dst q1, dst q2, a, c) of a per-source
    expansion result whose states 0..n-1 are the batch's sources, sorted,
    with their weights."""
    q1s = np.asarray(q1s, np.int64); q2s = np.asarray(q2s, np.int64)
    src = np.asarray(res.src, np.int64); dst = np.asarray(res.dst, np.int64)
    rows = np.stack([src, q1s[src], q2s[src], np.asarray(res.q1, np.int64)[dst],
                     np.asarray(res.q2, np.int64)[dst], np.asarray(res.a, np.int64),
                     np.asarray(res.c, np.int64)], 1) if len(src) else np.zeros((0, 7), np.int64)
    order = np.lexsort(rows.T[::-1]) if len(rows) else np.zeros(0, np.int64)
    return rows[order], np.asarray(res.w, np.float32)[order]
