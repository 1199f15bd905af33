"""Tie-aware comparison of Algorithm 1's discrete decisions (Sec. III-C)
between the library and the oracle.

The library and the oracle evaluate the same quantities in different orders
(the library's average linkage is a size-weighted update of cluster
distances, the oracle's a mean over member pairs; the greedy cost is
sigma^2 * h / h_i on one side and sigma^2 / (h_i / h) on the other), so two
candidates that are equal in exact arithmetic can be ordered differently by
rounding.  The rule applied here:

  * at every decision, the library's choice must be the oracle's best, or a
    candidate whose oracle key lies within a relative MARGIN of the oracle's
    best key (a near-tie);
  * outside near-ties the choices must be identical, so a path with no
    near-tie deviation must end at exactly the oracle's result.

MARGIN = 1e-12 is far above the rounding of either evaluation order (a few
ulps of quantities of order one, ~1e-15) and far below any real gap between
candidates of the random and planted inputs used in the tests.
"""

from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

import numpy as np

from oracle import compress as oc

MARGIN = 1e-12


def _near(x: float, best: float, margin: float) -> bool:
    return x <= best + margin * max(1.0, abs(best))


def check_merges(S: np.ndarray, merges: Sequence[Tuple[int, int, float]],
                 margin: float = MARGIN) -> int:
    """Replay the library's merge sequence against the oracle's linkage.

    Each merge must join the oracle's closest pair of the current clusters,
    or a pair within the margin of it; its reported height must equal the
    oracle's distance of that pair to the margin.  Returns the index of the
    first merge that took a near-tie alternative (len(merges) if none), so
    that every cut before it must equal the oracle's clustering exactly."""
    h = S.shape[0]
    D = 1.0 - np.asarray(S, dtype=np.float64)
    clusters: Dict[int, List[int]] = {i: [i] for i in range(h)}
    first_dev = len(merges)
    for s, (a, b, height) in enumerate(merges):
        assert a in clusters and b in clusters and a < b, (s, a, b)
        names = sorted(clusters)
        best = None
        for i, x in enumerate(names):
            for y in names[i + 1:]:
                key = (oc.linkage_distance(D, clusters[x], clusters[y]), x, y)
                if best is None or key < best:
                    best = key
        d_lib = oc.linkage_distance(D, clusters[a], clusters[b])
        assert abs(height - d_lib) <= margin * max(1.0, abs(d_lib)), (s, height, d_lib)
        if (a, b) != best[1:]:
            assert _near(d_lib, best[0], margin), (
                f"merge {s}: library joined {a},{b} at {d_lib!r}; oracle's best "
                f"{best[1]},{best[2]} at {best[0]!r} is not a near-tie")
            first_dev = min(first_dev, s)
        clusters[a] = sorted(clusters[a] + clusters.pop(b))
    return first_dev


def cut(merges: Sequence[Tuple[int, int, float]], h: int, K: int) -> List[int]:
    """Group id of each head after the first h - K merges (groups numbered by
    their smallest head)."""
    root = list(range(h))
    for a, b, _ in merges[:h - K]:
        root = [a if x == b else x for x in root]
    names = sorted(set(root))
    return [names.index(x) for x in root]


def greedy_reachable(init: Sequence[int], sigmas: Sequence[np.ndarray], heads: Sequence[int],
                     r: int, target: Sequence[int], margin: float = MARGIN) -> Tuple[bool, bool]:
    """Whether the oracle's greedy budget step, allowed to take any near-tie
    alternative, can end at `target` from `init`.  Returns (reachable, the
    oracle's own greedy_adjust result equals target)."""
    h = sum(heads)
    target = tuple(target)
    seen = set()

    def done(rk):
        return oc.budget_holds(rk, heads, r) and sum(rk) <= r

    def walk(rk: Tuple[int, ...]) -> bool:
        if rk in seen:
            return False
        seen.add(rk)
        if done(rk):
            return rk == target
        costs = [(oc.greedy_cost(sigmas[i], rk[i], heads[i], h), i) for i in range(len(rk)) if rk[i] > 1]
        if not costs:
            return rk == target
        best = min(costs)
        for c, i in sorted(costs):
            if (c, i) != best and not _near(c, best[0], margin):
                break
            nxt = list(rk)
            nxt[i] -= 1
            if walk(tuple(nxt)):
                return True
        return False

    exact = tuple(oc.greedy_adjust(list(init), sigmas, heads, r)) == target
    return (exact or walk(tuple(init))), exact


def init_ranks_agree(lib_init: Sequence[int], energies: Sequence[float], energy_total: float,
                     caps: Sequence[int], r: int, margin: float = MARGIN) -> bool:
    """The energy rule round(r E_i / E) (half up, clipped to [1, cap_i]),
    allowing either neighbour where r E_i / E lies within the margin of a
    rounding boundary."""
    for got, e, cap in zip(lib_init, energies, caps):
        x = r * e / energy_total
        opts = {int(np.floor(x + 0.5))}
        frac = x + 0.5 - np.floor(x + 0.5)
        if frac < margin * max(1.0, x):
            opts.add(int(np.floor(x + 0.5)) - 1)
        if 1.0 - frac < margin * max(1.0, x):
            opts.add(int(np.floor(x + 0.5)) + 1)
        if got not in {max(1, min(o, cap)) for o in opts}:
            return False
    return True
