"""Power of the oracle's pins: every planted mistake must fail one of them.

Each case copies one oracle module, replaces one line with a plausible
mistake (a dropped term, a wrong sign, index or abscissa, a transposed
order, a quantity summed over the wrong set), and runs the pins of
tests/test_oracle.py against the copy.  The mistake is planted only in that
in-memory copy, on the CPU; the oracle itself is never modified.  A case
passes when some pin fails on the mutant.
"""
import importlib.util
import os
import sys

import pytest

import tests.test_oracle as TO

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (module, original line, planted mistake, what the mistake is)
MUTATIONS = [
    ("tactic", "x1 = (geo.s1 + geo.t1) / 2.0", "x1 = float(geo.s1)",
     "window 1 placed at its first position instead of its middle"),
    ("tactic", "x2 = (geo.s2 + geo.t2) / 2.0", "x2 = float(geo.t2)",
     "window 2 placed at its last position instead of its middle"),
    ("tactic", "mu1 = float(np.mean(np.exp(l_pos[geo.s1 - 1:geo.t1] - m)))",
     "mu1 = float(np.exp(np.mean(l_pos[geo.s1 - 1:geo.t1] - m)))",
     "window 1 mean taken over logits (exp of the mean) instead of over scores"),
    ("tactic", "mu2 = float(np.mean(np.exp(l_pos[geo.s2 - 1:geo.t2] - m)))",
     "mu2 = float(np.exp(np.mean(l_pos[geo.s2 - 1:geo.t2] - m)))",
     "window 2 mean taken over logits"),
    ("tactic", "p_sel = float(s[r.sel[h]].sum())", "p_sel = float(s[r.union].sum())",
     "p(I_h) summed over the group union instead of the head's selection"),
    ("tactic", "cs = np.add.accumulate(s[r.rows[h]])", "cs = np.add.accumulate(np.sort(s)[::-1])",
     "Cluster-Optimal taken along the descending order (= Optimal)"),
    ("tactic", "bound = 2.0 * (1.0 - p_union)", "bound = (1.0 - p_union)",
     "Eq. 6 bound without its factor 2"),
    ("tactic", "eps = float(np.linalg.norm(o - r.out[h]))", "eps = float(np.max(np.abs(o - r.out[h])))",
     "attention distance as max-abs instead of the Euclidean norm (Eq. 4)"),
    ("tactic", "s1 = max(c1 - W // 2, N + 1)", "s1 = max(c1 - W // 2, N)",
     "window 1 allowed to overlap the exact head"),
    ("tactic", "b = mu1 - a / x1", "b = mu1 + a / x1", "wrong sign in the intercept"),
    ("tactic", "order = np.lexsort((np.arange(len(s)), -s))", "order = np.lexsort((np.arange(len(s)), s))",
     "clusters ranked in ascending score"),
    ("tactic", "int(np.argmax(S >= T)) + 1", "int(np.argmax(S > T)) + 1",
     "cutoff needs the sum to exceed the target instead of reaching it"),
    ("tactic", "w = np.concatenate([e, np.maximum(0.0, a / i + b)])", "w = np.concatenate([e, a / i + b])",
     "negative fitted scores not clamped"),
    ("tactic", "N = min(n, max(1, _ceil_div(n * prm.exact_bp, 10000)))",
     "N = min(n, max(1, (n * prm.exact_bp) // 10000))", "exact head rounded down"),
    ("tactic", "idx = union if use_union else np.sort(sels[h])", "idx = np.sort(sels[h])",
     "every head attends over its own selection even with the union"),
    ("tactic", "parts = [np.arange(offsets[c], offsets[c + 1], dtype=np.int64) for c in order]",
     "parts = [np.arange(offsets[c], offsets[c + 1], dtype=np.int64)[::-1] for c in order]",
     "a cluster's tokens unpacked in reverse stored order"),
    ("tactic", "S = E_t + S", "S = S", "recent tokens' mass left out of the cumulative sum"),
    ("tactic", "info[\"S_n\"] = float(S[-1])\n    if P >= 1.0:\n        k = n",
     "info[\"S_n\"] = float(S[-1])\n    if P >= 1.0:\n        k = n - 1", "P = 1 drops the last token"),
    ("attention", "return (K @ q) / np.sqrt(d)", "return (K @ q) / d", "logits scaled by 1/d instead of 1/sqrt(d)"),
    ("attention", "return dense_attention(q, K[idx], V[idx])", "return dense_attention(q, K, V)",
     "subset attention over every token"),
    ("kmeans", "C[nz] = sums[nz] / cnt[nz][:, None]", "C[nz] = sums[nz] / (cnt[nz][:, None] + 1)",
     "centroid mean with an extra count"),
    ("kmeans", "a = np.argmin(D, axis=1).astype(np.int64)", "a = np.argmax(D, axis=1).astype(np.int64)",
     "assignment to the farthest centroid"),
    ("kmeans", "C[m:] = K[init_idx[m:]]", "C[m:] = K[init_idx[m:] - 1]", "initial centroids off by one token"),
    ("kmeans", "perm[fill[c]] = t", "perm[fill[c]] = len(assign) - 1 - t", "layout not in ascending token order"),
    ("tactic", "union = np.unique(np.concatenate(sels))", "union = np.unique(sels[0])",
     "union of the first head's selection only"),
    ("tactic", "sels.append(np.concatenate([rows[:k], tail]))", "sels.append(rows[:k])",
     "recent tokens left out of the selection"),
    ("tactic", "T = P * S[-1]", "T = P * (S[-1] - E_t)", "target taken on the listed tokens' mass only"),
    ("tactic", "k = 0 if (has_tail and E_t >= T) else int(np.argmax(S >= T)) + 1", "k = int(np.argmax(S >= T)) + 1",
     "recent tokens that alone meet the target still take a listed token"),
    ("kmeans", "C = C_prev.copy()", "C = np.zeros_like(C_prev)", "an empty cluster's centroid reset to zero"),
    ("tactic", "t1 = min(s1 + W - 1, n)", "t1 = min(s1 + W, n)", "window 1 one position too long"),
    ("tactic", "W = max(prm.win_min, _ceil_div(n * prm.win_bp, 10000))", "W = _ceil_div(n * prm.win_bp, 10000)",
     "window width without its minimum"),
    ("tactic", "c2 = (n * prm.p2_bp + 5000) // 10000", "c2 = (n * prm.p2_bp) // 10000",
     "window 2 centre truncated instead of rounded"),
    ("tactic", "exact = (N == n) or (s1 > t1) or (s2 > t2) or (t1 >= s2)", "exact = (N == n) or (s1 > t1) or (s2 > t2)",
     "overlapping windows not sent to exact mode"),
]

# which module object of tests/test_oracle.py each oracle module replaces
_ATTR = {"tactic": "T", "attention": "A", "kmeans": "KM"}


def _mutant(module: str, old: str, new: str):
    path = os.path.join(ROOT, "oracle", module + ".py")
    with open(path) as f:
        src = f.read()
    assert src.count(old) == 1, f"mutation anchor not found once in oracle/{module}.py: {old!r}"
    name = f"oracle._mutant_{module}"
    spec = importlib.util.spec_from_loader(name, loader=None)
    mod = importlib.util.module_from_spec(spec)
    mod.__package__ = "oracle"  # its relative imports resolve to the real oracle modules
    sys.modules[name] = mod     # dataclasses look their module up while the class is built
    try:
        exec(compile(src.replace(old, new), f"{path} (mutant)", "exec"), mod.__dict__)
    finally:
        del sys.modules[name]
    return mod


def _pins():
    """Every test of tests/test_oracle.py as a no-argument call, one per
    parameter set of a parametrized test."""
    calls = []
    for name in sorted(dir(TO)):
        fn = getattr(TO, name)
        if not name.startswith("test_") or not callable(fn):
            continue
        marks = [m for m in getattr(fn, "pytestmark", []) if m.name == "parametrize"]
        if not marks:
            calls.append((name, fn))
            continue
        assert len(marks) == 1, name
        argnames, argvalues = marks[0].args[0], marks[0].args[1]
        names = [a.strip() for a in argnames.split(",")] if isinstance(argnames, str) else list(argnames)
        for vals in argvalues:
            vals = vals if len(names) > 1 else (vals,)
            calls.append((name, lambda fn=fn, kw=dict(zip(names, vals)): fn(**kw)))
    return calls


@pytest.mark.parametrize("module,old,new,what", MUTATIONS, ids=[m[3] for m in MUTATIONS])
def test_planted_mistake_fails_a_pin(module, old, new, what):
    attr = _ATTR[module]
    real = getattr(TO, attr)
    setattr(TO, attr, _mutant(module, old, new))
    failed = []
    try:
        for name, pin in _pins():
            try:
                pin()
            except Exception as e:  # an assertion, or arithmetic the mistake broke
                failed.append((name, type(e).__name__))
                break
    finally:
        setattr(TO, attr, real)
    assert failed, f"no pin fails with the planted mistake: {what}"


def test_unmutated_oracle_passes_every_pin():
    """Control: the same harness with the anchors replaced by themselves."""
    for module, old, _, _ in MUTATIONS[:1] + MUTATIONS[18:19] + MUTATIONS[20:21]:
        attr = _ATTR[module]
        real = getattr(TO, attr)
        setattr(TO, attr, _mutant(module, old, old))
        try:
            for _, pin in _pins():
                pin()
        finally:
            setattr(TO, attr, real)
