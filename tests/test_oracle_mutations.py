"""The oracle's pins catch plausible mistakes (CPU only).

Each case plants one mistake in a copy of an oracle module's source (a
dropped term, a wrong sign, index, operand or constant), loads the copy as
a module of its own, and runs the pin tests of that module against it with
the oracle swapped for the copy.  The case passes when at least one pin
fails.  The oracle on disk is never modified; nothing here runs on a GPU.
"""

import importlib
import inspect
import itertools
import os
import sys
import types

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

NS = "oracle/muonbp_oracle.py"
SC = "oracle/scalar_oracle.py"

# (file, what the mistake is, text in the file, text it becomes)
MUTANTS = [
    # Algorithm 2 (Orthogonalize-via-NS)
    (NS, "quintic term dropped", "gram @ (b * eye + c * gram)", "gram @ (b * eye)"),
    (NS, "cubic term sign", "gram @ (b * eye + c * gram)", "gram @ (-b * eye + c * gram)"),
    (NS, "linear term dropped", "q = a * eye + gram", "q = gram"),
    (NS, "Gram of the wrong side", "gram = X @ X.T", "gram = X.T @ X"),
    (NS, "spectral instead of Frobenius norm", 'np.linalg.norm(G, "fro") + eps',
     "np.linalg.norm(G, 2) + eps"),
    (NS, "no normalisation", 'X = G / (np.linalg.norm(G, "fro") + eps)', "X = G.copy()"),
    (NS, "one iteration short", "for a, b, c in table:", "for a, b, c in table[1:]:"),
    (NS, "quintic constant b", "NS_A, NS_B, NS_C = 2.0, -1.5, 0.5", "NS_A, NS_B, NS_C = 2.0, -1.25, 0.5"),
    (NS, "coefficient table off by one", "arr[min(k, arr.shape[0] - 1)]", "arr[min(k + 1, arr.shape[0] - 1)]"),
    (NS, "tall result not transposed back", "return X.T.copy() if transposed else X",
     "return X"),
    # Algorithm 1 (MuonBP step)
    (NS, "full step on t mod P = 1", "return period > 0 and t % period == 0",
     "return period > 0 and t % period == 1"),
    (NS, "P = infinity treated as P = 1", "return period > 0 and t % period == 0",
     "return period == 0 or t % period == 0"),
    (NS, "block rows and columns swapped",
     "return [(slice(i * mb, (i + 1) * mb), slice(j * nb, (j + 1) * nb))",
     "return [(slice(j * nb, (j + 1) * nb), slice(i * mb, (i + 1) * mb))"),
    (NS, "momentum as an EMA of the gradient", "return mu * np.asarray(M, dtype=np.float64) + np.asarray(G",
     "return mu * np.asarray(M, dtype=np.float64) + (1 - mu) * np.asarray(G"),
    (NS, "Nesterov input mixed the wrong way", "Y = G + cfg.momentum * self.M[k] if cfg.nesterov",
     "Y = self.M[k] + cfg.momentum * G if cfg.nesterov"),
    (NS, "block and full learning rates swapped", "eta = cfg.lr_full if full else cfg.lr_block",
     "eta = cfg.lr_block if full else cfg.lr_full"),
    (NS, "weight decay not scaled by the learning rate",
     "out.append(X - eta * (cfg.weight_decay * X + U))",
     "out.append(X - cfg.weight_decay * X - eta * U)"),
    (NS, "update sign", "out.append(X - eta * (cfg.weight_decay * X + U))",
     "out.append(X - eta * (cfg.weight_decay * X - U))"),
    (NS, "block step orthogonalizes the whole matrix",
     "U = orthogonalize_blockwise(Y, (spec.grid_rows, spec.grid_cols), **ns)",
     "U = orthogonalize_via_ns(Y, **ns)"),
    (NS, "RMS scale from the smaller side", "return beta * math.sqrt(max(p, q))",
     "return beta * math.sqrt(min(p, q))"),
    (NS, "cost model with S and L swapped", "return 2.0 * K * (2.0 * l * s * s + s ** 3)",
     "return 2.0 * K * (2.0 * s * l * l + s ** 3)"),
    # Scalar optimizer and schedules
    (SC, "AdamW without bias correction of m", "p = p - lr * (mi / bc1) / (np.sqrt(vi / bc2) + eps)",
     "p = p - lr * mi / (np.sqrt(vi / bc2) + eps)"),
    (SC, "AdamW eps inside the square root", "p = p - lr * (mi / bc1) / (np.sqrt(vi / bc2) + eps)",
     "p = p - lr * (mi / bc1) / np.sqrt(vi / bc2 + eps)"),
    (SC, "AdamW decay applied after the step", "p = p * (1.0 - lr * weight_decay)\n        p = p - lr * (mi / bc1)",
     "p = p - lr * (mi / bc1)"),
    (SC, "clipping never clips", "return min(1.0, max_norm / (global_norm(grads) + CLIP_EPS))",
     "return 1.0"),
    (SC, "clipping by the largest tensor norm",
     "return math.sqrt(sum(float(np.sum(np.asarray(g, dtype=np.float64) ** 2)) for g in grads))",
     "return max(math.sqrt(float(np.sum(np.asarray(g, dtype=np.float64) ** 2))) for g in grads)"),
    (SC, "Lion direction from beta2", "direction = np.sign(beta1 * mi + (1.0 - beta1) * g)",
     "direction = np.sign(beta2 * mi + (1.0 - beta2) * g)"),
    (SC, "Lion momentum from beta1", "out_m.append(beta2 * mi + (1.0 - beta2) * g)",
     "out_m.append(beta1 * mi + (1.0 - beta1) * g)"),
    (SC, "Lion without decoupled decay", "out_p.append(p * (1.0 - lr * weight_decay) - lr * direction)",
     "out_p.append(p - lr * direction)"),
    (SC, "cosine with sine", "0.5 * (1.0 + math.cos(math.pi * x))", "0.5 * (1.0 + math.sin(math.pi * x))"),
    (SC, "WSD decay spread over one step too many", "((t - (total - decay)) / decay)",
     "((t - (total - decay)) / (decay + 1))"),
    (SC, "warmup off by one", "    if t < warmup:\n        return lr_max * (t + 1) / warmup\n    span",
     "    if t < warmup:\n        return lr_max * t / warmup\n    span"),
]

# Pin modules of each oracle file and the name they import it under.
PINS = {NS: ("tests.test_oracle", "O"), SC: ("tests.test_oracle_scalar", "S")}


def _load_source(path, src, name):
    """Module from source text (registered while it runs: its dataclasses
    look their module up by name)."""
    mod = types.ModuleType(name)
    mod.__file__ = os.path.join(ROOT, path)
    sys.modules[name] = mod
    try:
        exec(compile(src, mod.__file__, "exec"), mod.__dict__)
    finally:
        del sys.modules[name]
    return mod


def _load_mutant(path, old, new):
    with open(os.path.join(ROOT, path)) as fh:
        src = fh.read()
    assert src.count(old) == 1, f"mutation site not unique in {path}: {old!r}"
    return _load_source(path, src.replace(old, new), "oracle_mutant")


def _cases(fn):
    """Keyword sets of a pin function from its parametrize marks (None when
    it needs a fixture)."""
    marks = [m for m in getattr(fn, "pytestmark", []) if m.name == "parametrize"]
    axes = []
    for m in marks:
        names = [n.strip() for n in m.args[0].split(",")] if isinstance(m.args[0], str) else list(m.args[0])
        vals = []
        for v in m.args[1]:
            v = v.values if hasattr(v, "values") else v
            vals.append(dict(zip(names, v if len(names) > 1 else (v,))))
        axes.append(vals)
    params = set(inspect.signature(fn).parameters)
    covered = set().union(*[set(a[0]) for a in axes]) if axes else set()
    if params - covered:
        return None
    return [dict(kv for d in combo for kv in d.items()) for combo in itertools.product(*axes)]


def _first_failing_pin(pins, attr, mutant):
    real = getattr(pins, attr)
    setattr(pins, attr, mutant)
    try:
        for name, fn in inspect.getmembers(pins, inspect.isfunction):
            if not name.startswith("test_") or fn.__module__ != pins.__name__:
                continue
            cases = _cases(fn)
            if cases is None:
                continue
            for kw in cases:
                try:
                    fn(**kw)
                except Exception:  # a failing assertion, or the mutant breaking outright
                    return f"{name}{kw or ''}"
        return None
    finally:
        setattr(pins, attr, real)


@pytest.mark.parametrize("path,what,old,new", MUTANTS, ids=[m[1] for m in MUTANTS])
def test_pins_catch_planted_mistake(path, what, old, new):
    mutant = _load_mutant(path, old, new)
    pins = importlib.import_module(PINS[path][0])
    caught = _first_failing_pin(pins, PINS[path][1], mutant)
    assert caught is not None, f"no pin fails with the mistake '{what}' planted in {path}"


def test_unmutated_oracle_passes_every_pin():
    """The harness itself: with the oracle's own source loaded the same way,
    no pin fails (so a failure above is the planted mistake's)."""
    for path, (mod, attr) in PINS.items():
        with open(os.path.join(ROOT, path)) as fh:
            clean = _load_source(path, fh.read(), "oracle_clean")
        assert _first_failing_pin(importlib.import_module(mod), attr, clean) is None, path
