"""The oracle's pins must reject a wrong oracle: each plausible mistake below is planted in a
copy of the C oracle (compiled here, on the CPU), the copy is swapped in, and the pins that
check the recurrence against the paper and the mathematics are run against it.  Every
mutation has to fail several of them; the real oracle passes them all (test_oracle_pins.py)."""
import os
import subprocess
import sys

import pytest

import oracle

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import test_oracle_pins as pins  # noqa: E402

SRC = os.path.join(os.path.dirname(oracle.__file__), "gdn_oracle.c")
UPDATE = "row[c] = a * (row[c] - b * sk * kt[c]) + b * vt * kt[c];"
MUTATIONS = {
    "decay applied after the write": (UPDATE, "row[c] = a * (row[c] - b * sk * kt[c] + b * vt * kt[c]);"),
    "erase term with the wrong sign": (UPDATE, "row[c] = a * (row[c] + b * sk * kt[c]) + b * vt * kt[c];"),
    "write without beta": (UPDATE, "row[c] = a * (row[c] - b * sk * kt[c]) + vt * kt[c];"),
    "half the log-decay": ("const double  a  = exp(g[t * H + h]);", "const double  a  = exp(0.5 * g[t * H + h]);"),
    "output read with the key": ("oj += row[c] * (scale * qt[c]);", "oj += row[c] * (scale * kt[c]);"),
}
PINS = [
    (pins.test_golden_handworked_example, ()),
    (pins.test_brute_force_exact_rationals, (1,)),
    (pins.test_beta_zero_is_pure_decay, ()),
    (pins.test_alpha_one_beta_one_orthonormal_keys_write_columns, ()),
    (pins.test_alpha_one_matches_lms_update, ()),
    (pins.test_alpha_to_zero_forgets_everything, ()),
    (pins.test_spectral_norm_bound, ()),
    (pins.test_retrieval_identity_per_step, ()),
    (pins.test_chunked_equals_sequential_every_chunk_size, (7,)),
    (pins.test_chunked_ragged_and_fast_decay, ()),
]


def _build(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, name
    path = tmp_path / ("mut_%d.c" % abs(hash(name)))
    path.write_text(src.replace(old, new))
    so = str(path) + ".so"
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", str(path), "-o", so, "-lm"])
    return so


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_reject_a_planted_mistake(tmp_path, monkeypatch, name):
    import ctypes
    so = _build(tmp_path, name, *MUTATIONS[name])
    real = oracle._load()
    lib = ctypes.CDLL(so)
    lib.oracle_gdn_recurrence.argtypes = real.oracle_gdn_recurrence.argtypes
    lib.oracle_gdn_recurrence.restype = real.oracle_gdn_recurrence.restype
    lib.oracle_max_threads.restype = ctypes.c_int
    monkeypatch.setattr(oracle, "_lib", lib)
    failed = []
    for fn, args in PINS:
        try:
            fn(*args)
        except AssertionError:
            failed.append(fn.__name__)
    print("%s: %d of %d pins fail" % (name, len(failed), len(PINS)))
    assert len(failed) >= 3, (name, failed)


def test_the_real_oracle_passes_the_same_pins():
    for fn, args in PINS:
        fn(*args)


# --------------------------------------------------------------------------- the attention oracle
from oracle import attention as att  # noqa: E402

ATT_MUTATIONS = {
    "mask keeps the next key": ("np.arange(T)[None, :] > idx[:, None]", "np.arange(T)[None, :] > idx[:, None] + 1"),
    "mask drops the own key": ("np.arange(T)[None, :] > idx[:, None]", "np.arange(T)[None, :] >= idx[:, None]"),
    "scale left out": ("s = scale * (q[b, idx, h] @ k[b, :, kh].T)", "s = (q[b, idx, h] @ k[b, :, kh].T)"),
    "query heads mapped round-robin": ("kh = h // (H // Hkv)", "kh = h % Hkv"),
    "softmax over the queries": ("s -= s.max(axis=1, keepdims=True)\n            p = np.exp(s)\n            p /= p.sum(axis=1, keepdims=True)",
                                 "s -= s.max(axis=1, keepdims=True)\n            p = np.exp(s)\n            p /= p.sum(axis=0, keepdims=True)"),
}
ATT_PINS = [
    (pins.test_attention_brute_force, (4, 2)),
    (pins.test_attention_brute_force, (2, 1)),
    (pins.test_attention_closed_forms, ()),
    (pins.test_attention_invariances_and_sampled_rows, ()),
]


@pytest.mark.parametrize("name", sorted(ATT_MUTATIONS))
def test_attention_pins_reject_a_planted_mistake(monkeypatch, name):
    import inspect
    src = inspect.getsource(att.causal_attention)
    old, new = ATT_MUTATIONS[name]
    assert src.count(old) == 1, name
    ns = {"np": att.np}
    exec(src.replace(old, new), ns)
    monkeypatch.setattr(att, "causal_attention", ns["causal_attention"])
    failed = []
    for fn, args in ATT_PINS:
        try:
            fn(*args)
        except (AssertionError, FloatingPointError, ValueError):
            failed.append(fn.__name__)
    print("%s: %d of %d pins fail" % (name, len(failed), len(ATT_PINS)))
    assert len(failed) >= 1, (name, failed)


# ------------------------------------------------------------------ the parity metric
import inspect  # noqa: E402

import test_metric_pins as mpins  # noqa: E402

METRIC_SRC = inspect.getsource(oracle.max_rel_err)
METRIC_MUTATIONS = {
    "abs dropped from the error": ("num = float(np.max(np.abs(x - ref)))", "num = float(np.max(x - ref))"),
    "scale taken from the result": ("den = float(np.max(np.abs(ref)))", "den = float(np.max(np.abs(x)))"),
    "abs dropped from the scale": ("den = float(np.max(np.abs(ref)))", "den = float(np.max(ref))"),
    "mean error instead of the largest": ("num = float(np.max(np.abs(x - ref)))", "num = float(np.mean(np.abs(x - ref)))"),
    "shape check dropped": ("if x.shape != ref.shape:", "if False:"),
    "zero reference gives zero": ("        return num\n    return num / den", "        return 0.0\n    return num / den"),
}
METRIC_PINS = [getattr(mpins, n) for n in dir(mpins) if n.startswith("test_")]


@pytest.mark.parametrize("name", sorted(METRIC_MUTATIONS))
def test_metric_pins_reject_a_planted_mistake(monkeypatch, name):
    import numpy as np
    old, new = METRIC_MUTATIONS[name]
    assert METRIC_SRC.count(old) == 1, name
    ns = {"np": np}
    exec(METRIC_SRC.replace(old, new), ns)
    monkeypatch.setattr(oracle, "max_rel_err", ns["max_rel_err"])
    failed = []
    for fn in METRIC_PINS:
        try:
            fn()
        except (KeyboardInterrupt, SystemExit):
            raise
        except BaseException:   # assertion errors and pytest.raises failures alike
            failed.append(fn.__name__)
    assert failed, "no metric pin caught: " + name
