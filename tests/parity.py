"""Comparison rules shared by the GPU parity tests.

Floating point: relative error ||x - x*|| / ||x*|| per vector, 1e-5 for fp32
inputs and 2e-2 for bf16 inputs; gaps use the denominator max(gap*, 1e-6 *
||o*||) so that exact zeros compare.  Index sets: equal, or a tie case that the
caller classifies from the float64 values (counted and reported).
"""
import numpy as np

TOL = {"f32": 1e-5, "bf16": 2e-2}


def rel_vec(x, ref, floor=0.0):
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    num = np.linalg.norm(x - ref, axis=-1)
    den = np.maximum(np.linalg.norm(ref, axis=-1), floor)
    return num / np.maximum(den, 1e-300)


def rel_scalar(x, ref, floor):
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    return np.abs(x - ref) / np.maximum(np.maximum(np.abs(ref), floor), 1e-300)


def t2np(t):
    return None if t is None else t.detach().cpu().numpy()


class Tally:
    def __init__(self):
        self.exact = 0
        self.ties = 0
        self.fail = 0
        self.notes = []

    def add(self, ok_exact, ok_tie, note=""):
        if ok_exact:
            self.exact += 1
        elif ok_tie:
            self.ties += 1
        else:
            self.fail += 1
            if len(self.notes) < 10:
                self.notes.append(note)

    def __repr__(self):
        return f"exact={self.exact} ties={self.ties} fail={self.fail} {self.notes[:3]}"


# test name -> what it measured (worst relative errors, tallies); written out
# at the end of the session by tests/conftest.py
SUMMARY = {}


def record(name, **values):
    SUMMARY[name] = {k: (v if not isinstance(v, Tally) else dict(exact=v.exact, ties=v.ties, fail=v.fail))
                     for k, v in values.items()}


def same_bits(a, b) -> bool:
    """Two results are bitwise identical (NaNs included)."""
    a, b = np.ascontiguousarray(a), np.ascontiguousarray(b)
    return a.shape == b.shape and a.dtype == b.dtype and a.tobytes() == b.tobytes()
