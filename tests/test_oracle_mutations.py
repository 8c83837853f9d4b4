"""The oracle's pins catch plausible mistakes (planted in the oracle, on the CPU).

Each case swaps one piece of the oracle for a subtly wrong version and checks
that at least one pin of ``test_oracle`` fails.  This guards the pins
themselves: a pin set that a dropped term or a wrong tie-break survives would
not pin the oracle.
"""

import types

import numpy as np
import pytest

import oracle.bmu as ob
import test_oracle as pins


def _dist_drop_nnz(W, norms, feats, N=None):
    n = norms.shape[0] if N is None else int(N)
    dot = np.asarray(W[feats, :n], np.float64).sum(0) if feats.size else np.zeros(n)
    return np.asarray(norms[:n], np.float64) - 2.0 * dot


def _dist_drop_norms(W, norms, feats, N=None):
    n = norms.shape[0] if N is None else int(N)
    dot = np.asarray(W[feats, :n], np.float64).sum(0) if feats.size else np.zeros(n)
    return float(feats.size) - 2.0 * dot


def _dist_sign(W, norms, feats, N=None):
    n = norms.shape[0] if N is None else int(N)
    dot = np.asarray(W[feats, :n], np.float64).sum(0) if feats.size else np.zeros(n)
    return float(feats.size) + np.asarray(norms[:n], np.float64) + 2.0 * dot


def _dist_half_dot(W, norms, feats, N=None):
    n = norms.shape[0] if N is None else int(N)
    dot = np.asarray(W[feats, :n], np.float64).sum(0) if feats.size else np.zeros(n)
    return float(feats.size) + np.asarray(norms[:n], np.float64) - dot


def _dist_shifted_row(W, norms, feats, N=None):
    n = norms.shape[0] if N is None else int(N)
    f = np.minimum(feats + 1, W.shape[0] - 1)
    dot = np.asarray(W[f, :n], np.float64).sum(0) if feats.size else np.zeros(n)
    return float(feats.size) + np.asarray(norms[:n], np.float64) - 2.0 * dot


def _norms_unsquared(W, N=None):
    n = W.shape[1] if N is None else int(N)
    return np.asarray(W[:, :n], np.float64).sum(0)


class _LastArgmin(types.ModuleType):
    """numpy with argmin returning the LAST minimiser (wrong tie-break)."""

    def __getattr__(self, name):
        return getattr(np, name)

    @staticmethod
    def argmin(a, *args, **kw):
        a = np.asarray(a)
        return a.size - 1 - int(np.argmin(a[::-1]))


PINS = [
    lambda: pins.test_hand_examples(0),
    pins.test_hand_examples_match_dense_brute_force,
    lambda: pins.test_random_tiny_vs_dense_brute_force(0),
    lambda: pins.test_random_tiny_vs_dense_brute_force(1),
    lambda: pins.test_fp64_equals_exact_integer(0),
    pins.test_empty_document_is_argmin_of_norms,
    pins.test_neuron_equal_to_document_has_zero_distance,
    pins.test_invariant_to_codebook_layout,
    pins.test_norms_definition_and_blocks,
]


def _some_pin_fails():
    for pin in PINS:
        try:
            pin()
        except (AssertionError, IndexError, ValueError):
            return True
    return False


@pytest.mark.parametrize("name,fn", [
    ("drop |S|", _dist_drop_nnz),
    ("drop ||w||^2", _dist_drop_norms),
    ("sign of dot", _dist_sign),
    ("dot not doubled", _dist_half_dot),
    ("wrong feature row", _dist_shifted_row),
])
def test_planted_distance_mistake_is_caught(monkeypatch, name, fn):
    monkeypatch.setattr(ob, "doc_distances", fn)
    assert _some_pin_fails(), name


def test_planted_norm_mistake_is_caught(monkeypatch):
    monkeypatch.setattr(ob, "codebook_norms", _norms_unsquared)
    assert _some_pin_fails()


def test_planted_tie_break_mistake_is_caught(monkeypatch):
    monkeypatch.setattr(ob, "np", _LastArgmin("numpy_last_argmin"))
    assert _some_pin_fails()


def test_unmutated_oracle_passes_every_pin():
    assert not _some_pin_fails()
