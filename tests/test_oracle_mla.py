"""The MLA decode oracle against its pins (tests/mla_pins.py), and a check
that plausible mistakes in its reduction to the attention oracle are caught:
each planted mistake must make some pin fail."""
import numpy as np
import pytest

import oracle
import mla_pins


@pytest.fixture(scope="module")
def lib():
    return oracle.load()


@pytest.mark.parametrize("name", sorted(mla_pins.PINS))
def test_mla_pin(lib, name):
    mla_pins.PINS[name](lib)


def _swap_query_parts(q, q_pe, kv, k_pe):        # rotary part first on one side only
    qf = np.concatenate([q_pe, q], axis=2)[:, :, None, :]
    kf = np.ascontiguousarray(np.concatenate([kv, k_pe], axis=3).transpose(0, 2, 1, 3))
    return qf, kf, q.shape[2]


def _drop_rotary(q, q_pe, kv, k_pe):             # scores from the latent part only
    qf = q[:, :, None, :]
    kf = np.ascontiguousarray(kv.transpose(0, 2, 1, 3))
    return qf, kf, q.shape[2]


def _wrong_cache_axes(q, q_pe, kv, k_pe):        # cache read as [B, Hkv, Skv, D]
    B, Skv, Hkv = kv.shape[:3]
    qf = np.concatenate([q, q_pe], axis=2)[:, :, None, :]
    kf = np.ascontiguousarray(np.concatenate([kv, k_pe], axis=3).reshape(B, Hkv, Skv, -1))
    return qf, kf, q.shape[2]


def _rotary_first_both(q, q_pe, kv, k_pe):      # scores right, value columns wrong
    qf = np.concatenate([q_pe, q], axis=2)[:, :, None, :]
    kf = np.ascontiguousarray(np.concatenate([k_pe, kv], axis=3).transpose(0, 2, 1, 3))
    return qf, kf, q.shape[2]


MUTANTS = {"swap_query_parts": _swap_query_parts, "drop_rotary": _drop_rotary,
           "wrong_cache_axes": _wrong_cache_axes, "rotary_first_both": _rotary_first_both}


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_mla_pins_catch_mutant(lib, monkeypatch, mutant):
    monkeypatch.setattr(oracle, "_mla_bits", MUTANTS[mutant])
    failed = []
    for name, pin in mla_pins.PINS.items():
        try:
            pin(lib)
        except (AssertionError, ValueError, IndexError):
            failed.append(name)
    assert failed, f"no MLA pin catches the mutant {mutant}"
