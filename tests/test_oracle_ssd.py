"""The SSD chunk oracle against its pins (tests/ssd_pins.py), and a mutation
check: plausible mistakes planted in a copy of the oracle's source, on the
CPU, must each fail at least one pin."""
import types

import pytest

import oracle.ssd as ssd
from tests import ssd_pins


@pytest.mark.parametrize("pin", ssd_pins.ALL_PINS, ids=[p.__name__ for p in ssd_pins.ALL_PINS])
def test_pin(pin):
    pin(ssd)


def test_recurrence_other_chunk_sizes():
    for Q in (1, 32, 300, 512):
        ssd_pins.pin_recurrence(ssd, B=1, L=300, H=2, G=1, Q=Q, seed=11)


MUTANTS = {
    "exclusive_cumsum": ("return np.cumsum(dtc * A, axis=2).transpose(0, 3, 1, 2)",
                         "return (np.cumsum(dtc * A, axis=2) - dtc * A).transpose(0, 3, 1, 2)"),
    "state_decay_sign": ("w = np.exp(a[:, :, :, -1:] - a)", "w = np.exp(a - a[:, :, :, -1:])"),
    "state_no_dt": ("w = np.exp(a[:, :, :, -1:] - a) * dtc.transpose(0, 3, 1, 2)",
                    "w = np.exp(a[:, :, :, -1:] - a)"),
    "group_map_modulo": ("return np.arange(H) // (H // G)", "return np.arange(H) % G"),
    "passing_prev_decay": ("h = np.exp(a[:, :, c, -1])[:, :, None, None] * h + S[:, c]",
                           "h = np.exp(a[:, :, max(c - 1, 0), -1])[:, :, None, None] * h + S[:, c]"),
    "passing_enter_after": ("        prev[:, c] = h\n        h = np.exp(a[:, :, c, -1])[:, :, None, None] * h + S[:, c]",
                            "        h = np.exp(a[:, :, c, -1])[:, :, None, None] * h + S[:, c]\n        prev[:, c] = h"),
    "scan_strict_causal": ("causal = np.tril(np.ones((Qn, Qn), dtype=bool))",
                           "causal = np.tril(np.ones((Qn, Qn), dtype=bool), -1)"),
    "scan_no_enter_decay": ("y = np.einsum(\"bchpn,bclhn->bclhp\", Hin, Cc) * np.exp(a).transpose(0, 2, 3, 1)[..., None]",
                            "y = np.einsum(\"bchpn,bclhn->bclhp\", Hin, Cc)"),
    "scan_dt_at_l": ("* dtc.transpose(0, 2, 1, 3)[:, :, :, None, :]",
                     "* dtc.transpose(0, 2, 1, 3)[:, :, :, :, None]"),
    "scan_decay_reversed": ("a[..., :, None] - a[..., None, :], 0.0)), 0.0)",
                            "a[..., None, :] - a[..., :, None], 0.0)), 0.0)"),
    "bmm_transposed": ('return np.einsum("bclgn,bcsgn->bcgls", Cc, Bc)',
                       'return np.einsum("bclgn,bcsgn->bcgsl", Cc, Bc)'),
    "scan_no_skip": ("y = y + np.asarray(D, dtype=np.float64)[None, None, None, :, None] * Xc",
                     "y = y"),
    # the tolerance scales (chunk_scan_abs / chunk_state_abs)
    "scan_abs_growth": ("np.asarray(A), np.abs(prev_states)", "np.abs(A), np.abs(prev_states)"),
    "scan_abs_signed_cb": ("np.abs(cb), dt", "cb, dt"),
    "scan_abs_signed_states": ("np.asarray(A), np.abs(prev_states)", "np.asarray(A), prev_states"),
    "scan_abs_signed_skip": ("np.abs(D), Q)", "D, Q)"),
    "state_abs_signed_x": ("return chunk_state(absbits(x), absbits(Bm), dt, A, Q)",
                           "return chunk_state(x, absbits(Bm), dt, A, Q)"),
    "widen_truncate": ("return (b.astype(np.uint32) << np.uint32(16))",
                       "return ((b & np.uint16(0xFF00)).astype(np.uint32) << np.uint32(16))"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_some_pin_catches_mutant(name):
    old, new = MUTANTS[name]
    src = open(ssd.__file__).read()
    assert src.count(old) == 1, f"mutant {name}: anchor not found once"
    mod = types.ModuleType(f"ssd_mutant_{name}")
    exec(compile(src.replace(old, new), f"<ssd mutant {name}>", "exec"), mod.__dict__)
    caught = []
    for pin in ssd_pins.ALL_PINS:
        try:
            pin(mod)
        except (AssertionError, ValueError, IndexError):
            caught.append(pin.__name__)
    assert caught, f"no pin catches mutant {name}"
