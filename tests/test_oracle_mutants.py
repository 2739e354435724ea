"""Plant plausible mistakes in the oracle's C source (on the CPU, in a temp
directory) and check that at least one pin catches each: evidence that the
pins constrain every step of the oracle, not just its happy path."""
import os
import tempfile

import pytest

import oracle
from oracle import build as obuild
from oracle_pins import PINS

MUTANTS = {
    "drop_scale": ("s[j] = p->scale * dot;", "s[j] = dot;"),
    "transposed_k": ("widen(k[j * D + d])", "widen(k[d * p->Sk + j])"),
    "v_from_k": ("const uint16_t *v = p->V +", "const uint16_t *v = p->K +"),
    "transposed_v": ("widen(v[j * D + d])", "widen(v[d * p->Sk + j])"),
    "gqa_modulo_map": ("const int64_t hk = h / (p->Hq / p->Hkv);", "const int64_t hk = h % p->Hkv;"),
    "causal_off_by_one": ("int64_t n = i + 1 + (p->Sk - p->Sq);", "int64_t n = i + (p->Sk - p->Sq);"),
    "causal_top_left": ("int64_t n = i + 1 + (p->Sk - p->Sq);", "int64_t n = i + 1;"),
    "causal_ignored": ("if (!p->causal)\n        return p->Sk;", "if (1)\n        return p->Sk;"),
    "min_not_max": ("if (s[j] > m)", "if (s[j] < m)"),
    "no_max_shift": ("double m = -INFINITY;", "double m = 0.0;\n    if (0) m = -INFINITY;"),
    "lse_sign": ("*lse = m + log(z);", "*lse = m - log(z);"),
    "lse_without_max": ("*lse = m + log(z);", "*lse = log(z);"),
    "no_normalise": ("o[d] /= z;", "o[d] /= 1.0;"),
    "drop_last_key_in_sum": ("z += exp(s[j] - m);", "z += (j + 1 < n) ? exp(s[j] - m) : 0.0;"),
    "drop_first_key_in_o": ("o[d] += w * widen(v[j * D + d]);",
                            "o[d] += (j > 0) ? w * widen(v[j * D + d]) : 0.0;"),
    "truncated_dot": ("for (int64_t d = 0; d < D; ++d)\n            dot +=",
                      "for (int64_t d = 0; d + 1 < D; ++d)\n            dot +="),
    "row_index_swap": ("h = (r / p->Sq) % p->Hq;", "h = (r / p->Sq) % p->Hkv;"),
    "bf16_widen_shift": ("uint32_t w = (uint32_t)bits << 16;", "uint32_t w = (uint32_t)bits << 15;"),
}


def _mutant_lib(tmp, name, old, new):
    with open(obuild.SRC) as f:
        src = f.read()
    assert src.count(old) == 1, f"mutation site for {name} not unique/present"
    path = os.path.join(tmp, f"{name}.c")
    with open(path, "w") as f:
        f.write(src.replace(old, new))
    lib_path = os.path.join(tmp, f"lib{name}.so")
    obuild.build(path, lib_path, extra=("-Wno-unused-parameter", "-Wno-unused-variable"))
    return oracle.load(lib_path)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_some_pin_catches_mutant(name):
    old, new = MUTANTS[name]
    with tempfile.TemporaryDirectory() as tmp:
        lib = _mutant_lib(tmp, name, old, new)
        caught = []
        for pin_name, pin in PINS.items():
            try:
                pin(lib)
            except (AssertionError, oracle.OracleError, FloatingPointError):
                caught.append(pin_name)
        assert caught, f"no pin catches mutant {name}"
