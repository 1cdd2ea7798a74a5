"""The pins have teeth: plausible mistakes planted in a *copy* of the oracle
source (compiled to a temporary library on the CPU) must each fail at least
one pin.  The real oracle is never modified."""
import os
import subprocess

import numpy as np
import pytest

import oracle
import workloads
from msa_pins import dense_reference, positions_of, to_f64

SRC = os.path.join(os.path.dirname(oracle.__file__), "msa_oracle.c")

MUTANTS = {
    "drop_last_key_in_weights": ("for (int32_t j = 0; j <= p; ++j) {\n    const double w",
                                 "for (int32_t j = 0; j < p; ++j) {\n    const double w"),
    "drop_scale": ("s[j] = J->scale * dot;", "s[j] = dot;"),
    "strided_gqa_groups": ("h / (J->num_q_heads / J->num_kv_heads)", "h % J->num_kv_heads"),
    "shifted_block_offset": ("(int64_t)(j % bs) * J->kst", "(int64_t)((j + 1) % bs) * J->kst"),
    "transposed_v_operand": ("vv[(int64_t)c * J->vsd]", "vv[c]"),
    "lse_without_log_sum": ("*lse = m + log(l);", "*lse = m;"),
    "unnormalized_output": ("for (int32_t c = 0; c < d; ++c) o[c] /= l;", ""),
    "wrong_sign_exponent": ("exp(s[j] - m)", "exp(m - s[j])"),
    "positions_collapsed": ("row_pos[r] = seg_start[s] + t;", "row_pos[r] = seg_start[s];"),
    "max_not_subtracted": ("exp(s[j] - m)", "exp(s[j])"),
}


def _build_mutant(tmp_path, name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation anchor for {name} not found"
    src = src.replace(old, new)
    c = tmp_path / f"{name}.c"
    so = tmp_path / f"{name}.so"
    c.write_text(src)
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                           "-pthread", str(c), "-o", str(so), "-lm"])
    return oracle.load_library(str(so))


def _pins_pass(lib) -> bool:
    """A compact battery of the pins in test_oracle_pins.py."""
    cases = [
        workloads.make_random(2, num_seqs=3, num_q_heads=4, num_kv_heads=2, head_dim=64,
                              max_len=200, max_segs=5),
        workloads.make_random(3, num_seqs=2, num_q_heads=8, num_kv_heads=2, head_dim=128,
                              max_len=260, max_segs=3),
    ]
    for inst in cases:
        o, lse = oracle.forward(inst, lib=lib)
        ro, rlse = dense_reference(inst)
        if not (np.allclose(o, ro, rtol=0, atol=1e-9) and np.allclose(lse, rlse, rtol=0, atol=1e-9)):
            return False
    # zero query closed form
    inst = workloads.make_layout(24, [130], [[(5, 3), (64, 17), (129, 1)]], 4, 1, 64)
    inst.q = np.zeros_like(inst.q)
    o, lse = oracle.forward(inst, lib=lib)
    _, pos = positions_of(inst)
    v = to_f64(inst.v_logical[0]).numpy()
    for r, p in enumerate(pos):
        if not np.allclose(o[r, 0], v[:p + 1, 0].mean(axis=0), rtol=0, atol=1e-12):
            return False
        if abs(lse[r, 0] - np.log(p + 1)) > 1e-12:
            return False
    return True


def test_unmutated_copy_passes(tmp_path):
    src = open(SRC).read()
    c = tmp_path / "same.c"
    so = tmp_path / "same.so"
    c.write_text(src)
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                           "-pthread", str(c), "-o", str(so), "-lm"])
    assert _pins_pass(oracle.load_library(str(so)))


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(tmp_path, name):
    lib = _build_mutant(tmp_path, name)
    assert not _pins_pass(lib), f"mutant {name} survived the pins"
