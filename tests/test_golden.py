"""The oracle against numbers printed in the paper (tests/golden/paper_numbers.json)."""
import json
import math
import os
from fractions import Fraction

import numpy as np

GOLDEN = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_numbers.json")))


def test_sawtooth_sequence(orc):
    g = GOLDEN["sawtooth"]
    got = [orc.sawtooth_dilation(layer, g["period"]) for layer in range(len(g["first_layers"]))]
    assert got == g["first_layers"]
    # the closed form (layer mod P) + 1 used to pick each workload's dilations
    for P in range(1, 9):
        assert [orc.sawtooth_dilation(l, P) for l in range(3 * P)] == [(l % P) + 1 for l in range(3 * P)]


def _stack_receptive_field(orc, dilations, k, T=24):
    """Number of input steps that reach the last output of a stack of linear
    charges (taps +1, no bias), found by pushing one impulse per input step."""
    reach = 0
    for tau in range(T):
        x = np.zeros((T, 1, 1), np.float32)
        x[tau] = 1.0
        for d in dilations:
            x, _ = orc.forward_f32(x, np.ones((1, k), np.int8), np.zeros((1, k), np.int8),
                                   np.zeros(1, np.float32), k, d, 1.0)
        reach += int(x[T - 1, 0, 0] != 0.0)
    return reach


def test_receptive_field_example(orc):
    g = GOLDEN["receptive_field"]
    fixed = [1] * g["layers"]
    saw = [orc.sawtooth_dilation(l, 3) for l in range(g["layers"])]
    assert _stack_receptive_field(orc, fixed, g["k"]) == g["fixed_dilation_steps"]
    assert _stack_receptive_field(orc, saw, g["k"]) == g["sawtooth_steps"]


def test_energy_table_operation_counts(orc):
    g = GOLDEN["energy_table"]
    T, k = g["T"], g["k"]
    # neurons of the sequential-CIFAR network: three SN layers of 128 channels
    # at height 32, three at height 16 after the 2x2 average pool, and FC256-SN
    neurons = 3 * g["channels"] * g["height"] + 3 * g["channels"] * (g["height"] // 2) + g["fc_neurons"]
    assert neurons == 18688
    x = np.ones((T, 1, 1), np.float32)
    _, _, taps = orc.forward_f32(x, np.ones((1, k), np.int8), np.zeros((1, k), np.int8),
                                 np.zeros(1, np.float32), k, 1, 1.0, with_tap_count=True)
    shift_ops = taps * neurons
    add_ops = (taps + T) * neurons  # one accumulate per tap plus the bias per step
    assert shift_ops == 7_325_696 and add_ops == 7_923_712
    # the table prints its figures cut (not rounded) to three significant
    # digits: 7,325,696 appears as 7.32e6 and 88.566 uJ as 88.56
    def cut(v, scale):
        return math.floor(v / scale * 100 + 1e-9) / 100

    assert cut(shift_ops, 1e6) == g["ours_shift"] / 1e6
    assert cut(add_ops, 1e6) == g["ours_add"] / 1e6
    energy = (shift_ops * g["e_shift_pJ"] + add_ops * g["e_add_pJ"]) / 1e6
    assert cut(energy, 1) == g["ours_energy_uJ"]
    psn_mul, psn_add = T * T * neurons, (T * T + T) * neurons
    assert cut(psn_mul, 1e7) == g["psn_mul"] / 1e7
    assert cut(psn_add, 1e7) == g["psn_add"] / 1e7
    assert cut((psn_mul * g["e_mul_pJ"] + psn_add * g["e_add_pJ"]) / 1e6, 1) == g["psn_energy_uJ"]


def test_max_order_energy_formula(orc):
    g = GOLDEN["max_order_energy"]
    e = GOLDEN["energy_table"]
    for T in [2, 8, 17, 32]:
        x = np.ones((T, 1, 1), np.float32)
        _, _, taps = orc.forward_f32(x, np.ones((1, T), np.int8), np.zeros((1, T), np.int8),
                                     np.zeros(1, np.float32), T, 1, 1.0, with_tap_count=True)
        energy = Fraction(str(e["e_shift_pJ"])) * taps + Fraction(str(e["e_add_pJ"])) * (taps + T)
        assert energy == Fraction(str(g["quadratic"])) * T * T + Fraction(str(g["linear"])) * T


def test_paper_surrogates_peak(orc):
    g = GOLDEN["surrogates"]
    for a in g["arctan_alphas"]:
        assert orc.surrogate("atan", a, 0.0) == np.float32(a / 2)
    assert orc.surrogate("rational", g["rational_alpha"], 0.0) == np.float32(1.0)
