"""Planted mistakes in the oracle's LM-head functions (on the CPU) must each
fail a pin of ``test_oracle_lmhead_pins.py``. The comparison with the
pure-Python mini oracle's dot products is left out, so what catches a mistake
is a closed form, a second path to the same logits (indexing h directly) or
the finite differences of the loss."""

import numpy as np
import pytest

import oracle
from tests import test_oracle_lmhead_pins as pins

_widen = oracle.bf16_bits_to_f64
_logits = oracle.lmhead_logits
_dlogits = oracle.dlogits


def _widen_off_by_one_bit(bits):
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 15
    return b.view(np.float32).astype(np.float64)


def _weight_read_as_d_by_v(h_bits, w_bits):
    V, d = w_bits.shape
    return np.ascontiguousarray(_widen(h_bits) @ _widen(w_bits).reshape(d, V))


def _hidden_rows_shifted(h_bits, w_bits):
    return _logits(np.roll(h_bits, 1, axis=0), w_bits)


def _dz_negated(*a, **k):
    return -_dlogits(*a, **k)


def _dz_without_target_term(z, target, lse, logp, g, **k):
    out = _dlogits(z, target, lse, logp, g, **k)
    out[np.arange(out.shape[0]), target] += np.asarray(g, np.float64) * -1.0
    return out


def _dz_with_next_rows_lse(z, target, lse, logp, g, **k):
    return _dlogits(z, target, np.roll(np.asarray(lse), 1), logp, g, **k)


def _dz_without_temperature_factor(z, target, lse, logp, g, inv_temp=1.0, **k):
    return _dlogits(z, target, lse, logp, g, inv_temp=inv_temp, **k) / inv_temp


MUTATIONS = {
    "bf16_widening_off_by_one_bit": ("bf16_bits_to_f64", _widen_off_by_one_bit),
    "weight_read_as_d_by_v": ("lmhead_logits", _weight_read_as_d_by_v),
    "hidden_rows_shifted": ("lmhead_logits", _hidden_rows_shifted),
    "dlogits_negated": ("dlogits", _dz_negated),
    "dlogits_without_onehot": ("dlogits", _dz_without_target_term),
    "dlogits_with_other_rows_lse": ("dlogits", _dz_with_next_rows_lse),
    "dlogits_without_temperature_factor": ("dlogits", _dz_without_temperature_factor),
}


def _pins():
    """(name, callable) for every LM-head pin except the mini-oracle comparison."""
    out = [("zero_weight", pins.test_zero_weight_gives_uniform_rows),
           ("one_hot_weight", pins.test_one_hot_weight_rows_select_hidden_features),
           ("rank_one", pins.test_rank_one_closed_form)]
    out += [(f"finite_differences[{s}-{it}]",
             (lambda s=s, it=it: pins.test_grads_finite_differences(s, it)))
            for s, it in ((0, 1.0), (1, 1.0), (2, 1.0), (3, 0.7))]
    return out


def test_pins_pass_unmutated():
    for _, pin in _pins():
        pin()


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name, monkeypatch):
    attr, fn = MUTATIONS[name]
    monkeypatch.setattr(oracle, attr, fn)
    caught = []
    for pin_name, pin in _pins():
        try:
            # a planted mistake may overflow on the way to a failed pin
            with np.errstate(over="ignore", invalid="ignore"):
                pin()
        except (AssertionError, ValueError):
            caught.append(pin_name)
    assert caught, f"mutation {name} passed every pin"
