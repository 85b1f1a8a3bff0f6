"""Planted mistakes in the oracle (CPU): each mutant changes one line of one
oracle function by a plausible index slip (a dropped base, a dropped factor,
transposed operands, a wrong subscript), and the pins of
test_oracle_pins.py must fail on it.  The original function is put back
after each case.
"""
import inspect
import textwrap

import pytest

from oracle import cmm, repack
from synth import configs
from tests import test_oracle_pins as pins

TINY = [configs.get(1), configs.get(1, kv_layout="token")]


def _packed():
    pins.pin_packed_words(TINY + pins.random_cfgs(12, seed=21))


def _outbound():
    pins.pin_outbound(TINY + pins.random_cfgs(40, seed=22))


def _kv():
    pins.pin_kv_invariant(TINY + pins.random_cfgs(6, seed=23))


MUTANTS = [
    # (module, function, original text, planted text, pin expected to fail)
    (repack, "expected_packed_weight_words", "gi, gj = a * t.unit + e // t.cols, e % t.cols",
     "gi, gj = a + e // t.cols, e % t.cols", _packed),
    (repack, "expected_packed_weight_words", "gi, gj = e // w, a * t.unit + e % w",
     "gi, gj = e % w, a * t.unit + e // w", _packed),
    (repack, "expected_packed_weight_words", "w = (b - a) * t.unit", "w = b - a", _packed),
    (repack, "packed_weight_outbound", "(a - o0, b - o0)", "(a, b)", _outbound),
    (repack, "_outbound_pieces", "for a, b in cmm.iv_subtract([(x.begin, x.end)], mine):",
     "for a, b in [(x.begin, x.end)]:", _outbound),
    (repack, "packed_kv_outbound", "part = _heads_slice(view, pb, a - o0, b - o0, live)",
     "part = _heads_slice(view, pb, a, b, live)", _outbound),
    (repack, "kv_arena", "tok = full[s, lb * bt:(lb + 1) * bt, a:b, :]",
     "tok = full[s, lb * bt:(lb + 1) * bt, :b - a, :]", _kv),
    (repack, "kv_arena", "view[p] = tok.transpose(1, 0, 2)", "view[p] = tok.reshape(view[p].shape)",
     pins.pin_hand_words),
    (repack, "_block_view", "g = layer * 2 + kv", "g = kv * 2 + layer", _kv),
    (repack, "kv_full", "shape = (c[\"n_seq\"], c[\"seq_tokens\"], pb.n_kv, pb.head_dim)",
     "shape = (c[\"seq_tokens\"], c[\"n_seq\"], pb.n_kv, pb.head_dim)", pins.pin_hand_words),
    (repack, "expected_kv_words", "* pb.n_kv + (a + h)) * hd + d", "* pb.n_kv + h) * hd + d", pins.pin_hand_words),
    (cmm, "retained_weight", "space_old[sp][owner_old]", "space_old[sp][j]", pins.pin_inorder_strict),
]


def _planted(mod, name, old, new):
    src = textwrap.dedent(inspect.getsource(getattr(mod, name)))
    assert src.count(old) == 1, f"{name}: the text to replace must occur once"
    code = compile(src.replace(old, new), f"<planted mistake in {mod.__name__}.{name}>", "exec")
    return code


@pytest.mark.parametrize("case", range(len(MUTANTS)),
                         ids=[f"{m[1]}:{i}" for i, m in enumerate(MUTANTS)])
def test_pin_catches_planted_mistake(case):
    mod, name, old, new, pin = MUTANTS[case]
    code = _planted(mod, name, old, new)
    saved = mod.__dict__[name]
    try:
        exec(code, mod.__dict__)  # rebinds `name` in the oracle module
        assert mod.__dict__[name] is not saved
        with pytest.raises(Exception):
            pin()
    finally:
        mod.__dict__[name] = saved
    pin()  # the original passes
