"""The RNN-head pins catch plausible mistakes (no GPU).

Each case below compiles a copy of the oracle with one mistake planted in its
RNN-head function (a swapped gate, the candidate and output parts exchanged,
z_k assembled in the wrong order, the recurrence dropped, a sigmoid where the
equation has tanh) and runs every pin of tests/test_oracle_rnn.py against it:
at least one pin must fail.  The unmodified source must pass them all.
"""
import contextlib
import os
import shutil
import subprocess
import tempfile

import pytest

import oracle
import test_oracle_rnn as pins

PINS = [getattr(pins, n) for n in dir(pins) if n.startswith("test_")]

MUTANTS = {
    "swapped gate": ("st[j] = g * st[j] + (1.0 - g) * tanh(act[rank + j]);",
                     "st[j] = (1.0 - g) * st[j] + g * tanh(act[rank + j]);"),
    "candidate and output exchanged": (
        "st[j] = g * st[j] + (1.0 - g) * tanh(act[rank + j]);\n                o[j] = tanh(act[2 * rank + j]);",
        "st[j] = g * st[j] + (1.0 - g) * tanh(act[2 * rank + j]);\n                o[j] = tanh(act[rank + j]);"),
    "state and embedding exchanged in z": (
        "for (int j = 0; j < rank; ++j) zin[j] = st[j];\n            for (int j = 0; j < rank; ++j) zin[rank + j] = bf16_to_f64(W1[(int64_t)prev * rank + j]);",
        "for (int j = 0; j < rank; ++j) zin[rank + j] = st[j];\n            for (int j = 0; j < rank; ++j) zin[j] = bf16_to_f64(W1[(int64_t)prev * rank + j]);"),
    "recurrence dropped": ("st[j] = g * st[j] + (1.0 - g) * tanh(act[rank + j]);",
                           "st[j] = (1.0 - g) * tanh(act[rank + j]);"),
    "sigmoid output": ("o[j] = tanh(act[2 * rank + j]);", "o[j] = sigmoid(act[2 * rank + j]);"),
}


@contextlib.contextmanager
def _oracle_from(text):
    d = tempfile.mkdtemp(prefix="oracle_mutant_")
    src, lib = os.path.join(d, "oracle.c"), os.path.join(d, "liboracle.so")
    with open(src, "w") as f:
        f.write(text)
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off",
                           "-fno-fast-math", "-shared", "-fPIC", src, "-o", lib, "-lm"])
    saved = (oracle._SRC, oracle._LIB, oracle._lib)
    oracle._SRC, oracle._LIB, oracle._lib = src, lib, None
    try:
        yield
    finally:
        oracle._SRC, oracle._LIB, oracle._lib = saved
        shutil.rmtree(d, ignore_errors=True)


def _failures():
    failed = []
    for pin in PINS:
        try:
            pin()
        except AssertionError:
            failed.append(pin.__name__)
    return failed


def _source():
    with open(oracle._SRC) as f:
        return f.read()


def test_unmodified_source_passes_every_pin():
    with _oracle_from(_source()):
        assert _failures() == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_fails_a_pin(name):
    old, new = MUTANTS[name]
    text = _source()
    assert text.count(old) == 1, f"mutation site for {name!r} not found once"
    with _oracle_from(text.replace(old, new)):
        assert _failures(), f"no pin caught: {name}"
