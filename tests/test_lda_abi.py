"""The LDA C ABI without a GPU: exported symbols, argument checks, and the host-side token
layout (minibatch blocks and processing order) against the oracle's, bit for bit."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_1410_8043_amd import ps_lda
from paper_1410_8043_amd.synth import lda_corpus as lc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_declared_lda_symbol():
    text = open(os.path.join(ROOT, "include", "ps_lda.h")).read()
    names = sorted(set(re.findall(r"\b(ps_lda_[a-z_]+)\s*\(", text)))
    lib = ctypes.CDLL(ps_lda.LIB_PATH)
    assert len(names) == 11
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(ps_lda.SYMBOLS)


def test_option_and_export_keys_match_the_header():
    text = open(os.path.join(ROOT, "include", "ps_lda.h")).read()
    keys = dict(re.findall(r"#define PS_LDA_((?:OPT|X)_[A-Z_]+) (\d+)", text))
    assert len(keys) == 11
    for name, value in keys.items():
        assert getattr(ps_lda, name) == int(value), name


@pytest.mark.parametrize("args", [
    (0, 5, 2, 1, 0, 0.1, 0.1), (5, 0, 2, 1, 0, 0.1, 0.1), (5, 5, 0, 1, 0, 0.1, 0.1), (5, 5, 513, 1, 0, 0.1, 0.1),
    (5, 5, 2, 0, 0, 0.1, 0.1), (5, 5, 2, 1, -1, 0.1, 0.1), (5, 5, 2, 1, 0, 0.0, 0.1), (5, 5, 2, 1, 0, 0.1, -1.0),
    (5, 5, 2, 1, 0, float("nan"), 0.1), (5, 5, 2, 1, 0, 0.1, float("inf")), (2**31, 5, 2, 1, 0, 0.1, 0.1)])
def test_create_rejects_bad_arguments(args):
    with pytest.raises(ps_lda.PsLdaError) as e:
        ps_lda.ps_lda_create(*args)
    assert e.value.code == ps_lda.EINVAL


def test_options_and_load_are_checked():
    with pytest.raises(ps_lda.PsLdaError) as e:
        ps_lda.PsLda(4, 4, 2, 1, 0, 0.1, 0.1, policy=3, host_only=True)
    assert e.value.code == ps_lda.EINVAL
    with pytest.raises(ps_lda.PsLdaError):
        ps_lda.PsLda(4, 4, 2, 1, 0, 0.1, 0.1, B=0, host_only=True)
    h = ps_lda.PsLda(4, 4, 2, 2, 1, 0.1, 0.1, host_only=True)
    for doc, word, z in (([4], [0], [0]), ([0], [4], [0]), ([0], [0], [2]), ([-1], [0], [0])):
        with pytest.raises(ps_lda.PsLdaError) as e:
            h.load(doc, word, z)
        assert e.value.code == ps_lda.EINVAL
    with pytest.raises(ps_lda.PsLdaError) as e:
        h.clock(1)
    assert e.value.code == ps_lda.ESTATE
    h.load([0, 1, 3], [0, 1, 2], [0, 1, 1])
    with pytest.raises(ps_lda.PsLdaError) as e:
        h.load([0], [0], [0])
    assert e.value.code == ps_lda.ESTATE
    for call in (lambda: h.clock(1), h.loglik, h.z):  # host-only: no device state
        with pytest.raises(ps_lda.PsLdaError) as e:
            call()
        assert e.value.code == ps_lda.ESTATE
    with pytest.raises(ps_lda.PsLdaError) as e:
        h.export(ps_lda.X_BLOCK_ORDER, 2)
    assert e.value.code == ps_lda.EINVAL


@pytest.mark.parametrize("P,B,seed", [(4, 2, 0), (7, 3, 12345), (1, 1, 9), (64, 2, 2**63 + 5)])
def test_block_order_matches_the_oracle(P, B, seed):
    spec = lc.scaled(lc.CORPORA["tiny"], 1.0, P=P, B=B, seed=seed)
    corpus = lc.generate(spec)
    h = ps_lda.PsLda(spec.D, spec.V, spec.K, P, spec.s, spec.alpha, spec.beta, B=B, seed=seed, host_only=True)
    h.load(corpus.doc, corpus.word, corpus.z0)
    o = oracle.LdaOracle(spec.D, spec.V, spec.K, P, spec.s, spec.alpha, spec.beta, oracle.ESSP, B, seed)
    o.load(corpus.doc, corpus.word, corpus.z0)
    for b in range(B):
        np.testing.assert_array_equal(h.export(ps_lda.X_BLOCK_ORDER, b), o.export(oracle.LDA_BLOCK_ORDER, b))


def test_empty_load_has_empty_blocks():
    h = ps_lda.PsLda(3, 3, 2, 2, 1, 0.1, 0.1, B=3, host_only=True)
    h.load([], [], [])
    assert all(h.export(ps_lda.X_BLOCK_ORDER, b).size == 0 for b in range(3))


def test_export_and_option_errors():
    h = ps_lda.PsLda(4, 4, 2, 2, 1, 0.1, 0.1, B=2, host_only=True)
    h.load([0, 1, 2, 3], [0, 1, 2, 3], [0, 1, 0, 1])
    with pytest.raises(ps_lda.PsLdaError) as e:  # an option after the load
        ps_lda._check(h._h, "ps_lda_set_option", ps_lda._lib.ps_lda_set_option(h._h, ps_lda.OPT_POLICY, 0))
    assert e.value.code == ps_lda.ESTATE
    n = ctypes.c_int64()
    assert ps_lda._lib.ps_lda_export(h._h, 9, 0, None, 0, ctypes.byref(n)) == ps_lda.EINVAL  # unknown kind
    assert b"unknown export" in ps_lda._lib.ps_lda_last_error(h._h)
    assert ps_lda._lib.ps_lda_export(h._h, ps_lda.X_BLOCK_ORDER, 0, None, 0, ctypes.byref(n)) == ps_lda.OK
    if n.value > 0:  # a buffer one element short
        buf = np.empty(n.value, np.int64)
        assert ps_lda._lib.ps_lda_export(h._h, ps_lda.X_BLOCK_ORDER, 0, buf.ctypes.data, n.value - 1,
                                         ctypes.byref(n)) == ps_lda.EINVAL
    assert h.export(ps_lda.X_VERSION_LOG).size == 0  # no clock run
    assert h.get_clock() == 0


def test_null_handle_calls_are_rejected():
    n = ctypes.c_int64()
    assert ps_lda._lib.ps_lda_clock(None, 1) == ps_lda.EINVAL
    assert ps_lda._lib.ps_lda_export(None, 0, 0, None, 0, ctypes.byref(n)) == ps_lda.EINVAL
    assert ps_lda._lib.ps_lda_last_error(None) == b"null handle"
    ps_lda._lib.ps_lda_destroy(None)  # NULL-safe


@pytest.mark.parametrize("alpha,beta", [(0.1, 1e-300), (1e300, 1e300)])
def test_weight_range_is_checked_on_both_sides(alpha, beta):
    # every p_k must be a normal fp64 number (its exponent sets the token's weight scale):
    # alpha beta / (n + V beta) below 2^-1000, or (longest document + alpha)(n + beta) /
    # (V beta) above 2^1000, is refused by library and oracle alike
    doc, word, z = [0] * 50, [0, 1] * 25, [0] * 50
    h = ps_lda.PsLda(1, 2, 4, 1, 1, alpha, beta, host_only=True)
    with pytest.raises(ps_lda.PsLdaError) as e:
        h.load(doc, word, z)
    assert e.value.code == ps_lda.EINVAL and b"2^700" in ps_lda._lib.ps_lda_last_error(h._h)
    o = oracle.LdaOracle(1, 2, 4, 1, 1, alpha, beta)
    with pytest.raises(oracle.OracleError):
        o.load(doc, word, z)
    # the same corpus with alpha = 0.1 and beta = 0.01 is accepted by both
    ps_lda.PsLda(1, 2, 4, 1, 1, 0.1, 0.01, host_only=True).load(doc, word, z)
    oracle.LdaOracle(1, 2, 4, 1, 1, 0.1, 0.01).load(doc, word, z)


def test_library_keeps_weights_numerators_and_denominators_in_its_division_range():
    # beta = 1e-215 gives weights between about 2^-722 and 2^724: normal numbers, which the
    # oracle accepts, but outside [2^-700, 2^700], where the library's short division is exact
    doc, word, z = [0] * 50, [0, 1] * 25, [0] * 50
    oracle.LdaOracle(1, 2, 4, 1, 1, 0.1, 1e-215).load(doc, word, z)
    h = ps_lda.PsLda(1, 2, 4, 1, 1, 0.1, 1e-215, host_only=True)
    with pytest.raises(ps_lda.PsLdaError) as e:
        h.load(doc, word, z)
    assert e.value.code == ps_lda.EINVAL and b"2^700" in ps_lda._lib.ps_lda_last_error(h._h)
    # inside the range on every count: accepted
    ps_lda.PsLda(1, 2, 4, 1, 1, 1e-100, 1e-100, host_only=True).load(doc, word, z)
