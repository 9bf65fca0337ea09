"""Pins of the policy semantics through the two-parameter model (App. B.1).

Every expected value below is printed in the paper (App. B.1 and the values it
quotes): the expected loss has its unique minimum 9/32 at gamma = 1/2, w = 1;
at that minimum R/R's average update is (1/2, 0) and U/U's is (0, -1/4); R/R is
at rest at gamma = 1/3, w = 1, where the expected loss exceeds its minimum by
1/18; U/R and N/R follow the gradient of the expected loss everywhere.
"""
from fractions import Fraction as Fr

from oracle import model2p

H, ONE = Fr(1, 2), Fr(1)


def test_expected_loss_closed_form():
    for g in (Fr(1, 7), Fr(1, 3), H, Fr(9, 10), ONE):
        for w in (Fr(-1), Fr(0), Fr(1, 2), ONE, Fr(5, 3)):
            want = Fr(9, 32) + 2 * (g - H) ** 2 + (1 + g / 2) * (w - 1) ** 2
            assert model2p.expected_loss(g, w) == want


def test_minimum_and_value():
    assert model2p.expected_loss(H, ONE) == Fr(9, 32)
    assert model2p.grad_expected_loss(H, ONE) == (0, 0)


def test_updates_at_minimum():
    assert model2p.average_update(("R", "R"), H, ONE) == (H, 0)
    assert model2p.average_update(("U", "U"), H, ONE) == (0, Fr(-1, 4))
    assert model2p.average_update(("U", "R"), H, ONE) == (0, 0)
    assert model2p.average_update(("N", "R"), H, ONE) == (0, 0)


def test_reference_and_NR_follow_gradient_everywhere():
    for g in (Fr(1, 5), Fr(2, 3), ONE):
        for w in (Fr(-2), Fr(1, 3), Fr(2)):
            grad = model2p.grad_expected_loss(g, w)
            assert model2p.average_update(("U", "R"), g, w) == grad
            assert model2p.average_update(("N", "R"), g, w) == grad


def test_rr_rest_point_and_excess():
    g = Fr(1, 3)
    assert model2p.average_update(("R", "R"), g, ONE) == (0, 0)
    assert model2p.expected_loss(g, ONE) - Fr(9, 32) == Fr(1, 18)


def test_per_use_errors():
    # App. B.1: R at the gain use adds w^2 (1 - gamma); U or N at the weight use adds -w gamma (1 - gamma).
    for g in (Fr(1, 4), Fr(3, 5)):
        for w in (Fr(1, 2), Fr(3)):
            ref = model2p.average_update(("U", "R"), g, w)
            for pol in (("R", "R"), ("R", "U"), ("U", "U"), ("N", "N"), ("U", "N"), ("R", "N")):
                got = model2p.average_update(pol, g, w)
                eg = w * w * (1 - g) if pol[0] == "R" else 0
                ew = -w * g * (1 - g) if pol[1] in ("U", "N") else 0
                assert got == (ref[0] + eg, ref[1] + ew), pol


def test_uu_class_rest_point_solves_quintic():
    # U/U, U/N, N/U, N/N: weight component vanishes at w = (2+g)/(2+g^2); the gain
    # component then vanishes where 8(g - 1/2)(g^2 + 2)^2 + g^2 (1 - g)^2 = 0.
    for g in (Fr(1, 10), Fr(2, 5), Fr(7, 10)):
        w = (2 + g) / (2 + g * g)
        dg, dw = model2p.average_update(("U", "U"), g, w)
        assert dw == 0
        quint = 8 * (g - H) * (g * g + 2) ** 2 + g * g * (1 - g) ** 2
        # the gain component is proportional to the quintic with a positive factor
        assert (dg > 0) == (quint > 0) and (dg == 0) == (quint == 0)
