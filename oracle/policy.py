"""Backward-state policies: which value each use reads.

Test infrastructure (see ``oracle/__init__``).

A use is a gradient computation that reads a rounded tensor; the policy chooses
per use between the original (U), the rounding the forward used (R) and a new
rounding from the same law (N) (Sec. 1; Sec. 3.1; App. B, first paragraph).
Policies over two uses are written "first use / second use", the first being
the use that needs the original (App. B).
"""
U, R, N = "U", "R", "N"
LETTERS = (U, R, N)


def read(letter, original, forward_rounding, fresh):
    """The value a use reads under policy letter ``letter``."""
    if letter == U:
        return original
    if letter == R:
        return forward_rounding
    if letter == N:
        return fresh
    raise ValueError(letter)


def parse(code):
    """'U/R' -> ('U', 'R')."""
    a, b = code.split("/")
    assert a in LETTERS and b in LETTERS, code
    return a, b
