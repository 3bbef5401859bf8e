"""The JS kernels' float64 exp (table-driven, Tang's method) rests on a
256-entry table of 2^(j/256) and a two-part ln2/256 written as literals in the
HIP source; this pins them to their exact values (Python's decimal module at
50 digits), independently of any GPU."""

import decimal
import os
import re

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2606_22768_amd", "csrc",
                   "js.hip")

decimal.getcontext().prec = 50


def _source():
    with open(SRC) as f:
        return f.read()


def _constant(text, name):
    m = re.search(r"constexpr double " + name + r" = ([0-9a-fA-Fx.p+-]+);", text)
    assert m, name
    return float.fromhex(m.group(1))


def test_exp2_fraction_table_is_correctly_rounded():
    text = _source()
    body = re.search(r"kExp2Frac\[kTab\] = \{(.*?)\};", text, re.S).group(1)
    vals = [float.fromhex(t) for t in re.findall(r"0x[0-9a-fA-F.]+p[+-]\d+", body)]
    assert len(vals) == 256 and re.search(r"constexpr int kTabBits = 8;", text)
    for j, v in enumerate(vals):
        exact = decimal.Decimal(2) ** (decimal.Decimal(j) / 256)
        assert v == float(exact), j          # float(Decimal) rounds to nearest
        assert abs(decimal.Decimal(v) - exact) <= decimal.Decimal(2) ** -53


def test_reduction_constants():
    text = _source()
    l1, l2 = _constant(text, "kExpL1"), _constant(text, "kExpL2")
    inv = _constant(text, "kExpInvL")
    part = decimal.Decimal(2).ln() / 256
    # the two parts carry ln2/256 to 2^-80 relative: times |n| < 2^19 that is
    # still far below a double's rounding of the reduced argument
    assert abs(decimal.Decimal(l1) + decimal.Decimal(l2) - part) < part * decimal.Decimal(2) ** -80
    # n * l1 is exact for |n| < 2^21 (the reduced arguments reach |n| < 2^19)
    mant = int.from_bytes(__import__("struct").pack(">d", l1), "big") & ((1 << 52) - 1)
    assert mant % (1 << 21) == 0
    assert inv == float(256 / decimal.Decimal(2).ln())
    assert _constant(text, "kExpRound") == 1.5 * 2.0 ** 52
