"""Values printed in the paper (tests/golden/paper_constants.txt, each with its citation)
against the oracle's constants and the storage accounting."""
import os

import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_constants.txt")


def _constants():
    out = {}
    with open(GOLDEN) as fh:
        for line in fh:
            if line.strip() and not line.startswith("#"):
                name, value, _cite = line.split(maxsplit=2)
                out[name] = float(value)
    return out


def test_algorithm1_constants():
    c, p = _constants(), oracle.Params()
    assert p.log_lo == c["log_lo"] and p.log_hi == c["log_hi"]
    assert p.imb_floor == c["imb_floor"]
    assert p.varn_iters == int(c["varn_iters"])


def _bits_per_element(code_bits, aux_bits_per_group, group):
    return code_bits + aux_bits_per_group / group


def test_paper_bits_accounting():
    """App. D's figure follows from its stated contents: 2 + (8 + 8 + 16) / 128 = 2.25."""
    c = _constants()
    assert _bits_per_element(2, 8 + 8 + 16, int(c["group"])) == c["paper_bits_per_element"]


@pytest.mark.parametrize("bits,expect", [(2, 2.75), (4, 4.75)])
def test_library_format_accounting(bits, expect):
    """The library's tile stores three fp32 vectors of 128 per 128 x 128 tile (a, b per group,
    s2 per other-axis index), i.e. three fp32 values per group of 128 elements."""
    c = _constants()
    g = int(c["group"])
    assert oracle.tile_bytes(bits) * 8 / (g * 128) == expect
    assert _bits_per_element(bits, 3 * 32, g) == expect
