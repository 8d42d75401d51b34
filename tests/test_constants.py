"""Constants baked into the kernels, pinned to independent computations."""
import re
from decimal import Decimal, getcontext
from pathlib import Path

ROOT = Path(__file__).resolve().parents[1]


def _header_words():
    text = (ROOT / "paper_2402_01964_amd" / "csrc" / "nlb_internal.h").read_text()
    body = re.search(r"kInv2PiBits\[6\]\s*=\s*\{([^}]*)\}", text).group(1)
    return [int(w.strip().rstrip("u"), 16) for w in body.split(",") if w.strip()]


def _pi_gauss_legendre(digits: int) -> Decimal:
    """pi by the Gauss-Legendre (arithmetic-geometric mean) iteration, which
    doubles the correct digits per step -- a different algorithm from the
    arctangent series the table generator uses."""
    getcontext().prec = digits + 10
    a, b, t, p = Decimal(1), Decimal(1) / Decimal(2).sqrt(), Decimal(1) / 4, Decimal(1)
    for _ in range(10):                      # 2^10 > digits / 1.4 correct digits
        a_next = (a + b) / 2
        b = (a * b).sqrt()
        t -= p * (a - a_next) ** 2
        a, p = a_next, 2 * p
    return (a + b) ** 2 / (4 * t)


def test_inv2pi_bits_match_gauss_legendre_pi():
    """The 192 fraction bits of 1 / (2 pi) used by the wide-argument cosine
    equal floor(2^192 / (2 pi)) for pi to 90 decimal digits (about 299 bits)."""
    pi = _pi_gauss_legendre(90)
    getcontext().prec = 100
    want = int((Decimal(2) ** 192) / (2 * pi))
    words = _header_words()
    got = 0
    for w in words:
        got = (got << 32) | w
    assert len(words) == 6
    assert got == want


def test_inv2pi_generator_agrees_with_header():
    import importlib.util
    spec = importlib.util.spec_from_file_location(
        "inv2pi_bits", ROOT / "paper_2402_01964_amd" / "csrc" / "inv2pi_bits.py")
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    assert mod.inv2pi_words() == _header_words()
