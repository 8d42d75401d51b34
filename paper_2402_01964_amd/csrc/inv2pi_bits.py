"""Print the first 192 bits of the binary fraction of 1 / (2 pi) as the six
32-bit words of kInv2PiBits (nlb_internal.h), most significant first.

pi comes from Machin's formula pi = 16 atan(1/5) - 4 atan(1/239), summed in
exact integer arithmetic with 400 fraction bits plus guard bits, far more
than the 192 bits kept (the series truncation leaves an error of a few units
of 2^-400)."""

FRACTION_BITS = 400
GUARD_BITS = 32


def _atan_inv(n: int) -> int:
    """atan(1 / n) * 2^FRACTION_BITS (Gregory series, truncated)."""
    one = 1 << (FRACTION_BITS + GUARD_BITS)
    x = one // n
    total, k, sign = x, 1, -1
    while x:
        x //= n * n
        total += sign * (x // (2 * k + 1))
        sign, k = -sign, k + 1
    return total >> GUARD_BITS


def inv2pi_words(words: int = 6) -> list:
    pi = 16 * _atan_inv(5) - 4 * _atan_inv(239)          # pi * 2^FRACTION_BITS
    frac = (1 << (32 * words + FRACTION_BITS)) // (2 * pi)  # floor(2^(32 words) / (2 pi))
    return [(frac >> (32 * (words - 1 - i))) & 0xFFFFFFFF for i in range(words)]


if __name__ == "__main__":
    print(", ".join(f"0x{w:08x}u" for w in inv2pi_words()))
