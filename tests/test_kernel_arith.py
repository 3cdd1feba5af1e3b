"""Integer identities the HIP kernels rely on, checked exhaustively on the CPU
over the domains the kernels use them on (test infrastructure: no GPU)."""


def test_entry_split_multiply_shift_is_exact():
    """The stage DP splits entry e of a stage's (segment, end layer) list into
    segment e // wd and end layer e % wd as (e * ceil(2^16 / wd)) >> 16; exact
    for every band width 1..128 and every e below 4 wd + 64 (four segments'
    entries plus the lanes past the last one)."""
    for wd in range(1, 129):
        m = (65536 + wd - 1) // wd
        assert m < 1 << 24   # a 24-bit multiply operand
        for e in range(4 * wd + 64):
            q = (e * m) >> 16
            assert q == e // wd and e - q * wd == e % wd, (wd, e)


def test_ceil_third_matches_definition():
    """ceil(c / 3) as (c + 2) // 3 for the non-negative stage costs."""
    for c in list(range(0, 1000)) + [10**12 + k for k in range(6)]:
        assert (c + 2) // 3 == -(-c // 3)
