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


def test_reciprocal_floor_division_is_exact():
    """The stage DP's sweep bound floor(x / d), d = B - 1 in 1..63, taken as the
    truncated double product x * RN(1 / d) corrected by one integer step either
    way, equals the floor for x below 2^52 (IEEE double products on both sides:
    numpy's float64 multiply rounds to nearest like the GPU's)."""
    import numpy as np

    rng = np.random.default_rng(7)
    xs = np.concatenate([
        np.arange(0, 4096, dtype=np.int64),
        rng.integers(0, 1 << 52, size=200_000, dtype=np.int64),
        (1 << 52) - 1 - np.arange(0, 4096, dtype=np.int64),
    ])
    for d in range(1, 64):
        rd = np.float64(1.0) / np.float64(d)
        # near-multiples of d, where a truncation error would show first
        k = rng.integers(0, ((1 << 52) - 1) // d, size=20_000, dtype=np.int64)
        x = np.concatenate([xs, k * d, k * d - 1, k * d + d - 1])
        x = x[(x >= 0) & (x < (1 << 52))]
        q = (x.astype(np.float64) * rd).astype(np.int64)
        r = x - q * d
        assert np.all(np.abs(q - x // d) <= 1), d
        q = np.where(r < 0, q - 1, np.where(r >= d, q + 1, q))
        assert np.array_equal(q, x // d), d


def test_cap_count_estimate_is_corrected_to_the_floor():
    """The class split's count floor(room / act), act <= room < 64 act: both
    shifted right until room fits 32 bits, an fp32 product with act's
    approximate reciprocal (taken here with a relative error of 2^-20 either
    way, well beyond the hardware's), clamped to [1, 63], then corrected by one
    integer step either way, equals the floor."""
    import numpy as np

    rng = np.random.default_rng(11)
    n = 200_000
    act = rng.integers(1, 1 << 45, size=n, dtype=np.int64)
    mult = rng.uniform(1.0, 64.0, size=n)
    room = np.minimum((act.astype(np.float64) * mult).astype(np.int64), act * 64 - 1)
    # exact multiples and their neighbours, where the estimate's error shows first
    k = rng.integers(1, 64, size=n, dtype=np.int64)
    act = np.concatenate([act, act, act])
    room = np.concatenate([room, np.minimum(k * act[:n], act[:n] * 64 - 1), np.maximum(k * act[:n] - 1, act[:n])])
    ok = (room >= act) & (room < 64 * act)
    room, act = room[ok], act[ok]
    hi = (room.astype(np.uint64) >> np.uint64(32)).astype(np.int64)
    sh = np.where(hi > 0, np.floor(np.log2(np.maximum(hi, 1))).astype(np.int64) + 1, 0)
    r32 = (room >> sh).astype(np.float32)
    a32 = (act >> sh).astype(np.float32)
    for err in (1.0 - 2.0 ** -20, 1.0 + 2.0 ** -20):
        rcp = (np.float32(1.0) / a32) * np.float32(err)
        m = (r32 * rcp).astype(np.float32).astype(np.int64)
        m = np.clip(m, 1, 63)
        m = np.where(m * act > room, m - 1, np.where((m + 1) * act <= room, m + 1, m))
        assert np.array_equal(m, room // act)
