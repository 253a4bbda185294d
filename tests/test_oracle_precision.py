"""Pins of the oracle's bfloat16 rounding: closed-form values around 1 and
at the format's edges, and brute-force nearest-neighbour search on the
bfloat16 grid for random float32 values."""
import numpy as np

from oracle.precision import round_bf16


def test_closed_form_values():
    u = 2.0 ** -7                      # bfloat16 spacing on [1, 2)
    cases = {
        1.0: 1.0,
        1.0 + u: 1.0 + u,              # representable
        1.0 + u / 2: 1.0,              # tie, even neighbour is 1.0
        1.0 + 3 * u / 2: 1.0 + 2 * u,  # tie, even neighbour is 1 + 2u
        1.0 + u / 2 + 2.0 ** -20: 1.0 + u,   # just above the tie
        -(1.0 + u / 2 + 2.0 ** -20): -(1.0 + u),
        2.0 - u / 4: 2.0,              # rounds up into the next binade
        0.0: 0.0,
        3.4e38: np.inf,                # past halfway above the largest finite bfloat16
    }
    for x, want in cases.items():
        got = round_bf16(np.float32(x))
        assert got == want, (x, got, want)
    assert np.isnan(round_bf16(np.float32(np.nan)))
    assert np.signbit(round_bf16(np.float32(-0.0)))


def _nearest_on_grid(x):
    """Brute force: the bfloat16 neighbours of x are multiples of its
    binade's spacing; pick the nearer, the even multiple on a tie."""
    x = float(x)
    if x == 0.0:
        return x
    e = np.floor(np.log2(abs(x)))
    sp = 2.0 ** (e - 7)
    lo = np.floor(abs(x) / sp) * sp
    hi = lo + sp
    d_lo, d_hi = abs(x) - lo, hi - abs(x)
    if d_lo < d_hi:
        m = lo
    elif d_hi < d_lo:
        m = hi
    else:
        m = lo if int(round(lo / sp)) % 2 == 0 else hi
    return np.copysign(m, x)


def test_matches_brute_force():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(3000).astype(np.float32),
        (rng.standard_normal(1000) * 1e-20).astype(np.float32),
        (rng.standard_normal(1000) * 1e20).astype(np.float32),
        # exact ties: a bfloat16 value plus half its spacing
        (np.float32(1.5) + np.float32(2.0 ** -8)) * np.float32(2.0) ** rng.integers(-30, 30, 500)
        .astype(np.float32),
    ])
    got = round_bf16(x)
    want = np.array([_nearest_on_grid(v) for v in x])
    assert np.array_equal(got, want)
    # the result is representable: its low 16 bits are zero as float32
    assert np.all((got.astype(np.float32).view(np.uint32) & 0xFFFF) == 0)
