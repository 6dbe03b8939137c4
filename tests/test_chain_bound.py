"""The exactness bound behind chained binary32 accumulation in the NVFP4 products.

The GPU products add the MFMA results of a group of 16-element blocks in one
binary32 register when rho * sigma < 2^48, with (per row, over the group's
blocks) rho = sum_b n2_b 4^(e_b - e_min), n2_b = sum (2q)^2 M^2 and the E4M3
scale written M 2^(e - 10).  The claim: every partial sum of the group's
products, in any order, is then an integer multiple of
u = 2^(ea_min + eb_min - 22) below 2^24 u in magnitude, so binary32 holds it
exactly.  These tests check the claim with integer arithmetic (independent of
the GPU code), including rows that meet Cauchy-Schwarz with equality, and that
a binary32 accumulation in random orders then equals the exact sum.
"""
import numpy as np
import pytest

K2 = np.array([0, 1, 2, 3, 4, 6, 8, 12])   # 2q for the eight E2M1 magnitudes


def scale_parts(code):
    """(M, e) of a non-zero E4M3 code: value = M 2^(e - 10)."""
    ef, mf = (code >> 3) & 15, code & 7
    return (8 + mf, ef) if ef else (mf, 1)


def rho_of(k2, codes):
    """rho of one row over a group: k2 [G, 16] signed 2q values, codes [G] scale codes."""
    parts = [scale_parts(int(c)) for c in codes]
    emin = min(e for (_, e) in parts)
    return sum(int(np.sum(k2[b].astype(np.int64) ** 2)) * parts[b][0] ** 2 * 4 ** (parts[b][1] - emin)
               for b in range(len(codes))), emin


def products_in_units(ka, ca, kb, cb):
    """Exact products of the two rows over the group, in units u (Python ints)."""
    pa = [scale_parts(int(c)) for c in ca]
    pb = [scale_parts(int(c)) for c in cb]
    ea0 = min(e for (_, e) in pa)
    eb0 = min(e for (_, e) in pb)
    out = []
    for b in range(len(ca)):
        (ma, ea), (mb, eb) = pa[b], pb[b]
        f = ma * mb * 2 ** ((ea - ea0) + (eb - eb0))
        out += [int(x) * int(y) * f for x, y in zip(ka[b], kb[b])]
    return out, ea0, eb0


def random_row(rng, groups, spread):
    k2 = rng.choice(K2, size=(groups, 16)) * rng.choice([-1, 1], size=(groups, 16))
    e = rng.integers(1, 1 + spread + 1, size=groups)
    m = rng.integers(0, 8, size=groups)
    codes = (np.minimum(e, 15) << 3) | m
    return k2, codes


def check_pair(ka, ca, kb, cb, rng):
    rho, _ = rho_of(ka, ca)
    sigma, _ = rho_of(kb, cb)
    prods, ea0, eb0 = products_in_units(ka, ca, kb, cb)
    total_abs = sum(abs(p) for p in prods)
    # Cauchy-Schwarz: sum |a b| <= sqrt(rho sigma) in units of u
    assert total_abs * total_abs <= rho * sigma
    if rho * sigma >= 2 ** 48:
        return False
    assert total_abs < 2 ** 24
    exact = sum(prods)
    u = 2.0 ** (ea0 + eb0 - 22)
    for _ in range(4):
        order = rng.permutation(len(prods))
        acc = np.float32(0.0)
        for i in order:
            acc = np.float32(acc + np.float32(prods[i] * u))   # each product is a binary32 value
        assert float(acc) == exact * u
    return True


@pytest.mark.parametrize("groups", [4, 8])
def test_chain_bound_random_rows(groups):
    rng = np.random.default_rng(11 + groups)
    chained = 0
    for t in range(300):
        spread = int(rng.integers(0, 6))
        ka, ca = random_row(rng, groups, spread)
        kb, cb = random_row(rng, groups, spread)
        chained += check_pair(ka, ca, kb, cb, rng)
    assert chained > 50   # the bound is exercised, not vacuous


def test_chain_bound_tight_rows():
    """Aligned maximal rows reach Cauchy-Schwarz with equality; raising one block's
    exponent walks rho sigma up to and past 2^48."""
    rng = np.random.default_rng(5)
    seen_close = False
    for lift in range(0, 6):
        k = np.full((4, 16), 12)
        codes = np.array([(1 + lift) << 3 | 7, 1 << 3 | 7, 1 << 3 | 7, 1 << 3 | 7])
        rho, _ = rho_of(k, codes)
        prods, _, _ = products_in_units(k, codes, k, codes)
        assert sum(prods) ** 2 == rho * rho          # equality case of Cauchy-Schwarz
        if check_pair(k, codes, k, codes, rng) and rho * rho > 2 ** 46:
            seen_close = True
    assert seen_close


def test_chain_bound_single_block_always_exact():
    """One block alone never needs the bound: its sum stays below 2^19 units."""
    k = np.full((1, 16), 12)
    codes = np.array([15 << 3 | 6])   # largest finite E4M3 scale, 448
    rho, _ = rho_of(k, codes)
    assert rho == 16 * 144 * 196 and rho < 2 ** 19
