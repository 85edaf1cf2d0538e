"""Host logic of the CU shares (the GPU shares of section 4.1, enforced by a
partitioning layer as in section 5): the mask ekya_partition_mask builds for
a CU range.  Checked by brute force over both ways a driver may number CU
mask bits -- die by die (bit b on XCD b // R) or dealt round-robin over the
dies and then the shader engines (bit b on XCD b % X, engine (b // X) % S,
the amdgpu driver's order) -- that every XCD receives the same number of
CUs, that under the round-robin order the engines of every XCD differ by at
most one CU, that the count is the range's groups times the dies, and that
disjoint ranges never share a CU."""
import numpy as np
import pytest

from paper_2012_10557_amd import binding


def _bits(words, n_cu):
    return [b for b in range(n_cu) if (int(words[b // 32]) >> (b % 32)) & 1]


def _per_xcd(bits, n_cu, n_xcd, mapping):
    R = n_cu // n_xcd
    counts = [0] * n_xcd
    for b in bits:
        counts[b // R if mapping == "blocked" else b % n_xcd] += 1
    return counts


def _per_engine(bits, n_xcd, n_se):
    """(XCD, engine) -> CUs under the driver's round-robin order."""
    counts = {}
    for b in bits:
        key = (b % n_xcd, (b // n_xcd) % n_se)
        counts[key] = counts.get(key, 0) + 1
    return counts


SHAPES = [(256, 8, 4), (304, 8, 4), (32, 1, 4), (80, 2, 4), (64, 2, 4)]


@pytest.mark.parametrize("n_cu,n_xcd,n_se", SHAPES)
@pytest.mark.parametrize("begin,share", [(0.0, 1.0), (0.0, 0.1), (0.1, 0.3), (0.5, 0.5),
                                         (0.25, 0.25), (0.9, 0.1), (0.0, 0.02), (0.3, 0.7)])
def test_every_xcd_gets_the_groups_of_the_range(n_cu, n_xcd, n_se, begin, share):
    R = n_cu // n_xcd
    g0, g1 = round(begin * R), min(R, round((begin + share) * R))
    if g1 <= g0:
        with pytest.raises(ValueError):
            binding.ekya_partition_mask(n_cu, n_xcd, n_se, begin, share)
        return
    n, words = binding.ekya_partition_mask(n_cu, n_xcd, n_se, begin, share)
    bits = _bits(words, n_cu)
    assert n == len(bits) == (g1 - g0) * n_xcd
    assert _per_xcd(bits, n_cu, n_xcd, "blocked") == [g1 - g0] * n_xcd
    if R % n_xcd == 0:
        assert _per_xcd(bits, n_cu, n_xcd, "round_robin") == [g1 - g0] * n_xcd
    if R == n_xcd * n_se:
        # engines of every die differ by at most one CU under the driver's order
        pe = _per_engine(bits, n_xcd, n_se)
        for x in range(n_xcd):
            c = [pe.get((x, e), 0) for e in range(n_se)]
            assert max(c) - min(c) <= 1, (x, c)
            assert sum(c) == g1 - g0


def test_disjoint_ranges_select_disjoint_cus():
    """Delta = 0.1 steps (the evaluation's quantum): the ten shares of one GPU
    cover it without overlap; any split point gives complementary masks."""
    seen = set()
    for i in range(10):
        n, words = binding.ekya_partition_mask(256, 8, 4, i / 10, 0.1)
        bits = set(_bits(words, 256))
        assert not (bits & seen)
        seen |= bits
    assert seen == set(range(256))
    for cut in np.arange(0.1, 1.0, 0.1):
        _, a = binding.ekya_partition_mask(256, 8, 4, 0.0, float(cut))
        _, b = binding.ekya_partition_mask(256, 8, 4, float(cut), 1.0 - float(cut))
        A, B = set(_bits(a, 256)), set(_bits(b, 256))
        assert not (A & B) and A | B == set(range(256))


@pytest.mark.parametrize("args", [(256, 8, 4, -0.1, 0.5), (256, 8, 4, 1.0, 0.1),
                                  (256, 8, 4, 0.5, 0.6), (256, 8, 4, 0.0, 0.0),
                                  (250, 8, 4, 0.0, 1.0), (0, 1, 4, 0.0, 1.0), (256, 8, 0, 0.0, 1.0)])
def test_invalid_ranges_are_rejected(args):
    with pytest.raises(ValueError):
        binding.ekya_partition_mask(*args)


def test_groups_fill_engines_in_turn():
    """On the MI355X shape (8 dies of 4 engines of 8 CUs) group g = 4 k + s
    takes CU k of engine s on every die under the driver's order: the first
    four groups cover every (die, engine) pair once, and the range's CU
    indices per engine are the groups' k."""
    n, words = binding.ekya_partition_mask(256, 8, 4, 0.0, 4 / 32)
    bits = _bits(words, 256)
    assert sorted((b % 8, (b // 8) % 4) for b in bits) == [(x, e) for x in range(8) for e in range(4)]
    for g0, g1 in [(0, 32), (5, 13), (30, 32), (7, 8)]:
        _, words = binding.ekya_partition_mask(256, 8, 4, g0 / 32, (g1 - g0) / 32)
        bits = _bits(words, 256)
        want = sorted((x, g % 4) for g in range(g0, g1) for x in range(8))
        assert sorted((b % 8, (b // 8) % 4) for b in bits) == want
