"""Schedules of the level products (CPU only; the schedule is built on the host).

Every schedule the library would run is exported and checked against the
oracle's definition of the levels (section 2, equation (3)): level t is the sum
of DA_p DB_q over the pairs p + q = t (``exact.pairs_of_level``).  The check is
symbolic: the schedule is a bilinear form in the digits, and its coefficient of
DA_p DB_q in level t must be 1 for those pairs and 0 otherwise.  It also checks
that every combination is the sum of its two parents (disjoint digit sets),
that every GEMM job stays exact (k times its digit weight times (2^w - 1)^2
below 2^53), and that a planted mistake in a schedule is caught.
"""

import numpy as np
import pytest

from oracle import exact
from paper_2607_06881_amd import mdgemm as md

KARA = md.MDGEMM_KARATSUBA
KMIN = md.MDGEMM_KARATSUBA_MIN_TERMS

# (m, n, k, S, T, w): the workloads' shapes, digit counts and cutoffs (dd all
# pairs, dd, qd, td, od, hd, range-balanced dd, adaptive widths) and small odd cases
CASES = [
    (1024, 1024, 1024, 8, 14, 13), (4096, 4096, 4096, 8, 7, 13), (2048, 2048, 1024, 16, 15, 13),
    (8192, 8192, 512, 12, 11, 13), (256, 8192, 128, 32, 31, 13), (128, 8192, 64, 64, 63, 13),
    (2048, 2048, 2048, 13, 17, 13), (4096, 4096, 4096, 6, 5, 19), (2048, 2048, 1024, 11, 10, 19),
    (8192, 8192, 512, 8, 7, 20), (16, 16, 16, 1, 0, 13), (40, 50, 16, 2, 2, 13), (70, 9, 40, 3, 4, 13),
    (5000, 3000, 100, 5, 3, 13), (900, 1000, 300, 7, 9, 13), (64, 64, 33, 9, 16, 13), (512, 512, 70000, 10, 4, 13),
    (3, 3, 1, 4, 6, 25), (2048, 2048, 2048, 24, 23, 13), (4096, 300, 256, 20, 38, 13),
]


def popcount(x: int) -> int:
    return bin(int(x)).count("1")


def digits_of(mask: int, S: int):
    return [p for p in range(S) if (int(mask) >> p) & 1]


def coefficients(sch: dict, S: int, T: int) -> np.ndarray:
    """coef[t, p, q]: the schedule's coefficient of DA_p DB_q in level t.  With a
    k split every job appears once per k chunk, each covering a share of k:
    the chunks of one job together count once."""
    coef = np.zeros((T + 1, S, S), dtype=np.int64)
    vec_a = np.array([[(int(m) >> p) & 1 for p in range(S)] for m in sch["mask_a"]], dtype=np.int64)
    vec_b = np.array([[(int(m) >> q) & 1 for q in range(S)] for m in sch["mask_b"]], dtype=np.int64)
    pf, ent = sch["plane_first"], sch["entries"]
    for first, count, plane, chunk in sch["jobs"]:
        if chunk != 0:
            continue  # chunk 0 stands for the job; check_chunks sees that all chunks are there
        outer = np.zeros((S, S), dtype=np.int64)
        for a, b in sch["pairs"][first:first + count]:
            outer += np.outer(vec_a[a], vec_b[b])
        for e in range(pf[plane], pf[plane + 1]):
            level, c = ent[e]
            coef[level] += c * outer
    return coef


def check_chunks(sch: dict):
    """Every job appears with k chunks 0 .. ksplit-1, each chunk with the same
    pairs and level entries."""
    sigma = sch["info"]["ksplit"]
    groups = {}
    pf, ent = sch["plane_first"], sch["entries"]
    for first, count, plane, chunk in sch["jobs"]:
        key = (int(first), int(count), tuple(map(tuple, ent[pf[plane]:pf[plane + 1]].tolist())))
        groups.setdefault(key, []).append(int(chunk))
    for key, chunks in groups.items():
        assert sorted(chunks) == list(range(sigma)) * (len(chunks) // sigma), (key, chunks)


def expected(S: int, T: int) -> np.ndarray:
    want = np.zeros((T + 1, S, S), dtype=np.int64)
    for t in range(T + 1):
        for p, q in exact.pairs_of_level(t, S):
            want[t, p, q] = 1
    return want


def check_combinations(mask, parents, S):
    assert len(mask) >= S
    for c in range(S):
        assert int(mask[c]) == 1 << c and tuple(parents[c]) == (-1, -1)
    for c in range(S, len(mask)):
        a, b = parents[c]
        assert 0 <= a < c and 0 <= b < c, (c, a, b)
        assert int(mask[a]) & int(mask[b]) == 0
        assert int(mask[a]) | int(mask[b]) == int(mask[c])


@pytest.mark.parametrize("m,n,k,S,T,w", CASES)
@pytest.mark.parametrize("flags", [0, KARA, KMIN])
def test_schedule_computes_the_levels(m, n, k, S, T, w, flags):
    sch = md.mdgemm_schedule_export(m, n, k, S, T, bits=w, flags=flags)
    info = sch["info"]
    np.testing.assert_array_equal(coefficients(sch, S, T), expected(S, T))
    check_chunks(sch)
    check_combinations(sch["mask_a"], sch["parents_a"], S)
    check_combinations(sch["mask_b"], sch["parents_b"], S)
    # every pair belongs to exactly one job (per k chunk); planes are distinct
    assert sum(int(c) for _, c, _, ch in sch["jobs"] if ch == 0) == info["terms"]
    assert info["terms"] * info["ksplit"] == sum(int(c) for _, c, _, _ in sch["jobs"]) or info["ksplit"] == 1
    assert len({int(p) for _, _, p, _ in sch["jobs"]}) == len(sch["jobs"])
    # exactness of every job: k * sum |comb a| |comb b| * (2^w - 1)^2 < 2^53
    dmax = (1 << w) - 1
    for first, count, _, _ in sch["jobs"]:
        weight = sum(popcount(sch["mask_a"][a]) * popcount(sch["mask_b"][b]) for a, b in sch["pairs"][first:first + count])
        # (a pair schedule's jobs are its levels, covered by the library's level check)
        if not info["direct_levels"]:
            assert k * weight * dmax * dmax < 2**53
        assert weight <= info["max_job_weight"]


@pytest.mark.parametrize("m,n,k,S,T", [(4096, 4096, 4096, 8, 7), (1024, 1024, 1024, 8, 14),
                                       (2048, 2048, 1024, 16, 15), (8192, 8192, 512, 12, 11),
                                       (256, 8192, 128, 32, 31), (128, 8192, 64, 64, 63), (2048, 2048, 2048, 13, 17)])
def test_karatsuba_schedule_uses_fewer_products(m, n, k, S, T):
    pairs = md.mdgemm_schedule_info(m, n, k, S, T)
    kara = md.mdgemm_schedule_info(m, n, k, S, T, flags=KARA)
    kmin = md.mdgemm_schedule_info(m, n, k, S, T, flags=KMIN)
    assert pairs["terms"] == sum(len(exact.pairs_of_level(t, S)) for t in range(T + 1))
    # (a k split turns the pair schedule's level planes into planes with entries)
    assert pairs["direct_levels"] == int(pairs["ksplit"] == 1) and kmin["direct_levels"] == 0
    # the fewest products: well under the pair count; the cost model's choice
    # trades some products for fewer planes, entries and combinations, and keeps
    # the pair schedule for octo and hexa doubles at their short k (128, 64),
    # where the level accumulation of many planes would cost more
    assert kmin["terms"] < 0.8 * pairs["terms"], (kmin, pairs)
    if k >= 512:
        assert kara["direct_levels"] == 0 and kmin["terms"] <= kara["terms"] < pairs["terms"]
    else:
        assert kara == pairs


def test_cost_model_keeps_pairs_for_small_products():
    # 64^3 double-double: a combination panel costs about as much as a GEMM term
    assert md.mdgemm_schedule_info(64, 64, 64, 8, 14, flags=KARA)["direct_levels"] == 1
    assert md.mdgemm_schedule_info(64, 64, 64, 8, 14, flags=KMIN)["direct_levels"] == 0


def test_schedule_on_random_digits():
    """The schedule evaluated on random integer digits (Python ints) equals the
    oracle's level products of the same digits."""
    rng = np.random.default_rng(7)
    S, T, k = 16, 15, 1024
    sch = md.mdgemm_schedule_export(2048, 2048, k, S, T, flags=KMIN)
    da = [int(x) for x in rng.integers(-8191, 8192, size=S)]
    db = [int(x) for x in rng.integers(-8191, 8192, size=S)]
    comb_a = [sum(da[p] for p in digits_of(m, S)) for m in sch["mask_a"]]
    comb_b = [sum(db[q] for q in digits_of(m, S)) for m in sch["mask_b"]]
    planes = {}
    for first, count, plane, chunk in sch["jobs"]:
        if chunk == 0:
            planes[int(plane)] = sum(comb_a[a] * comb_b[b] for a, b in sch["pairs"][first:first + count])
    levels = [0] * (T + 1)
    pf, ent = sch["plane_first"], sch["entries"]
    for plane, v in planes.items():
        for e in range(pf[plane], pf[plane + 1]):
            levels[ent[e][0]] += int(ent[e][1]) * v
    DA = np.array(da, dtype=np.int64).reshape(S, 1, 1)
    DB = np.array(db, dtype=np.int64).reshape(S, 1, 1)
    want = [int(G[0][0]) for G in exact.level_products(DA, DB, T)]
    assert levels == want


def test_planted_schedule_mistakes_are_caught():
    S, T, k = 8, 7, 4096
    base = md.mdgemm_schedule_export(4096, 4096, k, S, T, flags=KARA)
    want = expected(S, T)
    # a wrong coefficient
    bad = {key: (v.copy() if isinstance(v, np.ndarray) else v) for key, v in base.items()}
    bad["entries"][0, 1] = -bad["entries"][0, 1]
    assert not np.array_equal(coefficients(bad, S, T), want)
    # a dropped pair (job count one short)
    bad = {key: (v.copy() if isinstance(v, np.ndarray) else v) for key, v in base.items()}
    j = int(np.argmax(bad["jobs"][:, 1] * (bad["jobs"][:, 3] == 0)))
    bad["jobs"][j, 1] -= 1
    assert not np.array_equal(coefficients(bad, S, T), want)
    # a combination whose digit set is off by one digit
    bad = {key: (v.copy() if isinstance(v, np.ndarray) else v) for key, v in base.items()}
    c = S  # first derived combination
    bad["mask_a"][c] = np.uint64(int(bad["mask_a"][c]) ^ 1)
    assert not np.array_equal(coefficients(bad, S, T), want)


def test_karatsuba_workspace_and_plan():
    m = n = k = 256
    pw = md.mdgemm_workspace_bytes(m, n, k, 2)
    kw = md.mdgemm_workspace_bytes(m, n, k, 2, flags=KMIN)
    assert 0 < pw < kw < 2**40
    # the adaptive width with the Karatsuba schedule picks a width whose schedule stays exact
    w, S, T = md.mdgemm_plan(4096, 4096, 4096, 2, slice_bits=md.MDGEMM_SLICE_BITS_AUTO, flags=KARA)
    info = md.mdgemm_schedule_info(4096, 4096, 4096, S, T, bits=w, flags=KARA)
    assert 13 <= w <= 26 and S * w >= 104 and T == S - 1
    assert 4096 * info["max_job_weight"] * ((1 << w) - 1) ** 2 < 2**53
    with pytest.raises(md.MdgemmError):
        md.mdgemm_schedule_info(64, 64, 4096, 8, 15, flags=KARA)  # cutoff beyond 2S - 2


def test_fp32_panels_only_when_exact():
    # the library keeps digit panels in FP32 exactly when every panel value, at
    # most (digits in the largest combination) (2^w - 1), is below 2^24
    for m, n, k, S, T, w, flags in [(4096, 4096, 4096, 8, 7, 13, 0), (4096, 4096, 4096, 8, 7, 13, KARA),
                                    (512, 512, 512, 4, 3, 24, 0), (512, 512, 512, 4, 3, 25, 0),
                                    (512, 512, 64, 8, 7, 20, KMIN), (512, 512, 16, 8, 7, 22, KMIN),
                                    (128, 8192, 64, 64, 63, 13, KMIN)]:
        info = md.mdgemm_schedule_info(m, n, k, S, T, bits=w, flags=flags)
        sch = md.mdgemm_schedule_export(m, n, k, S, T, bits=w, flags=flags)
        digits = max(popcount(x) for x in list(sch["mask_a"]) + list(sch["mask_b"]))
        assert info["max_digits"] == digits
        assert info["panels_f32"] == int(digits * (2**w - 1) < 2**24), (m, n, k, S, T, w, flags, digits)


def test_small_products_split_k():
    # 1024^3 double-double at 19-bit digits: 6 level jobs x 64 tiles would fill
    # only 384 of the 512 resident blocks; k is split so that the chip fills
    info = md.mdgemm_schedule_info(1024, 1024, 1024, 6, 5, bits=19)
    assert info["ksplit"] > 1 and info["direct_levels"] == 0
    assert info["jobs"] == 6 * info["ksplit"] and info["planes"] == info["jobs"]
    # big products keep whole k
    assert md.mdgemm_schedule_info(4096, 4096, 4096, 8, 7)["ksplit"] == 1
    # short k cannot be split below 8 k steps a chunk
    assert md.mdgemm_schedule_info(128, 128, 100, 8, 7)["ksplit"] == 1
    # the split schedule still computes the levels
    sch = md.mdgemm_schedule_export(1024, 1024, 1024, 6, 5, bits=19)
    np.testing.assert_array_equal(coefficients(sch, 6, 5), expected(6, 5))
    check_chunks(sch)
    sch = md.mdgemm_schedule_export(1024, 1024, 1024, 6, 5, bits=18, flags=KARA)
    assert sch["info"]["ksplit"] > 1
    np.testing.assert_array_equal(coefficients(sch, 6, 5), expected(6, 5))
    check_chunks(sch)
