"""The synthetic workloads at full size, in the benchmark's launch
configuration (caller workspace from PyTorch, PyTorch's current stream).

Full-size outputs are checked where the oracle can follow them: exponents of
every row and column; digits of sampled rows of A and columns of B; level
products and final limbs of sampled output entries, bit-exact; the tolerance
4 k 2^-(53L-4) (|A||B|) against the exact rational product on those entries
(every limb count: the octo and hexa doubles take their default digit count,
34 and 66); and the nonoverlap property of every output element.  The
64^3 workload is checked on every entry.
"""

import numpy as np
import pytest
import torch

from checks import nonoverlap_all
from oracle import coracle, exact, pipeline
from paper_2607_06881_amd import mdgemm as md
from paper_2607_06881_amd import workloads

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _run(w):
    A_h, B_h = workloads.make_workload(w)
    A, B = torch.from_numpy(A_h).to(DEV), torch.from_numpy(B_h).to(DEV)
    opts = w.options()
    assert md.mdgemm_plan(w.m, w.n, w.k, w.limbs, **opts) == (13, w.slices, w.cutoff)
    ws = torch.empty(md.mdgemm_workspace_bytes(w.m, w.n, w.k, w.limbs, **opts), dtype=torch.uint8, device=DEV)
    C = md.mdgemm_ex(A, B, workspace=ws, **opts)
    torch.cuda.synchronize()
    return A_h, B_h, A, B, C


def _sample_entries(EA, EB, count, seed):
    rng = np.random.default_rng(seed)
    m, n = len(EA), len(EB)
    rows = {0, m - 1, int(np.argmin(EA)), int(np.argmax(EA))}
    cols = {0, n - 1, int(np.argmin(EB)), int(np.argmax(EB))}
    entries = {(i, j) for i in rows for j in cols}
    while len(entries) < count:
        entries.add((int(rng.integers(m)), int(rng.integers(n))))
    return sorted(entries)


@pytest.mark.parametrize("name", ["c0", "c1", "c2", "c3", "c4", "c5", "c6", "c7"])
def test_workload_full_size(name):
    w = workloads.WORKLOADS[name]
    print(f"[case] workload {name}: {w.description}", flush=True)
    A_h, B_h, A, B, C = _run(w)
    C_h = C.cpu().numpy()
    del C
    S, T, L = w.slices, w.cutoff, w.limbs

    # a1: every exponent
    EA_g = md.mdgemm_exponents(A[0], 0)
    EB_g = md.mdgemm_exponents(B[0], 1)
    EA = coracle.exponents(A_h[0], 0)
    EB = coracle.exponents(B_h[0], 1)
    assert np.array_equal(EA_g.cpu().numpy(), EA) and np.array_equal(EB_g.cpu().numpy(), EB)

    assert nonoverlap_all(C_h)
    assert np.isfinite(C_h).all()

    if name == "c0":
        ref = pipeline.full_reference(A_h, B_h, S, T)
        assert np.array_equal(C_h, ref["C"])
        entries = [(i, j) for i in range(0, w.m, 3) for j in range(0, w.n, 5)]
    else:
        entries = _sample_entries(EA, EB, 40, w.seed)
        ref = pipeline.reference_entries(A_h, B_h, S, T, entries)
        for (i, j), r in ref.items():
            assert C_h[:, i, j].tolist() == r["limbs"], (i, j)

        # a2: digits of sampled rows of A / columns of B
        rows = sorted({i for i, _ in entries})[:12]
        cols = sorted({j for _, j in entries})[:12]
        DA = md.mdgemm_split(A, EA_g, S, 0)
        DB = md.mdgemm_split(B, EB_g, S, 1)
        DA_rows = DA[:, rows, :].cpu().numpy()
        DB_cols = DB[:, :, cols].cpu().numpy()
        assert np.array_equal(DA_rows, coracle.split(np.ascontiguousarray(A_h[:, rows, :]), EA[rows], S, 0))
        assert np.array_equal(DB_cols, coracle.split(np.ascontiguousarray(B_h[:, :, cols]), EB[cols], S, 1))
        # a3: level products of the sampled entries
        DA_p = md.mdgemm_split_panel(A, EA_g, S, 0)
        DB_p = md.mdgemm_split_panel(B, EB_g, S, 1)
        # the panels hold the same digits (A transposed), zeros elsewhere
        assert torch.equal(DA_p[:, :w.k, :w.m], DA.transpose(1, 2))
        assert torch.equal(DB_p[:, :w.k, :w.n], DB)
        assert DA_p[:, w.k:, :].abs().sum().item() == 0 and DA_p[:, :, w.m:].abs().sum().item() == 0
        assert DB_p[:, w.k:, :].abs().sum().item() == 0 and DB_p[:, :, w.n:].abs().sum().item() == 0
        del DA, DB
        G = md.mdgemm_slice_gemm(DA_p, DB_p, w.m, w.n, w.k, T)
        ii = torch.tensor([i for i, _ in entries], device=DEV)
        jj = torch.tensor([j for _, j in entries], device=DEV)
        G_s = G[:, ii, jj].cpu().numpy()
        del DA_p, DB_p, G
        torch.cuda.empty_cache()
        for e, (i, j) in enumerate(entries):
            assert G_s[:, e].astype(np.int64).tolist() == ref[(i, j)]["levels"], (i, j)

    # final limbs against the exact product
    worst = 0.0
    for (i, j) in entries[:40]:
        want, mag = exact.exact_product(A_h, B_h, i, j)
        err = abs(exact.value(C_h[:, i, j]) - want)
        bound = exact.tolerance(w.k, L, mag)
        assert err <= bound, (i, j, float(err / bound))
        worst = max(worst, float(err / bound))
    print(f"[result] {name}: max |C - C_exact| / bound over {min(len(entries), 40)} entries = {worst:.3e}",
          flush=True)


def _tile_entries(m, n, seed, tile=128):
    """One random output entry inside every tile x tile block, plus the corners."""
    rng = np.random.default_rng(seed)
    out = {(0, 0), (m - 1, n - 1), (0, n - 1), (m - 1, 0)}
    for ti in range(0, m, tile):
        for tj in range(0, n, tile):
            out.add((ti + int(rng.integers(min(tile, m - ti))), tj + int(rng.integers(min(tile, n - tj)))))
    return sorted(out)


@pytest.mark.parametrize("name,k", [("c2", 64), ("c4", 32)])
def test_hot_path_levels_on_the_full_tile_grid(name, k):
    """The stages mdgemm_ex itself runs (read back from its caller workspace:
    exponents, the FP32 digit panels of slice_gemm32_kernel, the level planes),
    compared over the whole matrix with the oracle, on the workload's full grid
    of output tiles (c2: 32 x 32 tiles of 128 x 128, c4: 64 x 64) in the
    benchmark's launch configuration, at a reduced k so that the oracle's level
    products take seconds."""
    w = workloads.WORKLOADS[name]
    m, n, L, S, T = w.m, w.n, w.limbs, w.slices, w.cutoff
    print(f"[case] hot-path levels, full tile grid: {name} {m}x{k}x{n} L={L} S={S} T={T}", flush=True)
    A_h, B_h = workloads.make_workload(w, k=k)
    opts = w.options()
    info = md.mdgemm_schedule_info(m, n, k, S, T)
    assert info["panels_f32"] == 1 and info["ksplit"] == 1  # no k split: the full-size launch shape
    ws = torch.empty(md.mdgemm_workspace_bytes(m, n, k, L, **opts), dtype=torch.uint8, device=DEV)
    A, B = torch.from_numpy(A_h).to(DEV), torch.from_numpy(B_h).to(DEV)
    C = md.mdgemm_ex(A, B, workspace=ws, **opts)
    torch.cuda.synchronize()
    parts = md.workspace_parts(ws, m, n, k, L, **opts)
    lay = parts["layout"]
    assert lay["panel_bytes"] == 4 and lay["direct_levels"] == 1 and lay["planes"] == T + 1

    EA, EB = coracle.exponents(A_h[0], 0), coracle.exponents(B_h[0], 1)
    assert np.array_equal(parts["EA"].cpu().numpy(), EA) and np.array_equal(parts["EB"].cpu().numpy(), EB)
    DA = coracle.split(A_h, EA, S, 0)
    DB = coracle.split(B_h, EB, S, 1)
    DA_p = parts["DA"][:S].cpu().numpy()
    DB_p = parts["DB"][:S].cpu().numpy()
    assert np.array_equal(DA_p[:, :k, :m], DA.transpose(0, 2, 1)) and np.array_equal(DB_p[:, :k, :n], DB)
    assert not DA_p[:, k:, :].any() and not DA_p[:, :, m:].any()
    assert not DB_p[:, k:, :].any() and not DB_p[:, :, n:].any()
    del DA_p, DB_p
    G = parts["G"].cpu().numpy()
    del parts, ws
    torch.cuda.empty_cache()
    G_ref = pipeline.levels_rewritten(DA, DB, T)
    bad = np.argwhere((G != G_ref).any(axis=0))
    assert len(bad) == 0, f"{len(bad)} entries differ, first {bad[:5].tolist()}"
    del G, G_ref
    # the limbs of one entry per tile
    C_h = C.cpu().numpy()
    assert nonoverlap_all(C_h)
    entries = _tile_entries(m, n, w.seed)[::4]
    ref = pipeline.reference_entries(A_h, B_h, S, T, entries)
    for (i, j), r in ref.items():
        assert C_h[:, i, j].tolist() == r["limbs"], (i, j)


@pytest.mark.parametrize("name", ["c2", "c4"])
def test_hot_path_levels_full_size(name):
    """At the benchmark's full size: the level planes mdgemm_ex forms with
    slice_gemm32_kernel equal, over the whole matrix, those of the FP64-panel
    kernel run from the stage entry points, and equal the oracle's levels at
    one entry of every 128 x 128 output tile."""
    w = workloads.WORKLOADS[name]
    m, n, k, L, S, T = w.m, w.n, w.k, w.limbs, w.slices, w.cutoff
    print(f"[case] hot-path levels, full size: {name} {m}x{k}x{n} L={L} S={S} T={T}", flush=True)
    A_h, B_h = workloads.make_workload(w)
    opts = w.options()
    ws = torch.empty(md.mdgemm_workspace_bytes(m, n, k, L, **opts), dtype=torch.uint8, device=DEV)
    A, B = torch.from_numpy(A_h).to(DEV), torch.from_numpy(B_h).to(DEV)
    C = md.mdgemm_ex(A, B, workspace=ws, **opts)
    torch.cuda.synchronize()
    parts = md.workspace_parts(ws, m, n, k, L, **opts)
    assert parts["layout"]["panel_bytes"] == 4 and parts["layout"]["direct_levels"] == 1
    entries = _tile_entries(m, n, w.seed + 7)
    ii = torch.tensor([i for i, _ in entries], device=DEV)
    jj = torch.tensor([j for _, j in entries], device=DEV)
    G_s = parts["G"][:, ii, jj].cpu().numpy()
    # the FP64-panel kernel from the stage entry points, compared on the GPU
    EA_g = md.mdgemm_exponents(A[0], 0)
    EB_g = md.mdgemm_exponents(B[0], 1)
    assert torch.equal(EA_g, parts["EA"]) and torch.equal(EB_g, parts["EB"])
    DA_p = md.mdgemm_split_panel(A, EA_g, S, 0)
    DB_p = md.mdgemm_split_panel(B, EB_g, S, 1)
    kp = parts["layout"]["kp"]
    assert torch.equal(DA_p[:, :k, :].float(), parts["DA"][:S, :k, :])
    assert torch.equal(DB_p[:, :k, :].float(), parts["DB"][:S, :k, :])
    assert not parts["DA"][:S, k:kp, :].any().item() and not parts["DB"][:S, k:kp, :].any().item()
    G64 = md.mdgemm_slice_gemm(DA_p, DB_p, m, n, k, T)
    del DA_p, DB_p
    same = torch.equal(G64, parts["G"])
    del G64
    assert same, "level planes of slice_gemm32_kernel and slice_gemm_kernel differ"
    C_h = C.cpu().numpy()
    del parts, ws, C
    torch.cuda.empty_cache()
    ref = pipeline.reference_entries(A_h, B_h, S, T, entries)
    for e, (i, j) in enumerate(entries):
        assert G_s[:, e].astype(np.int64).tolist() == ref[(i, j)]["levels"], (i, j)
        assert C_h[:, i, j].tolist() == ref[(i, j)]["limbs"], (i, j)
    print(f"[result] {name}: {len(entries)} entries (one per tile) bit-exact; full planes equal the FP64-panel "
          f"kernel's", flush=True)


@pytest.mark.parametrize("name", ["c2", "c3", "c4", "c7"])
def test_workload_adaptive_width(name):
    # The same workloads with the adaptive width: fewer, wider digits, sampled
    # entries bit-exact against the oracle's chain at that width, within the
    # stated tolerance.
    w = workloads.WORKLOADS[name]
    opts = w.options(adaptive=True)
    bits, S, T = md.mdgemm_plan(w.m, w.n, w.k, w.limbs, **opts)
    assert (bits, S, T) == exact.plan(w.limbs, w.k, **opts)
    print(f"[case] workload {name} adaptive width: w={bits} S={S} T={T}", flush=True)
    A_h, B_h = workloads.make_workload(w)
    A, B = torch.from_numpy(A_h).to(DEV), torch.from_numpy(B_h).to(DEV)
    ws = torch.empty(md.mdgemm_workspace_bytes(w.m, w.n, w.k, w.limbs, **opts), dtype=torch.uint8, device=DEV)
    C_h = md.mdgemm_ex(A, B, workspace=ws, **opts).cpu().numpy()
    del ws
    assert nonoverlap_all(C_h) and np.isfinite(C_h).all()
    EA, EB = coracle.exponents(A_h[0], 0), coracle.exponents(B_h[0], 1)
    entries = _sample_entries(EA, EB, 24, w.seed + 50)
    ref = pipeline.reference_entries(A_h, B_h, S, T, entries, bits)
    worst = 0.0
    for (i, j), r in ref.items():
        assert C_h[:, i, j].tolist() == r["limbs"], (i, j)
        want, mag = exact.exact_product(A_h, B_h, i, j)
        err = abs(exact.value(C_h[:, i, j]) - want)
        bound = exact.tolerance(w.k, w.limbs, mag)
        assert err <= bound, (i, j, float(err / bound))
        worst = max(worst, float(err / bound))
    print(f"[result] {name} adaptive width: max |C - C_exact| / bound = {worst:.3e}", flush=True)


def test_workload_line_spread():
    # the measured range of the wide-range workload's lines, against the oracle
    w = workloads.WORKLOADS["c7"]
    print("[case] line spread c7", flush=True)
    A_h, B_h = workloads.make_workload(w)
    EA, SA = md.mdgemm_line_spread(torch.from_numpy(A_h[0]).to(DEV), 0)
    EB, SB = md.mdgemm_line_spread(torch.from_numpy(B_h[0]).to(DEV), 1)
    assert np.array_equal(EA.cpu().numpy(), coracle.exponents(A_h[0], 0))
    assert np.array_equal(EB.cpu().numpy(), coracle.exponents(B_h[0], 1))
    rows, cols = [0, 5, 1000, w.m - 1], [0, 77, w.n - 1]
    assert SA.cpu().numpy()[rows].tolist() == exact.line_spread(A_h[0, rows, :], 0).tolist()
    assert SB.cpu().numpy()[cols].tolist() == exact.line_spread(B_h[0][:, cols], 1).tolist()
    assert w.range_bits - 10 <= int(SA.min()) and int(SA.max()) <= w.range_bits + 30  # N(0,1) tails add bits


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c7"])
def test_workload_karatsuba(name):
    # The same workloads with the Karatsuba schedule of the level products
    # (fewer GEMMs of digit sums, levels formed exactly from their planes):
    # sampled entries bit-exact against the oracle's chain, which does not
    # depend on the schedule.  (For the octo/hexa-double workloads the cost
    # model keeps the pair schedule.)
    w = workloads.WORKLOADS[name]
    opts = w.options()
    info = md.mdgemm_schedule_info(w.m, w.n, w.k, w.slices, w.cutoff, flags=md.MDGEMM_KARATSUBA)
    print(f"[case] workload {name} karatsuba: {info['terms']} products instead of {w.pairs}, "
          f"{info['planes']} planes", flush=True)
    assert info["terms"] < w.pairs
    A_h, B_h = workloads.make_workload(w)
    A, B = torch.from_numpy(A_h).to(DEV), torch.from_numpy(B_h).to(DEV)
    ws = torch.empty(md.mdgemm_workspace_bytes(w.m, w.n, w.k, w.limbs, flags=md.MDGEMM_KARATSUBA, **opts),
                     dtype=torch.uint8, device=DEV)
    C_h = md.mdgemm_ex(A, B, workspace=ws, flags=md.MDGEMM_KARATSUBA, **opts).cpu().numpy()
    del ws
    torch.cuda.empty_cache()
    assert nonoverlap_all(C_h) and np.isfinite(C_h).all()
    EA, EB = coracle.exponents(A_h[0], 0), coracle.exponents(B_h[0], 1)
    entries = _sample_entries(EA, EB, 16, w.seed + 90)
    ref = pipeline.reference_entries(A_h, B_h, w.slices, w.cutoff, entries)
    for (i, j), r in ref.items():
        assert C_h[:, i, j].tolist() == r["limbs"], (i, j)


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5", "c7"])
def test_workload_int8(name):
    # The same workloads with the int8 level products (7-bit digits, exact int32
    # sums): sampled entries bit-exact against the oracle's chain at that width
    # and within the stated tolerance, and the whole C bit-identical to the FP64
    # path run with the same digits (hexa-double needs more than 64 digits of
    # 7 bits and is refused).
    w = workloads.WORKLOADS[name]
    rb = {"range_bits": w.range_bits} if w.range_bits else {}
    bits, S, T = md.mdgemm_plan(w.m, w.n, w.k, w.limbs, flags=md.MDGEMM_INT8, **rb)
    assert (bits, S, T) == exact.plan(w.limbs, w.k, int8=True, **rb)
    print(f"[case] workload {name} int8: w={bits} S={S} T={T}", flush=True)
    A_h, B_h = workloads.make_workload(w)
    A, B = torch.from_numpy(A_h).to(DEV), torch.from_numpy(B_h).to(DEV)
    C8 = md.mdgemm_ex(A, B, flags=md.MDGEMM_INT8, **rb).cpu().numpy()
    torch.cuda.empty_cache()
    D = -(-w.range_bits // bits) if w.range_bits else 0
    C64 = md.mdgemm_ex(A, B, slice_bits=bits, slices=S - D, cutoff=T, **rb).cpu().numpy()
    torch.cuda.empty_cache()
    assert np.array_equal(C8, C64)
    assert nonoverlap_all(C8) and np.isfinite(C8).all()
    EA, EB = coracle.exponents(A_h[0], 0), coracle.exponents(B_h[0], 1)
    entries = _sample_entries(EA, EB, 12, w.seed + 95)
    ref = pipeline.reference_entries(A_h, B_h, S, T, entries, bits)
    for (i, j), r in ref.items():
        assert C8[:, i, j].tolist() == r["limbs"], (i, j)
        if w.limbs <= 4:
            want, mag = exact.exact_product(A_h, B_h, i, j)
            assert abs(exact.value(C8[:, i, j]) - want) <= exact.tolerance(w.k, w.limbs, mag), (i, j)
