"""The host planner's choices at the benchmarked shapes (no GPU): the planner
source is compiled with its kernel launchers stubbed out (tests/planner) and
asked for the plan of each descriptor. These pin the execution paths that the
measurements in the design notes were taken on, and check that every plan
fits one compute unit's LDS and the chip's resident workgroup slots."""
import json
import random
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_10805_amd", "csrc")
LDS_FLOATS = 160 * 1024 // 4


def lds_wgs(floats):
    """Workgroups per CU an LDS size allows: 128 granules of 1280 bytes per CU
    (measured on MI355X: three workgroups of 53760 bytes fit, of 53888 two)."""
    return 128 // -(-floats // 320)


@pytest.fixture(scope="module")
def planner(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("needs g++")
    exe = str(tmp_path_factory.mktemp("planner") / "plan_dump")
    subprocess.run([gxx, "-O1", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include",
                    "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-x", "c++",
                    os.path.join(ROOT, "tests", "planner", "plan_dump.cpp"), "-o", exe,
                    "-L", "/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"], check=True,
                   capture_output=True)

    def plan(B, C, H, W, k, L, dtype=0):
        out = subprocess.run([exe], input=f"{B} {C} {H} {W} {k} {L} {dtype}\n", capture_output=True, text=True,
                             check=True, timeout=60).stdout
        return json.loads(out.strip().splitlines()[-1])
    return plan


def test_headline_workload_plan(planner):
    """B64 C96 56x56 k5 L3 fp32: the forward holds one plane per workgroup in
    one round of 4x4 tiles, levels >= 3 sharing level 1's round; the backward
    is the gradient pass (one resident plane, one block round) plus dx by the
    forward with rotated taps; no workspace for the forward."""
    p = planner(64, 96, 56, 56, 5, 3)
    assert p["fwd_mode"] == "resident" and p["fwd_PP"] == 1 and p["fwd_one_round"] == 1
    assert p["fwd_merge_deep"] == 1
    # 14 output tiles per row, laid out over 16 lanes (one round, four wavefronts either way)
    assert p["fwd_tiles_x"] == 14 and p["fwd_tiles_xl"] == 16
    assert p["fwd_ws"] == 0
    assert p["grad_pass"] == 1 and p["grad_levels"] == 3 and p["grad_coarse"] == 0
    assert p["grad_PP"] == 1 and p["grad_rounds"] == 1
    # four workgroups per CU fit in LDS
    assert lds_wgs(p["fwd_lds_floats"]) >= 4


@pytest.mark.parametrize("C,H,L,fwd_mode", [(96, 56, 5, "resident"), (192, 28, 4, "resident"),
                                            (192, 28, 5, "split"), (384, 14, 3, "resident"),
                                            (384, 14, 4, "split"), (768, 7, 3, "tiny")])
def test_convnext_stage_modes(planner, C, H, L, fwd_mode):
    p = planner(128, C, H, H, 5, L)
    assert p["fwd_mode"] == fwd_mode


def test_tile_row_padding_keeps_the_busy_wavefronts(planner):
    """Padding tile rows to 8 lanes is skipped where it would put work on more
    wavefronts: 12 x 12 planes have 3 tiles per row (at L = 4, 16 planes: 144
    tiles on three wavefronts; padded, more)."""
    p = planner(128, 192, 12, 12, 5, 4)
    assert p["fwd_mx_rounds"] == 0 and p["fwd_one_round"] == 1
    assert p["fwd_tiles_xl"] == p["fwd_tiles_x"] == 3
    p = planner(64, 192, 28, 28, 5, 1)
    assert p["fwd_tiles_xl"] == 8


def test_small_planes_take_mixed_rounds(planner):
    """Planes of at most 16 x 16 run the forward with mixed task rounds: at
    14 x 14 L = 1, eight planes' 128 output tiles and 128 level-1 tiles fill
    one round of 256 lanes; the split 14 x 14 L = 4 forward's level-1 pass is
    the same plan. Larger planes keep the fused kernel."""
    p = planner(128, 384, 14, 14, 5, 1)
    assert p["fwd_mode"] == "resident" and p["fwd_mx_rounds"] == 1 and p["fwd_PP"] == 8
    assert sorted(map(tuple, p["fwd_mx_seg"][0])) == [(1, 0, 0, 128)] + [(2, 1, q, 32) for q in range(4)]
    p = planner(128, 384, 14, 14, 5, 4)
    assert p["fwd_mode"] == "split" and p["fwd_mx_rounds"] == 1
    for H, L in [(56, 3), (28, 3), (20, 3)]:
        assert planner(64, 96, H, H, 5, L)["fwd_mx_rounds"] == 0


def test_gradient_pass_level1_tiles_and_shed(planner):
    """The gradient pass takes level 1 in 2 x 2 site tiles where the smaller
    footprint fits three workgroups per CU (B64 C192 28 x 28 L1: four planes
    in 13440 floats instead of five in 16800), not where it would trade
    workgroups for planes (B128 C384 12 x 12 L2 keeps ten planes at three per
    CU). A single level above m = 2 goes to the coarse sub-problem from
    18432 planes on (28 x 28 L3: B128 C192 yes, B64 C192 no)."""
    p = planner(64, 192, 28, 28, 5, 1)
    assert p["grad_PP"] == 4 and lds_wgs(p["grad_lds_floats"]) == 3
    p = planner(128, 384, 12, 12, 5, 2)
    assert p["grad_PP"] == 10 and lds_wgs(p["grad_lds_floats"]) == 3
    p = planner(128, 192, 28, 28, 5, 3)
    assert p["grad_levels"] == 2 and p["grad_coarse"] == 1
    p = planner(64, 192, 28, 28, 5, 3)
    assert p["grad_levels"] == 3 and p["grad_coarse"] == 0


@pytest.fixture(scope="module")
def mixed_check(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("needs g++")
    exe = str(tmp_path_factory.mktemp("mixed") / "mixed_check")
    subprocess.run([gxx, "-O1", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include",
                    "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-x", "c++",
                    os.path.join(ROOT, "tests", "planner", "mixed_check.cpp"), "-o", exe,
                    "-L", "/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"], check=True,
                   capture_output=True)
    return exe


def test_mixed_round_plans_hold_their_invariants(mixed_check):
    """Every mixed-round plan over 3000 seeded random small-plane problems
    (and the ConvNeXt-T 14 x 14 stage) keeps what the kernel relies on: whole
    (level, band) groups per round before the output rounds, every tile and
    group covered once, at most 256 tasks a round, every window and write-back
    inside its array and the LDS (tests/planner/mixed_check.cpp)."""
    rng = random.Random(7)
    lines = [f"{rng.randint(1, 140)} {rng.randint(1, 400)} {rng.randint(9, 16)} {rng.randint(9, 16)} "
             f"{rng.choice([1, 3, 5, 7, 9])} {rng.randint(1, 8)} {rng.randint(0, 2)}" for _ in range(3000)]
    lines += [f"128 384 14 14 {k} {L} 0" for k in (3, 5, 7, 9) for L in range(1, 6)]
    out = subprocess.run([mixed_check], input="\n".join(lines) + "\n", capture_output=True, text=True,
                         check=True, timeout=120).stdout.split("\n")[:len(lines)]
    fails = [(l, o) for l, o in zip(lines, out) if not (o.startswith("ok") or o == "fused")]
    assert not fails, fails[:5]
    assert sum(o.startswith("ok") for o in out) > 1000


def test_odd_shape_block_rounds(planner):
    """63 x 95 planes have 384 4x4 blocks: the gradient pass takes them in
    two rounds over one resident plane."""
    p = planner(32, 128, 63, 95, 5, 3)
    assert p["grad_pass"] == 1 and p["grad_PP"] == 1 and p["grad_rounds"] == 2


def test_large_planes_take_the_region_path(planner):
    """Planes larger than one CU's LDS run in region tiles; their backward is
    the gradient pass over the tiles plus the rotated forward for dx (64 x 64
    regions: 56 x 56 tiles at k = 3, 5, 48 x 48 at k = 7, 9), and the fused
    region backward when there is no level (L = 0)."""
    p = planner(16, 64, 224, 224, 5, 3)
    assert p["fwd_mode"] == "region" and p["fwd_ws"] > 0 and p["bwd_ws"] > 0
    assert p["bwd_mode"] == "region" and p["bwd_region_grad"] == 1
    assert planner(8, 32, 512, 512, 3, 3)["bwd_region_grad"] == 1
    assert planner(8, 128, 128, 128, 5, 1)["bwd_region_grad"] == 1
    assert planner(1, 1, 300, 300, 7, 4)["bwd_region_grad"] == 1
    assert planner(1, 2, 130, 126, 9, 3)["bwd_region_grad"] == 1
    assert planner(1, 2, 130, 126, 5, 0)["bwd_region_grad"] == 0  # no level: the fused region backward


def test_lds_granule_model():
    assert lds_wgs(53760 // 4) == 3 and lds_wgs(53888 // 4) == 2 and lds_wgs(81920 // 4) == 2
    assert lds_wgs(40960 // 4) == 4 and lds_wgs(9656) == 4


@pytest.mark.parametrize("B,C,H,W,k,L", [(64, 96, 56, 56, 5, 3), (128, 192, 28, 28, 5, 2), (128, 384, 14, 14, 5, 1),
                                         (32, 128, 63, 95, 5, 5), (8, 64, 100, 100, 3, 2), (64, 96, 40, 40, 7, 4)])
def test_plans_fit_the_chip(planner, B, C, H, W, k, L):
    """Every resident plan fits one CU's LDS, and the gradient pass is one
    round of resident workgroups (at most three per CU on 256 CUs)."""
    p = planner(B, C, H, W, k, L)
    if p["fwd_mode"] in ("resident", "split"):
        assert 0 < p["fwd_lds_floats"] <= LDS_FLOATS
        assert p["fwd_nb"] % p["fwd_PP"] == 0
    if p["grad_pass"]:
        assert 0 < p["grad_lds_floats"] <= LDS_FLOATS
        wgs = min(3, lds_wgs(p["grad_lds_floats"]))
        assert p["grad_nchunks"] * C <= max(256 * wgs, C)
