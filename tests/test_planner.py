"""The host planner's choices at the benchmarked shapes (no GPU): the planner
source is compiled with its kernel launchers stubbed out (tests/planner) and
asked for the plan of each descriptor. These pin the execution paths that the
measurements in the design notes were taken on, and check that every plan
fits one compute unit's LDS and the chip's resident workgroup slots."""
import json
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_10805_amd", "csrc")
LDS_FLOATS = 160 * 1024 // 4


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
    assert p["fwd_ws"] == 0
    assert p["grad_pass"] == 1 and p["grad_levels"] == 3 and p["grad_coarse"] == 0
    assert p["grad_PP"] == 1 and p["grad_rounds"] == 1
    # four workgroups per CU fit in LDS
    assert 4 * p["fwd_lds_floats"] <= LDS_FLOATS


@pytest.mark.parametrize("C,H,L,fwd_mode", [(96, 56, 5, "resident"), (192, 28, 4, "resident"),
                                            (192, 28, 5, "split"), (384, 14, 3, "split"), (768, 7, 3, "tiny")])
def test_convnext_stage_modes(planner, C, H, L, fwd_mode):
    p = planner(128, C, H, H, 5, L)
    assert p["fwd_mode"] == fwd_mode


def test_odd_shape_block_rounds(planner):
    """63 x 95 planes have 384 4x4 blocks: the gradient pass takes them in
    two rounds over one resident plane."""
    p = planner(32, 128, 63, 95, 5, 3)
    assert p["grad_pass"] == 1 and p["grad_PP"] == 1 and p["grad_rounds"] == 2


def test_large_planes_take_the_region_path(planner):
    p = planner(16, 64, 224, 224, 5, 3)
    assert p["fwd_mode"] == "region" and p["fwd_ws"] > 0 and p["bwd_ws"] > 0


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
        wgs = min(3, LDS_FLOATS // p["grad_lds_floats"])
        assert p["grad_nchunks"] * C <= max(256 * wgs, C)
