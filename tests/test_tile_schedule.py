"""Ordered-tile schedules of contiguous splices, checked on the CPU.

tests/tile_schedule_sim.cpp plans random multi-directive splices with the library's planner and
runs every tile launch of each plan under randomly interleaved workgroups (one tile each, or
persistent workgroups that prefetch their next tile as the kernel does), using the kernel's own
ticket-to-item lookup (tile_item_of, checked for every ticket) and wait rule (tile_wait_flags): no
load may see an overwritten row, no schedule may stall, and the rows must come out as the splice
defines them.  Planted mistakes in the wait rule or the planner's
wait lists (dropped cross-item waits, a missing tile of the shift, an off-by-one tile range) make
it fail."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_01065_amd", "csrc")


def _build(tmp_path_factory, name, defines):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path_factory.mktemp(name) / "tile_schedule_sim")
    subprocess.run([gxx, "-O2", "-std=c++17", "-Wall", "-Wextra", "-Werror"] + defines
                   + ["-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
                      os.path.join(ROOT, "tests", "tile_schedule_sim.cpp"), os.path.join(CSRC, "plan.cpp"),
                      "-o", exe], check=True)
    return exe


@pytest.fixture(scope="module")
def sim(tmp_path_factory):
    return _build(tmp_path_factory, "tile_sim", [])


@pytest.fixture(scope="module")
def sim_full_tiles(tmp_path_factory):
    """The planner with the quarter-size tiles of small calls switched off: every call here is
    small, so this build is the one that runs the full-size tiles of larger calls."""
    return _build(tmp_path_factory, "tile_sim_full", ["-DLEYLINE_TILE_SMALL_TICKETS=0"])


@pytest.fixture(scope="module")
def sim_packed(tmp_path_factory):
    """The planner and unit layout of the fp64-pair build, whose tile launches pack narrow
    interleaved bands (MLA K_pe) and cut those items into tiles of whole packed blocks."""
    return _build(tmp_path_factory, "tile_sim_packed", ["-DLEYLINE_PAIR_F64=1"])


@pytest.mark.parametrize("seed", [11, 12, 13, 14])
def test_tile_schedules_are_race_free_and_complete(sim, seed):
    r = subprocess.run([sim, str(seed), "3000"], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    ok, cases, tiles, gave_up = r.stdout.split()
    assert ok == "ok" and int(cases) > 2000 and int(tiles) > 50000 and int(gave_up) == 0


@pytest.mark.parametrize("persist", [0, 1])
def test_full_size_tile_schedules_are_race_free_and_complete(sim_full_tiles, persist):
    r = subprocess.run([sim_full_tiles, "19", "2500", "0", str(persist)], capture_output=True, text=True,
                       timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    ok, cases, tiles, gave_up = r.stdout.split()
    assert ok == "ok" and int(cases) > 2000 and int(tiles) > 10000 and int(gave_up) == 0


def test_persistent_workgroups_with_a_prefetched_tile_never_stall(sim):
    """The kernel's workgroups are persistent: each holds its current tile (published) and the
    next ticket's tile, whose loads it issues before it waits for the current tile's flags and
    stores it.  Under random interleavings of 1-64 such workgroups every schedule completes, no
    load (prefetched or not) sees an overwritten row, and the rows come out right."""
    r = subprocess.run([sim, "15", "2500", "0", "1"], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    ok, cases, tiles, gave_up = r.stdout.split()
    assert ok == "ok" and int(cases) > 2000 and int(tiles) > 50000 and int(gave_up) == 0


@pytest.mark.parametrize("persist", [0, 1])
def test_a_wait_that_cannot_end_gives_up_and_every_tile_exits(sim, persist):
    """A planted schedule fault (the first tile of every launch also waits for the launch's last
    tile, a later ticket) blocks launches whenever too few workgroups are in flight.  The kernel's
    bounded wait must then give up (the timeout status bit, no stores) so that every workgroup
    exits instead of hanging, with one tile per workgroup and with persistent workgroups."""
    r = subprocess.run([sim, "21", "300" if persist == 0 else "120", "1", str(persist)], capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    ok, cases, tiles, gave_up = r.stdout.split()
    assert ok == "ok" and int(cases) > 100 and int(gave_up) > 0


@pytest.mark.parametrize("persist", [0, 1])
def test_packed_tile_schedules_are_race_free_and_complete(sim_packed, persist):
    r = subprocess.run([sim_packed, "17", "2500", "0", str(persist)], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    ok, cases, tiles, gave_up = r.stdout.split()
    assert ok == "ok" and int(cases) > 2000 and int(tiles) > 50000 and int(gave_up) == 0
