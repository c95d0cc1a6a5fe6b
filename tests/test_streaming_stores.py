"""Every 16-byte data store of the splice kernels is a streaming (nontemporal) store, in both
builds (no GPU needed: the gfx950 assembly of the library's own kernels is compiled here and
read).  The kernels touch each moved byte once per call, so their loads and stores of rows and
bands are all nontemporal; the compiler can drop the hint when it merges stores from several
branches into one, which once turned a round kernel's main store into a cached one.  Table
writes (block tables, freed lists, row tables, sorted page lists) are not 16-byte data stores of
these kernels and are not checked."""

import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_01065_amd", "csrc")
DATA_KERNELS = ("contig_move_kernel", "contig_tile_kernel", "contig_chain_kernel", "paged_data_kernel",
                "rotate_rows_kernel")


def _stores_by_kernel(asm: str):
    """{kernel symbol: [16-byte global store lines]} from a device assembly listing."""
    out, cur = {}, None
    for line in asm.splitlines():
        m = re.match(r"^(_Z\w+):", line)
        if m:
            cur = m.group(1)
            out.setdefault(cur, [])
            continue
        if cur and re.search(r"\b(global|buffer)_store_dwordx4\b", line):
            out[cur].append(line.strip())
    return out


def test_data_stores_are_nontemporal(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    from paper_2606_01065_amd import build as B
    jobs = []
    for tag, defs in (("fp32", []), ("exact", ["-DLEYLINE_PAIR_F64=1"])):
        s = str(tmp_path / f"kernels_{tag}.s")
        cmd = [hipcc, *B.HIP_FLAGS, *defs, f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}",
               "--cuda-device-only", "-S", os.path.join(CSRC, "kernels.hip"), "-o", s]
        jobs.append((tag, s, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)))
    for tag, s, proc in jobs:
        log, _ = proc.communicate()
        assert proc.returncode == 0, log
        stores = _stores_by_kernel(open(s).read())
        for name in DATA_KERNELS:
            kernels = {k: v for k, v in stores.items() if name in k}
            assert kernels, f"{tag}: no {name} in the assembly"
            for k, lines in kernels.items():
                assert lines, f"{tag}: {k} has no 16-byte stores"
                plain = [x for x in lines if not re.search(r"\bnt\b", x)]
                assert not plain, f"{tag}: {k}: stores without the nontemporal hint: {plain}"
