"""Per-kernel register, spill, LDS and occupancy table of the built library.

The compiler reports, for every kernel instance it emits for gfx950, the
vector and accumulation registers it allots, any spills, the static LDS and
the waves per SIMD those allow; the build keeps these reports in
``_build/resource_usage.log``.  This turns them into one row per instance
(the analogue of the paper's register study of its tiled convolution,
Section 4.1.1).  Run after a build: ``python -m paper_1904_05347_amd.resources``.
Dynamic LDS (the direct convolutions' patch and filter block) is sized at
launch and shows as 0 here.
"""
from __future__ import annotations

import os
import re
import subprocess
import sys

from .build import RESOURCE_LOG

_FIELDS = {"VGPRs": "vgpr", "AGPRs": "agpr", "TotalSGPRs": "sgpr", "ScratchSize [bytes/lane]": "scratch",
           "Occupancy [waves/SIMD]": "occupancy", "SGPRs Spill": "sgpr_spill", "VGPRs Spill": "vgpr_spill",
           "LDS Size [bytes/block]": "lds"}


def parse(path: str = RESOURCE_LOG):
    """{mangled kernel name: {field: int}} from the build's remark log."""
    kernels, cur = {}, None
    pat = re.compile(r"remark:\s+(.*?):\s+(\S+)\s+\[-Rpass-analysis")
    with open(path) as fh:
        for line in fh:
            m = pat.search(line)
            if not m:
                continue
            key, val = m.group(1).strip(), m.group(2)
            if key == "Function Name":
                cur = kernels.setdefault(val, {"file": os.path.basename(line.split(":", 1)[0])})
            elif cur is not None and key in _FIELDS and val.lstrip("-").isdigit():
                cur[_FIELDS[key]] = int(val)
    return kernels


def demangle(names):
    res = subprocess.run(["c++filt"], input="\n".join(names), capture_output=True, text=True, check=True)
    return res.stdout.splitlines()


def short(name: str) -> str:
    """pk::(anonymous namespace)::direct_tiled_kernel<8, 1, 2, 1>(pk::KernelArgs) -> direct_tiled_kernel<8, 1, 2, 1>"""
    name = name.replace("pk::(anonymous namespace)::", "").replace("pk::", "")
    if name.startswith("void "):
        name = name[5:]
    depth, out = 0, []
    for ch in name:
        if ch == "(" and depth == 0:
            break
        depth += ch == "<"
        depth -= ch == ">"
        out.append(ch)
    return "".join(out)


def table(path: str = RESOURCE_LOG) -> str:
    kernels = parse(path)
    names = sorted(kernels)
    plain = dict(zip(names, demangle(names)))
    rows = sorted(((kernels[n]["file"], short(plain[n]), kernels[n]) for n in names), key=lambda r: r[:2])
    out = ["%-22s %-96s %5s %5s %5s %6s %6s %6s %7s %4s" % ("file", "kernel", "vgpr", "agpr", "sgpr", "vspill",
                                                            "sspill", "scratch", "lds", "occ")]
    for f, k, d in rows:
        out.append("%-22s %-96s %5d %5d %5d %6d %6d %6d %7d %4d" % (
            f, k, d.get("vgpr", 0), d.get("agpr", 0), d.get("sgpr", 0), d.get("vgpr_spill", 0),
            d.get("sgpr_spill", 0), d.get("scratch", 0), d.get("lds", 0), d.get("occupancy", 0)))
    return "\n".join(out) + "\n"


if __name__ == "__main__":
    sys.stdout.write(table(sys.argv[1] if len(sys.argv) > 1 else RESOURCE_LOG))
