"""Compiler-reported resources of every HIP kernel (CPU only: a device-only
compile for gfx950).  A kernel that spills to scratch memory or asks for more
LDS than a CU holds is a performance bug even when its results are right."""
import os

import pytest

from paper_2604_01622_amd import build

LDS_PER_CU = 160 * 1024


@pytest.mark.parametrize("src", [s for s in build.SOURCES if s.endswith(".hip")])
def test_no_scratch_and_lds_fits(src):
    res = build.resource_usage(src)
    assert res, f"no kernels reported for {src}"
    for name, r in res.items():
        assert r.get("scratch", 0) == 0, f"{name} spills {r['scratch']} bytes/lane to scratch"
        assert r.get("lds", 0) <= LDS_PER_CU, f"{name} uses {r['lds']} bytes of LDS"
        assert r.get("occupancy", 1) >= 1, f"{name} cannot be resident"


def test_no_self_initialised_declarations():
    """`T x = x` compiles without a warning (clang treats it as an idiom) and
    leaves x undefined; in a kernel that is an address computed from garbage."""
    import glob
    import re
    pat = re.compile(r"(int|size_t|long|float|double|auto|bool|uint32_t|int32_t)\s+([A-Za-z_]\w*)\s*=\s*\2\s*[,;]"
                     r"|,\s*([A-Za-z_]\w*)\s*=\s*\3\s*[,;]")
    bad = []
    for f in glob.glob(os.path.join(build.CSRC, "*")):
        for n, line in enumerate(open(f), 1):
            if pat.search(line):
                bad.append(f"{os.path.basename(f)}:{n}: {line.strip()}")
    assert not bad, bad
