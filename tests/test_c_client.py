"""The C interface used from C (CPU only): a program written against
include/ec_moe.h alone, compiled as C11 and linked with the built library, calls
the host-side entry points (capacity rule, size queries, status and error
detail) and must agree with the oracle and with the Python binding."""
import os
import shutil
import subprocess

import pytest
import torch

from oracle import ec_ref as ref
from paper_2604_01622_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

PROGRAM = r"""
#include <stdio.h>
#include "ec_moe.h"

int main(void) {
  const int32_t L[3] = {2048, 1000, 7};
  const double t[3] = {0.25, 0.5, 1.0};
  int32_t k[3] = {-1, -1, -1};
  const int st = ec_capacity(3, L, 64, 0.0, t, 4.0, 12.0, EC_SCHED_LINEAR_REV, k);
  printf("%d %d %d %d\n", st, k[0], k[1], k[2]);
  const int32_t off[4] = {0, 2048, 3048, 3055};
  ec_problem p = {3055, 2048, 64, 1024, 3, off, k, 1.0f, EC_BF16, 0};
  printf("%lld %zu %zu %zu %zu\n", (long long)ec_total_capacity(&p), ec_saved_size(&p),
         ec_workspace_size(&p, 0), ec_workspace_size(&p, 2), ec_workspace_size(&p, 3));
  ec_problem bad = p;
  bad.d_model = 100;                     /* not a multiple of 64 */
  printf("%lld\n%s\n%s\n", (long long)ec_total_capacity(&bad), ec_status_string(EC_ERR_SHAPE),
         ec_last_error());
  return 0;
}
"""


@pytest.fixture(scope="module")
def c_client(tmp_path_factory):
    cc = shutil.which("gcc")
    if cc is None or not os.path.exists(binding.LIB_PATH):
        pytest.skip("needs gcc and the built library")
    d = tmp_path_factory.mktemp("c_client")
    src = d / "client.c"
    src.write_text(PROGRAM)
    exe = d / "client"
    libdir = os.path.dirname(binding.LIB_PATH)
    subprocess.run([cc, "-std=c11", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__",
                    "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"),
                    str(src), "-o", str(exe), "-L", libdir, "-l:" + os.path.basename(binding.LIB_PATH),
                    "-Wl,-rpath," + libdir, "-L", os.path.join(ROCM, "lib"),
                    "-Wl,-rpath," + os.path.join(ROCM, "lib")],
                   check=True, capture_output=True, text=True)
    r = subprocess.run([str(exe)], check=True, capture_output=True, text=True, timeout=60)
    return r.stdout.splitlines()


def test_capacity_from_c(c_client):
    st, *k = (int(x) for x in c_client[0].split())
    assert st == 0
    want = ref.capacity_ref([2048, 1000, 7], 64, t=[0.25, 0.5, 1.0], c_min=4.0, c_max=12.0,
                            sched="linear_rev")
    assert k == [int(x) for x in want]


def test_size_queries_from_c_match_the_binding(c_client):
    k = [int(x) for x in c_client[0].split()[1:]]
    total, saved, ws0, ws2, ws3 = (int(x) for x in c_client[1].split())
    P = binding.Problem(3055, 2048, 64, 1024, [0, 2048, 3048, 3055], k, 1.0, torch.bfloat16)
    assert total == sum(k) == P.K
    assert saved == P.saved_size()
    assert (ws0, ws2, ws3) == (P.workspace_size(0), P.workspace_size(2), P.workspace_size(3))


def test_errors_from_c(c_client):
    assert int(c_client[2]) == -1
    assert c_client[3] == binding.lib().ec_status_string(2).decode()
    assert "d_model" in c_client[4]
