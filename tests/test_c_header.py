"""The boundary as C: a C11 program includes include/som.h, links libsom.so and
calls the host entry points (no GPU): the workspace queries, the CSR validator,
the schedule, an argument check of a device entry point, and the error text."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2608_24067_amd")

PROGRAM = r"""
#include "som.h"

#include <stdio.h>
#include <string.h>

int main(void)
{
    som_bmu_config cfg;
    memset(&cfg, 0, sizeof cfg);
    const size_t a = som_bmu_workspace_bytes(1000, 4096, 30000, 12000, &cfg);
    const size_t b = som_bmu_workspace_bytes(1000, 4096, 30000, 12000, NULL);
    const size_t c = som_bmu2_workspace_bytes(1000, 4096, 30000, 12000, NULL);
    if (a == 0 || a != b || c < a || a % 256 != 0) return 1;
    if (som_bmu_workspace_bytes(1000, SOM_MAX_NEURONS + 1, 30000, 12000, NULL) != 0) return 2;
    cfg.tile_samples = 5;
    if (som_bmu_workspace_bytes(1000, 4096, 30000, 12000, &cfg) != 0) return 3;

    const int32_t row_ptr[4] = {0, 2, 2, 5};
    const int32_t col_idx[5] = {1, 7, 0, 3, 9};
    if (som_validate_csr_host(row_ptr, col_idx, 3, 10) != SOM_OK) return 4;
    if (som_last_error()[0] != '\0') return 5;
    const int32_t unsorted[5] = {7, 1, 0, 3, 9};
    if (som_validate_csr_host(row_ptr, unsorted, 3, 10) != SOM_ERR_BAD_CSR) return 6;
    if (strstr(som_last_error(), "row 0") == NULL) return 7;

    if (som_codebook_norms(NULL, 10, 10, NULL, NULL) != SOM_ERR_INVALID_ARG) return 8;
    if (som_radius(som_sigma(1, 512.0, 0.5, 0.3)) != 512) return 9;
    if (som_update_workspace_bytes(30000, 64, 1000, 0) == 0) return 10;
    const som_status st = SOM_ERR_HIP;
    printf("workspace %zu, two-best %zu, status %d\n", a, c, (int)st);
    return 0;
}
"""


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_header_compiles_as_c11_and_links(tmp_path):
    lib = os.path.join(PKG, "libsom.so")
    if not os.path.exists(lib):
        pytest.fail("libsom.so is not built: run __graft_entry__.build()")
    src = tmp_path / "use_som.c"
    src.write_text(PROGRAM)
    exe = str(tmp_path / "use_som")
    r = subprocess.run(["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", "-pedantic", f"-I{ROOT}/include", str(src),
                        "-o", exe, f"-L{PKG}", "-lsom", f"-Wl,-rpath,{PKG}"], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, (r.returncode, r.stdout, r.stderr)
    assert r.stdout.startswith("workspace ")
