"""The public header is plain C: it compiles as C99 with warnings as errors,
and a C program that calls every entry point links against the library and
runs (CPU only: every call there is rejected or a no-op before any device
work, so no GPU is touched)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB_DIR = os.path.join(ROOT, "paper_2507_07114_amd")

C_SOURCE = r"""
#include "lossy.h"
#include <stdio.h>
int main(void) {
    ll_loss loss = {LL_LOSS_BERNOULLI, 0.1, 0.0, 0.0, 0.0, 0.0, 0};
    ll_opt opt = {LL_ADAM, 3e-4f, 0.0f, 0.9f, 0.95f, 1e-8f, 0.0f};
    ll_ext ext = {LL_EST_ARRIVED_MEAN, -1, NULL, NULL, NULL, 0.0, 0};
    ll_drift drift;
    (void)drift;
    int rc = 0;
    rc |= ll_masks(4, 0, 0, LL_DIR_GRAD, &loss, NULL, NULL, NULL, 0, &ext, NULL);
    rc |= lossy_aggregate(0, 0, 8, LL_F32, NULL, 0, NULL, 0.0f, NULL, NULL, NULL, NULL, NULL);
    rc |= ll_ages_update(4, 0, NULL, NULL, NULL);
    rc |= shard_step(&opt, 0, 0, NULL, NULL, NULL, NULL, NULL);
    rc |= lossy_broadcast(0, 0, 8, NULL, LL_BF16, NULL, 0, NULL, NULL);
    rc |= drift_stats(0, 0, 8, LL_BF16, NULL, 0, NULL, NULL, NULL, 0, NULL, NULL);
    rc |= lossy_step_fused(0, 0, 8, 0, &loss, &loss, NULL, NULL, LL_BF16, NULL, 0, &opt,
                           NULL, NULL, NULL, LL_BF16, NULL, 0, NULL, NULL, NULL, NULL, 0,
                           NULL, &ext, NULL);
    printf("%zu %zu %d %s\n", ll_workspace_bytes(64, 1000, 8), ll_masks_workspace_bytes(4, 8),
           rc, ll_last_error());
    return 0;
}
"""


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_header_is_c99_and_links(tmp_path):
    src = tmp_path / "use_lossy.c"
    src.write_text(C_SOURCE)
    exe = tmp_path / "use_lossy"
    cmd = ["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic",
           f"-I{os.path.join(ROOT, 'include')}", str(src), f"-L{LIB_DIR}", "-llossy",
           f"-Wl,-rpath,{LIB_DIR}", "-Wl,--allow-shlib-undefined", "-o", str(exe)]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert run.returncode == 0, run.stderr
    ws, ws_masks, rc, *msg = run.stdout.split()
    import paper_2507_07114_amd as ll
    assert int(ws) == ll.ll_workspace_bytes(64, 1000, 8)
    assert int(ws_masks) == ll.ll_masks_workspace_bytes(4, 8)
    assert int(rc) != 0 and " ".join(msg)  # the invalid calls reported an error
