"""Checks on the gfx950 assembly of the kernels that copy tiles global -> LDS
(latent-attention decode, bf16 prefill; CPU only: hipcc cross-compiles).

These kernels copy tiles into LDS with global->LDS loads written as inline
assembly, each preceded by its own write of M0 (the LDS destination); the
compiler does not preserve M0 across inline assembly, so the kernels rely on
no other instruction reading M0.  The test pins that: every instruction that
names M0 is one of those writes, immediately followed by its load."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2506_05345_amd", "csrc")


def _hipcc():
    exe = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(exe):
        pytest.skip("hipcc not available")
    return exe


@pytest.mark.parametrize("src", ["dms_mla.hip", "dms_prefill.hip"])
def test_m0_is_only_the_lds_copy_destination(tmp_path, src):
    from paper_2506_05345_amd import build
    out = tmp_path / (src + ".s")
    cmd = [_hipcc(), "-O3", "-std=c++17", f"--offload-arch={build.ARCH}", *build.GPU_FLAGS,
           *build.PER_SOURCE.get(src, []), "-munsafe-fp-atomics", "--cuda-device-only", "-S",
           os.path.join(CSRC, src), "-o", str(out)]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    assert r.returncode == 0, r.stdout.decode(errors="replace")
    lines = [l.split(";")[0].strip() for l in out.read_text().splitlines()]
    lines = [l for l in lines if l and not l.startswith(".") and not l.endswith(":")]
    copies = 0
    for i, l in enumerate(lines):
        if re.search(r"\bm0\b", l):
            assert re.fullmatch(r"s_mov_b32 m0, s\d+", l), l
            assert lines[i + 1].startswith("global_load_lds_dword"), (l, lines[i + 1])
            copies += 1
    assert copies > 0
    # and every global->LDS load has its own M0 write just before it
    loads = sum(1 for l in lines if l.startswith("global_load_lds"))
    assert loads == copies
