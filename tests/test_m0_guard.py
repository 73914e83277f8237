"""The attention kernels' chunk stream writes M0 itself: each piece is one
inline-assembly statement that sets M0 to the wave's LDS destination and
issues the global_load_lds_dwordx4 that reads it.  The compiler treats M0 as a
reserved register and does not protect a value of its own across such a
statement, so the code is correct only while nothing else in the translation
unit uses M0.  This test compiles the attention translation unit for gfx950
to assembly (on the CPU) and checks exactly that: every instruction that names
M0 is one of those writes, immediately followed by its load."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    return None


@pytest.mark.skipif(_hipcc() is None, reason="hipcc not available")
def test_m0_is_only_the_chunk_streams(tmp_path):
    out = tmp_path / "attn.s"
    cmd = [_hipcc(), "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Xclang", "-target-feature", "-Xclang",
           "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"), "--cuda-device-only", "-S", "-x", "hip",
           os.path.join(ROOT, "paper_2607_04302_amd", "csrc", "hifa4_attn.hip"), "-o", str(out)]
    subprocess.run(cmd, check=True, capture_output=True, timeout=600)
    lines = [l.strip() for l in out.read_text().splitlines()]
    code = [l for l in lines if l and not l.startswith((";", ".", "_")) and not l.endswith(":")]
    writes = 0
    for i, l in enumerate(code):
        if not re.search(r"\bm0\b", l):
            continue
        assert l.startswith("s_mov_b32 m0,"), f"M0 used outside the chunk stream: {l}"
        assert i + 1 < len(code) and code[i + 1].startswith("global_load_lds_dwordx4"), \
            f"an M0 write not followed by its load: {l} / {code[i + 1] if i + 1 < len(code) else ''}"
        writes += 1
    assert writes > 0, "no chunk-stream loads found"
    # the stream loads are all the scalar-base form written by hand
    loads = [l for l in code if l.startswith("global_load_lds")]
    assert loads and all(", s[" in l for l in loads), [l for l in loads if ", s[" not in l][:3]
