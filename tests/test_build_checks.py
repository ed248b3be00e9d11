"""Checks on the generated gfx950 code (CPU only: compiles to assembly).

The phase-A kernels write M0 in inline asm right before each LDS copy; that
is only sound while nothing else in the kernels relies on M0.  Packed-FP32
VALU instructions are kept out of the build as well.
"""

import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2608_25523_amd", "csrc", "pfx_kernels.hip")
HIPCC = "/opt/rocm/bin/hipcc"


@pytest.fixture(scope="module")
def isa(tmp_path_factory):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("isa") / "k.s"
    from paper_2608_25523_amd.build import FLAGS
    flags = [f for f in FLAGS if f not in ("-shared", "-fPIC")]
    subprocess.run([HIPCC, *flags, "-S", "--cuda-device-only", "-I", os.path.join(ROOT, "include"), SRC,
                    "-o", str(out)], check=True, capture_output=True)
    return out.read_text()


def test_m0_only_feeds_lds_copies(isa):
    lines = [l.strip() for l in isa.splitlines() if l.strip() and not l.strip().startswith(";")]
    for i, l in enumerate(lines):
        if re.search(r"\bm0\b", l):
            assert l.startswith("s_mov_b32 m0,"), l
            assert lines[i + 1].startswith("global_load_lds_dwordx4"), (l, lines[i + 1])


def test_no_packed_fp32(isa):
    assert not re.search(r"v_pk_(add|mul|fma)_f32", isa)


def test_no_scratch_in_attention_kernels(isa):
    kernels = re.findall(r"^(_ZN3pfx\w*(?:decode|extend|merge_rows)_kernel\w*):", isa, flags=re.M)
    # extend; decode with and without the folded-in append and the wide
    # prefix blocks, and on the vector ALU with and without the append; merge
    # with and without the append; head dims 64 and 128
    assert len(kernels) == 18
    for kernel in kernels:
        body = isa.split(kernel + ":", 1)[1].split("s_endpgm", 1)[0]
        assert "scratch_" not in body, kernel

