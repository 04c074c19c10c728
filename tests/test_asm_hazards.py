"""The inline-asm MFMAs of the matrix-core kernels keep the wait states and
register lifetimes the compiler does not manage for them (CPU only: the
sources are compiled to gfx950 assembly with the library's own flags and the
listing is scanned; see tests/asm_hazards.py for the two rules)."""
import concurrent.futures as cf
import os
import shutil
import subprocess

import pytest

from paper_2607_20501_amd import build
from tests import asm_hazards

MFMA_SOURCES = ["k_attn.hip", "k_gemm_mfma.hip"]


def _assembly(src, tmp):
    out = os.path.join(tmp, src + ".s")
    flags = [f for f in build.HIP_FLAGS if f != "-fPIC"]
    subprocess.run([build.HIPCC] + flags + ["--cuda-device-only", "-S",
                                            os.path.join(build.CSRC, src), "-o", out],
                   check=True, capture_output=True, text=True)
    return open(out).read()


@pytest.fixture(scope="module")
def listings(tmp_path_factory):
    if not (os.path.exists(build.HIPCC) or shutil.which(build.HIPCC)):
        pytest.skip("hipcc not available")
    tmp = str(tmp_path_factory.mktemp("asm"))
    with cf.ThreadPoolExecutor(len(MFMA_SOURCES)) as ex:
        texts = list(ex.map(lambda s: _assembly(s, tmp), MFMA_SOURCES))
    return dict(zip(MFMA_SOURCES, texts))


@pytest.mark.parametrize("src", MFMA_SOURCES)
def test_inline_mfma_hazards(listings, src):
    text = listings[src]
    assert text.count("v_mfma") > 0
    bad = asm_hazards.check(text)
    assert not bad, f"{len(bad)} violations, first: " + "\n".join(bad[:5])


def test_checker_flags_planted_cases():
    """The checker itself: a VALU write one instruction before an inline-asm
    MFMA source, and an accumulator input overwritten right after, are found;
    the same code with s_nop 1 in front and the write moved away passes."""
    head = "kern:\n"
    bad1 = head + ("\tv_accvgpr_write_b32 a4, v1\n\t;;#ASMSTART\n"
                   "\tv_mfma_f32_32x32x16_bf16 v[10:25], v[2:5], a[4:7], v[10:25]\n\t;;#ASMEND\n")
    ok1 = head + ("\tv_accvgpr_write_b32 a4, v1\n\t;;#ASMSTART\n\ts_nop 1\n"
                  "\tv_mfma_f32_32x32x16_bf16 v[10:25], v[2:5], a[4:7], v[10:25]\n\t;;#ASMEND\n")
    bad2 = head + ("\t;;#ASMSTART\n\tv_mfma_f32_32x32x16_bf16 v[10:25], v[2:5], a[4:7], v[30:45]\n"
                   "\t;;#ASMEND\n\tv_add_f32_e32 v31, v1, v2\n")
    ok2 = head + ("\t;;#ASMSTART\n\tv_mfma_f32_32x32x16_bf16 v[10:25], v[2:5], a[4:7], v[30:45]\n"
                  "\t;;#ASMEND\n\tv_add_f32_e32 v50, v1, v2\n")
    # An MFMA the compiler emitted itself (no asm markers) is its own business.
    compiler = head + ("\tv_accvgpr_write_b32 a4, v1\n"
                       "\tv_mfma_f32_32x32x16_bf16 v[10:25], v[2:5], a[4:7], v[10:25]\n")
    assert len(asm_hazards.check(bad1)) == 1
    assert asm_hazards.check(ok1) == []
    assert len(asm_hazards.check(bad2)) == 1
    assert asm_hazards.check(ok2) == []
    assert asm_hazards.check(compiler) == []
