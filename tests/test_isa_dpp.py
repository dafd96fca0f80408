"""The built library's gfx950 code: every v_fmac_f64_dpp (inline assembly in
the G' build's cut kernels, which the compiler's hazard recognizer does not
look into) follows an s_nop of at least two wait states, directly or after
other DPP FMAs of the same block, and no VALU write of EXEC (v_cmpx) comes
within the five instructions before it.  CPU only: it reads the code object
that the build produced, with the ROCm LLVM tools."""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

LIB = os.path.join(os.path.dirname(__file__), "..", "paper_1809_00072_amd", "librxnn.so")
LLVM = "/opt/rocm/llvm/bin"
MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"
TARGET = "hipv4-amdgcn-amd-amdhsa--gfx950"


def _tools():
    need = [shutil.which("objcopy"), os.path.join(LLVM, "clang-offload-bundler"),
            os.path.join(LLVM, "llvm-objdump")]
    return all(t and os.path.exists(t) for t in need)


def _disassembly():
    with tempfile.TemporaryDirectory() as d:
        fb = os.path.join(d, "fb.bin")
        subprocess.check_call(["objcopy", "--dump-section", ".hip_fatbin=" + fb, LIB])
        data = open(fb, "rb").read()
        starts = [m.start() for m in re.finditer(re.escape(MAGIC), data)]
        lines = []
        for k, o in enumerate(starts):
            e = starts[k + 1] if k + 1 < len(starts) else len(data)
            b = os.path.join(d, "b%d.bin" % k)
            co = os.path.join(d, "b%d.co" % k)
            open(b, "wb").write(data[o:e])
            subprocess.check_call([os.path.join(LLVM, "clang-offload-bundler"), "--unbundle",
                                   "--type=o", "--input=" + b, "--targets=" + TARGET,
                                   "--output=" + co])
            out = subprocess.run([os.path.join(LLVM, "llvm-objdump"), "-d", "--mcpu=gfx950", co],
                                 capture_output=True, text=True, check=True).stdout
            lines += [ln.split("//")[0].strip() for ln in out.splitlines()]
        return [ln for ln in lines if ln and not ln.endswith(":") and not ln.startswith("Disassembly")]


@pytest.mark.skipif(not os.path.exists(LIB) or not _tools(), reason="library or ROCm tools absent")
def test_dpp_fma_wait_states():
    ins = _disassembly()
    checked = 0
    for i, t in enumerate(ins):
        if not t.startswith("v_fmac_f64_dpp"):
            continue
        checked += 1
        j = i - 1
        while j >= 0 and ins[j].startswith("v_fmac_f64_dpp"):
            j -= 1
        m = re.match(r"s_nop (\d+)", ins[j]) if j >= 0 else None
        assert m and int(m.group(1)) >= 1, "DPP FMA without its s_nop: %r after %r" % (t, ins[j])
        for k in range(max(0, i - 5), i):
            assert not ins[k].startswith("v_cmpx"), "VALU write of EXEC before %r: %r" % (t, ins[k])
    assert checked > 1000, "expected the cut kernels' DPP FMAs, found %d" % checked
