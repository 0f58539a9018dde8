"""Host-side checks of the built gfx950 code (the device code objects inside
build.py's objects: kernel metadata and disassembly; no GPU needed): no
kernel spills registers to scratch memory (every kernel runs from registers
and LDS alone), and the FP4 kernel's inline-assembly MFMAs keep the
matrix-core wait states (its own s_nop fences around the main loop, the
compiler's placement of everything else)."""
import os
import re
import subprocess

import pytest

import mfma_hazards
from paper_2007_06919_amd import build


LLVM = "/opt/rocm/llvm/bin"


def _device_code(obj, workdir):
    """The gfx950 code object inside a host object file built by build.py."""
    fatbin, co = workdir / (obj + ".fatbin"), workdir / (obj + ".co")
    for cmd in ([f"{LLVM}/llvm-objcopy", "--dump-section", f".hip_fatbin={fatbin}",
                 os.path.join(build.BUILD, obj)],
                [f"{LLVM}/clang-offload-bundler", "--unbundle", "--type=o", f"--input={fatbin}",
                 "--targets=hipv4-amdgcn-amd-amdhsa--gfx950", f"--output={co}"]):
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, (cmd, r.stderr[-2000:])
    notes = subprocess.run([f"{LLVM}/llvm-readelf", "--notes", str(co)], capture_output=True, text=True)
    dis = subprocess.run([f"{LLVM}/llvm-objdump", "-d", "--mcpu=gfx950", str(co)], capture_output=True,
                         text=True)
    assert notes.returncode == 0 and dis.returncode == 0
    return notes.stdout, dis.stdout


@pytest.fixture(scope="module")
def device_asm(tmp_path_factory):
    """{source: (kernel metadata notes, disassembly)} of the built objects."""
    objs = [os.path.splitext(s)[0] + ".o" for s in build.SOURCES]
    if not all(os.path.exists(os.path.join(build.BUILD, o)) for o in objs) or \
            not os.path.exists(f"{LLVM}/clang-offload-bundler"):
        pytest.skip("the library is not built here (run __graft_entry__.build())")
    work = tmp_path_factory.mktemp("co")
    return {src: _device_code(obj, work) for src, obj in zip(build.SOURCES, objs)}


@pytest.fixture(scope="module")
def fp4_asm(device_asm):
    return device_asm["qconv_b16.hip"][1]


def test_no_kernel_uses_scratch(device_asm):
    bad = []
    for src, (text, _) in device_asm.items():
        for m in re.finditer(r"\.name:\s+(\S+)\n(.*?)\.vgpr_spill_count:\s+(\d+)", text, re.S):
            priv = re.search(r"\.private_segment_fixed_size:\s+(\d+)", m.group(2))
            if int(m.group(3)) or (priv and int(priv.group(1))):
                bad.append(f"{src}: {m.group(1)} spills {m.group(3)} VGPRs")
    assert not bad, "\n".join(bad)


def test_scan_flags_known_hazards():
    """The scan itself: a VALU write right before an MFMA and a read right
    after it are reported; the same code with enough s_nop is not."""
    bad = """
    v_add_u32_e32 v0, s0, v0
    v_mfma_scale_f32_16x16x128_f8f6f4 v[8:11], v[0:3], v[4:7], v[8:11], v13, v14 op_sel_hi:[0,0,0] cbsz:4 blgp:4
    v_add_f32_e32 v8, 1.0, v8
    """
    found, n = mfma_hazards.scan(bad)
    assert n == 1 and len(found) == 2
    good = """
    v_add_u32_e32 v0, s0, v0
    s_nop 1
    v_mfma_scale_f32_16x16x128_f8f6f4 v[8:11], v[0:3], v[4:7], v[8:11], v13, v14 op_sel_hi:[0,0,0] cbsz:4 blgp:4
    v_mfma_scale_f32_16x16x128_f8f6f4 v[8:11], v[0:3], v[4:7], v[8:11], v13, v14 op_sel_hi:[0,0,0] cbsz:4 blgp:4
    s_nop 7
    s_nop 7
    v_add_f32_e32 v8, 1.0, v8
    """
    found, n = mfma_hazards.scan(good)
    assert n == 2 and found == []


def test_fp4_kernel_has_no_mfma_hazards(fp4_asm):
    found, n = mfma_hazards.scan(fp4_asm)
    assert n >= 5 * 128, n          # five kernel variants, 128 MFMAs in each main loop
    assert found == [], "\n".join(found[:10])
