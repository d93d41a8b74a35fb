"""Code the run-time compiler makes from the wave-pipeline kernel's headers
(no GPU needed: compile and read back the AMD assembly).

The LDS DMAs are inline asm, so the compiler's hazard checks do not see
them as vector-memory instructions.  A VMEM instruction needs 5 wait states
after a VALU write of an SGPR it reads; the run-time build rebuilds the
descriptor with read-first-lanes (VALU writes), so each DMA must carry its
own wait.  The test compiles with the hipRTC the library itself would use in
a process that imported torch first (torch ships an older copy) and checks
that no LDS DMA reads a descriptor SGPR written by a VALU instruction fewer
than 5 wait states before it."""
import ctypes
import os
import re
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2004_11250_amd", "csrc")
OBJDUMP = "/opt/rocm/llvm/bin/llvm-objdump"
HEADERS = (("conv_pp_wave.hpp", CSRC), ("conv_pp_kernel.hpp", CSRC), ("conv_pp.hpp", CSRC),
           ("pp.h", os.path.join(ROOT, "include")))
PRELUDE = (
    "typedef __hip_internal::int8_t int8_t; typedef __hip_internal::uint8_t uint8_t;\n"
    "typedef __hip_internal::int16_t int16_t; typedef __hip_internal::uint16_t uint16_t;\n"
    "typedef __hip_internal::int32_t int32_t; typedef __hip_internal::uint32_t uint32_t;\n"
    "typedef __hip_internal::int64_t int64_t; typedef __hip_internal::uint64_t uint64_t;\n"
    "typedef __hip_internal::uint64_t uintptr_t;\n"
    "namespace std { template <class T, T v> struct integral_constant { static constexpr T value = v;\n"
    "  constexpr operator T() const { return v; } };\n"
    "using true_type = integral_constant<bool, true>; using false_type = integral_constant<bool, false>; }\n")
OPTS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-mllvm", "-structurizecfg-skip-uniform-regions", "-mllvm", "-simplifycfg-sink-common=false",
        "-Wno-pass-failed"]


@pytest.fixture(scope="module")
def hiprtc():
    try:
        import torch  # noqa: F401  (loads torch's own ROCm libraries first, as in the GPU tests)
    except ImportError:
        pass
    if not os.path.exists(OBJDUMP):
        pytest.skip("no llvm-objdump")
    try:
        return ctypes.CDLL("libhiprtc.so.7")
    except OSError:
        pytest.skip("no hipRTC")


def _compile(lib, inst):
    texts = [open(os.path.join(d, n)).read().encode() for n, d in HEADERS]
    names = [n.encode() for n, _ in HEADERS]
    src = (PRELUDE + "#define PP_JIT_LIBRARY 0x1B0, 0x03A, 0x0B8, 0x01B, 0x09A, 0x0D8, 0x0B2, 0x036\n"
           "#include \"conv_pp_wave.hpp\"\n"
           f"template __global__ void pp::kern::pp_conv3x3_wave_kernel<{inst}>(pp::ConvParams);\n")
    prog = ctypes.c_void_p()
    hs = (ctypes.c_char_p * len(texts))(*texts)
    ns = (ctypes.c_char_p * len(names))(*names)
    assert lib.hiprtcCreateProgram(ctypes.byref(prog), src.encode(), b"jit_test.hip", len(texts), hs, ns) == 0
    opts = (ctypes.c_char_p * len(OPTS))(*[o.encode() for o in OPTS])
    r = lib.hiprtcCompileProgram(prog, len(OPTS), opts)
    n = ctypes.c_size_t()
    lib.hiprtcGetProgramLogSize(prog, ctypes.byref(n))
    log = ctypes.create_string_buffer(n.value + 1)
    lib.hiprtcGetProgramLog(prog, log)
    assert r == 0, log.value.decode(errors="replace")[:2000]
    lib.hiprtcGetCodeSize(prog, ctypes.byref(n))
    code = ctypes.create_string_buffer(n.value)
    lib.hiprtcGetCode(prog, code)
    lib.hiprtcDestroyProgram(ctypes.byref(prog))
    with tempfile.TemporaryDirectory() as d:
        path = os.path.join(d, "k.co")
        with open(path, "wb") as fh:
            fh.write(code.raw)
        return subprocess.run([OBJDUMP, "-d", "--mcpu=gfx950", path], check=True, capture_output=True,
                              text=True).stdout


def _sregs(tok):
    m = re.match(r"s\[(\d+):(\d+)\]$", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"s(\d+)$", tok)
    return {int(m.group(1))} if m else set()


def dma_hazards(asm):
    """(writer, DMA) pairs where a VALU instruction writes an SGPR of the
    DMA's descriptor fewer than 5 wait states before it."""
    ins = []
    for line in asm.splitlines():
        t = line.split("//")[0].strip()
        if t and not t.endswith(":") and not t.startswith("."):
            ins.append(t)
    found, n_dma = [], 0
    for i, t in enumerate(ins):
        if not re.match(r"buffer_load_dword\w*\s.*\blds\b", t):
            continue
        n_dma += 1
        srsrc = _sregs(t.split(None, 1)[1].split(",")[1].strip())
        waits = 0
        for p in reversed(ins[max(0, i - 6):i]):
            m = re.match(r"s_nop\s+(?:0x)?(\d+)", p)
            waits += int(m.group(1)) + 1 if m else 1
            if waits > 5:
                break
            if p.startswith("v_") and _sregs(p.split(None, 1)[1].split(",")[0].strip()) & srsrc:
                found.append((p, t))
                break
    return found, n_dma


def test_scanner_finds_the_hazard():
    # the pattern that faulted: a read-first-lane straight into the DMA's descriptor
    bad = ("v_readfirstlane_b32 s4, v4\n"
           "buffer_load_dwordx4 v83, s[4:7], 0 offen lds\n")
    good = ("v_readfirstlane_b32 s4, v4\n"
            "s_nop 4\n"
            "buffer_load_dwordx4 v83, s[4:7], 0 offen lds\n")
    assert len(dma_hazards(bad)[0]) == 1
    assert dma_hazards(good) == ([], 1)
    assert dma_hazards("v_mov_b32 v0, s4\nbuffer_load_dword v0, s[4:7], 0 offen lds\n") == ([], 1)


@pytest.mark.parametrize("inst", ["1, 1, 1, 2, 2, 8, 16, 3, false, float",   # 2 x 2 per lane, 16 waves, 16-byte DMAs
                                  "1, 2, 1, 2, 4, 8, 4, 3, true, float"])    # stride 2, 4-byte DMAs, pipelined
def test_run_time_kernels_wait_before_dma(hiprtc, inst):
    asm = _compile(hiprtc, inst)
    found, n_dma = dma_hazards(asm)
    assert n_dma > 0
    assert not found, found[:3]
