"""Code generation of the HIP kernels for gfx950, checked on the host.

The kernels keep every LDS access on the LDS instructions and everything
else in registers: a lambda the compiler does not inline turns the captured
LDS pointers into generic ones (flat accesses through a stack frame in
scratch), which both slows the pass and turns an LDS access beyond the
allocation, harmless for an LDS instruction, into a memory fault.  Register
spills are rejected too: the spill slots of 1024 lanes per workgroup live in
scratch memory, and while the pass streams the cache they are evicted from L2,
so a few dwords per lane add megabytes of HBM writes and re-reads per pass.
This test compiles the device code to assembly and rejects calls, flat
accesses and any stack frame.
"""
import os
import re
import subprocess

import pytest

from paper_2609_23314_amd import build as lib_build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_23314_amd", "csrc")
MAX_PRIVATE_BYTES = 0    # per lane


def _assembly(tmp_path_factory, defines=()):
    out = tmp_path_factory.mktemp("asm") / "vd_kernels.s"
    cmd = [lib_build.hipcc(), f"--offload-arch={lib_build.ARCH}", "--cuda-device-only", "-S",
           "-O3", "-std=c++17", "-I", os.path.join(ROOT, "include"), "-I", CSRC, *defines,
           *lib_build.DEVICE_FLAGS, os.path.join(CSRC, "vd_kernels.hip"), "-o", str(out)]
    subprocess.run(cmd, check=True, capture_output=True)
    return out.read_text()


def _kernel_body(text, part):
    """Assembly of the first kernel whose symbol contains `part`."""
    m = re.search(r"^(_Z\S*" + part + r"\S*):\s*;\s*@", text, flags=re.M)
    assert m, part
    return text[m.end():text.find(".end_amdhsa_kernel", m.end())]


@pytest.fixture(scope="module")
def kernels(tmp_path_factory):
    text = _assembly(tmp_path_factory)
    # split into functions: "name:" label lines that open a function body
    bodies = {}
    for m in re.finditer(r"^(_Z\S+):\s*;\s*@", text, flags=re.M):
        start = m.end()
        end = text.find(".end_amdhsa_kernel", start)
        nxt = text.find("\n_Z", start)
        stop = min(x for x in (end, nxt, len(text)) if x >= 0)
        bodies[m.group(1)] = (text[start:stop], text[stop:text.find("\n", end) if end >= 0 else stop])
    sizes = dict(re.findall(r"\.amdhsa_kernel (\S+)\n(?:.*\n)*?\s*\.amdhsa_private_segment_fixed_size (\d+)",
                            text))
    return text, bodies, {k: int(v) for k, v in sizes.items()}


def test_every_kernel_is_a_single_function(kernels):
    text, bodies, _ = kernels
    assert "s_swappc" not in text, "a device function was called instead of inlined"
    names = list(bodies)
    assert names and all("kernel" in n for n in names), names


def test_no_flat_memory_access(kernels):
    text, _, _ = kernels
    flat = re.findall(r"^\s*(flat_\w+)", text, flags=re.M)
    assert not flat, f"generic-pointer accesses in the kernels: {sorted(set(flat))}"


def test_no_stack_frame(kernels):
    _, _, sizes = kernels
    assert sizes, "no kernel descriptors found"
    big = {k: v for k, v in sizes.items() if v > MAX_PRIVATE_BYTES}
    assert not big, big


def test_lds_checks_only_in_the_debug_build(kernels, tmp_path_factory):
    """The debug build's LDS index checks are compiled in (they record a
    violation with a global atomic OR), and the release build has none."""
    text, _, _ = kernels
    assert "global_atomic_or" not in _kernel_body(text, "step_kernel")
    dbg = _assembly(tmp_path_factory, ["-DVD_DEBUG=1"])
    for part in ("step_kernel", "select_kernel", "compact_kernel", "geometry_kernel"):
        assert "global_atomic_or" in _kernel_body(dbg, part), part


def test_decode_split_keeps_three_workgroups_per_cu(kernels):
    """The host sizes the fused decode step's split launch for three 256-thread
    workgroups per CU (three waves per SIMD), which holds while each split
    kernel needs at most 168 registers per lane, AGPRs included (512 per SIMD
    lane over three waves, in steps of 8).  With four query heads per KV head
    and 16-lane rows the value sums run on the matrix cores, their
    accumulators in ordinary VGPRs."""
    text, bodies, _ = kernels
    regs = dict(re.findall(r"\.amdhsa_kernel (\S*attn_split_kernel\S*)\n(?:.*\n)*?"
                           r"\s*\.amdhsa_next_free_vgpr (\d+)", text))
    assert len(regs) >= 9, regs
    over = {k: int(v) for k, v in regs.items() if int(v) > 168}
    assert not over, over
    for part in ("attn_split_kernelILi0ELi128ELi4E", "attn_split_kernelILi1ELi64ELi4E"):
        body = _kernel_body(text, part)
        assert "v_mfma_f32_4x4x1_16b_f32" in body, part
        assert "v_accvgpr" not in body, part
