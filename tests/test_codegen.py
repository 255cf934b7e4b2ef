"""Code-generation checks of the GEMM mainloop (host only: hipcc emits the
gfx950 assembly of the forward kernels, nothing runs).

Every k-step of every mainloop instance (one per count of active 32-row
blocks) waits only for the DMA of the stage it is about to read (vmcnt(4): the two stages issued after it stay in flight).  A wait for
vmcnt(0) inside the loop drains the whole pipeline on every k-step; the
compiler inserts one when a loop-invariant vector register was reloaded from
scratch in front of the loop, which happens when other code keeps values live
across the mainloop.  A scratch access inside the loop is a spill in the
hottest code of the library.  Both are checked in every kernel that holds the
mainloop (the megakernel, its stacked form and the serial GEMM kernels).
"""
import os
import re
import subprocess

import pytest

from paper_2609_21483_amd import build as BLD

MFMA_PER_STEP = 16  # 32x32x16 MFMAs per wavefront in one unrolled k-step with every row block active


def _device_asm(tmp_path) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    flags = [f for f in BLD.HIPCC_FLAGS if f not in ("-shared", "-fPIC")]
    out = tmp_path / "forward.s"
    subprocess.run([hipcc, *flags, "-S", "--cuda-device-only", os.path.join(BLD.CSRC, "forward.hip"), "-o",
                    str(out)], check=True, capture_output=True)
    return out.read_text()


def _mainloop_blocks(asm: str):
    """(kernel, block label, instructions) of every basic block holding a
    whole k-step of the mainloop: the DMA issue of a later stage and the
    barrier of the ring."""
    for m in re.finditer(r"\n(_ZN3moe\w+):[^\n]*\n", asm):
        fn = m.group(1)
        end = asm.index(".Lfunc_end", m.end())
        label, ins = None, []
        for line in asm[m.end():end].split("\n") + [".LBBend:"]:
            lm = re.match(r"^(\.LBB\w+):", line)
            if lm:
                if label and any(i.startswith("global_load_lds") for i in ins) and \
                        any(i.startswith("s_barrier") for i in ins):
                    yield fn, label, ins
                label, ins = lm.group(1), []
            else:
                s = line.strip()
                if s and not s.startswith(";") and not s.startswith("."):
                    ins.append(s)


def test_mainloop_keeps_its_dma_in_flight(tmp_path):
    blocks = list(_mainloop_blocks(_device_asm(tmp_path)))
    for name in ("moe_megakernelENS_7FwdArgs", "moe_megakernel_stack", "serial_gemm0_kernel", "serial_gemm1_kernel"):
        # one mainloop instance per count of active 32-row blocks (0..4), each
        # with that many MFMAs per 16-deep slice
        counts = {sum(i.startswith("v_mfma") for i in ins) for fn, _, ins in blocks if name in fn}
        assert counts >= {0, 4, 8, 12, MFMA_PER_STEP}, f"{name}: mainloop instances with {sorted(counts)} MFMAs"
    for fn, label, ins in blocks:
        waits = [i for i in ins if i.startswith("s_waitcnt") and "vmcnt" in i]
        assert waits, f"{fn} {label}: no DMA wait in the k-step"
        assert all("vmcnt(0)" not in w for w in waits), f"{fn} {label}: full DMA drain in the k-step: {waits}"
        assert not any("scratch_" in i for i in ins), f"{fn} {label}: scratch access in the k-step"
