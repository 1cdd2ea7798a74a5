"""Code-generation checks of the gfx950 kernels (CPU only: hipcc cross-compiles).

The kernels' speed rests on properties of the generated code that a compiler
change could silently undo.  These tests compile the sources the way the
build does and check them in the assembly and the resource report:

* no kernel spills vector registers or uses scratch memory (at most two
  scalar registers may go to VGPR lanes);
* the attention kernels keep two waves per SIMD (their tiles assume it;
  32-row tiles need two workgroups per CU);
* in the attention kernels the MFMA operand reads run ahead: most LDS waits
  leave later reads outstanding (``lgkmcnt(N)`` with N >= 1).  When the
  compiler sees the global-to-LDS copies it waits for every LDS read before
  each MFMA instead, which costs 3-5%.
"""
import os
import re
import subprocess

import pytest

from paper_2606_02964_amd import build as B

pytestmark = pytest.mark.filterwarnings("ignore")


def _hipcc():
    try:
        return B.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not available")


@pytest.fixture(scope="module")
def compiled(tmp_path_factory):
    cc = _hipcc()
    out = {}
    tmp = tmp_path_factory.mktemp("isa")
    for src in ("attn.hip", "append.hip"):
        asm = tmp / (src + ".s")
        cmd = [cc, *B.common_flags(), "--cuda-device-only", "-S", "-Rpass-analysis=kernel-resource-usage",
               os.path.join(B.CSRC, src), "-o", str(asm)]
        res = subprocess.run(cmd, capture_output=True, text=True)
        assert res.returncode == 0, res.stderr[-2000:]
        out[src] = (asm.read_text(), res.stderr)
    return out


def _resources(remarks):
    """{kernel name: {field: value}} from the kernel-resource-usage remarks."""
    kernels, cur = {}, None
    for line in remarks.splitlines():
        m = re.search(r"remark: Function Name: (\S+)", line)
        if m:
            cur = kernels.setdefault(m.group(1), {})
            continue
        m = re.search(r"remark:\s+([A-Za-z ]+?)(?: \[[^\]]*\])?: (\d+)", line)
        if m and cur is not None:
            cur[m.group(1).strip()] = int(m.group(2))
    return kernels


def _body(asm, kernel):
    start = re.search(r"^" + re.escape(kernel) + r":", asm, re.M).start()
    return asm[start:asm.index("s_endpgm", start)]


@pytest.mark.parametrize("src", ["attn.hip", "append.hip"])
def test_no_spills_or_scratch(compiled, src):
    kernels = _resources(compiled[src][1])
    assert kernels, "no resource remarks parsed"
    for name, r in kernels.items():
        # a scalar spill lands in a VGPR lane (no memory); the persistent
        # attention loop keeps the launch arguments in SGPRs and may push one
        # of them out once per workgroup
        assert r.get("VGPRs Spill", 0) == 0 and r.get("SGPRs Spill", 0) <= 2, (name, r)
        assert r.get("ScratchSize", 0) == 0, (name, r)


def test_attention_occupancy(compiled):
    kernels = {k: v for k, v in _resources(compiled["attn.hip"][1]).items()
               if "msa_attn_kernel" in k or "msa_decode_kernel" in k}
    # d in {64, 128} x {4, 8 waves, 32-row tiles} x {bf16 weights, precise weights}
    assert len(kernels) == 12
    for name, r in kernels.items():
        assert r["Occupancy"] >= 2, (name, r)


def test_operand_reads_run_ahead(compiled):
    asm, remarks = compiled["attn.hip"]
    names = [k for k in _resources(remarks) if "msa_attn_kernel" in k]
    for name in names:
        body = _body(asm, name)
        waits = re.findall(r"s_waitcnt lgkmcnt\((\d+)\)", body)
        ahead = sum(1 for n in waits if int(n) >= 1)
        assert ahead >= 0.5 * len(waits), (name, ahead, len(waits))
        assert len(re.findall(r"v_mfma_f32_32x32x16_bf16", body)) >= 32, name
