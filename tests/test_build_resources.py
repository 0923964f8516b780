"""Register, scratch and occupancy of the compiled gfx950 kernels (CPU only).

Compiles the forward unit and the backward units of gradient modes 1 and 3
for the device only, with the compiler's per-kernel resource remarks, and
checks the promises the kernel configurations make:

* every forward kernel (single pass, split-K partial pass and the sigmoid
  forward, for head dims that are multiples of 64 and for padded ones, and
  the key-split configuration) fits the workgroups per CU its configuration
  is sized for, MINB workgroups of NW waves = ceil(MINB * NW / 4) waves per
  SIMD, without spilling;
* the student-gradient backward kernels (mode 1) for head dims that are
  multiples of 64 never spill, and those of the workload head dims
  (128, 128), (128, 64), (192, 64) run two workgroups (two waves) per SIMD;
  their instantiations for padded head dims (real rows narrower) spill at
  most a few bytes;
* the kernels for all four gradients (mode 3) never spill: they exist only
  for d1 + d2 < 448, and from there on the host runs the student (mode 1)
  and teacher (mode 2) kernels one after the other.
"""
import concurrent.futures as cf
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_20005_amd", "csrc")
UNITS = ("kl_fwd_inst", "kl_fwd_sigmoid_inst", "kl_bwd_dq_m1", "kl_bwd_dk_m1", "kl_bwd_dq_m3", "kl_bwd_dk_m3")


def _hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    pytest.skip("hipcc not available")


def _remarks(unit, outdir):
    cmd = [_hipcc(), "-O3", "-std=c++17", "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang",
           "-packed-fp32-ops", f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}", "--offload-device-only", "-c",
           os.path.join(CSRC, unit + ".hip"), "-o", os.path.join(outdir, unit + ".o"),
           "-Rpass-analysis=kernel-resource-usage"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return r.stderr


def _parse(text):
    """{mangled kernel name: {remark: value}} from the resource-usage remarks."""
    out, cur = {}, None
    for line in text.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            cur = out.setdefault(m.group(1), {})
            continue
        m = re.search(r"remark:\s+([A-Za-z /\[\]]+?):\s+(\d+)", line)
        if m and cur is not None:
            cur[m.group(1).strip()] = int(m.group(2))
    return out


@pytest.fixture(scope="module")
def kernels(tmp_path_factory):
    outdir = str(tmp_path_factory.mktemp("ru"))
    with cf.ThreadPoolExecutor(max_workers=len(UNITS)) as ex:
        texts = list(ex.map(lambda u: _remarks(u, outdir), UNITS))
    res = {}
    for t in texts:
        res.update(_parse(t))
    return res


# FwdTraits<DA, DB, NSTAGE, MINB, NW, PAD[, KS]> in the mangled name of a forward kernel
FWD_RE = re.compile(r"kl_fwd_(?:partial_|sigmoid_)?kernelINS_9FwdTraitsILi(\d+)ELi(\d+)ELi(\d+)ELi(\d+)ELi(\d+)ELb([01])")
# kl_bwd_{dq,dk}_kernel<DA, DB, CAUSAL, MODE, ACT, PD>
BWD_RE = re.compile(r"kl_bwd_(dq|dk)_kernelILi(\d+)ELi(\d+)ELb([01])ELi(\d+)ELi(\d+)ELb([01])E")
PD_SPILL_LIMIT = 16   # bytes per lane the padded-dim backward instantiations may spill


def test_forward_occupancy_as_configured(kernels):
    seen = 0
    for name, r in kernels.items():
        m = FWD_RE.search(name)
        if not m:
            continue
        da, db, _, minb, nw, _ = (int(x) for x in m.groups())
        seen += 1
        promised = (minb * nw + 3) // 4
        assert r["ScratchSize [bytes/lane]"] == 0, (da, db, minb, nw, r)
        assert r["Occupancy [waves/SIMD]"] >= promised, (da, db, minb, nw, r)
    assert seen >= 16 * 4 * 2


def test_backward_student_kernels(kernels):
    seen = 0
    for name, r in kernels.items():
        m = BWD_RE.search(name)
        if not m or int(m.group(5)) != 1:
            continue
        seen += 1
        da, db, pd = int(m.group(2)), int(m.group(3)), m.group(7) == "1"
        if pd:
            assert r["ScratchSize [bytes/lane]"] <= PD_SPILL_LIMIT, (name, r)
            continue
        assert r["ScratchSize [bytes/lane]"] == 0, (name, r)
        if (da, db) in ((128, 128), (128, 64), (192, 64)):
            assert r["Occupancy [waves/SIMD]"] >= 2, (name, r)
    assert seen == 2 * 16 * 2 * 2


def test_all_gradient_kernels_never_spill(kernels):
    built = set()
    for name, r in kernels.items():
        m = BWD_RE.search(name)
        if not m or int(m.group(5)) != 3 or m.group(7) == "1":
            continue
        da, db = int(m.group(2)), int(m.group(3))
        built.add((m.group(1), da, db, m.group(4)))
        assert r["ScratchSize [bytes/lane]"] == 0, (name, r)
    expected = {(k, da, db, c) for k in ("dq", "dk") for da in (64, 128, 192, 256) for db in (64, 128, 192, 256)
                for c in ("0", "1") if da + db < 448}
    assert built == expected
