"""Register, scratch and LDS budgets of the hot kernels (no GPU): the prefill,
decode and Q8_0 sources are compiled for gfx950 with the library's own flags
and the compiler's per-kernel resource report, and the figures the launch
code and the schedule rely on are checked.

* prefill, D = 64: four waves per SIMD (two 8-wave workgroups, or one
  16-wave eight-slot workgroup, per CU) and no scratch;
* prefill, D = 128: three waves per SIMD; at most 32 bytes of scratch per
  lane (a few values spilled around the key loop, not inside it);
* split-KV decode: four waves per SIMD at D = 64, two at D = 128, no scratch;
* the LSE merge and the Q8_0 products: no scratch;
* every kernel: no dynamic stack, no spilled SGPRs, no spilled VGPRs except
  those few, and no occupancy target the compiler could not meet (a warning
  in the build)."""
import concurrent.futures as cf
import os
import re
import subprocess

import pytest

from paper_2608_18656_amd import build as hip_build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SOURCES = ["fa_prefill.hip", "fa_decode.hip", "fa_q8.hip"]


def _report(src, tmpdir):
    flags = [*hip_build.HIPCC_FLAGS, *hip_build.PER_FILE_FLAGS.get(src, [])]
    cmd = [hip_build.hipcc(), *flags, "-I", os.path.join(ROOT, "include"), "--cuda-device-only", "-c",
           os.path.join(hip_build.CSRC, src), "-o", os.path.join(tmpdir, src + ".o"),
           "-Rpass-analysis=kernel-resource-usage"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return r.stderr


def _parse(text):
    kernels, cur = {}, None
    for line in text.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            cur = kernels.setdefault(m.group(1), {})
            continue
        m = re.search(r"remark:\s+(.+?): (\S+) \[-Rpass-analysis", line)
        if m and cur is not None:
            cur[m.group(1).strip()] = m.group(2)
    return kernels


@pytest.fixture(scope="module")
def reports(tmp_path_factory):
    d = str(tmp_path_factory.mktemp("resources"))
    with cf.ThreadPoolExecutor(len(SOURCES)) as ex:
        texts = dict(zip(SOURCES, ex.map(lambda s: _report(s, d), SOURCES)))
    return {s: (t, _parse(t)) for s, t in texts.items()}


def _num(k, key):
    return int(k[key])


def test_no_unmet_occupancy_and_no_dynamic_stack(reports):
    for src, (text, kernels) in reports.items():
        assert "failed to meet occupancy target" not in text, src
        assert kernels, f"{src}: no resource report"
        for name, k in kernels.items():
            assert k["Dynamic Stack"] == "False", name
            assert _num(k, "SGPRs Spill") == 0, name
            # spilled VGPRs (4 bytes of scratch each) only in the D = 128 prefill
            d128 = re.search(r"prefill_kernelI.*?Li128ELi4E", name) is not None
            assert _num(k, "VGPRs Spill") <= (8 if d128 else 0), name


def test_prefill_budgets(reports):
    kernels = reports["fa_prefill.hip"][1]
    seen = set()
    for name, k in kernels.items():
        m = re.search(r"prefill_kernelI.*?Li(\d+)ELi(\d+)ELb(\d)ELb(\d)E", name)
        assert m, name
        D, NS = int(m.group(1)), int(m.group(2))
        seen.add((D, NS))
        occ, scratch, lds = (_num(k, "Occupancy [waves/SIMD]"), _num(k, "ScratchSize [bytes/lane]"),
                             _num(k, "LDS Size [bytes/block]"))
        if NS in (4, 8):   # the layouts fa_fwd picks
            if D == 64:
                assert occ >= 4 and scratch == 0, (name, occ, scratch)
            else:
                assert occ >= 3 and scratch <= 32, (name, occ, scratch)
        # the workgroups a CU holds at that occupancy fit its 160 KiB of LDS
        waves = NS * (2 if D == 64 else 1)
        per_cu = max(1, 4 * occ // waves)
        assert per_cu * lds <= 160 * 1024, (name, per_cu, lds)
    assert seen == {(D, NS) for D in (64, 128) for NS in (1, 2, 4, 8)}


def test_decode_and_q8_budgets(reports):
    split = combine = 0
    for name, k in reports["fa_decode.hip"][1].items():
        occ, scratch = _num(k, "Occupancy [waves/SIMD]"), _num(k, "ScratchSize [bytes/lane]")
        assert scratch == 0, name
        m = re.search(r"decode_split_kernelI.*?Li(\d+)ELb\d", name)
        if m:
            split += 1
            assert occ >= (4 if m.group(1) == "64" else 2), (name, occ)
        elif "decode_combine_kernel" in name:
            combine += 1
    assert split >= 8 and combine >= 4
    q8 = reports["fa_q8.hip"][1]
    assert q8 and all(_num(k, "ScratchSize [bytes/lane]") == 0 for k in q8.values())
