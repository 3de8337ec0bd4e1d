"""ISA lint (CPU only): no work-group barrier inside an exec-masked region.

On CDNA a barrier is a wave-level instruction.  When the compiler cannot prove
that a branch around a barrier is uniform, it lays the code out as an
exec-masked region or an exec-masked loop; waves can then execute different
numbers of ``s_barrier`` and the work-group deadlocks.  The kernels move every
barrier-adjacent branch condition to a scalar register; this test compiles
the kernels to gfx950 assembly and checks, per kernel, that every
``s_barrier`` lies outside all regions opened by ``s_and_saveexec`` /
``s_or_saveexec`` and that no loop is continued through the exec mask.
"""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2607_07862_amd", "csrc", "mlp2_kernels.hip")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("isa") / "k.s"
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-S", "--cuda-device-only",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I" + os.path.join(ROOT, "include"), SRC, "-o", str(out)]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert r.returncode == 0, r.stdout
    return out.read_text()


def kernels(text):
    out = {}
    for m in re.finditer(r"^(_Z\w*k_(?:gemm1|gemm2|pipelined)\w*):", text, re.M):
        body = text[m.end():]
        end = body.find("s_endpgm")
        out[m.group(1)] = body[:end]
    return out


def violations(body):
    bad = []
    stack = []
    seen_labels = set()
    for ln, line in enumerate(body.splitlines()):
        s = line.split(";")[0].strip()
        if not s:
            continue
        if re.match(r"^\.LBB\w+:$", s):
            seen_labels.add(s[:-1])
            continue
        m = re.match(r"s_(?:and|or)_saveexec_b64\s+(s\[\d+:\d+\])", s)
        if m:
            stack.append(m.group(1))
            continue
        m = re.match(r"s_or_b64\s+exec,\s*exec,\s*(s\[\d+:\d+\])", s)
        if m and m.group(1) in stack:
            del stack[len(stack) - 1 - stack[::-1].index(m.group(1)):]
            continue
        if s.startswith("s_barrier") and stack:
            bad.append(f"line {ln}: s_barrier inside exec region(s) {stack}")
        # a loop continued through the exec mask: a backward exec-conditional branch,
        # or lanes retired from exec inside a loop
        m = re.match(r"s_cbranch_exec(?:nz|z)\s+(\.LBB\w+)", s)
        if m and m.group(1) in seen_labels:
            bad.append(f"line {ln}: backward exec-masked branch '{s}'")
        if re.match(r"s_andn2_b64\s+exec,\s*exec", s):
            bad.append(f"line {ln}: lanes retired from exec '{s}'")
    return bad


def test_every_kernel_keeps_barriers_in_uniform_control_flow(asm):
    ks = kernels(asm)
    assert len(ks) >= 3 * 18, f"expected the full kernel table, found {len(ks)}"
    problems = {}
    for name, body in ks.items():
        assert "s_barrier" in body, name
        v = violations(body)
        if v:
            problems[name] = v[:5]
    assert not problems, problems
