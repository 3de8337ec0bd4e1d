"""ISA lint (CPU only): no work-group barrier inside an exec-masked region.

On CDNA a barrier is a wave-level instruction.  When the compiler cannot prove
that a branch around a barrier is uniform, it lays the code out as an
exec-masked region or an exec-masked loop; waves can then execute different
numbers of ``s_barrier`` and the work-group deadlocks.  The kernels move every
barrier-adjacent branch condition to a scalar register; this test compiles
the kernels to gfx950 assembly and checks, per kernel, that every
``s_barrier`` lies outside all regions opened by ``s_and_saveexec`` /
``s_or_saveexec`` and that no loop holding a barrier is continued through the
exec mask (a loop without one, such as the sentinel mode's re-read loop, may
be: its waves need not agree on a trip count).
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
    from paper_2607_07862_amd.build import DEVICE_FLAGS  # lint exactly what the library build compiles

    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-S", "--cuda-device-only", *DEVICE_FLAGS,
           "-I" + os.path.join(ROOT, "include"), SRC, "-o", str(out)]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert r.returncode == 0, r.stdout
    return out.read_text()


def kernels(text):
    out = {}
    for m in re.finditer(r"^(_Z\w*k_mlp2\w*):", text, re.M):
        body = text[m.end():]
        end = body.find(".Lfunc_end")
        out[m.group(1)] = body[:end]
    return out


def loop_headers(body):
    """Labels the compiler annotates as loop headers."""
    heads = set()
    lines = body.splitlines()
    for i, line in enumerate(lines):
        m = re.match(r"^(\.LBB\w+):", line)
        if m and any("Loop Header" in l for l in lines[i : i + 4]):
            heads.add(m.group(1))
    return heads


def parse_blocks(body):
    """Basic blocks of a kernel: list of (label, [instructions]) in layout order."""
    blocks = [["<entry>", []]]
    for line in body.splitlines():
        code = line.split(";")[0].strip()
        if not code:
            continue
        m = re.match(r"^(\.LBB\w+):$", code)
        if m:
            blocks.append([m.group(1), []])
            continue
        if code.startswith(".") or code.startswith("#"):
            continue
        blocks[-1][1].append(code)
        if re.match(r"s_(c?branch|endpgm)", code):
            blocks.append([f"<after{len(blocks)}>", []])
    return [(l, ins) for l, ins in blocks if ins or l.startswith(".LBB")]


def successors(blocks, i):
    ins = blocks[i][1]
    last = ins[-1] if ins else ""
    nxt = [i + 1] if i + 1 < len(blocks) else []
    index = {l: j for j, (l, _) in enumerate(blocks)}
    m = re.match(r"s_branch\s+(\.LBB\w+)", last)
    if m:
        return [index[m.group(1)]]
    m = re.match(r"s_cbranch_\w+\s+(\.LBB\w+)", last)
    if m:
        return [index[m.group(1)]] + nxt
    if last.startswith("s_endpgm"):
        return []
    return nxt


def violations(body):
    """Barriers reached with an open exec-masked region, found by dataflow over the CFG.

    State: the stack of SGPR pairs saved by s_and_saveexec / s_or_saveexec that
    have not yet been restored by s_or_b64 exec, exec, <pair>.
    """
    blocks = parse_blocks(body)
    heads = loop_headers(body)
    bad = []
    entry = {0: ((), ())}
    work = [0]
    seen_state = {}
    while work:
        i = work.pop()
        state = list(entry[i][0])
        alias = dict(entry[i][1])  # complement masks from s_xor, mapped to their region

        def region_of(reg):
            return alias.get(reg, reg)

        for ins in blocks[i][1]:
            # else entry: s_or_saveexec / s_andn2_saveexec on a region's own mask
            m = re.match(r"s_(?:or|andn2)_saveexec_b64\s+(s\[\d+:\d+\]),\s*(s\[\d+:\d+\])", ins)
            if m and region_of(m.group(2)) in state:
                r = region_of(m.group(2))
                del state[len(state) - 1 - state[::-1].index(r):]
                state.append(m.group(1))
                continue
            m = re.match(r"s_(?:and|or)_saveexec_b64\s+(s\[\d+:\d+\])", ins)
            if m:
                state.append(m.group(1))
                continue
            m = re.match(r"s_xor_b64\s+(s\[\d+:\d+\]),\s*(?:exec,\s*(s\[\d+:\d+\])|(s\[\d+:\d+\]),\s*exec)", ins)
            if m:
                src = m.group(2) or m.group(3)
                if region_of(src) in state:
                    alias[m.group(1)] = region_of(src)
                continue
            m = re.match(r"s_or_b64\s+exec,\s*exec,\s*(s\[\d+:\d+\])", ins)
            if m and region_of(m.group(1)) in state:
                r = region_of(m.group(1))
                del state[len(state) - 1 - state[::-1].index(r):]
                continue
            if ins.startswith("s_barrier") and state:
                bad.append(f"{blocks[i][0]}: s_barrier inside exec region(s) {state}")
            m = re.match(r"s_cbranch_exec(?:nz|z)\s+(\.LBB\w+)", ins)
            if m and m.group(1) in heads:
                # a loop continued through the exec mask may let waves run its
                # body different numbers of times: a fault only if that body
                # (the blocks from its header to this back-edge) holds a barrier
                h = next(k for k, blk in enumerate(blocks) if blk[0] == m.group(1))
                if any(x.startswith("s_barrier") for blk in blocks[min(h, i): max(h, i) + 1] for x in blk[1]):
                    bad.append(f"{blocks[i][0]}: exec-masked loop back-edge '{ins}' around a barrier")
            if re.match(r"s_andn2_b64\s+exec,\s*exec", ins):
                bad.append(f"{blocks[i][0]}: lanes retired from exec '{ins}'")
        out = (tuple(state), tuple(sorted(alias.items())))
        for j in successors(blocks, i):
            if j in entry:
                if entry[j][0] != out[0] and (j, out[0]) not in seen_state:
                    seen_state[(j, out[0])] = True
                    bad.append(f"{blocks[j][0]}: reached with exec regions {entry[j][0]} and {out[0]}")
                continue
            entry[j] = out
            work.append(j)
    return sorted(set(bad))


def m0_misuse(body):
    """M0 holds only the LDS addresses of the direct-to-LDS loads.

    The loads take it as an asm operand bound to M0, so the compiler writes
    the register itself (s_mov / s_add into m0) before each load; no other
    instruction may name M0 as a source (an indexed move or a second use
    would mean the compiler kept a value of its own there), and every kernel
    that issues direct-to-LDS loads writes M0."""
    bad = []
    lines = [l.split(";")[0].strip() for l in body.splitlines()]
    lines = [l for l in lines if l and not l.startswith(".") and not l.startswith("#")]
    writes = 0
    for s in lines:
        if re.match(r"s_\w+\s+m0,", s):
            writes += 1
            if re.search(r",.*\bm0\b", s):
                bad.append(f"m0 read by '{s}'")
        elif re.search(r"\bm0\b", s):
            bad.append(f"m0 used by '{s}'")
    if any(l.startswith("global_load_lds") for l in lines) and writes == 0:
        bad.append("direct-to-LDS loads without an M0 write")
    return bad


def test_m0_only_feeds_direct_to_lds_loads(asm):
    problems = {n: m0_misuse(b)[:3] for n, b in kernels(asm).items() if m0_misuse(b)}
    assert not problems, problems


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
