"""The register-streamed MFMA GEMM loads its weight fragments with inline-asm
global loads whose completion the compiler cannot see (the kernel waits for
them with explicit s_waitcnt).  That is only correct if, in the compiled
code, nothing but the MFMAs reads a destination register between the load
and its use, and nothing writes it (a spill copy or a reuse would read or
clobber data still in flight).  This test compiles csrc/gemm.hip for gfx950
with the library's own flags and walks every control path from each such
load to the first instruction that touches its registers: it must be an MFMA
that only reads them, or a full vmcnt(0) wait."""

import os
import re
import shutil
import subprocess

import pytest

from paper_2607_20507_amd import build as B

BRANCHES = ('s_branch', 's_cbranch_scc0', 's_cbranch_scc1', 's_cbranch_vccz', 's_cbranch_vccnz',
            's_cbranch_execz', 's_cbranch_execnz')


def _regs(tok):
    m = re.match(r'v\[(\d+):(\d+)\]', tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r'v(\d+)$', tok)
    return {int(m.group(1))} if m else set()


def check_register_loads(asm_lines, pattern):
    """{kernel: (register loads, list of bad first touches)} for the kernels
    whose symbol matches `pattern`."""
    out = {}
    i = 0
    while i < len(asm_lines):
        if re.match(r'^_Z\S*' + pattern + r'\S*:', asm_lines[i]):
            name = asm_lines[i].split(':')[0]
            j = i + 1
            body = []
            while j < len(asm_lines) and not asm_lines[j].startswith('.Lfunc_end'):
                body.append(asm_lines[j].strip())
                j += 1
            labels = {b.split(':')[0]: k for k, b in enumerate(body) if re.match(r'^\.LBB\S+:', b)}
            nload, bad = 0, []
            for k, b in enumerate(body):
                t = b.split(None, 1)
                if len(t) != 2 or t[0] != 'global_load_dwordx4':
                    continue
                dst = _regs(t[1].split(',')[0].strip())
                if not dst:
                    continue
                nload += 1
                stack, seen, verdicts = [k + 1], set(), []
                while stack:
                    p = stack.pop()
                    while p < len(body) and p not in seen:
                        seen.add(p)
                        tt = body[p].split(None, 1)
                        op = tt[0] if tt else ''
                        if op == 's_endpgm' or (op == 's_waitcnt' and 'vmcnt(0)' in body[p]):
                            verdicts.append('ok')
                            break
                        if op in BRANCHES and len(tt) == 2:
                            if tt[1].strip() in labels:
                                stack.append(labels[tt[1].strip()] + 1)
                            if op == 's_branch':
                                break
                            p += 1
                            continue
                        if not op or op.startswith(('.', ';', 's_')) or op.endswith(':'):
                            p += 1
                            continue
                        ops = [o.strip() for o in tt[1].split(',')] if len(tt) == 2 else []
                        touched = set().union(*[_regs(o) for o in ops]) if ops else set()
                        if touched & dst:
                            first = _regs(ops[0]) if ops else set()
                            verdicts.append('ok' if op.startswith('v_mfma') and not (first & dst) else body[p])
                            break
                        p += 1
                bad += [v for v in verdicts if v != 'ok'] or ([] if verdicts else ['no use found'])
            out[name] = (nload, bad)
            i = j
        i += 1
    return out


def test_checker_flags_a_copy():
    """The walk itself: a load consumed by an MFMA passes, one copied first fails."""
    good = ["_Zgemm_mfma3_x:", "global_load_dwordx4 v[2:5], v9, s[0:1]", "s_waitcnt vmcnt(0)",
            ".LBB0_1:", "v_mfma_f32_16x16x32_bf16 a[0:3], v[10:13], v[2:5], a[0:3]", "s_endpgm", ".Lfunc_end0:"]
    bad = ["_Zgemm_mfma3_y:", "global_load_dwordx4 v[2:5], v9, s[0:1]", "v_mov_b32_e32 v20, v3",
           "v_mfma_f32_16x16x32_bf16 a[0:3], v[10:13], v[2:5], a[0:3]", "s_endpgm", ".Lfunc_end1:"]
    r = check_register_loads(good + bad, "gemm_mfma3")
    assert r["_Zgemm_mfma3_x"] == (1, [])
    assert r["_Zgemm_mfma3_y"][1] == ["v_mov_b32_e32 v20, v3"]


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc not available")
def test_mfma3_register_loads_feed_only_mfmas(tmp_path):
    out = tmp_path / "gemm.s"
    cmd = [B.hipcc()] + B.flags() + ["--cuda-device-only", "-S", os.path.join(B.CSRC, "gemm.hip"), "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    res = check_register_loads(out.read_text().split('\n'), "gemm_mfma3")
    assert res, "no gemm_mfma3 kernel in the device code"
    for name, (nload, bad) in res.items():
        assert nload > 0, name
        assert not bad, (name, bad[:5])
