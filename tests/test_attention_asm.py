"""The bf16 attention kernel issues its score MFMAs as inline assembly, which
the compiler does not see as MFMAs: it inserts no wait states after them.
The kernel keeps the distance itself (the last MFMA pair of a tile and the
wait states after it are one asm statement).  This test compiles the kernel
for gfx950 with the library's own flags and checks, in every instance, that
no instruction reads, writes or copies a score register between an inline
MFMA that writes it and the wait states, and that those are at least the 12
the compiler itself puts between this MFMA and a vector read of its result.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2606_13501_amd import build as B

HIPCC = B.HIPCC
MIN_WAIT_STATES = 12


def _regs(text):
    out = set()
    for m in re.finditer(r"\bv\[(\d+):(\d+)\]", text):
        out.update(range(int(m.group(1)), int(m.group(2)) + 1))
    for m in re.finditer(r"\bv(\d+)\b", text):
        out.add(int(m.group(1)))
    return out


def scan(lines):
    """Hazards in one kernel's assembly, scanned in program order."""
    problems = []
    inflight = {}            # register -> line of the inline MFMA writing it
    in_asm = False
    nops = 0                 # wait states of the s_nop run inside the current asm statement
    for i, raw in enumerate(lines):
        l = raw.strip()
        if l.startswith(";;#ASMSTART"):
            in_asm, nops = True, 0
            continue
        if l.startswith(";;#ASMEND"):
            if nops and inflight:
                problems.append(f"line {i}: asm statement ends with an s_nop run of {nops} < {MIN_WAIT_STATES}")
            in_asm = False
            continue
        if not l or l.startswith((".", ";")) or l.endswith(":"):
            continue
        op = l.split()[0]
        if in_asm and op.startswith("v_mfma"):
            dst = l.split()[1].rstrip(",")
            d = _regs(dst)
            clash = (_regs(l[l.index(dst) + len(dst):]) - d) & set(inflight)
            if clash:
                problems.append(f"line {i}: inline MFMA reads in-flight v{min(clash)}")
            for r in d:
                inflight[r] = i
            nops = 0
            continue
        if in_asm and op == "s_nop":
            nops += int(l.split()[1], 0) + 1
            if nops >= MIN_WAIT_STATES:
                inflight.clear()
                nops = 0
            continue
        if op.startswith("s_"):
            continue
        touched = _regs(l) & set(inflight)
        if touched:
            problems.append(f"line {i}: '{l[:60]}' touches v{min(touched)} of the MFMA at line {inflight[min(touched)]}")
            for r in touched:
                inflight.pop(r, None)
    return problems


@pytest.fixture(scope="module")
def attention_asm(tmp_path_factory):
    if not os.path.exists(HIPCC) and shutil.which(HIPCC) is None:
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("asm") / "attention.s"
    flags = [f for f in B.FLAGS if f != "-fPIC"] + B.EXTRA.get("attention.hip", [])
    cmd = [HIPCC] + flags + ["-x", "hip", "--cuda-device-only", "-S", os.path.join(B.CSRC, "attention.hip"), "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return out.read_text().split("\n")


def _kernels(lines):
    heads = [i for i, l in enumerate(lines) if re.match(r"^_Z\S*attn_fwd_bf16\S*:", l)]
    for h in heads:
        end = next(i for i in range(h, len(lines)) if lines[i].startswith(".Lfunc_end"))
        yield lines[h].split(":")[0], lines[h:end]


def test_every_bf16_attention_kernel_is_scanned(attention_asm):
    names = [n for n, _ in _kernels(attention_asm)]
    assert len(names) == 4, names          # two shapes, with and without the fused q norm


def test_no_read_of_scores_before_the_wait_states(attention_asm):
    for name, body in _kernels(attention_asm):
        n_inline = sum(1 for l in body if l.strip().startswith("v_mfma"))
        assert n_inline > 0
        problems = scan(body)
        assert not problems, f"{name}:\n" + "\n".join(problems[:10])


def test_scanner_flags_a_copy_before_the_wait_states():
    body = [";;#ASMSTART", "v_mfma_f32_32x32x16_bf16 v[96:111], v[1:4], v[5:8], v[96:111]", ";;#ASMEND",
            "v_mov_b64_e32 v[200:201], v[96:97]",
            ";;#ASMSTART", "s_nop 7", "s_nop 4", ";;#ASMEND", "v_exp_f32_e32 v10, v96"]
    assert len(scan(body)) == 1
    fused = [";;#ASMSTART", "v_mfma_f32_32x32x16_bf16 v[96:111], v[1:4], v[5:8], v[96:111]", "s_nop 7", "s_nop 4",
             ";;#ASMEND", "v_mov_b64_e32 v[200:201], v[96:97]"]
    assert scan(fused) == []
    short = [";;#ASMSTART", "v_mfma_f32_32x32x16_bf16 v[96:111], v[1:4], v[5:8], v[96:111]", "s_nop 7",
             ";;#ASMEND", "v_exp_f32_e32 v10, v96"]
    assert len(scan(short)) >= 1
