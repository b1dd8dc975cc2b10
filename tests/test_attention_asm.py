"""The bf16 attention kernel issues its score MFMAs as inline assembly, which
the compiler does not see as MFMAs: it inserts no wait states after them.
The kernel keeps the distance itself (the last MFMA pair of a tile and the
wait states after it are one asm statement).  This test compiles the kernel
for gfx950 with the library's own flags and checks, in every instance, that
no instruction reads, writes or copies a score register between an inline
MFMA that writes it and the wait states, and that those are at least the 12
the compiler itself puts between this MFMA and a vector read of its result,
and that no inline MFMA reads a register a vector instruction wrote in the 2
wait states before it.  The scan follows every path of the control flow.
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


def _blocks(lines):
    """Basic blocks of one kernel: instructions (line, text, inside an asm
    statement) and successor block indices (branch targets and fallthrough)."""
    blocks = []

    def new(label):
        blocks.append({"label": label, "ins": [], "succ": [], "fall": True})
        return blocks[-1]

    cur, in_asm = new("entry"), False
    for i, raw in enumerate(lines):
        l = raw.strip()
        m = re.match(r"^(\.LBB\w+):", l) or re.match(r"^; %(bb\.\d+):", l)
        if m:
            cur = new(m.group(1))
            continue
        if l.startswith(";;#ASMSTART"):
            in_asm = True
            continue
        if l.startswith(";;#ASMEND"):
            in_asm = False
            continue
        if not l or l.startswith((".", ";")) or l.endswith(":"):
            continue
        op = l.split()[0]
        cur["ins"].append((i, l, in_asm))
        if op == "s_branch":
            cur["succ"].append(l.split()[1])
            cur["fall"] = False
            cur = new(None)
        elif op.startswith("s_cbranch"):
            cur["succ"].append(l.split()[1])      # and the fallthrough below
            cur = new(None)
        elif op in ("s_endpgm", "s_setpc_b64"):
            cur["fall"] = False
            cur = new(None)
    index = {b["label"]: k for k, b in enumerate(blocks) if b["label"]}
    for k, b in enumerate(blocks):
        succ = [index[s] for s in b["succ"] if s in index]
        if b["fall"] and k + 1 < len(blocks):
            succ.append(k + 1)
        b["succ"] = succ
    return blocks


def scan(lines):
    """Hazards of the inline MFMAs of one kernel, over every path.

    Each issued instruction counts one wait state (s_nop N counts N + 1).  An
    inline MFMA's result registers are in flight for MIN_WAIT_STATES after it;
    no other instruction may read or write them meanwhile.  A register written
    by a vector instruction may not be read by an inline MFMA within the next
    2 wait states.  States are merged over all predecessors to a fixpoint."""
    blocks = _blocks(lines)
    inflight_in = [dict() for _ in blocks]
    vwrite_in = [dict() for _ in blocks]
    problems = set()
    work = list(range(len(blocks)))
    while work:
        k = work.pop(0)
        inflight, vwrite = dict(inflight_in[k]), dict(vwrite_in[k])
        for i, l, in_asm in blocks[k]["ins"]:
            op = l.split()[0]
            ws = int(l.split()[1], 0) + 1 if op == "s_nop" else 1
            if in_asm and op.startswith("v_mfma"):
                dst = l.split()[1].rstrip(",")
                d = _regs(dst)
                srcs = _regs(l[l.index(dst) + len(dst):])
                bad = [r for r in srcs - d if inflight.get(r, 0) > 0]
                if bad:
                    problems.add((i, f"inline MFMA reads v{min(bad)} while an inline MFMA writes it"))
                bad = [r for r in srcs if vwrite.get(r, 0) > 0]
                if bad:
                    problems.add((i, f"inline MFMA reads v{min(bad)} within 2 wait states of a vector write"))
                inflight = {r: w - 1 for r, w in inflight.items() if w > 1}
                vwrite = {r: w - 1 for r, w in vwrite.items() if w > 1}
                for r in d:
                    inflight[r] = MIN_WAIT_STATES
                continue
            if not op.startswith("s_"):
                bad = [r for r in _regs(l) if inflight.get(r, 0) > 0]
                if bad:
                    problems.add((i, f"'{l[:60]}' touches v{min(bad)} of an inline MFMA in flight"))
            inflight = {r: w - ws for r, w in inflight.items() if w > ws}
            vwrite = {r: w - ws for r, w in vwrite.items() if w > ws}
            if op.startswith("v_") and not op.startswith("v_mfma"):
                for r in _regs(l.split()[1].rstrip(",")):
                    vwrite[r] = 2
        for s in blocks[k]["succ"]:
            changed = False
            for cur, into in ((inflight, inflight_in[s]), (vwrite, vwrite_in[s])):
                for r, w in cur.items():
                    if into.get(r, 0) < w:
                        into[r] = w
                        changed = True
            if changed and s not in work:
                work.append(s)
    return sorted(problems)


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
        assert not problems, f"{name}:\n" + "\n".join(f"line {i}: {m}" for i, m in problems[:10])


def test_scanner_flags_a_copy_before_the_wait_states():
    body = [";;#ASMSTART", "v_mfma_f32_32x32x16_bf16 v[96:111], v[1:4], v[5:8], v[96:111]", ";;#ASMEND",
            "v_mov_b64_e32 v[200:201], v[96:97]",
            ";;#ASMSTART", "s_nop 7", "s_nop 4", ";;#ASMEND", "v_exp_f32_e32 v10, v96"]
    assert len(scan(body)) == 1
    # over a loop back edge: the MFMA at the bottom, the read at the top
    loop = [".LBB0_1:", "v_exp_f32_e32 v10, v96",
            ";;#ASMSTART", "v_mfma_f32_32x32x16_bf16 v[96:111], v[1:4], v[5:8], v[96:111]", ";;#ASMEND",
            "s_cbranch_scc1 .LBB0_1", "s_endpgm"]
    assert len(scan(loop)) == 1
    # a vector write just before an inline MFMA reads it
    vw = ["v_mov_b32_e32 v5, 0", ";;#ASMSTART", "v_mfma_f32_32x32x16_bf16 v[96:111], v[1:4], v[5:8], v[96:111]",
          "s_nop 7", "s_nop 4", ";;#ASMEND"]
    assert len(scan(vw)) == 1
    fused = [";;#ASMSTART", "v_mfma_f32_32x32x16_bf16 v[96:111], v[1:4], v[5:8], v[96:111]", "s_nop 7", "s_nop 4",
             ";;#ASMEND", "v_mov_b64_e32 v[200:201], v[96:97]"]
    assert scan(fused) == []
    short = [";;#ASMSTART", "v_mfma_f32_32x32x16_bf16 v[96:111], v[1:4], v[5:8], v[96:111]", "s_nop 7",
             ";;#ASMEND", "v_exp_f32_e32 v10, v96"]
    assert len(scan(short)) >= 1


def _steady_loop(body):
    """The first loop (a backward branch) of a kernel holding exactly the 32
    MFMAs of one key tile: the steady key-tile loop."""
    labels = {}
    for i, l in enumerate(body):
        m = re.match(r"^(\.LBB\w+):", l)
        if m:
            labels[m.group(1)] = i
    for i, l in enumerate(body):
        m = re.match(r"\s+s_(cbranch_\w+|branch)\s+(\.LBB\w+)", l)
        if m and labels.get(m.group(2), i) < i:
            ins = [x.strip().split()[0] for x in body[labels[m.group(2)]:i + 1]
                   if x.strip() and not x.strip().startswith((".", ";")) and not x.strip().endswith(":")]
            if sum(1 for x in ins if x.startswith("v_mfma")) == 32:
                return ins
    return None


# Instructions of the steady key-tile loop as the library's flags compile it
# (8 waves: 233, 4 waves: 237), plus a small margin.  A change elsewhere in
# the kernel can make the compiler schedule this loop differently: a staged
# output store in the epilogue once grew the 4-wave loop to 257 instructions
# (each PV MFMA waiting for its own fragment reads) and made the 4-wave
# self-attention 8-12% slower.  A failure here asks for a timing check.
MAX_LOOP = {"ILi8ELi4E": 240, "ILi4ELi2E": 244}


def test_key_tile_loop_stays_compact(attention_asm):
    for name, body in _kernels(attention_asm):
        ins = _steady_loop(body)
        assert ins is not None, f"{name}: no loop of 32 MFMAs"
        limit = next(v for k, v in MAX_LOOP.items() if k in name)
        assert len(ins) <= limit, f"{name}: steady loop of {len(ins)} instructions (at most {limit})"
