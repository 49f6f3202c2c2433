"""Checks on the gfx950 assembly of the k-mer-local window attention (attn_kl).

attn_kl loads the next query tile's Q with inline-assembly global loads that
it does not wait for at once: the registers are written when the loads land,
and the kernel's own waits (a stage count of steps later) cover them.  That is
only correct while the compiler leaves those registers alone until the copy
at the query-tile boundary (no spill, no move, no other use).  Its global ->
LDS copies are inline assembly too, so the compiler inserts no wait of its own
in front of the step loop's LDS reads.  These tests compile the source to
assembly (no GPU needed) and check both facts, so a compiler change that
breaks them fails here before anything runs on a GPU.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2511_14694_amd import build as B

# head_dim -> (symbol, waves per workgroup, LDS stages) of the instantiations
KERNELS = {
    128: ("_ZN12_GLOBAL__N_17attn_klILi128ELi4ELi4EEEv15focus_attn_descfl", 4, 4),
    64: ("_ZN12_GLOBAL__N_17attn_klILi64ELi4ELi4EEEv15focus_attn_descfl", 4, 4),
}


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc is not available")
    out = tmp_path_factory.mktemp("isa") / "window_attn.s"
    src = os.path.join(B.CSRC, "window_attn.hip")
    cmd = [hipcc, *B.HIPCC_FLAGS, *B.EXTRA_FLAGS.get("window_attn.hip", []), "--cuda-device-only", "-S", src,
           "-o", str(out)]
    subprocess.run(cmd, check=True, capture_output=True)
    return out.read_text().split("\n")


def _body(lines, name):
    start = next(i for i, line in enumerate(lines) if line.startswith(name + ":"))
    end = next(i for i in range(start, len(lines)) if lines[i].startswith(".Lfunc_end"))
    return start, end


def _regs(text):
    used = set()
    for m in re.finditer(r"v\[(\d+):(\d+)\]", text):
        used |= set(range(int(m.group(1)), int(m.group(2)) + 1))
    for m in re.finditer(r"\bv(\d+)\b", text):
        used.add(int(m.group(1)))
    return used


@pytest.mark.parametrize("head_dim", [128, 64])
def test_prefetched_q_registers_untouched_until_copied(asm, head_dim):
    name, waves, stages = KERNELS[head_dim]
    start, end = _body(asm, name)
    # the asynchronous Q loads: inline-assembly blocks of plain global loads
    # with no wait inside
    prefetch, blocks = set(), 0
    i = start
    while i < end:
        if "ASMSTART" in asm[i]:
            j = i
            while "ASMEND" not in asm[j]:
                j += 1
            body = [x.strip() for x in asm[i + 1:j] if x.strip()]
            if body and all(b.startswith("global_load_dwordx4") for b in body):
                blocks += 1
                for b in body:
                    prefetch |= _regs(b.split(",")[0])
            i = j
        i += 1
    assert blocks > 0, "no asynchronous Q load found"
    assert len(prefetch) == 4 * (head_dim // 16)
    # Copies of the tiles in flight at a query-tile boundary: (stages - 1)
    # steps' copies of 2 x (tile bytes / 1 KB / waves) each.
    in_flight = (stages - 1) * 2 * (32 * head_dim * 2 // 1024 // waves)
    uses = 0
    in_asm = False
    last_wait = None  # vmcnt of the latest s_waitcnt in layout order
    for line in asm[start:end]:
        s = line.strip()
        if "ASMSTART" in s or "ASMEND" in s:
            in_asm = "ASMSTART" in s
            continue
        if not s or s.startswith((";", ".")) or s.endswith(":"):
            continue
        if in_asm and s.startswith("global_load_dwordx4") and _regs(s.split(",")[0]) & prefetch:
            last_wait = None  # a new prefetch: no wait covers it yet
            continue
        m = re.match(r"s_waitcnt\b.*vmcnt\((\d+)\)", s)
        if m:
            last_wait = int(m.group(1))
        if not in_asm and _regs(s) & prefetch:
            # the only other access: the copy into the working Q registers,
            # reading them as a source, after the wait that covers the loads
            assert s.startswith("v_mov_b"), s
            assert not (_regs(s.split(None, 1)[1].split(",", 1)[0]) & prefetch), s
            assert last_wait is not None and last_wait <= in_flight, (s, last_wait)
            uses += 1
    assert uses, "the prefetched Q is never copied"


@pytest.mark.parametrize("head_dim", [128, 64])
def test_no_spills_and_no_compiler_wait_before_lds_reads(asm, head_dim):
    name = KERNELS[head_dim][0]
    # kernel metadata: the fields after .name are in alphabetical order
    i = next(k for k, line in enumerate(asm) if re.search(r"\.name:\s+" + re.escape(name) + r"$", line))
    spill = next(line for line in asm[i:] if ".vgpr_spill_count:" in line)
    assert int(spill.split(":")[1]) == 0, spill
    start, end = _body(asm, name)
    prev, in_asm = None, False
    for line in asm[start:end]:
        s = line.strip()
        if "ASMSTART" in s or "ASMEND" in s:
            in_asm = "ASMSTART" in s
            prev = None
            continue
        if in_asm or not s or s.startswith((";", ".")) or s.endswith(":"):
            continue
        if prev is not None and prev.startswith("s_waitcnt") and "vmcnt" in prev:
            assert not s.startswith(("ds_read", "v_mfma")), f"compiler wait before an LDS read: {prev} -> {s}"
        prev = s
