"""Static check of the attention kernel's explicitly waited loads (CPU only).

`attn_tile_kernel` issues some loads as inline assembly so that the compiler
does not place its own (too early) waits: the Q and rotary-table loads before a
workgroup's first three tile DMAs, and the K operands of a tile before its first
Q.K^T product.  Each group is followed by an `s_waitcnt` that names the loaded
registers.  Correctness then rests on two facts about the code the compiler
emits, which this test checks in the gfx950 assembly of every instantiation:

* the wait counts: the Q/rotary loads are covered by `vmcnt(n)` with n the
  DMAs issued after them (three tiles: 12 at head dim 128, 6 at 64); the K
  reads by `lgkmcnt(half)` then `lgkmcnt(0)` (LDS reads complete in order);
* no instruction between a load and the wait that covers it reads or writes
  the load's destination registers (the compiler believes the value is there
  as soon as the asm statement issues), including code in out-of-line blocks
  branched to in between.
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2609_31224_amd", "csrc", "kernels.hip")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _regs(op):
    out = set()
    for a, b in re.findall(r"[va]\[(\d+):(\d+)\]", op):
        out |= set(range(int(a), int(b) + 1))
    for a in re.findall(r"(?<![\w\[:])v(\d+)\b", op):
        out.add(int(a))
    return out


def _dest(line):
    m = re.search(r"^\S+ v\[(\d+):(\d+)\]", line)
    return set(range(int(m.group(1)), int(m.group(2)) + 1))


def _addr(line):
    """Registers a load reads (its operands after the destination)."""
    return _regs(line.split(",", 1)[1])


def _no_pending_address(body, loads):
    """No load's address comes from a register an earlier load of the group
    is still writing."""
    pending = set()
    for k in loads:
        if _addr(body[k]) & pending:
            return False
        pending |= _dest(body[k])
    return True


def _uses(body, labels, lo, hi, regs, skip=()):
    """Instructions in (lo, hi), and in out-of-line blocks branched to from
    there, that touch ``regs``."""
    hits, seen, todo = [], set(), []
    for k in range(lo + 1, hi):
        if k in skip:
            continue
        l = body[k]
        if l and not l.startswith(".") and _regs(l) & regs:
            hits.append(l)
        m = re.search(r"s_c?branch\w* (\.LBB\w+)", l)
        if m and not lo < labels[m.group(1)] < hi:
            todo.append(m.group(1))
    while todo:
        t = todo.pop()
        if t in seen:
            continue
        seen.add(t)
        k = labels[t]
        while k < len(body):
            l = body[k]
            if l and not l.startswith(".") and _regs(l) & regs:
                hits.append(l)
            m = re.search(r"s_c?branch\w* (\.LBB\w+)", l)
            if m and not lo < labels[m.group(1)] < hi and m.group(1) not in seen:
                todo.append(m.group(1))
            if l.startswith(("s_branch", "s_endpgm", "s_setpc")):
                break
            k += 1
    return hits


@pytest.fixture(scope="module")
def kernels(tmp_path_factory):
    if not os.path.exists(HIPCC) and not shutil.which("hipcc"):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("asm") / "kernels.s"
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           f"-I{os.path.join(ROOT, 'include')}", "--cuda-device-only", "-S", SRC, "-o", str(out)]
    subprocess.run(cmd, check=True, capture_output=True)
    src = open(out).read().split("\n")
    found = {}
    for i, l in enumerate(src):
        if "attn_tile_kernel" in l and not l.startswith(".") and l.split(";")[0].strip().endswith(":"):
            j = i
            while ".amdhsa_kernel" not in src[j]:
                j += 1
            body = [x.split(";")[0].strip() for x in src[i:j]]
            found[l.split(":")[0]] = body
    # head dim {64, 128} x descriptor batches {1, 8, 64 in the kernel arguments, device memory}
    assert len(found) == 8, sorted(found)
    return found


def _head_dim(name):
    return 128 if "attn_tile_kernelILi128E" in name else 64


def test_q_loads_waited(kernels):
    for name, body in kernels.items():
        D = _head_dim(name)
        ks = D // 32
        n_q = 3 * ks        # Q (ks) + rotary rows (2 ks) per lane
        n_dma = 3 * ks      # three tiles of DMAs issued after them
        labels = {l[:-1]: k for k, l in enumerate(body) if re.match(r"^\.LBB\w+:$", l)}
        loads = [k for k, l in enumerate(body)
                 if re.match(r"global_load_dwordx4 v\[\d+:\d+\], v\[\d+:\d+\], off offset:", l)][:n_q]
        assert len(loads) == n_q, name
        wait = next(k for k in range(loads[-1] + 1, len(body)) if body[k].startswith("s_waitcnt"))
        assert body[wait] == f"s_waitcnt vmcnt({n_dma})", (name, body[wait])
        dmas = sum(1 for k in range(loads[-1] + 1, wait) if body[k].startswith("global_load_lds"))
        assert dmas >= n_dma, (name, dmas)  # both addressing paths are laid out in between
        regs = set().union(*(_dest(body[k]) for k in loads))
        assert _no_pending_address(body, loads), name
        assert not _uses(body, labels, loads[-1], wait, regs), name
        for i, (a, b) in enumerate(zip(loads, loads[1:])):
            # between two loads, the registers of the loads already issued are pending
            issued = set().union(*(_dest(body[k]) for k in loads[:i + 1]))
            assert not _uses(body, labels, a, b, issued), name


def test_k_operand_reads_waited(kernels):
    for name, body in kernels.items():
        D = _head_dim(name)
        n = 4 * (D // 32)   # K operands per tile and lane
        labels = {l[:-1]: k for k, l in enumerate(body) if re.match(r"^\.LBB\w+:$", l)}
        groups, k = [], 0
        while k < len(body):
            if body[k].startswith("ds_read_b128"):
                g, x = [k], k + 1
                while len(g) < n and x < len(body) and not body[x].startswith(("s_waitcnt", "v_mfma")):
                    if body[x].startswith("ds_read_b128"):
                        g.append(x)
                    x += 1
                if len(g) == n:
                    groups.append(g)
                    k = g[-1] + 1
                    continue
            k += 1
        assert groups, name
        for g in groups:
            dests = [_dest(body[x]) for x in g]
            assert _no_pending_address(body, g), name
            waits = [x for x in range(g[-1] + 1, len(body)) if "lgkmcnt" in body[x]]
            first = waits[0]
            regs = set().union(*dests)
            assert not _uses(body, labels, g[0], first, regs, skip=set(g)), name
            if n == 16:
                # two halves: lgkmcnt(8) covers the first eight reads, lgkmcnt(0) the rest
                assert body[first] == "s_waitcnt lgkmcnt(8)", (name, body[first])
                second = waits[1]
                assert body[second] == "s_waitcnt lgkmcnt(0)", (name, body[second])
                assert not _uses(body, labels, first, second, set().union(*dests[n // 2:])), name
            else:
                assert body[first] == "s_waitcnt lgkmcnt(0)", (name, body[first])
