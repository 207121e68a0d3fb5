"""The compiled gfx950 kernels keep every barrier loop uniform (CPU only: hipcc emits
the device assembly, nothing runs).

A workgroup barrier (s_barrier) inside a loop must be reached by every lane of every
wave on every trip. If a loop that holds a barrier leaves or repeats per lane (its
back edge lowered as an exec-mask update, `s_andn2_b64 exec, exec, ...`, rather than
a scalar branch), the lanes that leave early stop arriving at the barrier while the
others wait there: a hang. A copy loop written with thread-0 steps around its barrier
was compiled that way once. This test parses the loop nesting that LLVM writes into
the assembly comments and checks, for every kernel of the library, that no loop holding
a barrier has a per-lane back edge of its own (loops nested inside it, such as the
thread-0 polling of a ready flag, may be per lane as long as they hold no barrier).
"""
import os
import re
import subprocess
import tempfile

import pytest

from paper_2601_20595_amd import build as libbuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
KERNEL_SOURCES = ["chunk_gemm.hip", "chunk_attn.hip"]

_LABEL = re.compile(r"^(?:\.L(BB\d+_\d+)|; (%bb\.\d+)):")
_FUNC = re.compile(r"^(_Z\S+):")


def device_asm(src_path: str) -> str:
    """gfx950 assembly of one HIP source, with the library's own flags."""
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "k.s")
        cmd = [libbuild.hipcc()] + libbuild.compile_flags() + ["--cuda-device-only", "-S", "-x", "hip", src_path,
                                                               "-o", out]
        r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
        assert r.returncode == 0, r.stdout.decode(errors="replace")
        return open(out).read()


def divergent_barrier_loops(asm: str):
    """[(function, loop header)] of loops that hold an s_barrier (in their own blocks or
    nested loops) and whose own blocks take a per-lane back edge (s_andn2_b64 exec, exec)."""
    flagged = []
    funcs = []
    for line in asm.split("\n"):
        m = _FUNC.match(line)
        if m:
            funcs.append((m.group(1), []))
        elif funcs:
            funcs[-1][1].append(line)
    for fname, lines in funcs:
        blocks = []                  # [name, innermost loop header or None, [instructions]]
        parent = {}                  # loop header -> enclosing loop header (None at depth 1)
        cur = None
        pending = None               # annotations of the block being opened
        for line in lines:
            m = _LABEL.match(line)
            if m:
                cur = [m.group(1) or m.group(2), None, []]
                blocks.append(cur)
                pending = [line]
                continue
            if cur is None:
                continue
            stripped = line.strip()
            if pending is not None and stripped.startswith(";"):
                pending.append(line)
                continue
            if pending is not None:
                text = "\n".join(pending)
                parents = [(int(d), h) for h, d in re.findall(r"Parent Loop (BB\d+_\d+) Depth=(\d+)", text)]
                if "Loop Header" in text and cur[0].startswith("BB"):
                    cur[1] = cur[0]
                    if parents:
                        parent[cur[0]] = max(parents)[1]   # the deepest enclosing loop
                    else:
                        parent[cur[0]] = None
                else:
                    m2 = re.search(r"in Loop: Header=(BB\d+_\d+) Depth=\d+", text)
                    cur[1] = m2.group(1) if m2 else None
                pending = None
            cur[2].append(stripped)

        def chain(h):
            while h is not None:
                yield h
                h = parent.get(h)

        has_barrier, own_lane_exit = set(), set()
        for name, loop, insts in blocks:
            if loop is None:
                continue
            if any(i.startswith("s_barrier") for i in insts):
                has_barrier.update(chain(loop))
            if any(re.match(r"s_andn2_b64 exec, exec,", i) for i in insts):
                own_lane_exit.add(loop)
        for h in sorted(has_barrier & own_lane_exit):
            flagged.append((fname, h))
    return flagged


_BAD = r"""
#include <hip/hip_runtime.h>
// per-lane loop exit around a barrier: lanes leave at different trips
__global__ void per_lane_exit(const int* p, int* out) {
  int i = 0;
  for (;; ++i) {
    __syncthreads();
    if (p[threadIdx.x] <= i) break;
  }
  out[threadIdx.x] = i;
}
// the same loop with a workgroup-uniform exit: fine
__global__ void uniform_exit(const int* p, int* out) {
  __shared__ int s;
  int i = 0;
  for (;; ++i) {
    __syncthreads();
    if (threadIdx.x == 0) s = p[0] <= i;
    __syncthreads();
    if (__builtin_amdgcn_readfirstlane(s)) break;
  }
  out[threadIdx.x] = i;
}
"""


def test_checker_flags_a_per_lane_barrier_loop_and_passes_a_uniform_one():
    with tempfile.TemporaryDirectory() as d:
        src = os.path.join(d, "probe.hip")
        with open(src, "w") as f:
            f.write(_BAD)
        flagged = divergent_barrier_loops(device_asm(src))
    names = {f for f, _ in flagged}
    assert any("per_lane_exit" in f for f in names), flagged
    assert not any("uniform_exit" in f for f in names), flagged


@pytest.mark.parametrize("source", KERNEL_SOURCES)
def test_library_kernels_have_no_per_lane_barrier_loop(source):
    asm = device_asm(os.path.join(ROOT, "paper_2601_20595_amd", "csrc", source))
    kernels = re.findall(r"^(_Z\S+):", asm, re.M)
    assert kernels, "no kernels found in %s" % source
    assert divergent_barrier_loops(asm) == []
