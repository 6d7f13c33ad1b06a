"""Source-to-source elastic transformer for plain HIP kernels with 1-D or 2-D grids and
blocks (the paper's offline component, §6.4 and §5.2).

A plain kernel is written for one launch of gx x gy logical blocks of BX x BY threads (the
block given by a "// elastic: block BX" or "// elastic: block BXxBY" line above it) and reads
blockIdx, gridDim, threadIdx and blockDim in x and y.  Its elastic form NAME_elastic runs any
contiguous shard [begin, begin + len) of the G = gx * gy logical blocks, numbered
b = by * gx + bx, under any 1-D grid and any 1-D physical block:

* elastic grid: each physical block loops over the shard's logical blocks with a stride of
  the physical grid; blockIdx.x / .y become b mod gx and b div gx, gridDim.x / .y the logical
  gx and gy (so grid-stride loops inside the kernel keep their meaning);
* elastic block: a physical block of b threads (b dividing B = BX * BY) runs the B logical
  threads in B / b rounds; logical thread t = round * b + threadIdx.x has threadIdx.x / .y =
  t mod BX and t div BX, and blockDim.x / .y are BX and BY.  This needs logical threads that do
  not communicate, so a kernel that synchronises its block (__syncthreads) or declares
  block-shared memory keeps b = B;
* the body runs in a lambda per logical block (per logical thread for an elastic block), so
  its return statements end that logical block (thread) only; __shared__ declarations are
  hoisted to the kernel's scope.

Every logical thread executes the original body once with the original ids, so the outputs are
those of the plain launch whatever the shard plan, grid and block.  Ids in z are rejected.

For each kernel the generated file also holds two C-ABI launchers:
  int NAME_plain_launch(<params>, int grid_x, int grid_y, void *stream)
      (the plain kernel on a gx x gy grid of BX x BY blocks)
  int NAME_elastic_launch(<params>, int grid_x, int grid_y, long long begin, long long len,
                          int grid, int block, void *stream)
      (shard [begin, begin + len) of that logical launch on `grid` 1-D blocks of `block` threads)
returning 0, -3 for a shard / grid / block out of range, or the HIP error code.
"""
from __future__ import annotations

import os
import re
import subprocess
from dataclasses import dataclass

HERE = os.path.dirname(os.path.abspath(__file__))
PLAIN_DIR = os.path.join(HERE, "plain")

_KERNEL = re.compile(r"__global__\s+void\s+(\w+)\s*\(([^)]*)\)\s*\{")
_BLOCK_NOTE = re.compile(r"//\s*elastic:\s*block\s+(\d+)(?:\s*x\s*(\d+))?\s*$")
_Z_DIM = re.compile(r"\b(blockIdx|gridDim|threadIdx|blockDim)\.z\b")
_IDS = {"blockIdx.x": "__mi_bx", "blockIdx.y": "__mi_by", "gridDim.x": "__mi_gx", "gridDim.y": "__mi_gy",
        "threadIdx.x": "__mi_tx", "threadIdx.y": "__mi_ty", "blockDim.x": "__mi_bdx", "blockDim.y": "__mi_bdy"}


class TransformError(ValueError):
    pass


@dataclass
class Kernel:
    name: str
    params: str            # parameter list as written
    param_names: list      # forwarded argument names
    body: str              # text between the outer braces
    block: int             # logical block size (threads)
    bx: int                # logical block shape bx x by
    by: int
    shared_decls: list     # hoisted __shared__ declarations
    syncs: bool            # the body synchronises the block or shares memory

    @property
    def block_elastic(self) -> bool:
        return not self.syncs


def _match_brace(src: str, open_idx: int) -> int:
    """Index of the brace closing the one at open_idx (comments and strings skipped)."""
    depth, i, n = 0, open_idx, len(src)
    while i < n:
        ch = src[i]
        if src.startswith("//", i):
            i = src.find("\n", i)
            if i < 0:
                break
            continue
        if src.startswith("/*", i):
            i = src.find("*/", i) + 2
            continue
        if ch in "\"'":
            j = i + 1
            while j < n and src[j] != ch:
                j += 2 if src[j] == "\\" else 1
            i = j + 1
            continue
        if ch == "{":
            depth += 1
        elif ch == "}":
            depth -= 1
            if depth == 0:
                return i
        i += 1
    raise TransformError("unbalanced braces")


def _param_names(params: str) -> list:
    names = []
    for p in [p.strip() for p in params.split(",") if p.strip()]:
        p = re.sub(r"\[[^\]]*\]", "", p).strip()
        m = re.search(r"(\w+)\s*$", p)
        if not m or m.group(1) in ("int", "float", "const", "unsigned", "long", "double", "char", "void"):
            raise TransformError(f"unnamed parameter: {p!r}")
        names.append(m.group(1))
    return names


def _hoist_shared(body: str):
    decls = []

    def take(m):
        decls.append(m.group(0).strip())
        return ""

    body = re.sub(r"(?m)^[ \t]*__shared__[^;]*;[ \t]*\n?", take, body)
    return body, decls


def parse(src: str) -> list:
    """Plain kernels of `src`, in order."""
    kernels = []
    for m in _KERNEL.finditer(src):
        name, params = m.group(1), m.group(2).strip()
        # the annotation must be on one of the lines just above the kernel
        before = src[:m.start()].rstrip("\n").splitlines()[-4:]
        bx = by = None
        for line in reversed(before):
            bm = _BLOCK_NOTE.search(line.strip())
            if bm:
                bx, by = int(bm.group(1)), int(bm.group(2) or 1)
                break
        if bx is None:
            raise TransformError(f"{name}: no '// elastic: block N' line above the kernel")
        block = bx * by
        if block not in (64, 128, 256):
            raise TransformError(f"{name}: logical block must be 64, 128 or 256 threads")
        open_idx = m.end() - 1
        close = _match_brace(src, open_idx)
        body = src[open_idx + 1:close]
        md = _Z_DIM.search(body)
        if md:
            raise TransformError(f"{name}: id {md.group(0)} is not supported (grids and blocks in x and y)")
        body, shared = _hoist_shared(body)
        syncs = "__syncthreads" in body or bool(shared)
        kernels.append(Kernel(name, params, _param_names(params), body, block, bx, by, shared, syncs))
    return kernels


def _rewrite_ids(text: str) -> str:
    for k, v in _IDS.items():
        text = re.sub(r"\b" + re.escape(k) + r"\b", v, text)
    return text


PREAMBLE = """// Generated by paper_2307_04339_amd/transform/elastify.py from plain kernels: do not edit.
#include <hip/hip_runtime.h>

struct miriam_elastic_shard {
    long long begin, len;  // logical blocks [begin, begin + len), numbered by * gx + bx
    unsigned gx, gy;       // logical grid of the plain launch
};
"""


def emit(k: Kernel) -> str:
    body = _rewrite_ids(k.body)
    shared = "".join(f"    {d}\n" for d in k.shared_decls)
    tid = (f"            const unsigned __mi_tx = __mi_t % {k.bx}u, __mi_ty = __mi_t / {k.bx}u;\n"
           f"            (void)__mi_tx;\n"
           f"            (void)__mi_ty;\n")
    if k.block_elastic:
        inner = (f"        for (unsigned __mi_r = 0; __mi_r < {k.block}u / blockDim.x; ++__mi_r) {{\n"
                 f"            const unsigned __mi_t = __mi_r * blockDim.x + threadIdx.x;\n"
                 f"{tid}"
                 f"            [&]() {{{body}}}();\n"
                 f"        }}\n")
    else:
        # a kernel that synchronises or shares memory: the shared arrays are hoisted to kernel
        # scope, so every logical block ends at a barrier before the workgroup starts the next
        # one (its threads would otherwise overwrite shared data that others still read); the
        # trip count of the shard loop depends on blockIdx.x only, so the barrier is uniform
        barrier = "            __syncthreads();\n" if k.syncs else ""
        inner = (f"        {{\n"
                 f"            const unsigned __mi_t = threadIdx.x;\n"
                 f"{tid}"
                 f"            [&]() {{{body}}}();\n"
                 f"{barrier}"
                 f"        }}\n")
    kern = (f"__global__ void {k.name}_elastic({k.params}, miriam_elastic_shard __mi_sh) {{\n"
            f"{shared}"
            f"    const unsigned __mi_gx = __mi_sh.gx, __mi_gy = __mi_sh.gy;\n"
            f"    const unsigned __mi_bdx = {k.bx}u, __mi_bdy = {k.by}u;\n"
            f"    (void)__mi_bdx;\n"
            f"    (void)__mi_bdy;\n"
            f"    for (long long __mi_b = __mi_sh.begin + blockIdx.x; __mi_b < __mi_sh.begin + __mi_sh.len;\n"
            f"         __mi_b += gridDim.x) {{\n"
            f"        // logical block ids stay below 2^31 (checked by the launcher); 1-D grids need no division\n"
            f"        const unsigned __mi_bu = (unsigned)__mi_b;\n"
            f"        const unsigned __mi_by = __mi_gy == 1u ? 0u : __mi_bu / __mi_gx;\n"
            f"        const unsigned __mi_bx = __mi_bu - __mi_by * __mi_gx;\n"
            f"        (void)__mi_bx;\n"
            f"        (void)__mi_by;\n"
            f"{inner}"
            f"    }}\n"
            f"}}\n")
    args = ", ".join(k.param_names)
    block_ok = (f"(block == 64 || block == 128 || block == 256) && {k.block} % block == 0"
                if k.block_elastic else f"block == {k.block}")
    launchers = (
        f'extern "C" int {k.name}_plain_launch({k.params}, int grid_x, int grid_y, void *stream) {{\n'
        f"    if (grid_x < 1 || grid_y < 1 || grid_y > 65535) return -3;\n"
        f"    hipLaunchKernelGGL({k.name}, dim3(grid_x, grid_y), dim3({k.bx}, {k.by}), 0, (hipStream_t)stream, {args});\n"
        f"    return (int)hipGetLastError();\n"
        f"}}\n\n"
        f'extern "C" int {k.name}_elastic_launch({k.params}, int grid_x, int grid_y, long long begin,\n'
        f"        long long len, int grid, int block, void *stream) {{\n"
        f"    const long long num_blocks = (long long)grid_x * grid_y;\n"
        f"    if (grid_x < 1 || grid_y < 1 || num_blocks > 0x7fffffffLL || begin < 0 || len < 1 ||\n"
        f"        begin + len > num_blocks || grid < 1 || !({block_ok}))\n"
        f"        return -3;\n"
        f"    miriam_elastic_shard sh{{begin, len, (unsigned)grid_x, (unsigned)grid_y}};\n"
        f"    hipLaunchKernelGGL({k.name}_elastic, dim3(grid), dim3(block), 0, (hipStream_t)stream, {args}, sh);\n"
        f"    return (int)hipGetLastError();\n"
        f"}}\n")
    return kern + "\n" + launchers


def transform(src: str, plain_include: str | None = None) -> str:
    """Elastic forms (plus launchers) of every kernel in `src`.  The plain kernels themselves
    come from `plain_include` (an #include of the plain source) so both are in one library."""
    out = [PREAMBLE]
    if plain_include:
        out.append(f'#include "{plain_include}"\n')
    for k in parse(src):
        out.append(f"\n// ---- {k.name}: logical block {k.bx} x {k.by}, "
                   f"{'elastic block' if k.block_elastic else 'block fixed (it synchronises or shares memory)'}\n")
        out.append(emit(k))
    return "".join(out)


def build(out_so: str, build_dir: str, flags: list) -> str:
    """Transform every plain source and compile the plain and elastic kernels into out_so."""
    os.makedirs(build_dir, exist_ok=True)
    objs = []
    for f in sorted(os.listdir(PLAIN_DIR)):
        if not f.endswith(".hip"):
            continue
        path = os.path.join(PLAIN_DIR, f)
        with open(path) as fh:
            src = fh.read()
        gen = os.path.join(build_dir, f.replace(".hip", "_elastic.hip"))
        with open(gen, "w") as fh:
            fh.write(transform(src, plain_include=path))
        obj = gen + ".o"
        r = subprocess.run(["hipcc"] + flags + ["-c", gen, "-o", obj], capture_output=True, text=True)
        if r.returncode != 0:
            msg = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l)
            raise RuntimeError(f"hipcc failed for the elastic form of {f}:\n{msg}")
        objs.append(obj)
    tmp = out_so + ".tmp"
    arch = [f for f in flags if f.startswith("--offload-arch")]
    r = subprocess.run(["hipcc"] + arch + ["-shared", "-fPIC", "-o", tmp] + objs, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stderr)
    os.replace(tmp, out_so)
    return out_so
