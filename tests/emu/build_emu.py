"""Builds the decoder library's own sources for the host CPU on the SIMT stand-in of simt.h.

The HIP sources are copied with five mechanical substitutions, all device-to-host plumbing:
  * `#include <hip/hip_runtime.h>` -> `#include "simt.h"`;
  * `__builtin_amdgcn_*` -> `emu_amdgcn_*` (the stand-ins of the AMDGPU builtins);
  * the inline-assembly statements (direct global->LDS loads, vector-memory waits) -> calls;
  * the LDS address cast in `lds_addr` -> `emu_lds_off`;
  * `kernel<<<grid, block, smem, stream>>>(args)` -> `emu::launch(...)`, and
    `extern __shared__ T name[]` -> a pointer to the launch's dynamic LDS.
Everything else -- index arithmetic, loop structure, waits, barriers, the host library and its
launch sequence -- is compiled as written, so the emulated run exercises the same addresses the
GPU run computes. Test infrastructure: the product loads only the HIP build of the library.
"""
from __future__ import annotations

import os
import re
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_2601_09921_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
OUT = os.path.join(HERE, "_build")
LIB = os.path.join(OUT, "libpwdec_emu.so")
CLANG = "/opt/rocm/llvm/bin/clang++"


def _matching(text: str, i: int) -> int:
    """Index of the parenthesis closing the one at text[i]."""
    depth = 0
    for j in range(i, len(text)):
        if text[j] == "(":
            depth += 1
        elif text[j] == ")":
            depth -= 1
            if depth == 0:
                return j
    raise ValueError("unbalanced parentheses")


def _split_top(s: str) -> list[str]:
    """Splits on commas outside parentheses and angle brackets of template arguments."""
    parts, depth, cur = [], 0, ""
    for ch in s:
        if ch in "([{":
            depth += 1
        elif ch in ")]}":
            depth -= 1
        if ch == "," and depth == 0:
            parts.append(cur)
            cur = ""
        else:
            cur += ch
    parts.append(cur)
    return [p.strip() for p in parts]


def _operand(spec: str) -> str:
    """`"v"(expr)` -> expr."""
    i = spec.index("(")
    return spec[i + 1:_matching(spec, i)]


def rewrite_asm(text: str) -> str:
    out, pos = [], 0
    for m in re.finditer(r"asm\s+volatile\s*\(", text):
        if m.start() < pos:
            continue
        open_i = m.end() - 1
        close_i = _matching(text, open_i)
        body = text[open_i + 1:close_i]
        # the wait-state guard ahead of a direct-to-LDS load has no host meaning
        body = re.sub(r'^\s*LDS_DMA_GUARD\s*', "", body)
        tmpl = re.match(r'\s*"([^"]*)"', body).group(1)
        if tmpl.startswith("s_waitcnt vmcnt"):
            call = "emu_waitcnt_vm(0)"
        elif tmpl.startswith("global_load_lds_dword"):
            nbytes = {"global_load_lds_dwordx4": 16, "global_load_lds_dword": 4}[tmpl.split()[0]]
            ins = body.split("::", 1)[1].split(":")[0]
            ops = _split_top(ins)
            call = f"emu_lds_dma({nbytes}, {_operand(ops[0])}, {_operand(ops[1])}, {_operand(ops[2])})"
        else:
            raise ValueError(f"no host stand-in for inline assembly {tmpl!r}")
        out.append(text[pos:m.start()])
        out.append(call)
        pos = close_i + 1
    out.append(text[pos:])
    return "".join(out)


LAUNCH = re.compile(r"(\w+(?:<(?:[^<>;]|<[^<>;]*>)*>)?)<<<(.*?)>>>\(([^;]*)\);", re.S)


def rewrite_launches(text: str) -> str:
    def sub(m):
        name, cfg, args = m.group(1), _split_top(m.group(2)), m.group(3)
        cfg += ["0", "nullptr"][len(cfg) - 2:] if len(cfg) < 4 else []
        label = name.replace('"', "")
        return f'emu::launch("{label}", {name}, {", ".join(cfg)}, {args});'
    return LAUNCH.sub(sub, text)


def transform(text: str) -> str:
    text = text.replace("#include <hip/hip_runtime.h>", '#include "simt.h"')
    text = rewrite_asm(text)
    text = text.replace("__builtin_amdgcn_", "emu_amdgcn_")
    text = re.sub(r"\(uint32_t\)reinterpret_cast<uintptr_t>\(\(__attribute__\(\(address_space\(3\)\)\) T\*\)p\)",
                  "emu_lds_off(p)", text)
    text = re.sub(r"extern __shared__ (?:__align__\(\d+\) )?([\w ]+?) (\w+)\[\];",
                  r"\1* \2 = (\1*)emu::dyn_smem();", text)
    text = rewrite_launches(text)
    for bad in ("asm volatile", "<<<", "address_space(3)", "__builtin_amdgcn_"):
        if bad in text:
            raise ValueError(f"untranslated {bad!r} left")
    return text


def sources(csrc: str = CSRC) -> list[str]:
    return sorted(f for f in os.listdir(csrc) if f.endswith((".hip", ".cpp", ".h")))


def build(verbose: bool = False, opt: str = "-O2", csrc: str = CSRC, include: str = INCLUDE, out: str = OUT,
          lift: list[tuple[str, str]] = ()) -> str:
    """Translates and compiles every library source for the host; returns the library path.
    csrc / include / out default to the library's sources and tests/emu/_build. `lift`: extra
    (old, new) text substitutions, each of which must apply, e.g. to lift a configuration that
    the library rejects so that a test can replay it on the CPU."""
    src_out = os.path.join(out, "p", "csrc")
    inc_out = os.path.join(out, "include")
    os.makedirs(src_out, exist_ok=True)
    os.makedirs(inc_out, exist_ok=True)
    shutil.copy(os.path.join(include, "pwdec.h"), inc_out)
    units, used = [], set()
    for f in sources(csrc):
        with open(os.path.join(csrc, f)) as fh:
            t = transform(fh.read())
        for old, new in lift:
            if old in t:
                t = t.replace(old, new)
                used.add(old)
        dst = os.path.join(src_out, f)
        with open(dst, "w") as fh:
            fh.write(t)
        if not f.endswith(".h"):
            units.append(dst)
    if set(o for o, _ in lift) - used:
        raise ValueError(f"substitutions that matched nothing: {set(o for o, _ in lift) - used}")
    flags = [opt, "-g", "-std=c++20", "-fPIC", "-w", "-I", HERE, "-I", src_out, "-x", "c++"]
    objs, procs = [], []
    for u in units + [os.path.join(HERE, "simt.cpp"), os.path.join(HERE, "units.cpp")]:
        obj = os.path.join(out, os.path.basename(u) + ".o")
        cmd = [CLANG, *flags, "-c", u, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True), u))
        objs.append(obj)
    for p, u in procs:
        log, _ = p.communicate()
        if p.returncode != 0:
            raise RuntimeError(f"host build of {u} failed:\n{log}")
    lib = os.path.join(out, os.path.basename(LIB))
    r = subprocess.run([CLANG, "-shared", "-fPIC", *objs, "-o", lib + ".tmp"], capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(lib + ".tmp", lib)
    return lib


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
