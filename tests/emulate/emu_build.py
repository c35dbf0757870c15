"""Builds the plan emulator (``emu_main.cpp``) with gcc, AddressSanitizer and
UndefinedBehaviorSanitizer.

The plan kernels are taken from ``plan.hip`` as they are, minus the launchers at its
end (``emu_main.cpp`` launches them itself); the dynamic LDS array becomes the
emulator's per-workgroup buffer, and each static LDS array registers itself so that
it starts every workgroup filled with garbage.  The host code is ``api.hip`` itself.
"""
import os
import re
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_1906_07155_amd", "csrc")


def plan_kernels() -> str:
    src = open(os.path.join(CSRC, "plan.hip")).read()
    cut = src.index("hipError_t launch_level_map(")
    src = src[:cut] + "}  // namespace rex\n"
    src = src.replace("extern __shared__ int32_t smem[];", "int32_t *smem = emu_smem;")
    src, n = re.subn(r"__shared__ (\w+) (\w+)((?:\[\w+\])?);",
                     r"static \1 \2\3; emu_register(&\2, sizeof(\2));", src)
    assert n >= 1 and "__shared__" not in src, "unexpected LDS declarations in plan.hip"
    return ("extern int32_t *emu_smem;\nvoid emu_register(void *p, size_t n);\n" + src)


def build(outdir: str, edit=None) -> str:
    """Compile the emulator into outdir; `edit` (str -> str), if given, changes the
    kernels' source first (to plant a mistake the emulator must catch)."""
    src = plan_kernels()
    if edit is not None:
        changed = edit(src)
        assert changed != src, "the edit changed nothing"
        src = changed
    with open(os.path.join(outdir, "plan_kernels.inc"), "w") as f:
        f.write(src)
    out = os.path.join(outdir, "plan_emu")
    subprocess.check_call(["g++", "-std=c++17", "-O1", "-g", "-pthread", "-Wno-attributes",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                           "-fno-omit-frame-pointer", "-I" + HERE, "-I" + outdir, "-I" + CSRC,
                           "-I" + os.path.join(ROOT, "include"),
                           os.path.join(HERE, "emu_main.cpp"), "-o", out])
    return out


if __name__ == "__main__":
    print(build(sys.argv[1] if len(sys.argv) > 1 else os.getcwd()))
