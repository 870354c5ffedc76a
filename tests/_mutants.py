"""Builds copies of the C oracle with one planted mistake (test infrastructure for
the mutation tests: a pin that cannot tell a wrong oracle from the right one
pins nothing)."""
import os
import subprocess

from oracle import build_oracle


def build_mutant(tmp_dir: str, edits) -> str:
    """Apply (old, new) source replacements, each of a text found exactly once in
    the oracle source, and compile the result; returns the library path."""
    src = open(build_oracle.SOURCE).read()
    for old, new in edits:
        assert src.count(old) == 1, f"mutation site not unique: {old!r}"
        src = src.replace(old, new)
    c = os.path.join(tmp_dir, "mutant.c")
    so = os.path.join(tmp_dir, "libmutant.so")
    with open(c, "w") as fh:
        fh.write(src)
    subprocess.run(["gcc", *build_oracle.CFLAGS, "-o", so, c, "-lm"], check=True)
    return so
