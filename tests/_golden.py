"""Reader of the fixtures under tests/golden/: values the paper prints, one
record per line, '#' lines carry the citation."""
import os

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def records(name):
    """Whitespace-separated fields of every non-comment line of golden/<name>."""
    out = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                out.append(line.split())
    return out


def table(name):
    """First field -> remaining fields parsed as floats."""
    return {r[0]: [float(v) for v in r[1:]] for r in records(name)}
