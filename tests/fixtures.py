"""Readers of the cited text fixtures under tests/golden/ (values the paper
prints; each file names the passage it comes from)."""
import os

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def rows(name):
    """Whitespace-separated rows of a fixture, comments and blank lines dropped."""
    out = []
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.split("#", 1)[0].strip()
            if line:
                out.append(line.split())
    return out


def table(name):
    """A two-column fixture as a dict of floats."""
    return {k: float(v) for k, v in rows(name)}
