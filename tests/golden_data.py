"""Readers for the hand-written fixtures under tests/golden/."""
import os

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def clock_cycle(name="clock_cycle_m4_n3.txt"):
    """{kind: [[(i, j), ...] per clock, in file order]}."""
    out = {}
    for line in open(os.path.join(GOLDEN, name)):
        line = line.split("#", 1)[0].strip()
        if not line:
            continue
        head, tasks = line.split(":")
        kind, _clock = head.split()
        out.setdefault(kind, []).append(
            [tuple(int(v) for v in t.split(",")) for t in tasks.split()])
    return out
