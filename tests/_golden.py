"""Readers for the text fixtures under tests/golden/."""
import os

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def read_table(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                rows.append(line.split())
    return rows


def read_keyvals(name):
    out = {}
    for row in read_table(name):
        out[row[0]] = float(row[1]) if any(ch in row[1] for ch in ".e") else int(row[1])
    return out
