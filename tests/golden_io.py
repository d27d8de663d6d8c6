"""Reader for the small text fixtures under tests/golden/."""
import os

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def read_fixture(name):
    """Returns (rows, expect): numeric data rows and ``expect key values...`` lines."""
    rows, expect = [], {}
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            parts = line.split()
            if parts[0] == "expect":
                expect[parts[1]] = [float(p) for p in parts[2:]]
            elif parts[0] in ("x", "y"):
                expect[parts[0]] = [float(p) for p in parts[1:]]
            else:
                rows.append([float(p) for p in parts])
    return rows, expect
