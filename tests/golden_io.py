"""Reader for the small text fixtures under tests/golden/."""
import os

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def read_uniquify_example():
    keys, counts, values = [], {}, {}
    with open(os.path.join(GOLDEN, "uniquify_example.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            parts = line.split()
            if parts[0] == "keys":
                keys = [int(p, 16) for p in parts[1:]]
            elif parts[0] == "count":
                counts[int(parts[1], 16)] = int(parts[2])
            elif parts[0] == "value":
                values[int(parts[1], 16)] = float(parts[2])
    return keys, counts, values
