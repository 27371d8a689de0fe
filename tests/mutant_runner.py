"""Run every oracle pin against one compiled oracle library and print the
names of the pins that failed, as JSON (used by test_oracle_mutants.py)."""
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from tests.oracle_pins import ALL_PINS  # noqa: E402


def main(libpath):
    lib = oracle.load(libpath)
    caught = []
    for pin in ALL_PINS:
        try:
            pin(lib)
        except (AssertionError, ValueError, IndexError):
            caught.append(pin.__name__)
    print(json.dumps(caught))


if __name__ == "__main__":
    main(sys.argv[1])
