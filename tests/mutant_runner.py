"""Run the oracle pins against one planted mistake, in a process of its own.

Usage: python -m tests.mutant_runner "<mutation name>" <work dir>
Prints "CAUGHT <pin>" when a pin fails, "MISSED" when every pin passes.
"""
import os
import sys

import oracle
from tests import pins
from tests.test_oracle_mutations import MUTATIONS


def main():
    name, work = sys.argv[1], sys.argv[2]
    old, new = MUTATIONS[name]
    src = oracle.source()
    if src.count(old) != 1:
        print("ANCHOR-MISSING")
        return 3
    orc = oracle.compile_variant(src.replace(old, new), os.path.join(work, "mutant.so"))
    for pin in pins.ALL_PINS:
        try:
            pin(orc)
        except (AssertionError, ValueError):
            print("CAUGHT", pin.__name__)
            return 0
    print("MISSED")
    return 1


if __name__ == "__main__":
    sys.exit(main())
