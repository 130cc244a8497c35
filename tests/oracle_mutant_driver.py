"""Run every oracle pin against one compiled oracle library.

Usage: python oracle_mutant_driver.py <path-to-.so>
Exit status 0 when every pin passes, 1 when at least one fails (the names
of the failing pins are printed).
"""
import os
import sys

_HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, _HERE)
sys.path.insert(0, os.path.dirname(_HERE))

import oracle  # noqa: E402
import oracle_pins  # noqa: E402


def main(path):
    orc = oracle.load(path)
    failed = []
    for check in oracle_pins.ALL_CHECKS:
        try:
            check(orc)
        except AssertionError:
            failed.append(check.__name__)
            break
    print("failed:", ",".join(failed) if failed else "none", flush=True)
    return 1 if failed else 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1]))
