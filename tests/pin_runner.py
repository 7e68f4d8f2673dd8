"""Run every oracle pin against each oracle library named on the command line
and print one JSON line per library: {"lib": path, "caught": [pin names that
failed]}.  Used by the sanitizer test, which starts it in a child process
with the AddressSanitizer runtime preloaded (an instrumented shared library
cannot be loaded into an uninstrumented interpreter any other way)."""
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(HERE))
sys.path.insert(0, HERE)

import oracle  # noqa: E402
import oracle_pins  # noqa: E402


def main(paths):
    for path in paths:
        orc = oracle.Oracle(oracle.load(path))
        caught = []
        for pin in oracle_pins.ALL_PINS:
            try:
                pin(orc)
            except AssertionError:
                caught.append(pin.__name__)
        print(json.dumps({"lib": path, "caught": caught}), flush=True)


if __name__ == "__main__":
    main(sys.argv[1:])
