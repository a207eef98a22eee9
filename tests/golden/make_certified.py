"""Write tests/golden/certified_inputs.json: for every named parity case (tests/certified_cases.py),
the key positions that margin certification re-draws (tests/certify.py).  Runs only the CPU oracle
and the input generator.

    python tests/golden/make_certified.py [case ...]     (default: every case; existing entries of
                                                          other cases are kept)
"""
from __future__ import annotations

import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from tests import certified_cases, certify  # noqa: E402


def main(argv):
    names = argv or list(certified_cases.CASES)
    path = certified_cases.GOLDEN
    rec = {"cases": {}}
    if os.path.exists(path):
        with open(path) as f:
            rec = json.load(f)
    rec["params"] = {"eps_s": certify.EPS_S, "eps_c": certify.EPS_C, "factor": certify.FACTOR,
                     "max_rounds": certify.MAX_ROUNDS,
                     "written_by": "tests/golden/make_certified.py (CPU oracle only)"}
    for name in names:
        wl = certified_cases.workload(name)
        opts = certified_cases.options(name)
        t0 = time.time()
        print(f"{name}: {wl.name} options[{opts.key()}]", flush=True)
        red, rounds, certs = certify.certify_workload(wl, certified_cases.problems(name), opts=opts,
                                                      log=lambda m: print(m, flush=True))
        summary = certify.summarize(certs)
        print(f"  {summary} ({time.time() - t0:.0f} s)", flush=True)
        rec["cases"][name] = {
            "workload": wl.name, "options": opts.key(), "rounds": rounds,
            "redrawn_keys": sum(len(v) for d in red.values() for v in d.values()),
            "summary": summary,
            "redraw": {str(p): {str(g): v for g, v in sorted(d.items())}
                       for p, d in sorted(red.items())}}
        with open(path + ".tmp", "w") as f:
            json.dump(rec, f, indent=1, sort_keys=True)
        os.replace(path + ".tmp", path)


if __name__ == "__main__":
    main(sys.argv[1:])
