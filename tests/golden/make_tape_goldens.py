"""Write tests/golden/tape_sha256.json: SHA-256 of the tapes the reference
encoder (oracle/tape_ref.py) produces for the five benchmark programs at their
full sizes.  Calls only oracle/ and the seeded input generators."""
import hashlib
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import tape_ref  # noqa: E402
from workloads import configs  # noqa: E402


def main():
    out = {}
    for name in configs.ORDER[:4]:
        w = configs.build(name, L=1)
        out[name] = hashlib.sha256(tape_ref.encode(w.bytecode)).hexdigest()
    w = configs.random_programs(L=1)
    h = hashlib.sha256()
    for bc in w.programs:
        h.update(tape_ref.encode(bc))
    out["random_programs"] = h.hexdigest()
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tape_sha256.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1, sort_keys=True)
        f.write("\n")
    print(json.dumps(out, indent=1))


if __name__ == "__main__":
    main()
