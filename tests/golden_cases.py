"""Parser for tests/golden/hand_examples.txt (hand-worked clocked SGD examples)."""
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
POLICIES = {"LAZY": 0, "WORST": 1, "ESSP": 2, "VAP": 5}
STEPS = {"ROWMEAN": 0, "SUM": 1, "SEQ": 2}


def load_cases(fname="hand_examples.txt"):
    cases, cur = [], None
    with open(os.path.join(GOLDEN, fname)) as f:
        for raw in f:
            line = raw.split("#", 1)[0].strip()
            if not line:
                continue
            tok = line.split()
            if tok[0] == "case":
                kv = dict(t.split("=", 1) for t in tok[2:])
                cur = dict(name=tok[1], N=int(kv["N"]), M=int(kv["M"]), K=int(kv["K"]), P=int(kv["P"]),
                           s=int(kv["s"]), eta=float(kv["eta"]), lam=float(kv["lam"]),
                           policy=POLICIES[kv["policy"]], step=STEPS[kv["step"]], ratings=[], owner=None,
                           expect=[], strata=int(kv["strata"]) if "strata" in kv else None,
                           v0=float(kv["v0"]) if "v0" in kv else None)
            elif tok[0] == "rating":
                cur["ratings"].append((int(tok[1]), int(tok[2]), float(tok[3])))
            elif tok[0] in ("L0", "R0"):
                cur[tok[0]] = np.array([float(x) for x in tok[1:]], dtype=np.float32)
            elif tok[0] == "owner":
                cur["owner"] = np.array([int(x) for x in tok[1:]], dtype=np.int32)
            elif tok[0] == "expect":
                e, key, vals = {}, None, []
                for t in tok[1:]:
                    if "=" in t:
                        if key is not None:
                            e[key] = vals
                        key, v = t.split("=", 1)
                        vals = [float(v)]
                    else:
                        vals.append(float(t))
                e[key] = vals
                cur["expect"].append(dict(clock=int(e["clock"][0]), L=np.array(e["L"]), R=np.array(e["R"]),
                                          loss=e.get("loss", [None])[0]))
            elif tok[0] == "end":
                cases.append(cur)
                cur = None
    return cases
