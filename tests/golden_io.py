"""Readers for the hand-written fixtures in tests/golden (test-side parsing only)."""

import os

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        for raw in f:
            s = raw.split("#", 1)[0].strip()
            if s:
                yield s.split()


def read_tree(name):
    out = {"nodes": []}
    for t in _lines(name):
        if t[0] == "B":
            out["B"] = int(t[1])
        elif t[0] == "p":
            out["p"] = [int(x) for x in t[1:]]
        elif t[0] == "leaves":
            out["leaves"] = [int(x) for x in t[1:]]
        else:
            n, pos, path, par = (int(x) for x in t[:4])
            anc = {int(x) for x in t[4].split(",")}
            out["nodes"].append(dict(node=n, position=pos, path=path, parent=par, anc=anc))
    return out


def read_accept(name):
    cases, cur = [], None
    for t in _lines(name):
        if t[0] == "case":
            cur = {"name": t[1]}
            cases.append(cur)
        elif t[0] in ("argmax", "draft"):
            cur[t[0]] = [int(x) for x in t[1:]]
        elif t[0] == "expect":
            kv = dict(zip(t[1::2], t[2::2]))
            cur["L"] = int(kv["L"])
            cur["path"] = int(kv["path"])
            cur["node"] = int(kv["node"])
            cur["nodes"] = [int(x) for x in kv["nodes"].split(",")]
            cur["tokens"] = [int(x) for x in kv["tokens"].split(",")]
    return cases


def read_boundary(name):
    out = {}
    for t in _lines(name):
        out[t[0]] = [float(x) if "." in x else int(x) for x in t[1:]]
    return out
