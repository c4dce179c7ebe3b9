"""Write printed_plans.json from the deployment-plan tables of the E2LLM paper.

Run once, with the path of the paper's LaTeX source as the one argument:
    python tests/golden/extract_printed_plans.py <paper source>

It parses every plan table (Sec. 4 Tables 3-6 and the App. B tables): each
replica's mode (P/D), its devices, which device is the master (starred) and
the GPU--CPU block split per device.  The tests read only the JSON it writes.
"""
from __future__ import annotations

import json
import os
import re
import sys

ROW_MODE = re.compile(r"^\s*(?:\\multirow\{(\d+)\}\{\*\}\{([PD])\}|([PD]))\s*&\s*(.*)$")
ROW_CONT = re.compile(r"^\s*&\s*(.*)$")
DEV = re.compile(r"Dev\.(\d+)(\$\^\{\\star\}\$)?")
GC = re.compile(r"(\d+)\s*--\s*(\d+)")
MODEL = re.compile(r"(Gpt-Oss-20b|Qwen3)")
BLOCKS = {"Gpt-Oss-20b": 24, "Qwen3": 48}


def parse(path: str):
    lines = open(path, encoding="utf-8").read().splitlines()
    tables = []
    cur = None
    method = None
    pending = None
    model_ctx = None
    for line in lines:
        if "\\caption{Deployment plans" in line:
            mm = MODEL.search(line)
            model_ctx = mm.group(1) if mm else None
            cap_txt = re.search(r"\\caption\{(.*)\}\s*$", line.strip())
            cur = dict(table=None, caption=cap_txt.group(1) if cap_txt else line.strip(),
                       model=model_ctx, plans=[])
            tables.append(cur)
            continue
        lab = re.search(r"\\label\{([^}]*)\}", line)
        if cur is not None and cur["table"] is None and lab and not cur["plans"]:
            cur["table"] = lab.group(1)
            continue
        if cur is None:
            continue
        cap = re.search(r"\\caption\{(HG|ELS|SPW)\}", line)
        if cap:
            method = cap.group(1)
            cur["plans"].append(dict(method=method, replicas=[]))
            pending = None
            continue
        if not cur["plans"]:
            continue
        m = ROW_MODE.match(line)
        if m and "Dev." in line:
            nrows = int(m.group(1)) if m.group(1) else 1
            mode = m.group(2) or m.group(3)
            rest = m.group(4)
            rep = dict(mode=mode, devices=[])
            cur["plans"][-1]["replicas"].append(rep)
            pending = [rep, nrows]
            _add_dev(rep, rest)
            pending[1] -= 1
            continue
        c = ROW_CONT.match(line)
        if c and "Dev." in line and pending and pending[1] > 0:
            _add_dev(pending[0], c.group(1))
            pending[1] -= 1
    return tables


def _add_dev(rep, text):
    d = DEV.search(text)
    g = GC.search(text)
    if not d or not g:
        raise ValueError(f"unparsed row: {text}")
    rep["devices"].append(dict(dev=int(d.group(1)), master=bool(d.group(2)),
                               gpu_blocks=int(g.group(1)), cpu_blocks=int(g.group(2))))


def main():
    if len(sys.argv) != 2:
        sys.exit("usage: extract_printed_plans.py <path of the paper's LaTeX source>")
    src = sys.argv[1]
    tables = parse(src)
    out = []
    for t in tables:
        model = t["model"]
        if model is None:
            # Tables 3 and 6 mix models per column block; the model is named in
            # the subtable caption there, so those are skipped here.
            continue
        for p in t["plans"]:
            out.append(dict(table=t["table"], caption=t["caption"], method=p["method"],
                            model=model, n_blocks=BLOCKS[model], replicas=p["replicas"]))
    dst = os.path.join(os.path.dirname(os.path.abspath(__file__)), "printed_plans.json")
    doc = dict(
        source=("E2LLM (arXiv 2606.03770): deployment-plan tables of Sec. 4 and App. B; "
                "G--C columns give GPU and CPU blocks per device, a star marks the master; "
                "Gpt-Oss-20b has 24 blocks and Qwen3-30B-A3B 48 (Sec. 4.1)."),
        plans=out)
    with open(dst, "w") as f:
        json.dump(doc, f, separators=(",", ":"))
        f.write("\n")
    n_rep = sum(len(p["replicas"]) for p in out)
    print(f"wrote {dst}: {len(out)} plans, {n_rep} replicas")


if __name__ == "__main__":
    main()
