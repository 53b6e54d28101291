"""Writes tests/parity_rel_l2.md from the JSON lines that the GPU suite records
when SSM_PARITY_RECORD is set (tests/conftest.py).

usage: python tests/parity_record_md.py <parity.jsonl> tests/parity_rel_l2.md "<command>"
"""
import collections
import json
import sys

src, dst, cmd = sys.argv[1], sys.argv[2], sys.argv[3]
d = collections.OrderedDict()
for l in open(src):
    r = json.loads(l)
    d.setdefault(r["test"], []).append(r)
out = ["# Achieved parity (rel-L2 per output tensor against the fp64 oracle)", "",
       "MI355X (gfx950), one GPU.  Every check of the GPU test suite, as recorded by `tests/gpu_helpers.check` "
       "with `SSM_PARITY_RECORD` set; the command:", "", "    " + cmd, "",
       "Tolerances: 1e-5 for fp32 inputs; 1e-4 for the scan outputs of bf16-input calls (the oracle reads the same "
       "bf16 bits); 2e-2 for outputs downstream of the bf16 GEMM operands and for the stack; GEMM-only checks 1e-5 "
       "(1e-4 over 262,144-long reductions); the language head 2e-4 against the oracle with its bf16 operands "
       "rounded as the GPU rounds them, 2e-2 against the exact model.  `worst` is the output with the largest error/tolerance ratio.", "",
       "| test | checks | worst output | rel-L2 | tolerance |", "|---|---|---|---|---|"]
for t, rs in d.items():
    m = max(rs, key=lambda r: r["rel_l2"] / r["tol"])
    out.append(f"| `{t.split('::', 1)[1]}` ({t.split('::')[0].split('/')[-1]}) | {len(rs)} | {m['output']} | "
               f"{m['rel_l2']:.2e} | {m['tol']:.0e} |")
full = [t for t in d if "test_gpu_parity_full" in t]
out += ["", "## Full-size workloads, every output", ""]
for t in full:
    out.append(f"- `{t.split('::', 1)[1]}`: " + ", ".join(f"{r['output']} {r['rel_l2']:.1e}" for r in d[t]))
open(dst, "w").write("\n".join(out) + "\n")
