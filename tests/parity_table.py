"""Turn the figures that the GPU parity tests append to $MTGR_PARITY_LOG (JSON lines, one per
comparison) into a markdown table: per case and tensor, the literal max|gpu - ref| / rms and
the storage-adjusted figure (see tests/gpu_util.tensor_err).

    MTGR_PARITY_LOG=parity.jsonl python -m pytest tests -m gpu
    python tests/parity_table.py parity.jsonl              (every comparison)
    python tests/parity_table.py --summary parity.jsonl    (per workload and tensor)
"""
import json
import sys


def main(path: str) -> None:
    rows = []
    with open(path) as f:
        for line in f:
            rec = json.loads(line)
            for name, e in rec["errors"].items():
                rows.append((rec["case"], name, e))
    print("| case | tensor | literal max/rms | storage-adjusted | 2^-8 max/rms | literal asserted on |")
    print("|---|---|---|---|---|---|")
    for case, name, e in rows:
        if "users" in e:      # per-user figures: worst user of each column
            la = e.get("literal_asserted")
            asserted = f"{e['users_literal']}/{e['users']} users" + (f" (worst {la:.2e})" if la is not None else "")
        else:                 # one tensor (batch-summed gradients, fp32 outputs)
            asserted = "all" if e["checked"] == e["literal"] else "none"
        print(f"| {case} | {name} | {e['literal']:.2e} | {e['adjusted']:.2e} | {e['storage']:.2e} | {asserted} |")


SUMMARY_CASES = [("tiny", "tiny (fp32, 4 users)"), ("small", "small (32 users)"),
                 ("mtgr_small-whole", "mtgr_small, whole batch (128 users)"),
                 ("mtgr_large-full", "mtgr_large, full size, sampled users"),
                 ("mtgr_large-whole-gln", "mtgr_large, whole batch (Group-LN)"),
                 ("serving-full", "serving, full size, sampled users")]


def summary(path: str) -> None:
    """One row per workload and tensor, then the edge-case batches folded per dtype (worst
    figure over the cases): the literal figure, the storage-adjusted one, the storage rounding
    of the largest element (2^-8 max|ref| / rms) and whether the literal figure is within the
    stated bar (2e-2 bf16, 1e-4 fp32)."""
    recs = {}
    with open(path) as f:
        for line in f:
            rec = json.loads(line)
            recs[rec["case"]] = rec["errors"]
    print("| case | tensor | literal max/rms | storage-adjusted | 2^-8 max/rms | literal within bar |")
    print("|---|---|---|---|---|---|")
    for case, label in SUMMARY_CASES:
        if case not in recs:
            continue
        tol = 1e-4 if case == "tiny" else 2e-2
        for name, e in recs[case].items():
            print(f"| {label} | {name} | {e['literal']:.2e} | {e['adjusted']:.2e} | {e['storage']:.2e} | "
                  f"{'yes' if e['literal'] <= tol else 'no'} |")
    for dt, tol in (("bf16", 2e-2), ("fp32", 1e-4)):
        cases = [c for c in recs if c.endswith(tuple(f"-{dt}-{h}" for h in (16, 32, 64, 128)))]
        worst = {}
        for c in cases:
            for name, e in recs[c].items():
                w = worst.setdefault(name, {"literal": 0.0, "adjusted": 0.0, "storage": 0.0})
                for k in w:
                    w[k] = max(w[k], e[k])
        for name, w in worst.items():
            print(f"| edge cases {dt} ({len(cases)} batches) | {name} | {w['literal']:.2e} | {w['adjusted']:.2e} | "
                  f"{w['storage']:.2e} | {'yes' if w['literal'] <= tol else 'no'} |")


if __name__ == "__main__":
    if sys.argv[1] == "--summary":
        summary(sys.argv[2])
    else:
        main(sys.argv[1])
