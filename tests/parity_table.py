"""Turn the figures that the GPU parity tests append to $MTGR_PARITY_LOG (JSON lines, one per
comparison) into a markdown table: per case and tensor, the literal max|gpu - ref| / rms and
the storage-adjusted figure (see tests/gpu_util.tensor_err).

    MTGR_PARITY_LOG=parity.jsonl python -m pytest tests -m gpu
    python tests/parity_table.py parity.jsonl
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


if __name__ == "__main__":
    main(sys.argv[1])
