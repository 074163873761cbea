"""Table of the per-tensor errors a GPU parity run recorded.

Run the GPU tests with MOE_PARITY_LOG set (each parity test appends one JSON
line: the test, its largest error and every tensor's normwise relative error
against the oracle), then write the table:

    MOE_PARITY_LOG=gpurun_out/parity_errors.jsonl python -m pytest tests -m gpu -x -v -s
    python tests/parity_record.py gpurun_out/parity_errors.jsonl OUT --command "..."
"""
from __future__ import annotations

import argparse
import json

TOL = {"f32": 1e-5, "bf16": 2e-2}


def write(jsonl: str, out: str, command: str) -> None:
    rows = [json.loads(line) for line in open(jsonl) if line.strip()]
    lines = [f"# per-tensor errors of the GPU parity tests against the oracle ({len(rows)} tests)",
             f"# command: {command}",
             "# error = max|gpu - oracle| / max|oracle| per tensor (normwise); tolerance "
             f"{TOL['bf16']:g} in bf16, {TOL['f32']:g} in fp32 (logits and gate weights: 1e-5)",
             "# routing indices, mask, counts, offsets, permutations and gathered rows are "
             "compared bit-exact (not listed)",
             f"{'test':64s} {'max':>9s}  worst tensors"]
    for r in rows:
        errs = {k: v for k, v in r["errors"].items() if k != "excluded_near_ties"}
        worst = sorted(errs.items(), key=lambda kv: -kv[1])[:3]
        lines.append(f"{r['test'][:64]:64s} {r['max']:9.2e}  " +
                     ", ".join(f"{k} {v:.1e}" for k, v in worst))
    bf = [r["max"] for r in rows if r["max"] > 1e-4]
    f32 = [r["max"] for r in rows if r["max"] <= 1e-4]
    lines.append(f"# largest: bf16 tests {max(bf, default=0):.2e}, fp32 tests {max(f32, default=0):.2e}")
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")


def main() -> None:
    p = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    p.add_argument("jsonl")
    p.add_argument("out")
    p.add_argument("--command", required=True)
    a = p.parse_args()
    write(a.jsonl, a.out, a.command)


if __name__ == "__main__":
    main()
