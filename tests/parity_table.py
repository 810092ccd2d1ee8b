"""Markdown tables of the parity figures a GPU test run logged.

The GPU parity tests print one line per case that starts with ``PARITY`` and carries a
JSON record (reduced cases, full-size sampled sequences, same-input KV codes, weight
codes).  Run the tests with ``-s`` so the lines reach the log, then

    python tests/parity_table.py <log> > <summary.md>

The bar each figure is held to is stated in the test that produced it.
"""
import json
import sys


def _fmt(v):
    if v is None:
        return "—"
    if isinstance(v, float):
        return f"{v:.2e}"
    if isinstance(v, list):
        return ", ".join(_fmt(x) for x in v)
    return str(v)


def records(lines):
    out = []
    for line in lines:
        i = line.find("PARITY {")
        if i >= 0:
            out.append(json.loads(line[i + len("PARITY "):]))
    return out


def tables(recs):
    md = []
    red = [r for r in recs if r["kind"] == "reduced"]
    if red:
        md += ["### Reduced shapes (every sequence, teacher-forced)", "",
               "| case | prefill error per layer | prefill, chained | decode steps | decode max error |",
               "|---|---|---|---|---|"]
        md += [f"| {r['workload']} | {_fmt(r['prefill_layer_err']) or '—'} | {_fmt(r['prefill_chained_err'])} | "
               f"{r['decode_steps']} | {_fmt(r['decode_max_err'])} |" for r in red]
        md.append("")
    full = [r for r in recs if r["kind"] == "fullsize"]
    if full:
        md += ["### Full size (sampled sequences, graph-replayed decode to the cache's capacity)", "",
               "| workload | rows | prefill error per layer | chained (bound; fp32-oracle drift) | decode max / last | KV max Δcode | KV mismatch rate |",
               "|---|---|---|---|---|---|---|"]
        md += [f"| {r['workload']} | {_fmt(r['rows'])} | {_fmt(r['prefill_layer_err'])} | "
               f"{_fmt(r['prefill_chained_err'])} ({_fmt(r['chained_bound'])}; {_fmt(r['oracle_fp32_drift'])}) | "
               f"{_fmt(r['decode_max_err'])} / {_fmt(r['decode_last_err'])} | {_fmt(r['kv_max_code_delta'])} | "
               f"{_fmt(r['kv_mismatch_rate'])} |" for r in full]
        md.append("")
    other = [r for r in recs if r["kind"] in ("kv_same_input", "weight_codes")]
    if other:
        md += ["### Bit-exact checks at full size", "", "| check | workload | checked | mismatches |", "|---|---|---|---|"]
        for r in other:
            n = r.get("codes_checked", r.get("rows_checked"))
            what = "KV codes + scales, same quantiser input" if r["kind"] == "kv_same_input" else "weight rows (codes, scales, zeros)"
            md.append(f"| {what} | {r['workload']} | {n} | {r['mismatches']} |")
        md.append("")
    return "\n".join(md)


if __name__ == "__main__":
    with open(sys.argv[1]) as f:
        print(tables(records(f)))
