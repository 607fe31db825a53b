"""Result tables of README.md, generated from the committed run records.

    python -m paper_2608_15473_amd.report            # rewrite the tables in place
    python -m paper_2608_15473_amd.report --check    # exit 1 if a table differs from its records

A run record is ``profiles/bench_<workload>.json``: the list of JSON result lines that
``bench.py --record`` appended for that workload, each carrying where and on what code it was
measured (``env``).  Every number in the generated tables comes from those lines; the tables sit
between ``<!-- results:NAME -->`` and ``<!-- /results:NAME -->`` markers, and a test fails when
they no longer match the records.
"""

from __future__ import annotations

import glob
import hashlib
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
RECORDS = os.path.join(ROOT, "profiles")
SOURCE_FILES = ("bench.py", "workloads.py", "include/qfattn.h")

# Table order and the names the tables give the workloads.
WORKLOAD_LABELS = {
    "qwen3-0.6b_b32_n32768_s64_l28": "Qwen3-0.6B, 32 × 32,768 tokens, 28 layers (headline)",
    "qwen3-0.6b_b1_n1m_s16_l28_planted": "Qwen3-0.6B, 1 × 2²⁰ tokens, 28 layers, planted logits",
    "qwen3-4b_b16_n36480_s32_l36": "Qwen3-4B, 16 × 36,480 tokens, 36 layers",
    "qwen3-4b_ragged_b64": "Qwen3-4B, 64 ragged requests (512–131,072 tokens), 1 layer",
    "qwen3-0.6b_b1_n4608_s8": "Qwen3-0.6B, 1 × 4,608 tokens, 1 layer",
    "qwen3-0.6b_b1_n131072_s2_l28_planted":
        "Qwen3-0.6B, 1 × 131,072 tokens, 28 layers (one GPU's share of the 2²⁰-token request)",
    "qwen3-32b_b16_n32768_s32_l64": "Qwen3-32B heads (64 q / 8 KV), 16 × 32,768 tokens, 64 layers",
}


# The decode-stage workloads (bench.py --stage), their names in the tables.
STAGE_LABELS = {
    "qwen3-0.6b_stage_b1_n4608": "Qwen3-0.6B, 1 request, 4,608 tokens, 24 shards, 28 blocks",
    "qwen3-4b_stage_b1_n36480": "Qwen3-4B, 1 request, 36,480 tokens, 128 shards, 36 blocks",
    "qwen3-0.6b_stage_b8_n4608": "Qwen3-0.6B, 8 requests, 4,608 tokens, 16 shards, 28 blocks",
}


def source_digest() -> str:
    """sha256 over every source a measurement depends on: the library's sources, its header, the
    bench and the input generator (the same digest bench.py stamps on each result)."""
    csrc = os.path.join(ROOT, "paper_2608_15473_amd", "csrc")
    names = [os.path.join("paper_2608_15473_amd", "csrc", f) for f in sorted(os.listdir(csrc))
             if f.endswith((".hip", ".h", ".cpp"))] + list(SOURCE_FILES)
    h = hashlib.sha256()
    for name in names:
        with open(os.path.join(ROOT, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read() + b"\0")
    return h.hexdigest()


def load_records(stage: bool = False) -> dict:
    """{workload: runs} of the decode-attention records, or (stage) of the decode-stage ones
    (whose lines carry per-kernel times)."""
    recs = {}
    for path in sorted(glob.glob(os.path.join(RECORDS, "bench_*.json"))):
        with open(path) as f:
            rec = json.load(f)
        runs = [r for r in rec["runs"] if ("kernels" in r) == stage]
        if runs:
            recs[rec["workload"]] = runs
    return recs


def _span(vals, fmt):
    lo, hi = min(vals), max(vals)
    return fmt(lo) if fmt(lo) == fmt(hi) else f"{fmt(lo)}–{fmt(hi)}"


def _current(runs, digest):
    """The runs taken on the current sources (the whole record if none is)."""
    cur = [r for r in runs if r.get("env", {}).get("source_sha256") == digest]
    return (cur, True) if cur else (runs, False)


def readme_table(recs, digest) -> str:
    rows = ["| workload | whole step (bench `value`: sweep + combine, every layer) | "
            "sweep kernel (HIP events) | runs |",
            "|---|---|---|---|"]
    for name, label in WORKLOAD_LABELS.items():
        if name not in recs:
            continue
        runs, cur = _current(recs[name], digest)
        tbs = _span([r["value"] / 1000 for r in runs], lambda v: f"{v:.2f}")
        pct = _span([100 * r["hbm_peak_frac"] for r in runs], lambda v: f"{v:.1f}")
        kern = _span([100 * r["roofline"]["frac"] for r in runs], lambda v: f"{v:.1f}")
        boxes = len({r.get("env", {}).get("host") for r in runs})
        note = "" if cur else ", earlier sources"
        rows.append(f"| {label} | {tbs} TB/s, {pct}% of 8 TB/s | {kern}% | {len(runs)} on "
                    f"{boxes} box{'es' if boxes != 1 else ''}{note} |")
    return "\n".join(rows)


def design_table(recs, digest) -> str:
    rows = ["| workload | ms per step | bench `value` GB/s (% of 8 TB/s) | sweep µs per launch "
            "(% of 8 TB/s) | HBM traffic / algorithmic bytes | fp64 oracle on the host | runs "
            "(sources) |",
            "|---|---|---|---|---|---|---|"]
    for name in WORKLOAD_LABELS:
        if name not in recs:
            continue
        runs, cur = _current(recs[name], digest)
        ms = _span([r["ms_per_step"] for r in runs], lambda v: f"{v:.3f}")
        val = _span([r["value"] for r in runs], lambda v: f"{v:,.0f}")
        pct = _span([100 * r["hbm_peak_frac"] for r in runs], lambda v: f"{v:.1f}")
        us = _span([r["roofline"]["launch_avg_us"] for r in runs], lambda v: f"{v:.1f}")
        kf = _span([100 * r["roofline"]["frac"] for r in runs], lambda v: f"{v:.1f}")
        ratios = [r["roofline"]["traffic"] / r["roofline"]["algorithmic_bytes"] for r in runs
                  if r["roofline"].get("traffic")]
        tr = _span(ratios, lambda v: f"{v:.4f}") if ratios else "—"
        cpus = [r["cpu_baseline"] for r in runs if "cpu_baseline" in r]
        cpu = (f"{_span([c['value'] for c in cpus], lambda v: f'{v:.2f}')} GB/s "
               f"({cpus[-1]['cores']} threads)") if cpus else "—"
        srcs = sorted({r.get("env", {}).get("source_sha256", "")[:8] for r in runs})
        rows.append(f"| `{name}` | {ms} | {val} ({pct}%) | {us} ({kf}%) | {tr} | {cpu} | "
                    f"{len(runs)} ({', '.join(srcs)}{'' if cur else ', earlier'}) |")
    envs = [r.get("env", {}) for runs in recs.values() for r in runs]
    if envs:
        e = envs[-1]
        rows.append("")
        rows.append(f"Measured on {e.get('gpu')} ({e.get('gpu_arch')}, "
                    f"{e.get('gpu_compute_units')} compute units), ROCm {e.get('rocm')}, HIP "
                    f"{e.get('hip')}, torch {e.get('torch')}; host {e.get('cpu_model')}, "
                    f"{e.get('host_cores')} usable cores. Current sources: `{digest[:8]}`.")
    return "\n".join(rows)


def stage_table(recs, digest) -> str:
    rows = ["| workload | serial ms/step | two HIP streams | shared launch (tokens/s) | sweep alone | "
            "shared vs serial (sweep hidden) | shared launch kernel: µs, GB/s (% of 8 TB/s) | "
            "fp64 oracle on the host | runs (sources) |",
            "|---|---|---|---|---|---|---|---|---|"]
    for name, label in STAGE_LABELS.items():
        if name not in recs:
            continue
        runs, cur = _current(recs[name], digest)
        f3 = lambda v: f"{v:.3f}"
        serial = _span([r["serial_ms_per_step"] for r in runs], f3)
        streams = _span([r["streams_ms_per_step"] for r in runs], f3)
        fused = _span([r["fused_ms_per_step"] for r in runs], f3)
        tps = _span([r["value"] for r in runs], lambda v: f"{v:,.0f}")
        alone = _span([r["sweep_only_ms_per_step"] for r in runs], f3)
        speed = _span([r["speedup_vs_serial"] for r in runs], lambda v: f"{v:.2f}×")
        hidden = _span([100 * r["sweep_hidden_frac"] for r in runs], lambda v: f"{v:.0f}%")
        us = _span([r["roofline"]["launch_avg_us"] for r in runs], lambda v: f"{v:.1f}")
        gbs = _span([r["roofline"]["achieved"] for r in runs], lambda v: f"{v:,.0f}")
        pct = _span([100 * r["roofline"]["frac"] for r in runs], lambda v: f"{v:.0f}")
        cpus = [r["cpu_baseline"] for r in runs if "cpu_baseline" in r]
        cpu = (f"{_span([c['value'] for c in cpus], lambda v: f'{v:.3g}')} tokens/s"
               if cpus else "—")
        srcs = sorted({r.get("env", {}).get("source_sha256", "")[:8] for r in runs})
        rows.append(f"| {label} | {serial} | {streams} | **{fused}** ({tps}) | {alone} | "
                    f"{speed} ({hidden}) | {us}, {gbs} ({pct}%) | {cpu} | "
                    f"{len(runs)} ({', '.join(srcs)}{'' if cur else ', earlier'}) |")
    return "\n".join(rows)


def readme_stage(recs, digest) -> str:
    """One sentence on the decode stage, its numbers from the stage records."""
    def step(name):
        runs, _ = _current(recs[name], digest)
        ms = _span([r["fused_ms_per_step"] for r in runs], lambda v: f"{v:.2f}")
        tps = _span([r["value"] for r in runs], lambda v: f"{v:,.0f}")
        return ms, tps
    parts = []
    if "qwen3-0.6b_stage_b1_n4608" in recs:
        ms, tps = step("qwen3-0.6b_stage_b1_n4608")
        parts.append(f"a batch-1 Qwen3-0.6B step at 4,608 tokens in {ms} ms ({tps} tokens/s")
        if "qwen3-0.6b_stage_b8_n4608" in recs:
            parts[-1] += f"; eight requests: {step('qwen3-0.6b_stage_b8_n4608')[1]} tokens/s"
        parts[-1] += ")"
    if "qwen3-4b_stage_b1_n36480" in recs:
        ms, tps = step("qwen3-4b_stage_b1_n36480")
        parts.append(f"a batch-1 Qwen3-4B step at 36,480 tokens in {ms} ms ({tps} tokens/s)")
    if not parts:
        return ""
    return ("The decode stage (`bench.py --stage`, every block of the model with the sweep beside "
            "the feed-forward) runs " + " and ".join(parts) + ".")


TABLES = {("README.md", "readme"): readme_table, ("DESIGN.md", "design"): design_table,
          ("DESIGN.md", "stage"): stage_table, ("README.md", "readme-stage"): readme_stage}


def _replace(text, tag, body):
    begin, end = f"<!-- results:{tag} -->", f"<!-- /results:{tag} -->"
    i, j = text.find(begin), text.find(end)
    if i < 0 or j < i:
        raise ValueError(f"markers for results:{tag} not found")
    return text[:i + len(begin)] + "\n" + body + "\n" + text[j:]


STAGE_TAGS = ("stage", "readme-stage")


def render() -> dict:
    """{file: new text} with every table regenerated from the records."""
    recs, stage_recs, digest = load_records(), load_records(stage=True), source_digest()
    out = {}
    for (fname, tag), fn in TABLES.items():
        path = os.path.join(ROOT, fname)
        text = out.get(fname) or open(path).read()
        out[fname] = _replace(text, tag, fn(stage_recs if tag in STAGE_TAGS else recs, digest))
    return out


def main(argv) -> int:
    new = render()
    stale = [f for f, t in new.items() if open(os.path.join(ROOT, f)).read() != t]
    if "--check" in argv:
        if stale:
            print("tables differ from the run records: " + ", ".join(stale), file=sys.stderr)
            return 1
        return 0
    for f in stale:
        with open(os.path.join(ROOT, f), "w") as fh:
            fh.write(new[f])
    print("rewrote " + (", ".join(stale) if stale else "nothing"))
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
