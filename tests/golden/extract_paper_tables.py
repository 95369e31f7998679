"""Recipe that wrote ``paper_memory_tables.json`` and ``paper_oom_outcomes.json``.

It reads the LaTeX source of arXiv 2411.06465 (its path is the one required
argument) and copies, cell by cell, the values the paper prints in its
memory-estimate tables (Tables "a100-memory-table", "a100-memory-table-70b",
"h100-memory-table-8B-8192", "h100-memory-table-8B-16384",
"h100-memory-table-8B-32768") and the OOM / TFLOP/s outcomes of its
throughput tables.  Nothing here computes anything: the outputs are the
paper's printed numbers plus the table label, caption facts (model, sequence
length, GPU memory) and the colour of each cell.

Run:  python tests/golden/extract_paper_tables.py <LaTeX source of the paper>
"""
import json
import re
import sys
from pathlib import Path

# model / sequence / device facts stated in each table's caption
MEMORY_TABLES = {
    "tab:a100-memory-table": ("llama-3.1-8b", 8192, 40),
    "tab:a100-memory-table-70b": ("llama-3.1-70b", 8192, 40),
    "tab:h100-memory-table-8B-8192": ("llama-3.1-8b", 8192, 94),
    "tab:h100-memory-table-8B-16384": ("llama-3.1-8b", 16384, 94),
    "tab:h100-memory-table-8B-32768": ("llama-3.1-8b", 32768, 94),
}
TFLOPS_TABLES = {
    "tab:a100-tflops": ("llama-3.1-8b", 8192, 40),
    "tab:a100-tflops-70B": ("llama-3.1-70b", 8192, 40),
    "tab:h100-tflops-8192": ("llama-3.1-8b", 8192, 94),
    "tab:h100-tflops-8B-16384": ("llama-3.1-8b", 16384, 94),
    "tab:h100-tflops-8B-32768": ("llama-3.1-8b", 32768, 94),
}

ROW = re.compile(r"\((\d+),\s*(\d+),\s*(\d+),\s*(\d+)\)\s*&(.*?)\\\\")
CELL = re.compile(r"(?:\\cellcolor\{light(red|yellow|green)\})?\s*(?:\\textbf\{)?\s*([0-9.]+|OOM|-)\s*\}?")


def tables(text):
    """Yield (label, body) for every tabular environment that has a label."""
    for m in re.finditer(r"\\begin\{tabular\}(.*?)\\end\{tabular\}\s*\\label\{([^}]+)\}", text, re.S):
        yield m.group(2), m.group(1)


def gpu_columns(body):
    head = re.search(r"\(TP, CP, PP, MBS\)(.*?)\\\\", body).group(1)
    return [int(x) for x in re.findall(r"(\d+) GPUs", head)]


def parse(body):
    cols = gpu_columns(body)
    for m in ROW.finditer(body):
        tp, cp, pp, mbs = (int(m.group(i)) for i in range(1, 5))
        cells = [c.strip() for c in m.group(5).split("&")]
        for n_gpus, raw in zip(cols, cells):
            cm = CELL.fullmatch(raw.strip())
            if cm is None:
                raise ValueError(f"unparsed cell {raw!r}")
            colour, value = cm.group(1), cm.group(2)
            if value == "-":
                continue
            yield dict(tp=tp, cp=cp, pp=pp, mbs=mbs, n_gpus=n_gpus, colour=colour, printed=value)


def main(path):
    text = Path(path).read_text()
    lines = text.splitlines()
    mem, oom = [], []
    for label, body in tables(text):
        if label in MEMORY_TABLES or label in TFLOPS_TABLES:
            model, seq, gpu_gb = MEMORY_TABLES.get(label) or TFLOPS_TABLES[label]
            for cell in parse(body):
                cell.update(table=label, model=model, seq=seq, gpu_mem_gb=gpu_gb)
                (mem if label in MEMORY_TABLES else oom).append(cell)
    assert len(mem) == 454, len(mem)
    out = Path(__file__).parent
    note = ("Values printed in arXiv 2411.06465 (Fujii, Watanabe, Yokota), copied by "
            "extract_paper_tables.py. 'printed' is the cell text; 'colour' is the cell shading.")
    for name, cells in (("paper_memory_tables.json", mem), ("paper_oom_outcomes.json", oom)):
        rows = ",\n".join(json.dumps(c, separators=(",", ":")) for c in cells)
        (out / name).write_text('{"source": %s,\n"cells": [\n%s\n]}\n' % (json.dumps(note), rows))
    print(len(mem), "memory cells,", len(oom), "throughput/OOM cells")


if __name__ == "__main__":
    if len(sys.argv) != 2:
        sys.exit("usage: extract_paper_tables.py <LaTeX source of the paper>")
    main(sys.argv[1])
