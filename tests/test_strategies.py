"""Host logic of the strategy-grid study (the GPU part runs as a module on a device)."""
from paper_2507_01676_amd import strategies as S


def test_markdown_table_marks_fastest_and_inapplicable():
    rows = [dict(rows=512, pooling=8, table_bytes=512 * 256, lookups=100, lds=90.0, hot=None, dedup=120.0,
                 gather=9.5, stream=100.0, auto=10.0, auto_pick="GATHER", fastest="gather")]
    md = S.to_markdown(rows, "python -m paper_2507_01676_amd.strategies --rows 512")
    line = [ln for ln in md.splitlines() if ln.startswith("| 512")][0]
    cells = [c.strip() for c in line.strip("|").split("|")]
    assert cells[:2] == ["512 (0.12)", "8"]
    assert cells[3] == "-" and cells[5] == "9.5" and cells[7] == "gather" and cells[9] == "GATHER"
    assert "python -m paper_2507_01676_amd.strategies --rows 512" in md
