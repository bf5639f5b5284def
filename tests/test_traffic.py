"""Host logic of the rocprofv3 traffic summary (no GPU)."""
import csv
import os

import pytest

from paper_2606_07703_amd import traffic as T


def _write_run(d, counter, values, copy_kib):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name",
                                          "Counter_Value"])
        w.writeheader()
        did = 1
        for i, v in enumerate(values):
            # two counter instances per dispatch: the summary adds them
            for part in (v / 2, v / 2):
                w.writerow({"Dispatch_Id": did, "Kernel_Name": f"void sp::(anonymous namespace)::"
                            f"k{i}_kernel<1>(int)", "Counter_Name": counter,
                            "Counter_Value": part})
            did += 1
        w.writerow({"Dispatch_Id": did, "Kernel_Name": "__amd_rocclr_copyBuffer",
                    "Counter_Name": counter, "Counter_Value": copy_kib})


def _per_dispatch(stage_values):
    """Split each stage's value evenly over its kernel launches."""
    out = []
    for st, v in zip(T.STAGES, stage_values):
        nd = T.STAGE_DISPATCHES.get(st, 1)
        out += [v / nd] * nd
    return out


def test_summary_scales_by_copy_and_maps_stages(tmp_path):
    n = len(T.STAGES)
    fetch = [100.0 * (i + 1) for i in range(n)]
    write = [10.0 * (i + 1) for i in range(n)]
    _write_run(tmp_path / "f", "FETCH_SIZE", _per_dispatch(fetch), copy_kib=512 * 1024)
    _write_run(tmp_path / "w", "WRITE_SIZE", _per_dispatch(write), copy_kib=1024 * 1024)
    s = T.summarize(str(tmp_path / "f"), str(tmp_path / "w"), 1 << 30)
    assert s["fetch_factor"] == pytest.approx(2.0)
    assert s["write_factor"] == pytest.approx(1.0)
    for i, st in enumerate(T.STAGES):
        e = s["stages"][st]
        assert e["fetch_bytes"] == pytest.approx(fetch[i] * 1024 * 2)
        assert e["write_bytes"] == pytest.approx(write[i] * 1024)
        assert e["traffic_bytes"] == pytest.approx(e["fetch_bytes"] + e["write_bytes"])
    out = tmp_path / "t.md"
    T.write_md(str(out), s, "cmd-f", "cmd-w", "cmd-p")
    back = T.load_traffic(str(out))
    assert set(back) == set(T.STAGES)
    assert all(v["current"] for v in back.values())
    st = T.STAGES[3]
    assert T.stage_traffic(str(out), st) == pytest.approx(s["stages"][st]["traffic_bytes"],
                                                          rel=1e-6)


def test_changed_source_invalidates(tmp_path):
    files = T.kernel_sources(T.STAGE_KERNEL_FILE["block64.sparse_attn"])
    assert "paper_2606_07703_amd/csrc/sparse_block_mfma.hip" in files
    assert "paper_2606_07703_amd/csrc/attn_tile.hpp" in files   # included header
    p = tmp_path / "t.md"
    p.write_text("<!-- traffic block64.sparse_attn 1.0e9 0000000000000000 -->\n")
    assert T.load_traffic(str(p))["block64.sparse_attn"]["current"] is False
    assert T.stage_traffic(str(p), "block64.sparse_attn") is None


def test_ragged_dispatch_count_rejected(tmp_path):
    per_step = len(_per_dispatch([1.0] * len(T.STAGES)))
    _write_run(tmp_path / "f", "FETCH_SIZE", [1.0] * (per_step + 1), copy_kib=1.0)
    _write_run(tmp_path / "w", "WRITE_SIZE", [1.0] * per_step, copy_kib=1.0)
    with pytest.raises(ValueError):
        T.summarize(str(tmp_path / "f"), str(tmp_path / "w"), 1 << 20)
