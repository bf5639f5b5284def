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


def _write_mfma_run(d, per_dispatch, ns=100_000):
    """One bench step of dispatches, each with the three matrix-core counters."""
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name",
                                          "Counter_Value", "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        t = 1_000_000
        for i, (busy, gui) in enumerate(per_dispatch):
            for cname, v in (("SQ_VALU_MFMA_BUSY_CYCLES", busy), ("GRBM_GUI_ACTIVE", gui),
                             ("SQ_BUSY_CYCLES", 32 * gui / 8)):
                for part in (v / 2, v / 2):   # two instances, summed
                    w.writerow({"Dispatch_Id": i + 1, "Kernel_Name":
                                f"void sp::(anonymous namespace)::k{i}_kernel<1>(int)",
                                "Counter_Name": cname, "Counter_Value": part,
                                "Start_Timestamp": t, "End_Timestamp": t + ns})
            t += 2 * ns


def test_mfma_summary(tmp_path):
    # 100 us launches at 2.0 GHz: 200k cycles per XCD; stage i busy (i+1)/40 of them
    per = []
    busy_frac = []
    for i, st in enumerate(T.STAGES):
        f = (i + 1) / 40.0
        for _ in range(T.STAGE_DISPATCHES.get(st, 1)):
            per.append((f * T.N_SIMD * 200_000, 8 * 200_000))
        busy_frac.append(f)
    _write_mfma_run(tmp_path / "m", per)
    s = T.summarize_mfma(str(tmp_path / "m"))
    for i, st in enumerate(T.STAGES):
        e = s["stages"][st]
        assert e["clock_ghz"] == pytest.approx(2.0)
        assert e["mfma_busy"] == pytest.approx(busy_frac[i])
        assert e["mfma_busy_peak"] == pytest.approx(busy_frac[i] * 2.0 / 2.4)
        assert e["se_busy"] == pytest.approx(1.0)
    out = tmp_path / "m.md"
    T.write_mfma_md(str(out), s, "cmd", "parse")
    c = T.stage_counters(str(out), "dense.attn")
    assert c["mfma_busy"] == pytest.approx(s["stages"]["dense.attn"]["mfma_busy"], rel=1e-5)
    assert c["clock_ghz"] == pytest.approx(2.0)
