"""Host-side measurement logic of bench.py: the code hash that keys the
stored HBM-traffic records, and the trace summary's mean over
back-to-back launches (the launches the bench line's HIP events time).
Nothing here touches a GPU."""
import os
import sqlite3
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402

SRC = """// a kernel
__global__ void k(float* p) {  // one store
  /* block
     comment */
  p[0] = 1.f;

}
"""


def test_code_only_drops_comments_and_blank_lines():
    assert bench.code_only(SRC) == "__global__ void k(float* p) {\n  p[0] = 1.f;\n}"


def test_source_hash_ignores_comments_but_not_code():
    sym = "softmax_kernel<unsigned short, 2, true, 1, true, true>"
    files = {f: open(os.path.join(ROOT, f), encoding="utf-8").read()
             for f in bench.KERNEL_SOURCES["softmax_kernel"]}
    base = bench.kernel_source_hash(sym, files.__getitem__)
    assert base == bench.kernel_source_hash(sym)
    first = bench.KERNEL_SOURCES["softmax_kernel"][0]
    commented = dict(files)
    commented[first] = "// an added comment\n\n" + files[first].replace("\n", "  // note\n", 1)
    assert bench.kernel_source_hash(sym, commented.__getitem__) == base
    changed = dict(files)
    changed[first] = files[first] + "\nstatic int extra_symbol = 1;\n"
    assert bench.kernel_source_hash(sym, changed.__getitem__) != base


def _trace_db(path, rows):
    con = sqlite3.connect(path)
    con.execute("create table counters_collection (x int)")
    con.execute("create table kernels (name text, grid_x int, workgroup_x int, start int, "
                "end int)")
    con.executemany("insert into kernels values (?, ?, ?, ?, ?)", rows)
    con.commit()
    con.close()


def test_trace_summary_means_back_to_back_runs(tmp_path):
    rows, t = [], 0
    for _ in range(6):  # a step: A and B alternate (A 1 us, B 2 us)
        for name, dur in (("A", 1000), ("B", 2000)):
            rows.append((name, 512, 256, t, t + dur))
            t += 3000
    for _ in range(bench.REP_RUN):  # a stage loop: A alone, 1.5 us each
        rows.append(("A", 512, 256, t, t + 1500))
        t += 2000
    for _ in range(bench.REP_RUN - 1):  # a run too short to count
        rows.append(("B", 512, 256, t, t + 4000))
        t += 5000
    _trace_db(str(tmp_path / "run.db"), rows)
    out = bench.collect([str(tmp_path)])
    a, b = out[("A", 2)], out[("B", 2)]
    assert a["launches"] == 6 + bench.REP_RUN
    assert abs(a["avg_us"] - (6 * 1.0 + bench.REP_RUN * 1.5) / (6 + bench.REP_RUN)) < 1e-9
    assert a["rep_launches"] == bench.REP_RUN and abs(a["rep_avg_us"] - 1.5) < 1e-9
    assert "rep_launches" not in b and b["launches"] == 6 + bench.REP_RUN - 1


def test_fault_schedules_follow_the_workloads():
    import workloads as W
    c1 = bench.fault_lists("c1", W.C1, 4)
    assert [sorted(f.op for f in fl) for fl in c1] == [["AS", "CL", "Q"], [], ["AS", "CL", "Q"], []]
    c3 = bench.fault_lists("c3", W.C3, 30)
    assert all(bool(fl) == (k % 10 == 0) for k, fl in enumerate(c3))
    assert all(1 <= len(fl) <= 4 for fl in c3 if fl)
    c4 = bench.fault_lists("c4", W.C4, 8)
    assert all(len(fl) == 1 and fl[0].op in ("AS", "Q", "dWQ") for fl in c4)
    c5 = bench.fault_lists("c5", W.C5, 12)
    assert [len(fl) for fl in c5] == [0, 1, 4, 16] * 3
    mags = [{abs(f.value) for f in fl} for fl in c5]
    assert mags[1] == {1e6} and mags[5] == {1e10} and mags[11] == {1e30}
    # distinct rows and columns within one output of one step
    for fl in c5:
        rows = [(f.op, f.b, f.h, f.row) for f in fl]
        cols = [(f.op, f.b, f.h, f.col) for f in fl]
        assert len(set(rows)) == len(rows) and len(set(cols)) == len(cols)


def test_stage_tables_cover_each_path_once():
    for fused in (False, True):
        t = bench.stage_table(8, 1024, 768, 12, True, fused)
        fwd = [m for _, b, m, *_ in t if not b]
        bwd = [m for _, b, m, *_ in t if b]
        assert len(set(fwd)) == len(fwd) and len(set(bwd)) == len(bwd)
        names = {n for n, *_ in t}
        assert ("core_kv" in names) == fused and ("softmax_bwd" in names) != fused
        # every GEMM flop of the step is in some stage: the useful flops
        # plus, in the fused backward, the recomputations (S in both
        # passes, dP once more: three score-sized products)
        sq = 8 * 12 * (1024 * 1025 // 2)
        extra = 3 * 2 * sq * 64 if fused else 0
        assert sum(f for _, _, _, f, _, _ in t) == bench.useful_flops(8, 1024, 768, 12, True) + extra
