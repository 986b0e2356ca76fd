"""Host logic of bench.py's per-level-pass roofline: the work of each pass and its class."""
import types

import pytest

import bench
from paper_1702_02181_amd import gen


def _treelstm_workload(H, dtype, backward=True):
    return types.SimpleNamespace(
        hidden=H, dtype=dtype, backward=backward,
        ops=[gen.OpSpec(gen.KIND_TREELSTM, 0, 1, 0), gen.OpSpec(gen.KIND_TREELSTM, 2, 0, 0)],
        params=[types.SimpleNamespace(in_dim=H)])


def test_pass_work_treelstm_counts():
    H = 64
    w = _treelstm_workload(H, "f32")
    host = dict(group_op=[0, 1], group_rows=[4, 2])
    work = bench.pass_work(w, host, table_grad=False)
    S, Sg = 8 * H, 8 * H  # fp32 h + fp32 c; fp32 gradients of both
    # leaf: 4 rows, input width H, the 3 live gates (a leaf's forget gates multiply the zero state)
    assert work[("fwd", 0)] == (2.0 * 4 * H * 3 * H, 4 * (4 * H + S) + H * 3 * H * 4 + 3 * H * 4)
    # leaf backward without a trainable table: only the cell's elementwise part
    assert work[("bwd", 0)] == (0.0, 4 * Sg)
    # internal: 2 rows, two children
    assert work[("fwd", 1)] == (2.0 * 2 * 2 * H * 5 * H, 2 * (2 * S + S) + 2 * H * 5 * H * 4 + 5 * H * 4)
    assert work[("bwd", 1)] == (2.0 * 2 * 5 * H * 2 * H, 2 * (Sg + 2 * (S + Sg)) + 2 * H * 5 * H * 4)
    # weight gradients per op over all its rows
    assert work[("wgrad", 0)][0] == 2.0 * 4 * H * 3 * H
    assert work[("wgrad", 1)][0] == 2.0 * 2 * 2 * H * 5 * H


def test_pass_work_bf16_state_bytes_and_table_grad():
    H = 32
    w = _treelstm_workload(H, "bf16")
    # three leaves reading leaf-table rows 5, 9, 5 (two distinct) and one internal node
    w.node_op = [0, 0, 0, 1]
    w.node_input = [5, 9, 5, -1]
    host = dict(group_op=[0], group_rows=[3])
    work = bench.pass_work(w, host, table_grad=True)
    S = H * (2 + 4)  # bf16 h, fp32 c
    assert work[("fwd", 0)][1] == 3 * (2 * H + S) + H * 3 * H * 2 + 3 * H * 4
    # the leaf backward is the cell's elementwise part; the leaf-table gradient is a pass of its own: every
    # row's dz read once, then one contraction row per distinct leaf-table row, read and written
    assert work[("bwd", 0)] == (0.0, 3 * 8 * H)
    assert work[("tgrad", 0)] == (2.0 * 2 * 3 * H * H, 3 * 3 * H * 2 + 2 * H * 4 * 2 + H * 3 * H * 2)
    assert bench.table_runs(w) == {0: 2}
    assert bench.flops_by_kernel(w, host, True)["tgrad.bf16"] == 2.0 * 2 * 3 * H * H


def test_pass_of_routes_launches():
    assert bench.pass_of("cell_fwd.treelstm.f32", 3, 1) == [("fwd", 3)]
    assert bench.pass_of("embed_fwd", 0, 0) == [("fwd", 0)]
    assert bench.pass_of("cell_bwd.treelstm", 3, 1) == [("bwd", 3)]
    assert bench.pass_of("bwd_dx.bf16", 2, 1) == [("bwd", 2)]
    assert bench.pass_of("wgrad.bf16", -1, 1) == [("wgrad", 1)]
    assert bench.pass_of("wgrad_reduce", -1, 0) == [("wgrad", 0)]
    assert bench.pass_of("tgrad.bf16", -1, 0) == [("tgrad", 0)]
    assert bench.pass_of("tgrad_sum", -1, 0) == [("tgrad", 0)]
    assert bench.pass_of("bwd_init", -1, -1) == []
    assert bench.pass_of("roots", -1, -1) == []
    # a level launch over groups 4, 5, 6 (op = -1 - 3)
    assert bench.pass_of("cell_fwd.level.bf16", 4, -4) == [("fwd", 4), ("fwd", 5), ("fwd", 6)]
    assert bench.pass_of("cell_bwd.level", 4, -3) == [("bwd", 4), ("bwd", 5)]
    assert bench.pass_of("bwd_dx.level.bf16", 7, -2) == [("bwd", 7)]


def test_level_classes_split_and_fractions():
    P, BW = 100.0, 1000.0  # TFLOP/s, GB/s
    work = {
        ("fwd", 0): (1e9, 1e6),     # 10 us of MFMA vs 1 us of HBM: wide
        ("fwd", 1): (1e6, 1e7),     # 0.01 us vs 10 us: gather
        ("bwd", 1): (1e6, 1e3),     # roofline 0.01 us: narrow
        ("wgrad", 0): (2e9, 1e6),   # 20 us: wide
    }
    steps = 2
    launches = [
        ("cell_fwd.treelstm.f32", 0, 0, 0.020), ("cell_fwd.treelstm.f32", 0, 0, 0.020),   # 20 us a step
        ("cell_fwd.treelstm.f32", 1, 1, 0.025), ("cell_fwd.treelstm.f32", 1, 1, 0.025),   # 25 us
        ("cell_bwd.treelstm", 1, 1, 0.004), ("cell_bwd.treelstm", 1, 1, 0.004),           # 4 us
        ("wgrad.f32", -1, 0, 0.015), ("wgrad_reduce", -1, 0, 0.005),                      # 20 us a step
        ("wgrad.f32", -1, 0, 0.015), ("wgrad_reduce", -1, 0, 0.005),
        ("bwd_init", -1, -1, 0.002), ("bwd_init", -1, -1, 0.002),
    ]
    c = bench.level_classes(work, launches, steps, P, BW)
    assert c["wide"]["passes"] == 2
    assert c["wide"]["ms_per_step"] == pytest.approx(0.040)
    assert c["wide"]["frac"] == pytest.approx((0.010 + 0.020) / 0.040)
    assert c["wide"]["by_pass"]["fwd"]["frac"] == pytest.approx(0.5)
    assert c["wide"]["by_pass"]["wgrad"]["frac"] == pytest.approx(1.0)
    assert c["gather"]["passes"] == 1 and c["gather"]["frac"] == pytest.approx(0.010 / 0.025)
    assert c["gather"]["achieved_gbs"] == pytest.approx(1e7 / 25e-6 / 1e9, rel=1e-3)
    assert c["narrow"]["passes"] == 1 and c["narrow"]["us_per_pass"] == pytest.approx(4.0)
    assert c["other_ms_per_step"] == pytest.approx(0.002)


def test_rocprof_roles_of_kernel_names():
    f = "cell_fwd.treelstm.f32"
    assert bench.rocprof_role(f, "void fold::(anonymous namespace)::k_cell_fwd_w<float, 2>(fold::FwdArgs)") == "main"
    assert bench.rocprof_role(f, "void k_cell_fwd_w<float, 8>(fold::FwdArgs)") == "main"  # leaf kind
    assert bench.rocprof_role(f, "void k_cell_fwd<float, 8, 1, true>(fold::FwdArgs)") == "main"
    assert bench.rocprof_role(f, "void k_cell_epi<float, 8>(fold::FwdArgs, int)") == "extra"
    assert bench.rocprof_role(f, "void k_cell_fwd<float, 3, 1, false>(fold::FwdArgs)") is None  # LSTM
    assert bench.rocprof_role(f, "void k_cell_fwd_w<unsigned short, 2>(fold::FwdArgs)") is None  # bf16
    assert bench.rocprof_role("cell_fwd.lstm.bf16", "void k_cell_fwd<unsigned short, 3, 2, false>(x)") == "main"
    assert bench.rocprof_role("bwd_dx.bf16", "void k_bwd_dx_w<unsigned short>(fold::DxArgs)") == "main"
    assert bench.rocprof_role("bwd_dx.f32", "void k_bwd_dx2<float, 1, true>(fold::DxArgs)") == "main"
    assert bench.rocprof_role("wgrad.bf16", "void k_wgrad_bf16_w(fold::WgArgs)") == "main"
    assert bench.rocprof_role("wgrad.f32", "void k_wgrad_f32<128>(fold::WgArgs)") == "main"
    assert bench.rocprof_role("wgrad.f32", "k_wgrad_reduce(float const*, int)") is None


def test_counters_table_from_rocprof_csvs(tmp_path):
    """Per-kernel MFMA utilisation (weighted by active cycles) and HBM rate from four rocprofv3 csv files;
    the copy probe's counter value calibrates the byte counters."""
    import csv as _csv

    def write(name, header, rows):
        p = tmp_path / name
        with open(p, "w", newline="") as f:
            wr = _csv.writer(f)
            wr.writerow(header)
            wr.writerows(rows)
        return str(p)

    H = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]
    probe = "k_probe_copy(uint4 const*, uint4*, unsigned long)"
    kib = bench.PROBE_BYTES / 1024.0
    mfma = write("m.csv", H, [
        [1, "k_a", "GRBM_GUI_ACTIVE", 100], [1, "k_a", "MfmaUtil", 50], [1, "k_a", "SQ_INSTS_VALU_MFMA_MOPS_BF16", 1e6],
        [2, "k_a", "GRBM_GUI_ACTIVE", 300], [2, "k_a", "MfmaUtil", 10], [2, "k_a", "SQ_INSTS_VALU_MFMA_MOPS_BF16", 1e6]])
    fetch = write("f.csv", H, [[3, probe, "FETCH_SIZE", kib / 2], [1, "k_a", "FETCH_SIZE", 1e6], [2, "k_a", "FETCH_SIZE", 1e6]])
    wsz = write("w.csv", H, [[3, probe, "WRITE_SIZE", kib], [1, "k_a", "WRITE_SIZE", 5e5], [2, "k_a", "WRITE_SIZE", 5e5]])
    trace = write("t.csv", ["Kernel_Name", "Start_Timestamp", "End_Timestamp"],
                  [["k_a", 0, 1_000_000], ["k_a", 5_000_000, 6_000_000], [probe, 0, 10]])
    table = bench.counters_table(mfma, fetch, wsz, trace)
    row = [l for l in table.splitlines() if "`k_a`" in l][0].split("|")
    assert row[2].strip() == "2" and row[3].strip() == "2.0"         # dispatches, total ms
    assert row[4].strip() == "20.0"                                    # (50*100 + 10*300) / 400
    assert row[5].strip() == f"{2 * 512e6 / 2e-3 / 1e12:.0f}"          # executed MFMA TFLOP/s
    assert row[6].strip() == f"{2e6 * 1024 * 2 / 1e9:.1f}"             # FETCH_SIZE scaled by 2
    assert row[7].strip() == f"{1e6 * 1024 / 1e9:.1f}"                 # WRITE_SIZE scaled by 1


def test_attention_pass_bytes():
    """Feed-forward attention passes: an aggregate is acc (H pool values) + (m, s); a gradient dh (fp32) + ds."""
    H = 16
    w = types.SimpleNamespace(
        hidden=H, dtype="bf16", backward=True,
        ops=[gen.OpSpec(gen.KIND_ATTN_SCORE, 1, 0, 0), gen.OpSpec(gen.KIND_ATTN_SUM, 2, 0, 1),
             gen.OpSpec(gen.KIND_ATTN_OUT, 1, 0, 2)],
        params=[types.SimpleNamespace(in_dim=0)] * 3)
    host = dict(group_op=[0, 1, 2], group_rows=[8, 4, 1])
    work = bench.pass_work(w, host, table_grad=False)
    agg, grad = 2 * H + 8, 4 * H + 4
    assert work[("fwd", 0)] == (2.0 * 8 * H, 8 * (2 * H + agg) + 2 * H)     # item read, aggregate written, w
    assert work[("bwd", 0)] == (0.0, 8 * (grad + 2 * H + grad) + 2 * H)    # dh, ds, item in; item's gradient out
    assert work[("fwd", 1)] == (0.0, 4 * 3 * agg)                           # two aggregates in, one out
    assert work[("bwd", 1)] == (0.0, 4 * (grad + 16 + 2 * grad))
    assert work[("fwd", 2)] == (0.0, 1 * (agg + 2 * H))
    assert work[("bwd", 2)] == (0.0, 1 * (4 * H + agg + grad))
    assert work[("wgrad", 0)] == (2.0 * 8 * H, 8 * (4 + 2 * H) + (H + 1) * 4)
    assert ("wgrad", 1) not in work and ("wgrad", 2) not in work
    k = bench.attn_kernel_bytes(w, host)
    assert k == {"attn_fwd.score": work[("fwd", 0)][1], "attn_bwd.score": work[("bwd", 0)][1],
                 "attn_fwd.sum": work[("fwd", 1)][1], "attn_bwd.sum": work[("bwd", 1)][1],
                 "attn_fwd.out": work[("fwd", 2)][1], "attn_bwd.out": work[("bwd", 2)][1],
                 "attn_wgrad": work[("wgrad", 0)][1]}
    assert bench.pass_of("attn_fwd.sum", 1, 1) == [("fwd", 1)]
    assert bench.pass_of("attn_bwd.out", 2, 2) == [("bwd", 2)]
    assert bench.pass_of("attn_wgrad", -1, 0) == [("wgrad", 0)]


def test_rocprof_roles_follow_the_library_kind_ids():
    """The rocprof name matcher knows the Tree-LSTM leaf kernels by the library's internal leaf kind id."""
    import os
    import re
    src = open(os.path.join(os.path.dirname(bench.__file__), "paper_1702_02181_amd", "csrc", "common.h")).read()
    leaf = int(re.search(r"constexpr int kTreeLstmLeaf = (\d+);", src).group(1))
    assert leaf in bench.KERNEL_KINDS["treelstm"]
    ns = "void fold::(anonymous namespace)::"
    assert bench.rocprof_role("cell_fwd.treelstm.f32", f"{ns}k_cell_fwd_w<float, {leaf}>(fold::FwdArgs)") == "main"
    assert bench.rocprof_role("cell_fwd.treelstm.f32", f"{ns}k_cell_fwd_w<float, 2>(fold::FwdArgs)") == "main"
    assert bench.rocprof_role("cell_fwd.treelstm.bf16",
                              f"{ns}k_cell_fwd<unsigned short, 2, 1, true>(fold::FwdArgs)") == "main"
    assert bench.rocprof_role("cell_fwd.treelstm.f32", f"{ns}k_cell_epi<float, {leaf}>(fold::FwdArgs, int)") == "extra"
    assert bench.rocprof_role("cell_fwd.treelstm.f32", f"{ns}k_cell_fwd_w<float, 3>(fold::FwdArgs)") is None
    assert bench.rocprof_role("cell_fwd.treelstm.f32", f"{ns}k_cell_fwd_w<unsigned short, 2>(fold::FwdArgs)") is None
