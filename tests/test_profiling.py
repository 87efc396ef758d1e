"""The rocprofv3 summaries (host code, no GPU): copy-calibrated traffic,
the staleness check against the kernel sources, the generic counter table."""
import csv

from paper_2607_24062_amd import profiling as P


def _csv(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for k, c, v in rows:
            w.writerow({"Kernel_Name": k, "Counter_Name": c, "Counter_Value": v})


def test_traffic_is_scaled_by_the_copy_and_goes_stale(tmp_path):
    copy = "void at::native::vectorized_elementwise_kernel<8, at::native::neg_kernel_cuda>(int)"
    kern = "void acrl::(anonymous namespace)::score_kernel<0, 0, 8, true>(acrl::(anonymous namespace)::ScoreParams)"
    # the copy reads 2 GiB worth of FETCH_SIZE for its 1 GiB: fetch scale 1/2, write scale 1
    _csv(tmp_path / "f.csv", [(copy, "FETCH_SIZE", 2 * 1048576), (kern, "FETCH_SIZE", 1000), (kern, "FETCH_SIZE", 3000)])
    _csv(tmp_path / "w.csv", [(copy, "WRITE_SIZE", 1048576), (kern, "WRITE_SIZE", 10)])
    t = P.traffic(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"))
    assert abs(t["fetch_scale"] - 0.5) < 1e-12 and abs(t["write_scale"] - 1.0) < 1e-12
    k = t["kernels"]["score_kernel<0, 0, 8, true>"]
    assert abs(k["fetch_bytes"] - 2000 * 1024 * 0.5) < 1e-6 and abs(k["write_bytes"] - 10 * 1024) < 1e-6
    md = tmp_path / "t.md"
    md.write_text(P.traffic_markdown(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), "t", "c"))
    assert P.load_traffic(str(md))["kernels"]["score_kernel<0, 0, 8, true>"]["traffic_bytes"] == k["traffic_bytes"]
    # a summary taken from other kernel sources is ignored
    stale = md.read_text().replace(P.source_digest(), "0" * 64)
    md.write_text(stale)
    assert P.load_traffic(str(md)) is None


def test_counters_table(tmp_path):
    _csv(tmp_path / "c.csv", [("void a(int)", "X", 1), ("void a(int)", "X", 3), ("void a(int)", "Y", 5),
                              ("void b()", "X", 7)])
    md = P.counters_markdown(str(tmp_path / "c.csv"), "title", "cmd").splitlines()
    assert md[0] == "# title" and "| kernel | dispatches | X | Y |" in md
    assert "| b | 1 | 7 |  |" in md and "| a | 2 | 2 | 5 |" in md

