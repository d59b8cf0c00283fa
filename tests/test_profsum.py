"""Host logic of the profile summariser: kernel classification and the
per-workload HBM-traffic file (counter CSVs written here, no GPU)."""
import csv
import json
import types

from paper_2606_04415_amd import profsum


def test_kernel_roles():
    r = profsum.kernel_role
    assert r("void flexattn::decode_gqa_kernel<128, 4, 16, false, true>(flexattn::AttnParams)") == "decode"
    assert r("void flexattn::merge_kernel<512>(flexattn::AttnParams)") == "merge"
    assert r("void flexattn::flat_prefill_kernel<128, 4, 2, 32, 16, 3, 3>(flexattn::AttnParams)") == "prefill"
    # rowpar_kernel's seventh template argument is the row layout: 2 = latent decode rows
    assert r("void flexattn::rowpar_kernel<576, 512, 8, 1, 32, true, 2, 64, 3, 1>(flexattn::AttnParams)") == "decode"
    assert r("void flexattn::rowpar_kernel<576, 512, 8, 1, 32, true, 1, 64, 3, 1>(flexattn::AttnParams)") == "prefill"
    assert r("void flexattn::rowpar_kernel<128, 128, 16, 1, 64, false, 0, 16, 3, 2>(flexattn::AttnParams)") == "prefill"
    assert r("__amd_rocclr_copyBuffer") is None


def _counters(path, counter, per_kernel):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        d = 0
        for name, values in per_kernel.items():
            for v in values:
                d += 1
                w.writerow({"Dispatch_Id": d, "Kernel_Name": name, "Counter_Name": counter, "Counter_Value": v})


def test_traffic_scaling_and_merge(tmp_path):
    dec = "void flexattn::decode_gqa_kernel<128, 4, 16, false, true>(flexattn::AttnParams)"
    pre = "void flexattn::flat_prefill_kernel<128, 4, 2, 32, 16, 3, 3>(flexattn::AttnParams)"
    copy = "__amd_rocclr_copyBuffer"
    gib_kib = (1 << 30) / 1024
    _counters(tmp_path / "cf.csv", "FETCH_SIZE", {copy: [gib_kib / 2] * 3})    # fetch reads half the bytes
    _counters(tmp_path / "cw.csv", "WRITE_SIZE", {copy: [gib_kib] * 3})
    _counters(tmp_path / "df.csv", "FETCH_SIZE", {dec: [100.0, 300.0]})
    _counters(tmp_path / "dw.csv", "WRITE_SIZE", {dec: [10.0, 10.0]})
    _counters(tmp_path / "pf.csv", "FETCH_SIZE", {pre: [50.0]})
    _counters(tmp_path / "pw.csv", "WRITE_SIZE", {pre: [20.0]})

    def args(workload, f, w, into=""):
        return types.SimpleNamespace(workload=workload, fetch=str(tmp_path / f), write=str(tmp_path / w),
                                     copy_fetch=str(tmp_path / "cf.csv"), copy_write=str(tmp_path / "cw.csv"),
                                     command=[f"cmd {workload}"], into=into)

    t1 = profsum.traffic(args("decode", "df.csv", "dw.csv"))
    assert abs(t1["fetch_scale"] - 2.0) < 1e-12 and abs(t1["write_scale"] - 1.0) < 1e-12
    e = t1["entries"]["decode:decode"]
    assert e["fetch_bytes"] == int(200.0 * 1024 * 2.0) and e["write_bytes"] == int(10.0 * 1024)
    assert e["hbm_bytes_per_launch"] == e["fetch_bytes"] + e["write_bytes"]
    first = tmp_path / "t1.json"
    first.write_text(json.dumps(t1))
    t2 = profsum.traffic(args("prefill", "pf.csv", "pw.csv", into=str(first)))
    assert set(t2["entries"]) == {"decode:decode", "prefill:prefill"}
    assert t2["commands"] == ["cmd decode", "cmd prefill"]
    # entries measured on another kernel source are dropped, not merged
    stale = dict(t1, kernel_source_sha256_16="0" * 16)
    first.write_text(json.dumps(stale))
    t3 = profsum.traffic(args("prefill", "pf.csv", "pw.csv", into=str(first)))
    assert set(t3["entries"]) == {"prefill:prefill"}


def test_source_hash_ignores_comments_only(tmp_path):
    """The counter summary stays keyed to a kernel source whose comments
    change, and not to one whose code changes."""
    a = tmp_path / "a.hip"
    a.write_text("// kernel\n__global__ void k(int* p) { p[0] = 1; /* one */ }\n")
    b = tmp_path / "b.hip"
    b.write_text("// the kernel, reworded\n__global__ void k(int* p) {\n  p[0] = 1;   // still one\n}\n")
    c = tmp_path / "c.hip"
    c.write_text("__global__ void k(int* p) { p[0] = 2; }\n")
    assert profsum.source_hash(str(a)) == profsum.source_hash(str(b))
    assert profsum.source_hash(str(a)) != profsum.source_hash(str(c))
