"""Host logic of bench.py that needs no GPU: the kernel code hash that keys
the committed counter records, and the lookup of a workload's own record."""
import json
import os

import bench


def test_code_hash_ignores_comments_and_layout_only(tmp_path):
    a = tmp_path / "a.hip"
    b = tmp_path / "b.hip"
    c = tmp_path / "c.hip"
    a.write_text("// header\nint f(int x) {  /* twice */ return 2 * x; }\n")
    b.write_text("// another header, longer\n\nint f(int x) {\n  return 2 * x;  // twice\n}\n")
    c.write_text("// header\nint f(int x) { return 3 * x; }\n")
    assert bench.kernel_code_hash(str(a)) == bench.kernel_code_hash(str(b))
    assert bench.kernel_code_hash(str(a)) != bench.kernel_code_hash(str(c))


def test_traffic_record_is_per_workload_and_per_code():
    """Every committed record names its own workload; its traffic is reported
    only while its code hash is the current code's (else null), and a
    workload without a record gives none."""
    code = bench.kernel_code_hash()
    for w in ("wan13_6x", "wan14_6x", "hv15_2x_text", "hv15_2x", "hv15_2x_c21", "wan13_1x"):
        path = os.path.join(bench.PROFILES, f"attn_pmc_{w}.json")
        rec = json.load(open(path))
        assert rec["workload"] == w
        t = bench.traffic_from_profile(w, bench.SPARSE_KERNEL)
        if rec.get("attention_code_sha256") == code:
            assert t == rec["kernels"][bench.SPARSE_KERNEL]["hbm_bytes_per_launch"] and t > 0
        else:
            assert t is None
    assert bench.traffic_from_profile("tiny", bench.SPARSE_KERNEL) is None
