"""Host logic of the rocprofv3 summaries (no GPU): kernel names map to the
labels the library's own timing reports, instantiations that share a label
are merged, and the traffic figures are calibrated by the copy kernel's
counters."""
import csv
import json
import os

import pytest

from paper_2609_29395_amd import profile_summary as ps

HALO = "void (anonymous namespace)::conv_lds_kernel<256, 256, 4, 4, 0, false, true{}>(ConvArgs, FastDiv, " \
       "FastDiv, FastDiv, int, int)"


@pytest.mark.parametrize("flag", ["", ", false", ", true"])
def test_halo_forward_instantiations_share_a_label(flag):
    # the head conv that also writes the pooled features is one more
    # template flag on the same kernel
    assert ps.kernel_label(HALO.format(flag)) == "conv_fwd<bf16,256x256x64,w16,halo>"


def test_one_buffer_halo_label():
    for avg in ("false", "true"):
        assert ps.kernel_label("void (anonymous namespace)::conv_lds_kernel<256, 128, 4, 2, 0, false, true, "
                               f"{avg}, 1>(ConvArgs, FastDiv, FastDiv, FastDiv, int, int)") == \
            "conv_fwd<bf16,256x128x64,w8,halo1>"
    assert ps.kernel_label("void (anonymous namespace)::conv_lds_kernel<256, 256, 4, 4, 1, false, true, false, 2>"
                           "(ConvArgs, FastDiv, FastDiv, FastDiv, int, int)") == "conv_dgrad<bf16,256x256x64,w16,halo>"


def test_other_labels():
    assert ps.kernel_label("void (anonymous namespace)::conv_lds_kernel<256, 64, 8, 2, 1, false, true>"
                           "(ConvArgs, FastDiv, FastDiv, FastDiv, int, int)") == "conv_dgrad<bf16,256x64x192,w16,halo>"
    assert ps.kernel_label("void (anonymous namespace)::conv_lds_kernel<128, 64, 2, 4, 0, false>"
                           "(ConvArgs, FastDiv, FastDiv, FastDiv, int, int)") == "conv_fwd<bf16,128x64x64,w8,lds>"


def test_image_layer_labels():
    ns = "void (anonymous namespace)::"
    assert ps.kernel_label(ns + "conv_col_kernel<true>(ConvArgs, int)") == "conv_fwd<bf16,256x32x27,w4,img3>"
    assert ps.kernel_label(ns + "conv_col_kernel<false>(ConvArgs, int)") == "conv_fwd<bf16,256x32x32,w4,col>"
    assert ps.kernel_label(ns + "wgrad_col_kernel<true>(WgradArgs)") == "conv_wgrad<bf16,32x27,w4,img3>"
    assert ps.kernel_label(ns + "wgrad_col_kernel<false>(WgradArgs)") == "conv_wgrad<bf16,32x32,w4,col>"
    assert ps.kernel_label(ns + "conv_img_kernel<32, 64, 0, 2>(ConvArgs, int)") == "conv_fwd<bf16,512x64x288,w8,img>"
    assert ps.kernel_label(ns + "conv_img_kernel<64, 32, 1, 1>(ConvArgs, int)") == "conv_dgrad<bf16,256x32x576,w8,img>"
    assert ps.kernel_label(ns + "wgrad_img_kernel<3, false>(WgradArgs)") == "conv_wgrad<bf16,64x288,w8,img>"
    assert ps.kernel_label(ns + "sgd_seg_kernel<4>(float*, float*, float*)") == "sgd"
    assert ps.kernel_label(ns + "wgrad_img_kernel<3, true>(WgradArgs)") == "conv_wgrad<bf16,64x288,w8,img,pool>"
    assert ps.kernel_label(ns + "conv_img_pool_kernel<64>(ConvArgs, int, int)") == \
        "conv_fwd<bf16,512x64x288,w8,img,pool>"
    assert ps.kernel_label(ns + "conv_img_dgrad_kernel(ConvArgs, int, int)") == "conv_dgrad<bf16,256x32x576,w8,img,pool>"


@pytest.mark.parametrize("label,source", [
    ("conv_fwd<bf16,256x128x64,w8,halo1>", "k_conv_lds.hip"),
    ("conv_dgrad<bf16,256x128x64,w8,halo1>", "k_conv_lds.hip"),
    ("conv_dgrad<bf16,256x64x192,w16,halo>", "k_conv_lds.hip"),
    ("conv_wgrad<bf16,128x576,w8,halo>", "k_wgrad_lds.hip"),
    ("conv_fwd<bf16,256x32x27,w4,img3>", "k_conv_img.hip"),
    ("conv_wgrad<bf16,32x27,w4,img3>", "k_wgrad_lds.hip"),
    ("conv_wgrad<bf16,64x288,w8,img,pool>", "k_wgrad_lds.hip"),
    ("conv_fwd<bf16,512x64x288,w8,img>", "k_conv_img.hip"),
    ("conv_fwd<bf16,512x64x288,w8,img,pool>", "k_conv_img.hip"),
    ("conv_dgrad<bf16,256x32x576,w8,img,pool>", "k_conv_img.hip"),
    ("conv_fwd<f32,128x128x32,w4,vec>", "k_conv.hip"),
    ("sgd", "k_misc.hip"),
    ("fuse", "k_misc.hip"),
    ("chan_reduce", "k_norm.hip"),
    ("norm_apply_bwd", "k_norm.hip"),
    ("group_reduce", "k_norm.hip"),
    ("im2col", "k_block.hip"),
    ("zero_insert", "k_block.hip"),
])
def test_kernel_source_of_every_label_kind(label, source):
    # the file whose hash decides whether a kernel's committed counters are
    # still current
    assert ps.kernel_source(label) == source


def _write(path, header, rows):
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(header)
        w.writerows(rows)


def test_stats_merges_rows_with_one_label(tmp_path):
    d = tmp_path / "trace"
    _write(str(d / "host" / "run_kernel_stats.csv"), ["Name", "Calls", "TotalDurationNs", "AverageNs"],
           [[HALO.format(""), 3, 3000.0, 1000.0], [HALO.format(", true"), 1, 2000.0, 2000.0],
            ["sgd_kernel<4>", 2, 1000.0, 500.0]])
    # the trace: one sampler launch per step (steps at 0, 10000, 20000 ns);
    # with one warm-up step only the launches from 10000 ns on count for the
    # steady-state column: (1000 + 2000 + 2000) / 3 ns
    _write(str(d / "host" / "run_kernel_trace.csv"), ["Kernel_Name", "Start_Timestamp", "End_Timestamp"],
           [["sample_kernel(int const*)", 0, 100], ["sample_kernel(int const*)", 10000, 10100],
            ["sample_kernel(int const*)", 20000, 20100],
            [HALO.format(""), 200, 200 + 0], [HALO.format(""), 10200, 11200], [HALO.format(""), 20200, 22200],
            [HALO.format(", true"), 21000, 23000], ["sgd_kernel<4>", 500, 1000], ["sgd_kernel<4>", 20500, 21000]])
    out = tmp_path / "stats.md"
    ps.stats(str(d), "wl", str(out), ["bench.py --warmup 1"])
    rows = [l for l in out.read_text().splitlines() if l.startswith("| conv_fwd")]
    assert len(rows) == 1
    cells = [c.strip() for c in rows[0].strip("|").split("|")]
    # 4 calls, 5000 ns in all, 1250 ns = 1.25 us each, 5000 / 6000 of the time
    assert cells[1:] == ["4", "0.005", "1.25", "1.67", "83.33"]
    e = ps.profile_entry("wl", "conv_fwd<bf16,256x256x64,w16,halo>", "trace")
    assert e["calls"] == 4 and e["avg_us"] == pytest.approx(1.25)
    assert e["avg_us_steady"] == pytest.approx(5000 / 3 / 1e3)


@pytest.fixture(autouse=True)
def _private_profile(tmp_path, monkeypatch):
    # every summary writes profile.json: keep the committed one untouched
    monkeypatch.setattr(ps, "PROFILE_JSON", str(tmp_path / "profile.json"))


def test_a_new_summary_drops_labels_the_run_no_longer_has():
    ps._update_profile("wl", "trace", {"old": {"calls": 1, "avg_us": 1.0}, "sgd": {"calls": 1, "avg_us": 2.0}})
    ps._update_profile("wl", "mfma", {"old": {"launches": 1}})
    ps._update_profile("wl", "trace", {"sgd": {"calls": 2, "avg_us": 3.0}})
    assert ps.profile_entry("wl", "old", "trace") is None
    assert ps.profile_entry("wl", "old", "mfma") is not None  # another kind's entry stays
    assert ps.profile_entry("wl", "sgd", "trace")["avg_us"] == 3.0


def test_profile_entry_goes_stale_with_its_source(tmp_path, monkeypatch):
    ps._update_profile("wl", "trace", {"sgd": {"calls": 1, "avg_us": 2.0}})
    assert ps.profile_entry("wl", "sgd", "trace")["avg_us"] == 2.0
    monkeypatch.setattr(ps, "file_hash", lambda name: "changed")
    assert ps.profile_entry("wl", "sgd", "trace") is None


def test_mfma_busy_and_counted_flops(tmp_path):
    # two launches of one kernel: 800 ns each at 2.0 GHz per XCD (the CSV sums
    # the 8 XCDs: 8 x 1600 cycles), MFMA busy 512 x 1600 of 1024 x 1600
    # SIMD-cycles = 50 %, 1000 MOPS = 512,000 FLOPs each
    hdr = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]
    rows = []
    for disp in (1, 2):
        for c, v in (("SQ_VALU_MFMA_BUSY_CYCLES", 512 * 1600.0), ("GRBM_GUI_ACTIVE", 8 * 1600.0),
                     ("SQ_INSTS_VALU_MFMA_MOPS_BF16", 1000.0), ("SQ_INSTS_VALU_MFMA_MOPS_F32", 0.0)):
            rows.append([disp, HALO.format(""), c, v, 1000, 1800])
    _write(str(tmp_path / "m" / "a" / "run_counter_collection.csv"), hdr, rows)
    ps.mfma(str(tmp_path / "m"), "wl", str(tmp_path / "m.md"), ["cmd"])
    e = ps.profile_entry("wl", "conv_fwd<bf16,256x256x64,w16,halo>", "mfma")
    assert e["launches"] == 2
    assert e["mfma_busy_pct"] == pytest.approx(50.0)
    assert e["counted_flops_per_launch"] == pytest.approx(512000.0)
    assert e["gui_mhz"] == pytest.approx(2000.0)


def _counters(path, counter, per_kernel):
    rows = [[k, counter, v] for k, vs in per_kernel.items() for v in vs]
    _write(path, ["Kernel_Name", "Counter_Name", "Counter_Value"], rows)


def test_traffic_calibration_and_merge(tmp_path):
    kib = ps.COPY_MIB * 1024.0
    # the copy reads FETCH_SIZE = 0.5 x and writes WRITE_SIZE = 1.0 x its size
    _counters(str(tmp_path / "cf" / "a" / "run_counter_collection.csv"), "FETCH_SIZE", {"copy": [0.5 * kib] * 3})
    _counters(str(tmp_path / "cw" / "a" / "run_counter_collection.csv"), "WRITE_SIZE", {"copy": [kib] * 3})
    # three plain halo forward launches and one that also writes the pooled
    # features; counters in KiB per dispatch
    _counters(str(tmp_path / "f" / "a" / "run_counter_collection.csv"), "FETCH_SIZE",
              {HALO.format(""): [100.0, 100.0, 100.0], HALO.format(", true"): [140.0]})
    _counters(str(tmp_path / "w" / "a" / "run_counter_collection.csv"), "WRITE_SIZE",
              {HALO.format(""): [256.0, 256.0, 256.0], HALO.format(", true"): [260.0]})
    out = tmp_path / "traffic.md"
    ps.traffic(str(tmp_path / "f"), str(tmp_path / "w"), str(tmp_path / "cf"), str(tmp_path / "cw"), "wl", str(out))
    k = ps.profile_entry("wl", "conv_fwd<bf16,256x256x64,w16,halo>", "traffic")
    assert k["fetch_factor"] == pytest.approx(0.5) and k["write_factor"] == pytest.approx(1.0)
    assert k["launches"] == 4
    assert k["fetch_kib"] == pytest.approx(110.0) and k["write_kib"] == pytest.approx(257.0)
    assert k["bytes_per_launch"] == pytest.approx(1024.0 * (110.0 / 0.5 + 257.0))
    assert "conv_fwd<bf16,256x256x64,w16,halo>" in out.read_text()
