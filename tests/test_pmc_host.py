"""Host logic of the rocprofv3 summariser: dispatch classification, class
launches, copy-probe calibration and the per-launch figures, on synthetic
profiler CSV files."""
import csv
import json
import os

import pytest

from paper_2609_10018_amd import pmc

G = "void elasto::(anonymous namespace)::gemm_bf16_kernel<{}, {}, 2, 4, (elasto::Epi){}>(elasto::(anonymous namespace)::Params)"
LN = "elasto::(anonymous namespace)::layernorm_bf16_kernel(...)"
GP = "void elasto::(anonymous namespace)::gemm_bf16_persistent<(elasto::Epi){}, true>(elasto::(anonymous namespace)::Params)"
ATT = "void elasto::(anonymous namespace)::attention_bf16_kernel<13>(elasto::(anonymous namespace)::AttnP)"
COPY = "void at::native::vectorized_elementwise_kernel<4, at::native::BinaryFunctor<float, float, float, at::native::binary_internal::MulFunctor<float> > >(...)"


def forward_names(depth=2):
    n = [G.format(256, 256, 4), G.format(128, 256, 4)]
    for _ in range(depth):
        n += [LN, G.format(256, 256, 0), ATT, G.format(256, 256, 2), G.format(128, 256, 2), LN,
              G.format(256, 256, 1), G.format(128, 256, 1), G.format(256, 256, 2),
              G.format(128, 256, 2)]
    n += [LN, G.format(128, 128, 3)]
    return n


def test_classify_and_launches():
    names = forward_names(2)
    cls = pmc.classify(names)
    assert cls[:2] == ["patch", "patch"]
    assert cls[2:12] == ["ln", "qkv", "attn", "proj", "proj", "ln", "fc1", "fc1", "fc2", "fc2"]
    assert cls[-2:] == ["ln", "head"]
    runs = pmc.launches(cls)
    count = {}
    for c, idx in runs:
        count[c] = count.get(c, 0) + 1
    assert count == {"patch": 1, "ln": 5, "qkv": 2, "attn": 2, "proj": 2, "fc1": 2, "fc2": 2,
                     "head": 1}
    per = pmc.per_launch(cls, [1.0] * len(cls))
    assert per["fc1"] == (2, 2.0) and per["ln"] == (5, 1.0) and per["head"] == (1, 1.0)


def test_classify_persistent_and_folded_layernorm():
    # bf16 forward with LayerNorm folded into the GEMMs: the q/k/v and fc1
    # GEMMs run the persistent kernel (fc1 plus a 128x256 tail launch); only
    # the final LayerNorm remains.
    n = [G.format(256, 256, 4), G.format(128, 256, 4)]
    for _ in range(2):
        n += [GP.format(0), ATT, G.format(256, 256, 2), G.format(128, 256, 2), GP.format(1),
              G.format(128, 256, 1), G.format(256, 256, 2), G.format(128, 256, 2)]
    n += [LN, G.format(128, 128, 3)]
    cls = pmc.classify(n)
    assert cls[2:10] == ["qkv", "attn", "proj", "proj", "fc1", "fc1", "fc2", "fc2"]
    count = {}
    for c, idx in pmc.launches(cls):
        count[c] = count.get(c, 0) + 1
    assert count == {"patch": 1, "qkv": 2, "attn": 2, "proj": 2, "fc1": 2, "fc2": 2, "ln": 1,
                     "head": 1}


def _write_counters(path, names, counters):
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Correlation_Id", "Dispatch_Id", "Process_Id", "Kernel_Name", "Counter_Name",
                    "Counter_Value"])
        for i, (n, c) in enumerate(zip(names, counters)):
            for k, v in c.items():
                w.writerow([i + 1, i + 1, 7, n, k, v])
    with open(os.path.join(path, "run_agent_info.csv"), "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Agent_Type", "Simd_Count"])
        w.writerow(["CPU", 0])
        w.writerow(["GPU", 1024])


MARK = "void at::native::vectorized_elementwise_kernel<4, at::native::FillFunctor<float>, std::array<char*, 1> >(...)"


def test_after_mark_drops_the_tuning_dispatches():
    tuning = forward_names(1) * 3
    names = tuning + [MARK] + forward_names(2)
    kept, vals = pmc.after_mark(names, list(range(len(names))))
    assert kept == forward_names(2) and vals[0] == len(tuning) + 1
    assert pmc.after_mark(forward_names(1), [0] * 14)[0] == forward_names(1)  # no marker


def test_summarize_synthetic(tmp_path):
    # dispatches before the marker (create-time tuning) must not count
    names = [G.format(256, 256, 1)] * 5 + [MARK] + forward_names(2) + [COPY] * 3
    out = str(tmp_path)
    # trace: each dispatch 10 us, except fc1 dispatches 30 us
    os.makedirs(os.path.join(out, "trace"))
    with open(os.path.join(out, "trace", "run_kernel_trace.csv"), "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        t = 0
        for i, n in enumerate(names):
            d = 30000 if "Epi)1" in n else 10000
            w.writerow([i + 1, n, t, t + d])
            t += d + 100
    cls = pmc.classify(names)
    # counters read half the true bytes: calibration must double them
    kib = [{"FETCH_SIZE": (2**30 / 2 / 1024) if c == "copy" else 1000.0} for c in cls]
    _write_counters(os.path.join(out, "fetch"), names, kib)
    kib = [{"WRITE_SIZE": (2**30 / 1024) if c == "copy" else 500.0} for c in cls]
    _write_counters(os.path.join(out, "write"), names, kib)
    mf = [{"SQ_VALU_MFMA_BUSY_CYCLES": 1024 * 50.0, "GRBM_GUI_ACTIVE": 8 * 100.0} for _ in cls]
    _write_counters(os.path.join(out, "mfma"), names, mf)
    classes = {c: {"flops_per_launch": 1e9, "bytes_per_launch": 4096000.0,
                   "launches_per_forward": 1} for c in pmc.CLASSES}
    json.dump({"classes": classes, "dominant": "fc1", "dominant_avg_us": 60.5,
               "class_ms_mode0": {}, "source_hash": "abc"}, open(os.path.join(out, "work.json"), "w"))
    pmc.summarize(out, {"trace": ["x"], "fetch": ["y"]}, 3)
    tr = json.load(open(os.path.join(out, "traffic.json")))
    assert "DN mode 3" in tr["workload"]
    assert tr["kernel_class"] == "fc1" and tr["source_hash"] == "abc"
    assert tr["calibration"]["fetch_scale"] == pytest.approx(2.0)
    assert tr["calibration"]["write_scale"] == pytest.approx(1.0)
    # fc1 launch = 2 dispatches: fetch 2 x 1000 KiB x 2, write 2 x 500 KiB x 1
    assert tr["fetch_bytes_per_launch"] == pytest.approx(4000 * 1024)
    assert tr["write_bytes_per_launch"] == pytest.approx(1000 * 1024)
    assert tr["hbm_bytes_per_launch"] == pytest.approx(5000 * 1024)
    fc1 = tr["classes"]["fc1"]
    assert fc1["avg_us"] == pytest.approx(60.0) and fc1["launches"] == 2
    assert fc1["mfma_util"] == pytest.approx(0.5)
    # roofline: max(1e9 / 2.5e15, 4.096e6 / 8e12) s = 0.512 us over 60 us, memory-bound
    assert fc1["roofline_frac"] == pytest.approx(4.096e6 / 8e12 / 60e-6)
    assert fc1["roofline_bound"] == "hbm"
    assert "fc1" in open(os.path.join(out, "summary.md")).read()
