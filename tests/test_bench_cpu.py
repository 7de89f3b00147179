"""Host-side checks of bench.py (no GPU): the one-GPU refusal, the
algorithmic byte counts the roofline divides by, and the lookup of the
committed HBM-counter profiles."""

import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import math  # noqa: E402
from paper_2608_00814_amd import workload as wl  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)


def test_algorithmic_bytes_at_the_qwen3_8b_shape():
    cfg = wl.CONFIGS["qwen3-8b"]
    N = 64
    # K and V of 8 KV heads over the 4096 prefix rows and 64 node rows, plus
    # Q and O of 64 nodes x 32 heads, all head_dim 128 in bf16
    assert bench.attention_bytes(cfg, N) == 2 * 8 * (4096 + 64) * 128 * 2 + 2 * 64 * 32 * 128 * 2 == 18087936
    # the LM-head weight, the 64 hidden rows, and an id and a max logit per node
    assert bench.lmhead_bytes(cfg, N) == 151936 * 4096 * 2 + 64 * 4096 * 2 + 64 * 8 == 1245184512


def test_recorded_traffic_follows_the_sources(tmp_path, monkeypatch):
    """A counter profile counts only while the kernel sources it names are
    unchanged (comments aside)."""
    src = "paper_2608_00814_amd/csrc/tree_attn.hip"
    os.makedirs(tmp_path / "profiles")
    os.makedirs(tmp_path / os.path.dirname(src))
    (tmp_path / src).write_text(open(os.path.join(ROOT, src)).read())
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    rec = {"workload": "w", "ooo_tree_attn": {"bytes_per_launch": 123456, "sources": {src: bench._source_digest(src)}}}
    (tmp_path / "profiles" / "hbm_traffic_w.json").write_text(json.dumps(rec))
    assert bench.recorded_traffic("w", "ooo_tree_attn") == 123456
    assert bench.recorded_traffic("no-such-workload", "ooo_tree_attn") is None
    assert bench.recorded_traffic("w", "no-such-entry") is None
    # a kernel source that changed since the counters were taken voids them
    (tmp_path / src).write_text(open(os.path.join(ROOT, src)).read() + "\nint x;\n")
    assert bench.recorded_traffic("w", "ooo_tree_attn") is None


@pytest.mark.parametrize("path", ["paper_2608_00814_amd/csrc/tree_attn.hip"])
def test_source_digest_ignores_comments_and_layout(tmp_path, monkeypatch, path):
    text = open(os.path.join(ROOT, path)).read()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    (tmp_path / "a.hip").write_text(text)
    (tmp_path / "b.hip").write_text("// a new comment\n" + text.replace("\n", "\n\n") + "\n/* trailing */\n")
    (tmp_path / "c.hip").write_text(text + "\nint x;\n")
    assert bench._source_digest("a.hip") == bench._source_digest("b.hip")
    assert bench._source_digest("a.hip") != bench._source_digest("c.hip")


def test_step_time_statistics():
    st = bench.step_time_stats([0.001 * k for k in range(1, 101)])  # 1..100 ms
    assert st["median_ms"] == pytest.approx(50.5)
    assert st["p10_ms"] == pytest.approx(10.9)
    assert st["p90_ms"] == pytest.approx(90.1)


def test_host_cpu_reports_model_and_affinity():
    model, cores = bench.host_cpu()
    assert isinstance(model, str) and model
    assert cores == len(os.sched_getaffinity(0)) >= 1
    if os.path.exists("/proc/cpuinfo"):
        first = next(l for l in open("/proc/cpuinfo") if l.startswith("model name"))
        assert model == first.split(":", 1)[1].strip()


def test_paper_context_and_mat_tokens():
    # the paper's mean accepted tokens per call for Qwen3-8B on API-Bank (Table 2)
    assert bench.PAPER_MAT_QWEN3_8B == 8.35
    t = bench.tokens_at_mat(1000.0)
    assert t["tokens_per_s"] == 8350.0 and t["mean_accepted_tokens_per_call"] == 8.35
    ctx = bench.PAPER_CONTEXT
    assert ctx["speedup_over_autoregressive"].startswith("2.46x-5.34x")
    assert "H100" in ctx["hardware"] and "Table 2" in ctx["source"]
    assert ctx["qwen3_8b_api_bank"]["speedup"] == 5.34


def test_cpu_baseline_uses_every_core_of_the_affinity():
    """The oracle's BLAS pool is limited to the process affinity (not left at
    whatever size the pool happened to start with)."""
    threadpoolctl = pytest.importorskip("threadpoolctl")
    cores = len(os.sched_getaffinity(0))
    with bench._blas_limit(cores):
        sizes = [i.get("num_threads") for i in threadpoolctl.threadpool_info() if i.get("user_api") == "blas"]
    assert all(n == cores for n in sizes)


def _counter_csv(path, counter, rows):
    head = ("Correlation_Id,Dispatch_Id,Agent_Id,Queue_Id,Process_Id,Thread_Id,Grid_Size,Kernel_Id,Kernel_Name,"
            "Workgroup_Size,LDS_Block_Size,Scratch_Size,VGPR_Count,Accum_VGPR_Count,SGPR_Count,Counter_Name,"
            "Counter_Value,Start_Timestamp,End_Timestamp")
    lines = [head]
    for i, (name, value) in enumerate(rows):
        lines.append(f'{i},{i},"Agent 1",1,1,1,256,1,"{name}",256,0,0,4,0,16,"{counter}",{value},0,1')
    path.write_text("\n".join(lines) + "\n")


def test_traffic_record_from_counter_profiles(tmp_path):
    """Per-launch bytes = sum over an entry point's kernels of mean FETCH
    and WRITE KiB per dispatch, each scaled by what the counter reads for
    the calibration copy of known size."""
    attn = "void ooo::(anonymous namespace)::tree_attn_bf16_kernel<128, 4, true>(ooo::(anonymous namespace)::AttnArgs)"
    comb = "void ooo::(anonymous namespace)::tree_attn_combine_kernel<128, 13>(ooo::(anonymous namespace)::AttnArgs)"
    cal = ("void at::native::vectorized_elementwise_kernel<4, at::native::CUDAFunctorOnSelf_add<float>, "
           "std::array<char*, 2ul> >(int, at::native::CUDAFunctorOnSelf_add<float>, std::array<char*, 2ul>)")
    other = "void at::native::vectorized_elementwise_kernel<4, at::native::FillFunctor<int> >(int)"
    f, w = tmp_path / "fetch.csv", tmp_path / "write.csv"
    # the copy of 1 MiB: FETCH reads half its bytes (scale 2), WRITE all (scale 1)
    _counter_csv(f, "FETCH_SIZE", [(cal, 512.0), (attn, 100.0), (attn, 300.0), (comb, 10.0), (other, 7.0)])
    _counter_csv(w, "WRITE_SIZE", [(cal, 1024.0), (attn, 50.0), (attn, 50.0), (comb, 1.0), (other, 9.0)])
    rec = bench.traffic_record("w", str(f), str(w), calibrate_mib=1)
    assert rec["fetch_scale"] == 2.0 and rec["write_scale"] == 1.0
    e = rec["ooo_tree_attn"]
    assert set(e["kernels"]) == {"ooo::tree_attn_bf16_kernel<128, 4, true>", "ooo::tree_attn_combine_kernel<128, 13>"}
    assert e["bytes_per_launch"] == ((200.0 * 2 + 50.0) + (10.0 * 2 + 1.0)) * 1024
    assert "ooo_lmhead_argmax" not in rec  # no LM-head dispatch in these profiles
    assert e["sources"]["paper_2608_00814_amd/csrc/tree_attn.hip"] == bench._source_digest(
        "paper_2608_00814_amd/csrc/tree_attn.hip")


def test_traffic_record_of_the_model_projections(tmp_path):
    """Full-model workload: one "projections" entry, the bytes of every
    projection kernel of one verify step (mean per dispatch times the
    dispatches of a step: per-layer count times the layers)."""
    from paper_2608_00814_amd import model_workload as mw
    cal = ("void at::native::vectorized_elementwise_kernel<4, at::native::CUDAFunctorOnSelf_add<float>, "
           "std::array<char*, 2ul> >(int, at::native::CUDAFunctorOnSelf_add<float>, std::array<char*, 2ul>)")
    names = {"linear_bf16_kernel": "void ooo::(anonymous namespace)::linear_bf16_kernel<2, true>(int)",
             "linear_add_rmsnorm_kernel": "void ooo::(anonymous namespace)::linear_add_rmsnorm_kernel(int)",
             "linear_qk_norm_rope_kernel": "void ooo::(anonymous namespace)::linear_qk_norm_rope_kernel<128>(int)",
             "linear_reduce_kernel": "void ooo::(anonymous namespace)::linear_reduce_kernel(int)"}
    kib = {"linear_bf16_kernel": (40.0, 4.0), "linear_add_rmsnorm_kernel": (3.0, 2.0),
           "linear_qk_norm_rope_kernel": (2.0, 1.0), "linear_reduce_kernel": (5.0, 1.0)}
    attn = "void ooo::(anonymous namespace)::tree_attn_bf16_kernel<128, 4, true>(int)"
    f, w = tmp_path / "fetch.csv", tmp_path / "write.csv"
    # two dispatches of the streaming kernel with different sizes: the mean counts
    frows = [(cal, 512.0), (attn, 99.0)] + [(names[k], v[0]) for k, v in kib.items()]
    frows.append((names["linear_bf16_kernel"], 60.0))
    wrows = [(cal, 1024.0), (attn, 99.0)] + [(names[k], v[1]) for k, v in kib.items()]
    wrows.append((names["linear_bf16_kernel"], 6.0))
    _counter_csv(f, "FETCH_SIZE", frows)
    _counter_csv(w, "WRITE_SIZE", wrows)
    rec = bench.traffic_record("small-model", str(f), str(w), calibrate_mib=1)
    assert set(rec) == {"workload", "fetch_scale", "write_scale", "projections"}
    L = mw.MODEL_CONFIGS["small-model"].n_layers
    e = rec["projections"]
    want = L * 1024 * (4 * (50.0 * 2 + 5.0) + 2 * (3.0 * 2 + 2.0) + (2.0 * 2 + 1.0) + (5.0 * 2 + 1.0))
    assert e["bytes_per_launch"] == int(round(want))
    assert e["kernels"]["ooo::linear_bf16_kernel<2, true>"] == [50.0, 5.0, 4 * L]
    assert set(e["sources"]) == set(bench.MODEL_PROJECTION_SOURCES)


def test_kernel_record_at_the_other_workloads():
    """The other workloads' kernel figures use the headline's byte and flop
    counts: an HBM-bound shape is graded against 8 TB/s, an MFMA-bound one
    against the bf16 matrix peak."""
    q32b = wl.CONFIGS["qwen2.5-32b"]
    N = 128
    kv = 2 * q32b.n_kv_heads * (q32b.prefix_len + N) * q32b.head_dim * 2
    qo = 2 * N * q32b.n_q_heads * q32b.head_dim * 2
    flops = 4.0 * q32b.n_q_heads * N * q32b.prefix_len * q32b.head_dim
    rec = bench.kernel_record(q32b, N, attn_call_us=40.0, lm_us=300.0)
    assert rec["attention_bound"] == "mfma"  # 4 Hq N P D / bytes is above the 312 flop/B ridge
    assert math.isclose(rec["attention_mfma_frac"], flops / 40e-6 / 1e12 / 2500.0, rel_tol=1e-3)
    assert rec["attention_frac"] == rec["attention_mfma_frac"]
    assert math.isclose(rec["attention_hbm_frac"], (kv + qo) / 40e-6 / 1e9 / 8000.0, rel_tol=1e-3)
    lm = q32b.vocab * q32b.hidden * 2 + N * q32b.hidden * 2 + N * 8
    assert math.isclose(rec["lmhead_hbm_frac"], lm / 300e-6 / 1e9 / 8000.0, rel_tol=1e-3)
    q06b = wl.CONFIGS["qwen3-0.6b"]
    rec2 = bench.kernel_record(q06b, 32, attn_call_us=10.0, lm_us=60.0)
    assert rec2["attention_bound"] == "hbm"
    assert rec2["attention_frac"] == rec2["attention_hbm_frac"]
    assert set(bench.SECONDARY_WORKLOADS) <= set(wl.CONFIGS)


def test_tp8_shard_shape():
    """One GPU's share under 8-way tensor parallelism keeps the query heads
    per KV head and the trie, with an eighth of the heads and vocabulary."""
    q8b = wl.CONFIGS["qwen3-8b"]
    s = bench.tp8_shard_config()
    assert (s.n_kv_heads, s.n_q_heads, s.vocab) == (1, 4, q8b.vocab // 8)
    assert s.group == q8b.group and s.max_nodes == q8b.max_nodes and s.prefix_len == q8b.prefix_len
    assert bench.attention_bytes(s, 64) * 8 == bench.attention_bytes(q8b, 64)
