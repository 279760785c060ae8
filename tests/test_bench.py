"""Host logic of the benchmark (CPU only): attribution of kernel names to stages,
the source hash that keeps stored counter records valid, the work model of the
expert products, and the refusal of more than one GPU."""
import os
import re
import shutil
import subprocess
import sys

import pytest

import bench

ROOT = bench.ROOT


@pytest.mark.parametrize("name,stage", [
    ("void ec::(anonymous namespace)::gemm_dma_kernel<256, 256, 2, 4, 64, 2, true, true, 1, false, "
     "1, 0>(ec::(anonymous namespace)::GemmParams)", "gemm_w13_swiglu"),
    ("gemm_dma_kernel<192, 256, 2, 4, 64, 2, true, true, 1, false, 1, 0>", "gemm_w13_swiglu"),
    ("gemm_dma_kernel<192, 256, 2, 4, 64, 2, true, true, 0, false, 2, 0>", "gemm_w2"),
    ("gemm_dma_kernel<256, 256, 4, 2, 64, 2, true, false, 2, false, 3, 0>", "gemm_dA_swiglu_bwd"),
    ("gemm_dma_kernel<256, 256, 4, 2, 64, 2, false, false, 0, false, 6, 2>", "gemm_dW13"),
    ("gemm_dma_kernel<128, 256, 2, 4, 64, 2, false, false, 0, true, 8, 0>", "router_dwg"),
    ("gemm_dma_kernel<256, 256, 4, 2, 64, 2, true, true, 0, false, 16, 0>", None),   # token choice
    ("void ec::combine_kernel<unsigned short, 64, true>(int)", "bwd_combine"),
    ("combine_kernel<float, 64, false>", "combine"),
    ("router_softmax_bf16_kernel<4, 4>", "router"),
    ("router_softmax_f32_kernel", "router"),
    ("topk_col_kernel<8, 4>", "topk"),
    ("topk_kernel<true>", "topk"),
    ("router_dz_kernel<8>", "router_dz"),
    ("splitk_reduce_kernel", "router_dwg_reduce"),
    ("at::native::vectorized_elementwise_kernel<4, at::native::FillFunctor<float>>", None),
])
def test_stage_of_kernel(name, stage):
    assert bench.stage_of_kernel(name) == stage


def test_stage_tags_match_the_kernel_source():
    # the tags bench.py reads out of kernel names are the enum of the GEMM source
    src = open(os.path.join(ROOT, bench.CSRC, "gemm.hip")).read()
    body = re.search(r"enum\s*\{\s*(G_W13\s*=\s*1[^}]*)\}", src).group(1)
    names = [n.strip() for n in body.split(",") if n.strip()]
    tags = {n.split("=")[0].strip(): i + 1 for i, n in enumerate(names)}
    want = {"gemm_w13_swiglu": "G_W13", "gemm_w2": "G_W2", "gemm_dA_swiglu_bwd": "G_DA",
            "gemm_dXe": "G_DXE", "gemm_dW2": "G_DW2", "gemm_dW13": "G_DW13",
            "router_dx": "G_ROUTER_DX", "router_dwg": "G_ROUTER_DWG",
            "shared_w13_swiglu": "G_SH_W13", "shared_w2": "G_SH_W2",
            "shared_dA_swiglu_bwd": "G_SH_DA", "shared_dX": "G_SH_DXE",
            "shared_dW2": "G_SH_DW2", "shared_dW13": "G_SH_DW13"}
    for stage, sym in want.items():
        assert bench.GEMM_TAGS[stage] == tags[sym], stage


def test_sources_hash_ignores_comments_only(tmp_path, monkeypatch):
    src = os.path.join(ROOT, bench.CSRC)
    dst = tmp_path / bench.CSRC
    dst.mkdir(parents=True)
    for f in os.listdir(src):
        if f.endswith((".hip", ".h", ".cpp")):
            shutil.copy(os.path.join(src, f), dst / f)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    h0 = bench.sources_hash("router")
    assert h0 == bench.sources_hash("router")
    p = dst / "router.hip"
    text = p.read_text()
    p.write_text("// a comment added\n" + text.replace("namespace ec {", "namespace ec {  /* x */", 1))
    assert bench.sources_hash("router") == h0
    assert "constexpr int RT_PX = 4;" in text
    p.write_text(text.replace("constexpr int RT_PX = 4;", "constexpr int RT_PX = 2;", 1))
    assert bench.sources_hash("router") != h0
    # the shared header belongs to every stage's hash
    h1 = bench.sources_hash("topk")
    hdr = dst / "ec_common.h"
    hdr.write_text(hdr.read_text() + "\nconstexpr int kUnused = 1;\n")
    assert bench.sources_hash("topk") != h1


def test_work_model_of_the_expert_products():
    # the forward products do 6 P d h flops and the backward ones 12 P d h (SwiGLU:
    # three d x h matrices per expert, each used once forward and twice backward);
    # at 8 x 2048 tokens, 64 experts of 1024, k = 256 that is 1.649 TFLOP forward
    N, d, E, h, K = 16384, 2048, 64, 1024, 8 * 256
    P = E * K
    w = lambda n: bench.stage_work(n, N, d, E, h, K, 2, 64, True, 32)[0]
    fwd = w("gemm_w13_swiglu") + w("gemm_w2")
    bwd = w("gemm_dA_swiglu_bwd") + w("gemm_dW2") + w("gemm_dXe") + w("gemm_dW13")
    assert fwd == 6 * P * d * h and bwd == 12 * P * d * h
    assert abs(fwd / 1e12 - 1.649) < 5e-4
    # the combine reads every expert row once and writes every token row once
    by = bench.stage_work("combine", N, d, E, h, K, 2, 64, True, 32)[1]
    assert by == P * d * 2 + N * d * 2 + E * N * 4


@pytest.mark.parametrize("extra", [[], ["--routing", "tc"]])
def test_more_than_one_gpu_is_refused(extra):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"] + extra,
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr
    assert r.stdout == ""


@pytest.mark.parametrize("args", [["--workload", "static", "--mask-ratio", "0.5"],
                                  ["--workload", "decode", "--mask-ratio", "1.5"]])
def test_mask_ratio_needs_a_schedule_and_a_ratio_in_range(args):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py")] + args,
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "--mask-ratio needs" in r.stderr
