"""Host-side checks of the benchmark's command line (no GPU needed)."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and not r.stdout.strip()


def test_flop_and_byte_accounting():
    sys.path.insert(0, ROOT)
    import bench
    from synth import vision as SV
    from synth import workloads as W
    d = W.DIMS_FULL
    g = bench.gemm_flops(d, 1536)
    assert g["gate_up"] == 2 * 1536 * 12288 * 2048 and g["qkv"] == 2 * 1536 * 4096 * 2048
    assert sum(g.values()) * d.n_layers == 2 * 1536 * 1_409_286_144       # 2 flops per weight per token
    # e4m3 bytes: one byte per linear weight plus float row scales and fp32 gains
    assert bench.e4m3_weight_bytes(d) == d.n_layers * (50_331_648 + 4 * (4096 + 2048 + 12288 + 2048)
                                                       + 4 * (2 * 2048 + 2 * 128))
    v = SV.VDIMS_FULL
    per_block = 2 * 4096 * (4 * 1024 * 1024 + 2 * 4096 * 1024) + 16 * 4 * 256 * 256 * 1024
    assert bench.vision_flops(v, 16, 256, 256) == (2 * 4096 * 1024 * 768 + 24 * per_block
                                                  + 2 * 1024 * (4096 * 4096 + 2048 * 4096))


def test_per_kernel_algorithmic_bytes():
    """The bytes each kernel class must move at 16 frames of 96 tokens: weights once, fp16
    activations in and out, the fp32 residual stream read and written, and the fp16
    attention operands the QKV epilogue writes (q/k rows and V^T tiles)."""
    sys.path.insert(0, ROOT)
    import bench
    from synth import workloads as W
    d = W.DIMS_FULL
    T = 1536
    w = bench.kernel_work(d, [96] * 16)
    assert w[3][1] == 75_497_472 == 2 * 12288 * 2048 + 2 * T * 2048 + 2 * T * 6144   # gate/up
    assert w[0][1] == 2 * 4096 * 2048 + 2 * T * 2048 + 2 * T * 4096                   # QKV
    assert w[1][1] == 2 * T * 4096 + 2 * T * 2048                                      # attention
    assert w[2][1] == 2 * 2048 * 2048 + 2 * T * 2048 + 8 * T * 2048                   # O + residual
    assert w[4][1] == 2 * 2048 * 6144 + 2 * T * 6144 + 8 * T * 2048                   # down + residual
    # causal attention: 4 d flops per (query, visible key) pair and query head
    assert w[1][0] == 16 * 4 * 16 * 128 * (96 * 97 // 2)
