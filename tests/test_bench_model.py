"""The benchmark's work model (algorithmic bytes and flops per launch, roofline bound) and its
command line.  CPU only: no kernel runs."""
import json
import os
import subprocess
import sys

import pytest

import bench
from paper_1704_04560_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _work(name, site, layer, fused=()):
    wkl = wl.WORKLOADS[name]
    geo = bench.geometry(wkl.net)
    es = 2 if wkl.net.dtype == wl.BF16 else 4
    return bench._site_work(site, layer, geo, wkl, es, fused)


def test_gradient_average_moves_r_rows_plus_weights_and_momentum():
    # Sec. III-E: R shard gradients read; w and v read and written; the average written
    wkl = wl.WORKLOADS["alexnet"]
    P = bench.wkl_params(wkl)
    bound, nbytes, mm = _work("alexnet", "avg_update", -1)
    assert bound == "hbm" and mm == 0.0
    assert nbytes == (wkl.shards + 5) * 4 * P


def test_alexnet_conv3_is_a_matrix_bound_launch():
    # conv3: 256 x 13 x 13 outputs of 384 channels over a 3 x 3 x 256 window
    bound, flops, mm = _work("alexnet", "wgrad", 4)
    assert bound == "mfma"
    assert flops == mm == 2.0 * 256 * 13 * 13 * 384 * 256 * 9


def test_fully_connected_weight_gradient_is_bound_by_its_gradient_rows():
    # FC6 (9216 -> 4096): the R fp32 gradient rows it writes outweigh its flops at the peaks
    wkl = wl.WORKLOADS["alexnet"]
    bound, nbytes, mm = _work("alexnet", "wgrad", 8)
    assert bound == "hbm"
    assert mm == 2.0 * 256 * 9216 * 4096
    assert nbytes == (256 * 9216 + 256 * 4096) * 2 + wkl.shards * (9216 * 4096 + 4096) * 4


def test_fused_weight_gradient_adds_the_update_traffic():
    # FC6 fused with the average + update: w and v read, the average, v and w written
    wkl = wl.WORKLOADS["alexnet"]
    _, plain, _ = _work("alexnet", "wgrad", 8)
    bound, fused, mm = _work("alexnet", "wgrad_update", 8)
    assert bound == "hbm" and mm == 2.0 * 256 * 9216 * 4096
    assert fused - plain == (9216 * 4096 + 4096) * 20


def test_average_after_fused_layers_covers_the_rest():
    # with the three fc layers fused, the stand-alone average + update moves only the
    # convolutions' parameters (60,965,224 in all, 58,631,144 of them in the fc layers)
    wkl = wl.WORKLOADS["alexnet"]
    _, nbytes, _ = _work("alexnet", "avg_update", -1, fused=(8, 9, 10))
    fc = (9216 * 4096 + 4096) + (4096 * 4096 + 4096) + (4096 * 1000 + 1000)
    assert fc == 58631144
    assert nbytes == (wkl.shards + 5) * 4 * (60965224 - fc)


def test_one_by_one_convolution_data_gradient_is_memory_bound():
    # bottleneck layer 16: 1x1, 256 -> 128 channels at 32 x 32; dy, W, the mask and dx
    bound, nbytes, mm = _work("bottleneck", "dgrad", 16)
    assert bound == "hbm"
    pos = 256 * 32 * 32
    assert nbytes == (pos * 128 + 128 * 256 + 2 * pos * 256) * 2
    assert mm == 2.0 * pos * 128 * 256


def test_projection_counts_the_source_as_its_input():
    # bottleneck layer 22: 1x1 stride-2 projection of layer 15's 256 x 32 x 32 output to 512
    # channels at 16 x 16
    bound, nbytes, mm = _work("bottleneck", "fwd", 22)
    assert mm == 2.0 * 256 * 16 * 16 * 512 * 256
    assert nbytes == (256 * 256 * 32 * 32 + 512 * 256 + 256 * 512 * 16 * 16) * 2


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode != 0
    assert "--gpus 1" in r.stderr
    assert not r.stdout.strip()


def test_identity_shortcut_share_reads_the_source_mask():
    # bottleneck layer 15 adds layer 8's output (a projection block's ReLU output, 256 x 32 x 32):
    # the share added into layer 8's gradient is layer 15's own output gradient, times layer 8's
    # ReLU mask, so the launch reads three tensors and writes one
    bound, nbytes, mm = _work("bottleneck", "skip_add", 8)
    assert bound == "hbm" and mm == 0.0
    assert nbytes == 4 * 256 * 256 * 32 * 32 * 2



def test_batch_norm_apply_carries_the_following_addition():
    # bottleneck layer 14 (BN over 256 x 32 x 32) is followed by layer 15's identity addition,
    # computed in the same pass: x and the shortcut read, the BN output and the sum written
    bound, nbytes, mm = _work("bottleneck", "bn_fwd_apply", 14)
    assert bound == "hbm" and nbytes == 4 * 256 * 256 * 32 * 32 * 2
    # layer 12's BN (ReLU, then a convolution) moves x and y only
    assert _work("bottleneck", "bn_fwd_apply", 12)[1] == 2 * 256 * 64 * 32 * 32 * 2
