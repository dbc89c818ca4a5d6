"""The as-a-service latency model (paper §3.3) against the numbers the paper
prints for it and against its own closed forms."""

import json
import math
import os

import pytest

from paper_2009_04509_amd.sonic_model import SonicParams, transmit_seconds, travel_seconds

G = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "sonic_model.json")))


def paper(t_gpu, t_transmit, t_travel):
    return SonicParams(t_cpu=G["t_cpu_s"], p=G["p"], t_gpu=t_gpu, t_preproc=G["t_preproc_s"],
                       t_transmit=t_transmit, t_travel=t_travel)


def test_accelerated_fraction_from_module_time():
    # p = (ML module time - preprocessing) / total CPU time
    assert abs((G["ml_module_cpu_s"] - G["t_preproc_s"]) / G["t_cpu_s"] - G["p"]) < 0.006


def test_transmit_and_travel_terms():
    bits = G["patches_per_event"] * G["patch_bits"]
    assert abs(bits / 1e9 - G["event_input_gigabits"]) < 0.05
    for gbps, want in zip(G["link_gbps"], G["t_transmit_s"]):
        got = transmit_seconds(G["patches_per_event"], G["patch_bits"] / 8, gbps * 1e9)
        assert abs(got - want) < 0.06
    assert abs(travel_seconds(G["patches_per_event"], G["large_batch"], G["t_request_s"])
               - G["large_batch_travel_s"]) < 0.01
    assert G["large_batch_requests"] == -(-G["patches_per_event"] // G["large_batch"])
    # printed to two significant figures: 214 x 12 ms = 2.57 s
    assert abs(G["small_batch_requests"] * G["t_request_s"] - G["small_batch_travel_s"]) < 0.05
    for rate, t in zip(G["gpu_inferences_per_s"], G["t_gpu_s"]):
        assert abs(G["patches_per_event"] / rate - t) < 0.02


def test_saturation_ratio_near_the_measured_optimum():
    # large batch, dynamic batching on, 1-2 Gbit/s links: the model's
    # clients-per-GPU ratio brackets the measured 68 : 1 (270 processes, 4 GPUs)
    lo = paper(G["t_gpu_s"][1], G["t_transmit_s"][1], G["large_batch_travel_s"])
    hi = paper(G["t_gpu_s"][1], G["t_transmit_s"][0], G["large_batch_travel_s"])
    assert 65 < lo.saturation_ratio < hi.saturation_ratio < 80
    assert abs(lo.saturation_ratio - G["measured_optimal_cpu_per_gpu"]) / 68 < 0.1
    # small batch without dynamic batching saturates earlier (paper: ~190
    # processes on 4 GPUs against ~270)
    small = paper(G["t_gpu_s"][0], G["t_transmit_s"][1], G["small_batch_travel_s"])
    assert small.saturation_ratio < lo.saturation_ratio
    assert abs(4 * small.saturation_ratio - G["measured_saturation_processes_4gpu"][0]) / 190 < 0.1


def test_closed_forms():
    m = paper(1.77, 2.05, 0.38)
    assert m.t_ideal == pytest.approx((1 - 0.65) * 330 + 1.77 + 7 + 2.05 + 0.38)
    # flat below saturation, t_gpu * n_cpu / n_gpu above it, continuous at it
    assert m.t_sonic(1) == pytest.approx(m.t_ideal)
    assert m.t_sonic(0.5 * m.saturation_ratio) == pytest.approx(m.t_ideal)
    for n in (100, 270, 400, 1000):
        assert m.t_sonic(n, 1) == pytest.approx(max(m.t_ideal, m.t_gpu * n))
    assert m.t_sonic(400, 4) == pytest.approx(m.t_sonic(100, 1))
    assert m.t_sonic(m.saturation_ratio) == pytest.approx(m.t_ideal)
    # the saturated throughput is the GPU's own rate
    assert m.throughput(5000) == pytest.approx(1 / m.t_gpu)
    assert m.throughput(10) == pytest.approx(10 / m.t_ideal)
    assert math.isclose(m.throughput(m.saturation_ratio), 1 / m.t_gpu)
