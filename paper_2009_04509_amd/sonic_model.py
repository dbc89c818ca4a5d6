"""Latency model of the as-a-service deployment (paper §3.3, "Scale out
modeling", its equations for the ideal and the saturated processing time).

A CPU job spends (1 - p) * t_cpu on work that stays on the CPU; the offloaded
module costs t_gpu of GPU time per event plus t_latency = t_preproc +
t_transmit + t_travel of extra latency (preprocessing on the CPU, moving the
inputs, request round trips).  With a GPU always free, an event takes

    t_ideal = (1 - p) * t_cpu + t_gpu + t_latency.

The GPU saturates once n_cpu / n_gpu > t_ideal / t_gpu; past that point each
event waits for the requests of the other jobs:

    t_sonic = (1 - p) * t_cpu + t_gpu * (1 + max(0, n_cpu / n_gpu - t_ideal / t_gpu)) + t_latency,

which in the saturated regime reduces to t_gpu * n_cpu / n_gpu.  The
clients-per-GPU ratio that just saturates the GPU is t_ideal / t_gpu.

Host-side arithmetic only; nothing here runs on the GPU.
"""

from __future__ import annotations

from dataclasses import dataclass


@dataclass(frozen=True)
class SonicParams:
    t_cpu: float        # s per event, everything on the CPU
    p: float            # fraction of t_cpu that is offloaded
    t_gpu: float        # s of GPU inference per event
    t_preproc: float    # s of input preparation left on the CPU
    t_transmit: float   # s to move one event's inputs
    t_travel: float     # s of request round trips per event

    @property
    def t_latency(self) -> float:
        return self.t_preproc + self.t_transmit + self.t_travel

    @property
    def t_ideal(self) -> float:
        return (1.0 - self.p) * self.t_cpu + self.t_gpu + self.t_latency

    @property
    def saturation_ratio(self) -> float:
        """n_cpu / n_gpu above which the GPU is saturated."""
        return self.t_ideal / self.t_gpu

    def t_sonic(self, n_cpu: float, n_gpu: float = 1.0) -> float:
        """Processing time per event with n_cpu jobs sharing n_gpu GPUs."""
        excess = max(0.0, n_cpu / n_gpu - self.saturation_ratio)
        return (1.0 - self.p) * self.t_cpu + self.t_gpu * (1.0 + excess) + self.t_latency

    def throughput(self, n_cpu: float, n_gpu: float = 1.0) -> float:
        """Events per second of all the jobs together."""
        return n_cpu / self.t_sonic(n_cpu, n_gpu)


def transmit_seconds(n_inputs: int, bytes_per_input: float, link_bits_per_s: float) -> float:
    """Time to send an event's inputs over a link of the given rate."""
    return n_inputs * bytes_per_input * 8.0 / link_bits_per_s


def travel_seconds(n_inputs: int, batch: int, t_request: float) -> float:
    """Round trips of an event sent in requests of `batch` inputs."""
    return -(-n_inputs // batch) * t_request
