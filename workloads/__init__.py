"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke check."""

from .gen import (WORKLOADS, Workload, bf16_bits, gauss, haar, high_snr,
                  lowrank_plus_noise, stream, to_stored, zipf_rows)

__all__ = ["WORKLOADS", "Workload", "bf16_bits", "gauss", "haar", "high_snr",
           "lowrank_plus_noise", "stream", "to_stored", "zipf_rows"]
