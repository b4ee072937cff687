"""Seeded synthetic workloads: model shapes, device constants and grid rules.

Pure data, shared by the HIP path and by the tests' oracle calls.  Nothing in
here computes any part of the simulation.

The five workloads are the shapes the paper's evaluation works with, scaled
to this project's configurations:

* ``tiny_mlp``      4 dense 256-wide layers, batch 64, fp32, training with SGD;
                    D,H,P,K in {1,2,4}, D*H*P <= 4 devices.
* ``large_mlp``     16 dense 8192-wide layers, batch 8192, fp16, Adam;
                    power-of-two D,H,P with D*H*P <= 16, K = 1..64.
* ``gpt2_small``    12 layers, d_model 768, 12 heads, seq 1024, vocab 50257,
                    batch 512 sequences, fp16, inference (the paper's GPT-2
                    workload is inference, Sec. 4) -- also run in training;
                    power-of-two D,H,P,K, D*H*P <= 64, K <= 128.
* ``random_tables`` 1,000,000 random programs of 2,048 ops over 8 devices
                    (70% compute, 20% send, 10% all-reduce), seed 0.
* ``gpt3_175b``     96 layers, d_model 12288, 96 heads, seq 2048, vocab 50257,
                    batch 1536 sequences, fp16 with fp32 master weights and
                    Adam; power-of-two D,H,P with D*H*P <= 1024, K = 1..256,
                    a 288e9-byte per-device memory cap and top-16 selection.

The device constants (14e12 FLOP/s, 900e9 B/s memory, 25e9 B/s link, 5 us
latency, 5 us launch) are the same for every workload.
"""
import math
from dataclasses import dataclass, replace

MLP, TRANSFORMER = 0, 1
INFER, TRAIN_SGD, TRAIN_ADAM, TRAIN_ADAM_MIXED = 0, 1, 2, 3
SCHED_1F1B, SCHED_GPIPE = 0, 1


@dataclass(frozen=True)
class ModelSpec:
    family: int
    mode: int
    n_layers: int
    n_heads: int
    d_model: int
    d_ff: int
    seq_len: int
    vocab: int
    global_batch: int
    elem_bytes: int
    schedule: int = 0   # SCHED_1F1B or SCHED_GPIPE
    recompute: int = 0  # 1: activation recomputation (gradient checkpointing), training only
    zero: int = 0       # 1: ZeRO parameter/gradient partitioning over the data-parallel replicas, training only
    overlap: int = 0    # 1: two streams per GPU, the data-parallel gradient all-reduce overlapping the backward pass


@dataclass(frozen=True)
class DeviceSpec:
    flops_per_s: float = 14e12
    mem_bytes_per_s: float = 900e9
    link_bytes_per_s: float = 25e9
    link_latency_s: float = 5e-6
    launch_s: float = 5e-6
    mem_cap_bytes: int = 0
    # (c0, c1, c2, c3, floor): a matrix multiplication of reduction length k
    # costs max(floor, c0 + c1 * flops + c2 * bytes + c3 * k) (an empirical
    # regression fitted on microbenchmarks); (c0, c1, c2) is the linear form
    # (c3 = floor = 0); None: the roofline
    matmul: tuple = None
    # (node_size, bytes/s, latency s): devices d lie in node d // node_size,
    # and sends and collectives spanning nodes cross this network link;
    # None: one uniform interconnect
    network: tuple = None
    # (streams_per_gpu, bytes/s, latency s): devices d are streams of GPU
    # d // streams_per_gpu, and sends and collectives among the streams of
    # one GPU cost this (bytes/s may be inf); None: one device per GPU
    streams: tuple = None


@dataclass(frozen=True)
class GridSpec:
    max_devices: int
    exact_devices: int
    k_mode: int          # 0: powers of two <= k_max, 1: 1..k_max, 2: K=1 if P=1 else 2..k_max pow2
    k_max: int
    require_k_divides: int = 0


@dataclass(frozen=True)
class RandomTablesSpec:
    seed: int = 0
    n_cand: int = 1_000_000
    n_ops: int = 2048
    n_dev: int = 8


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelSpec = None
    grid: GridSpec = None
    device: DeviceSpec = DeviceSpec()
    top_k: int = 1
    tables: RandomTablesSpec = None


def mlp(n_layers, d, batch, elem_bytes, mode, schedule=0, recompute=0, zero=0, overlap=0):
    return ModelSpec(MLP, mode, n_layers, 1, d, d, 1, 1, batch, elem_bytes, schedule, recompute, zero, overlap)


def transformer(n_layers, d, heads, seq, vocab, batch, elem_bytes, mode, d_ff=None, schedule=0, recompute=0, zero=0,
                overlap=0):
    return ModelSpec(TRANSFORMER, mode, n_layers, heads, d, d_ff or 4 * d, seq, vocab, batch, elem_bytes, schedule,
                     recompute, zero, overlap)


TINY_MLP = Workload("tiny_mlp", mlp(4, 256, 64, 4, TRAIN_SGD), GridSpec(4, 0, 0, 4))
LARGE_MLP = Workload("large_mlp", mlp(16, 8192, 8192, 2, TRAIN_ADAM), GridSpec(16, 0, 1, 64))
GPT2_SMALL = Workload("gpt2_small", transformer(12, 768, 12, 1024, 50257, 512, 2, INFER),
                      GridSpec(64, 0, 0, 128))
GPT2_SMALL_TRAIN = replace(GPT2_SMALL, name="gpt2_small_train",
                           model=replace(GPT2_SMALL.model, mode=TRAIN_ADAM))
RANDOM_TABLES = Workload("random_tables", tables=RandomTablesSpec())
GPT3_175B = Workload("gpt3_175b",
                     transformer(96, 12288, 96, 2048, 50257, 1536, 2, TRAIN_ADAM_MIXED),
                     GridSpec(1024, 0, 1, 256),
                     DeviceSpec(mem_cap_bytes=288_000_000_000), top_k=16)

# the same grid under the GPipe schedule (all forwards, then all backwards)
GPT3_175B_GPIPE = replace(GPT3_175B, name="gpt3_175b_gpipe", model=replace(GPT3_175B.model, schedule=SCHED_GPIPE))
# the same grid with activation recomputation (gradient checkpointing)
GPT3_175B_RECOMPUTE = replace(GPT3_175B, name="gpt3_175b_recompute", model=replace(GPT3_175B.model, recompute=1))
# the same grid with ZeRO partitioning of weights, gradients and optimizer state
GPT3_175B_ZERO = replace(GPT3_175B, name="gpt3_175b_zero", model=replace(GPT3_175B.model, zero=1))
# the same grid with the data-parallel gradient all-reduce on a second stream
# per GPU, overlapping the last backward pass; hand-overs between a GPU's two
# streams cost nothing (they share its memory)
STREAMS_FREE = (2, math.inf, 0.0)
GPT3_175B_OVERLAP = replace(GPT3_175B, name="gpt3_175b_overlap", model=replace(GPT3_175B.model, overlap=1),
                            device=replace(GPT3_175B.device, streams=STREAMS_FREE))

# A cluster of MI355X: fp16 matrix multiplications take the regression fitted
# on this GPU by `python -m paper_2111_05426_amd.calibrate --dtype fp16`
# (max(floor, c0 + c1 flops + c2 bytes + c3 k): floor = 19.4 us per-product
# dispatch, 1/c1 = 1.81 PFLOP/s, 1/c2 = 4.6 TB/s, c3 = 2.8 ns per step of
# the reduction length); other compute ops the roofline with F = 1/c1, the
# bandwidth of a 4 GiB device-to-device copy measured on the same GPU
# (4.94 TB/s, read + write) and the dispatch floor as their launch cost;
# nodes of 8 GPUs joined by xGMI (one link's 153 GB/s, 5 us) and a network of
# one 400 Gb/s NIC per GPU between nodes (50 GB/s, 10 us) -- specification
# values: a single GPU cannot measure them; 288 GB of HBM per device.
MI355X = DeviceSpec(flops_per_s=1.810e15, mem_bytes_per_s=4.94e12, link_bytes_per_s=153e9, link_latency_s=5e-6,
                    launch_s=1.936e-5, mem_cap_bytes=288_000_000_000,
                    matmul=(3.996e-6, 5.524e-16, 2.190e-13, 2.840e-9, 1.936e-5), network=(8, 50e9, 10e-6))
GPT3_175B_MI355X = replace(GPT3_175B, name="gpt3_175b_mi355x", device=MI355X)
GPT3_175B_MI355X_OVERLAP = replace(GPT3_175B_MI355X, name="gpt3_175b_mi355x_overlap",
                                   model=replace(GPT3_175B.model, overlap=1),
                                   device=replace(MI355X, streams=STREAMS_FREE))

ALL = {w.name: w for w in (TINY_MLP, LARGE_MLP, GPT2_SMALL, GPT2_SMALL_TRAIN, RANDOM_TABLES, GPT3_175B,
                           GPT3_175B_GPIPE, GPT3_175B_RECOMPUTE, GPT3_175B_ZERO, GPT3_175B_OVERLAP, GPT3_175B_MI355X,
                           GPT3_175B_MI355X_OVERLAP)}
