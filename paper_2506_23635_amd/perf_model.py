"""Lower-bound per-token decode time of an expert-parallel DBRX deployment:
the performance model of the paper's Eq. (eq:pm) (Sec. "Performance
Modeling"), with its variables from Table tab:vars.

One node's time per generated token is the larger of the time to stream its
weights (the self-attention weights plus the expected number of experts the
node executes per layer) and the time to compute on them, plus the
communication: a fixed latency per layer and the all-reduced activations over
the link bandwidth.  With P-L_R-D every node carries the same load, so one
node's time is the system's.

The same function, re-parameterised with one MI355X's measured HBM bandwidth
and MFMA rate and an assumed collective latency over xGMI, predicts a
multi-GPU deployment of the full model from single-GPU measurements.

Host-side arithmetic only (no GPU).
"""
from __future__ import annotations

import itertools
from dataclasses import dataclass, replace


@dataclass(frozen=True)
class ModelVars:
    """Per-token work of the whole model (all layers), Table tab:vars."""
    n_layers: int
    precision: int            # bytes per parameter
    d_embed: int
    d_qkv_hidden: int
    d_ffn: int
    comm_data: float          # bytes all-reduced per token (all layers)
    params_sa: float          # self-attention weight bytes (all layers)
    flops_sa: float           # self-attention FLOPs per token (all layers)
    params_expert: float      # weight bytes of one expert across all layers
    flops_expert: float       # FLOPs of one expert per token across all layers


@dataclass(frozen=True)
class HardwareVars:
    """One node, Table tab:vars."""
    flops: float              # dense bf16 FLOP/s per node
    mem_bw: float             # bytes/s per node
    comm_bw: float            # bytes/s of the node's link
    comm_latency: float       # seconds per layer-wise collective


def dbrx_exact() -> ModelVars:
    """DBRX's variables from the formulas of Table tab:vars notes (a)-(e),
    unrounded (the paper prints them rounded to one significant figure)."""
    L, p, d, q, f = 40, 2, 6144, 8192, 10752
    params_sa = (q * d + d * d) * L * p                 # note (b)
    return ModelVars(n_layers=L, precision=p, d_embed=d, d_qkv_hidden=q, d_ffn=f,
                     comm_data=d * 4 * L * p,           # note (a)
                     params_sa=params_sa,
                     flops_sa=2 * params_sa,            # note (c)
                     params_expert=d * f * 3 * L * p,   # note (d)
                     flops_expert=2 * d * f * 3 * L)    # note (e)


def dbrx_as_printed() -> ModelVars:
    """The rounded values the paper prints in Table tab:vars (and uses for
    Table tab:predict)."""
    return replace(dbrx_exact(), comm_data=2e6, params_sa=7e9, flops_sa=14e9,
                   params_expert=16e9, flops_expert=16e9)


# The Mac Studio node and its 10 GbE link, Table tab:vars.
M2_ULTRA_10GBE = HardwareVars(flops=54e12, mem_bw=800e9, comm_bw=1.25e9, comm_latency=1e-3)

# E[#executed experts per node per layer] measured by the paper (Table
# tab:vars) for 2, 3, 4 nodes.
PAPER_EXEC_EXPERTS = {2: 2.65, 3: 2.32, 4: 1.57}


@dataclass(frozen=True)
class Estimate:
    load: float       # s: weight streaming (GPU Load term)
    compute: float    # s: arithmetic (GPU Compute term)
    latency: float    # s: per-layer collective latency
    transfer: float   # s: all-reduced bytes over the link
    time: float       # s per token, lower bound
    throughput: float  # tokens/s, upper bound


def estimate(exec_experts: float, model: ModelVars, hw: HardwareVars,
             n_nodes: int = 2) -> Estimate:
    """Eq. (eq:pm): max(load, compute) + latency x layers + data / bandwidth.
    exec_experts is E[#executed experts per node per layer].  A single node
    (n_nodes == 1) has no collective."""
    if exec_experts < 0 or n_nodes < 1:
        raise ValueError("exec_experts must be >= 0 and n_nodes >= 1")
    load = (model.params_sa + model.params_expert * exec_experts) / hw.mem_bw
    compute = (model.flops_sa + model.flops_expert * exec_experts) / hw.flops
    if n_nodes > 1:
        lat = hw.comm_latency * model.n_layers
        trans = model.comm_data / hw.comm_bw
    else:
        lat = trans = 0.0
    t = max(load, compute) + lat + trans
    return Estimate(load, compute, lat, trans, t, 1.0 / t)


def expected_busiest_node_experts(n_nodes: int, n_experts: int = 16, top_k: int = 4) -> float:
    """E[max over nodes of the experts a token selects on that node] for one
    token whose top-k set is uniform over the n_experts (experts split over
    the nodes as evenly as possible, in id order): under router-aided load
    balancing every node executes that many experts per layer.  Exact, by
    enumerating the C(n_experts, top_k) sets."""
    if not 1 <= n_nodes <= n_experts or not 1 <= top_k <= n_experts:
        raise ValueError("need 1 <= n_nodes <= n_experts and 1 <= top_k <= n_experts")
    node = []
    for i in range(n_nodes):
        node += [i] * (n_experts // n_nodes + (1 if i < n_experts % n_nodes else 0))
    total = count = 0
    for sel in itertools.combinations(range(n_experts), top_k):
        per = [0] * n_nodes
        for e in sel:
            per[node[e]] += 1
        total += max(per)
        count += 1
    return total / count


def mi355x_hardware(hbm_gbs: float, mfma_tflops: float, collective_latency_s: float,
                    link_gbs: float) -> HardwareVars:
    """One MI355X as a node: measured streaming bandwidth (GB/s) and bf16
    matrix rate (TFLOP/s); the collective latency and the link bandwidth of
    the all-reduce are inputs (a one-GPU build cannot measure them)."""
    return HardwareVars(flops=mfma_tflops * 1e12, mem_bw=hbm_gbs * 1e9,
                        comm_bw=link_gbs * 1e9, comm_latency=collective_latency_s)


def mi355x_predictions(hbm_gbs: float, mfma_tflops: float, gpus=(1, 2, 4, 8),
                       collective_latency_s: float = 20e-6, link_gbs: float = 150.0) -> dict:
    """Per-token lower bound of the full 40-layer DBRX on 1..8 MI355X by Eq.
    (eq:pm), with E[#executed experts] from uniform routing under router-aided
    balancing.  One GPU holds the whole model (264 GB of weights in 288 GB)."""
    model = dbrx_exact()
    hw = mi355x_hardware(hbm_gbs, mfma_tflops, collective_latency_s, link_gbs)
    out = {}
    for n in gpus:
        e = float(4 if n == 1 else expected_busiest_node_experts(n))
        est = estimate(e, model, hw, n_nodes=n)
        out[str(n)] = {"exec_experts": e, "load_ms": est.load * 1e3, "compute_ms": est.compute * 1e3,
                       "latency_ms": est.latency * 1e3, "transfer_ms": est.transfer * 1e3,
                       "ms_per_token": est.time * 1e3, "tokens_per_s": est.throughput}
    return out
