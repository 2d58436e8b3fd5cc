"""Expert placement across GPUs and the per-layer load plan of expert
parallelism (host side).

Two ideas of the paper, restated for GPUs that each hold a subset of the
experts:

* Router-aided dynamic loading, L_R (Sec. "Load balancing strategies"): in
  every layer the largest number of router-selected experts on any node is
  shared with all nodes, and a node that selected fewer fills the difference
  with its least recently used local experts, so every node does the same
  amount of work per layer.  The fill kept Metal's weights wired; on MI355X
  weights stay resident in HBM, so the fill is optional here (``fill``) and
  only the balancing survives.
* Overlapping expert replicas (Sec. "Scalability"): with spare memory an
  expert is held by several nodes and each selected expert runs on one of
  its holders, chosen to spread the work.  ``assign`` picks the holders that
  minimise the busiest GPU's number of executed experts (exact bottleneck
  assignment; ties broken deterministically, so every GPU that replicates
  the router computes the same plan from the same routing).

The load of a GPU in one layer is the number of distinct experts it executes
(each streams its weights once per layer, whatever its token count), so the
layer time of a synchronous expert-parallel step follows the busiest GPU;
``expected_busiest_load`` gives its expectation under uniform top-k routing,
the E[#exec. experts per node per layer] of Table tab:vars, which Eq. (eq:pm)
turns into a time per token.
"""
from __future__ import annotations

import itertools
import math
from dataclasses import dataclass, field


@dataclass(frozen=True)
class Placement:
    """holders[e]: the GPUs that hold expert e (ascending, at least one)."""
    n_gpus: int
    holders: tuple

    def __post_init__(self):
        if self.n_gpus < 1:
            raise ValueError("n_gpus must be >= 1")
        for e, h in enumerate(self.holders):
            if not h or list(h) != sorted(set(h)) or h[0] < 0 or h[-1] >= self.n_gpus:
                raise ValueError(f"expert {e}: holders must be distinct ascending GPU ids")

    @property
    def n_experts(self) -> int:
        return len(self.holders)

    def local(self, g: int) -> tuple:
        """Experts GPU g holds, ascending."""
        return tuple(e for e, h in enumerate(self.holders) if g in h)

    def experts_per_gpu(self) -> list:
        return [len(self.local(g)) for g in range(self.n_gpus)]


def contiguous(n_experts: int, n_gpus: int) -> Placement:
    """No replicas: experts split over the GPUs in id order, as evenly as
    possible (the first GPUs take one more), the layout of the paper's
    expert-parallel nodes."""
    if not 1 <= n_gpus <= n_experts:
        raise ValueError("need 1 <= n_gpus <= n_experts")
    owner = []
    for g in range(n_gpus):
        owner += [g] * (n_experts // n_gpus + (1 if g < n_experts % n_gpus else 0))
    return Placement(n_gpus, tuple((g,) for g in owner))


def replicated(n_experts: int, n_gpus: int, copies: int, shift: int = 1) -> Placement:
    """Each expert on `copies` GPUs: its contiguous owner p and p + shift,
    p + 2 shift, ... (mod n_gpus).  copies == n_gpus holds every expert on
    every GPU."""
    if not 1 <= copies <= n_gpus:
        raise ValueError("need 1 <= copies <= n_gpus")
    base = contiguous(n_experts, n_gpus)
    holders = []
    for e in range(n_experts):
        p = base.holders[e][0]
        hs = sorted({(p + i * shift) % n_gpus for i in range(copies)})
        if len(hs) != copies:
            raise ValueError("shift repeats a GPU before `copies` distinct holders")
        holders.append(tuple(hs))
    return Placement(n_gpus, tuple(holders))


def _assign_with_cap(experts, placement: Placement, cap: int):
    """Maximum bipartite matching of experts to GPU slots (cap slots per GPU)
    by augmenting paths (Kuhn's algorithm), experts in ascending id, slots
    tried in ascending (GPU, slot) order; None if some expert stays
    unplaced."""
    owner = {}   # (gpu, slot) -> expert

    def augment(e, seen):
        for g in placement.holders[e]:
            for i in range(cap):
                slot = (g, i)
                if slot in seen:
                    continue
                seen.add(slot)
                if slot not in owner or augment(owner[slot], seen):
                    owner[slot] = e
                    return True
        return False

    for e in experts:
        if not augment(e, set()):
            return None
    return {e: g for (g, _), e in owner.items()}


def assign(selected, placement: Placement) -> dict:
    """Selected expert -> executing GPU, minimising the busiest GPU's count
    of executed experts (the smallest feasible cap, found in increasing
    order).  The result depends on the set of selected experts only, not on
    their order."""
    experts = sorted(set(int(e) for e in selected))
    for e in experts:
        if not 0 <= e < placement.n_experts:
            raise ValueError(f"expert {e} outside [0, {placement.n_experts})")
    if not experts:
        return {}
    lo = math.ceil(len(experts) / placement.n_gpus)
    for cap in range(lo, len(experts) + 1):
        where = _assign_with_cap(experts, placement, cap)
        if where is not None:
            return dict(sorted(where.items()))
    raise AssertionError("a cap of len(experts) always fits")


def loads(where: dict, n_gpus: int) -> list:
    """Executed experts per GPU of an assignment."""
    out = [0] * n_gpus
    for g in where.values():
        out[g] += 1
    return out


@dataclass
class LRPlanner:
    """Router-aided dynamic loading across layers.  Per layer: assign the
    selected experts to holders (exact, as ``assign``), take the busiest
    GPU's count m, and (with fill) let every GPU with fewer than m executed
    experts add its least recently used held experts that were not selected
    until it executes m (or runs out).  Filled experts compute and their
    outputs are discarded (weighted by zero).  `use` records, per GPU and
    held expert, the last step that executed it (-1: never); ties in recency
    go to the lower expert id."""
    placement: Placement
    fill: bool = True
    step: int = 0
    use: dict = field(default_factory=dict)

    def plan(self, selected) -> dict:
        """One layer: returns {'assign': expert->gpu for the selected experts,
        'executed': per GPU the executed experts (ascending), 'filled': per
        GPU the fill experts, 'max_load': m}."""
        P = self.placement
        where = assign(selected, P)
        own = [sorted(e for e, g in where.items() if g == gg) for gg in range(P.n_gpus)]
        m = max((len(o) for o in own), default=0)
        sel = set(where)
        executed, filled = [], []
        for g in range(P.n_gpus):
            extra = []
            if self.fill and len(own[g]) < m:
                spare = [e for e in P.local(g) if e not in sel]
                spare.sort(key=lambda e: (self.use.get((g, e), -1), e))
                extra = spare[: m - len(own[g])]
            ex = sorted(own[g] + extra)
            for e in ex:
                self.use[(g, e)] = self.step
            executed.append(ex)
            filled.append(sorted(extra))
        self.step += 1
        return {"assign": where, "executed": executed, "filled": filled, "max_load": m}


def busy_full_loads(placement: Placement) -> list:
    """Busy full loading (L_B): every GPU executes every expert it holds, in
    every layer."""
    return placement.experts_per_gpu()


def expected_busiest_load(placement: Placement, top_k: int) -> float:
    """E[max over GPUs of executed experts] for one token whose top-k set is
    uniform over the experts, with the exact assignment; enumerates all
    C(n_experts, top_k) sets."""
    E = placement.n_experts
    if not 1 <= top_k <= E:
        raise ValueError("need 1 <= top_k <= n_experts")
    total = count = 0
    for sel in itertools.combinations(range(E), top_k):
        total += max(loads(assign(sel, placement), placement.n_gpus))
        count += 1
    return total / count


# One DBRX expert across its 40 layers (gate, up, down in bf16) and the
# replicated self-attention weights (Table tab:vars, note (b)), bytes.
DBRX_EXPERT_ALL_LAYERS = 3 * 6144 * 10752 * 2 * 40
DBRX_ATTENTION_ALL_LAYERS = (8192 * 6144 + 6144 * 6144) * 40 * 2
MI355X_HBM_BYTES = 288 * 10**9


def fits_mi355x(placement: Placement, hbm_bytes: int = MI355X_HBM_BYTES,
                reserve_bytes: int = 8 * 10**9) -> bool:
    """Whether every GPU holds its experts of all 40 DBRX layers plus the
    replicated attention weights, with reserve_bytes left for activations
    and the workspace."""
    per = max(placement.experts_per_gpu()) * DBRX_EXPERT_ALL_LAYERS
    return per + DBRX_ATTENTION_ALL_LAYERS + reserve_bytes <= hbm_bytes


def mi355x_placements(gpus=(2, 4, 8), top_k: int = 4, n_experts: int = 16) -> list:
    """For each GPU count, the placements from no replicas to every expert on
    every GPU that fit MI355X's HBM, with their expected busiest load."""
    rows = []
    for n in gpus:
        for copies in range(1, n + 1):
            p = contiguous(n_experts, n) if copies == 1 else replicated(n_experts, n, copies)
            if not fits_mi355x(p):
                continue
            rows.append({"gpus": n, "copies": copies,
                         "experts_per_gpu": max(p.experts_per_gpu()),
                         "exec_experts": expected_busiest_load(p, top_k)})
    return rows


def mi355x_placement_predictions(hbm_gbs: float, mfma_tflops: float, gpus=(2, 4, 8),
                                 collective_latency_s: float = 20e-6,
                                 link_gbs: float = 150.0) -> list:
    """Eq. (eq:pm) per token of the full 40-layer DBRX on 2..8 MI355X for
    every placement that fits, with E[#executed experts] from the exact
    assignment under uniform routing: what replicas buy once one GPU's
    streaming and matrix rates are measured."""
    from . import perf_model as pm
    model = pm.dbrx_exact()
    hw = pm.mi355x_hardware(hbm_gbs, mfma_tflops, collective_latency_s, link_gbs)
    rows = mi355x_placements(gpus)
    for r in rows:
        est = pm.estimate(r["exec_experts"], model, hw, n_nodes=r["gpus"])
        r["ms_per_token"] = est.time * 1e3
        r["tokens_per_s"] = est.throughput
    return rows
