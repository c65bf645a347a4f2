"""Oracle for plan-bundle annotations and load-driven variant switching: plain,
slow, obviously correct Python written from the paper.

TEST INFRASTRUCTURE ONLY: the test suite may use this module; the product path
never does.  It shares no code with the GPU library.

Annotations (Sec. 4.4 and Algorithm gen: each variant carries per-model demand
and a profile-based quality estimate; the model with the largest share of the
planned demand is the variant's dominant model, Sec. 5.2):
  demand[m]  = sum over LLM nodes n whose chosen implementation runs model m of
               its nominal duration tau (fp64, node order);
  dominant   = the model with the largest demand, equal demand to the lowest
               model id; -1 when no LLM node exists;
  quality    = product over LLM nodes of (1 - v_n (1 - q_n)), fp64 in node
               order (readings: the plan's chance of no impact-weighted error,
               f = v r with r = 1 - q, under independent nodes).

Switching (Sec. 5.2, "Switching plan variants"), one load sample at a time,
starting on variant 0 with no earlier switch:
  - within `dwell` of the last switch nothing changes;
  - if the active variant's dominant-model load exceeds `high`, take the first
    later variant j (in level order) whose dominant model differs from the
    active one's, is not itself above `high`, has load at most the active
    one's minus `margin`, and whose quality is at most `tolerance` below the
    active variant's;
  - otherwise, from a variant other than 0, return to the lowest-index variant
    whose dominant-model load is below `low` and that passes the same quality
    check;
  - when no transition is eligible the selection is retained.
A variant without an LLM node (dominant -1) sees load 0.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple


def annotate(prob, impl: Sequence[int], model, n_models: int, is_tool=None) -> Tuple[List[float], int, float]:
    """(per-model demand, dominant model, quality) of one plan."""
    demand = [0.0] * n_models
    quality = 1.0
    any_llm = False
    for n in range(prob.n_nodes):
        if is_tool is not None and is_tool[n]:
            continue
        any_llm = True
        i = int(impl[n])
        demand[int(model[n][i])] += float(prob.tau[n][i])
        t = 1.0 - float(prob.p[n][i])
        t = float(prob.w[n]) * t
        quality = quality * (1.0 - t)
    dominant = -1
    if any_llm:
        dominant = 0
        for m in range(1, n_models):
            if demand[m] > demand[dominant]:
                dominant = m
    return demand, dominant, quality


def simulate(dominant: Sequence[int], quality: Sequence[float], times: Sequence[float], loads,
             high: float, low: float, tolerance: float, margin: float, dwell: float) -> Tuple[List[int], int]:
    """(active variant after each sample, number of switches)."""
    K = len(dominant)

    def load_of(sample, v):
        d = dominant[v]
        return 0.0 if d < 0 else float(sample[d])

    def quality_ok(cur, j):
        return quality[cur] - quality[j] <= tolerance

    cur = 0
    last = None
    out = []
    switches = 0
    for t, sample in zip(times, loads):
        if last is not None and t - last < dwell:
            out.append(cur)
            continue
        nxt = cur
        if load_of(sample, cur) > high:
            for j in range(cur + 1, K):
                if dominant[j] == dominant[cur]:
                    continue
                if load_of(sample, j) > high:
                    continue
                if not load_of(sample, j) <= load_of(sample, cur) - margin:
                    continue
                if not quality_ok(cur, j):
                    continue
                nxt = j
                break
        elif cur > 0:
            for j in range(0, cur):
                if load_of(sample, j) < low and quality_ok(cur, j):
                    nxt = j
                    break
        if nxt != cur:
            cur = nxt
            last = t
            switches += 1
        out.append(cur)
    return out, switches
