"""Seeded request traces for the trajectory-task simulator.

The paper's traces are not available; these stand in for its two workloads
(section 6.1): a compact mixed-arrival period, and a foreground burst of short
requests arriving while longer ones are in flight.  Each request carries the
scheduler-visible deadline the paper defines, arrival + alpha_c * T_c, with T_c
the class's standalone service time (here: its steps at degree 1 from the cost
table) and alpha_c the paper's multiplier.  Arrival rates are set as a
fraction `load` of the capacity of `n_ranks` ranks serving requests alone at
degree 1.  Nothing here computes a schedule.
"""
from typing import Dict, List, Sequence

import numpy as np

from .workloads import REQUEST_CLASSES


def standalone_us(step_ms: Dict[str, float], cls_name: str) -> int:
    c = REQUEST_CLASSES[cls_name]
    return int(round(c.n_steps * step_ms[f"{cls_name}@1"] * 1000))


def make_trace(kind: str, model: str, step_ms: Dict[str, float], n_ranks: int, duration_s: float,
               load: float, seed: int) -> Dict[str, List[int]]:
    """kind: "mixed" (Poisson arrivals, S/M/L equally likely) or "burst" (M/L
    in the background at half the load, plus bursts of 2 * n_ranks short
    requests every duration/4).  Returns arrival_us, cls (index into
    `classes`), n_steps, deadline_us and the class names."""
    names = [n for n, c in REQUEST_CLASSES.items() if c.model == model]
    rng = np.random.default_rng([13501, 31, seed, 0 if kind == "mixed" else 1])
    T = {n: standalone_us(step_ms, n) for n in names}
    dur = int(duration_s * 1e6)
    arrival, cls = [], []
    if kind == "mixed":
        mean_T = float(np.mean([T[n] for n in names]))
        rate = load * n_ranks / mean_T                  # requests per us
        t = 0.0
        while True:
            t += rng.exponential(1.0 / rate)
            if t >= dur:
                break
            arrival.append(int(t))
            cls.append(int(rng.integers(0, len(names))))
    elif kind == "burst":
        bg = [n for n in names if not n.endswith("_S")]
        mean_T = float(np.mean([T[n] for n in bg]))
        rate = 0.5 * load * n_ranks / mean_T
        t = 0.0
        while True:
            t += rng.exponential(1.0 / rate)
            if t >= dur:
                break
            arrival.append(int(t))
            cls.append(names.index(bg[int(rng.integers(0, len(bg)))]))
        short = names.index(next(n for n in names if n.endswith("_S")))
        for b in range(1, 4):
            t0 = b * dur // 4
            for k in range(2 * n_ranks):
                arrival.append(t0 + int(rng.integers(0, 200_000)))
                cls.append(short)
    else:
        raise ValueError(kind)
    order = np.argsort(np.asarray(arrival), kind="stable")
    arrival = [arrival[i] for i in order]
    cls = [cls[i] for i in order]
    n_steps = [REQUEST_CLASSES[names[c]].n_steps for c in cls]
    deadline = [a + int(REQUEST_CLASSES[names[c]].alpha * T[names[c]]) for a, c in zip(arrival, cls)]
    return {"arrival_us": arrival, "cls": cls, "n_steps": n_steps, "deadline_us": deadline, "classes": names}


def cost_matrix(step_ms: Dict[str, float], classes: Sequence[str], degrees: Sequence[int]) -> List[List[int]]:
    """Integer microseconds per (class, degree) from the measured table."""
    return [[int(round(step_ms[f"{c}@{d}"] * 1000)) for d in degrees] for c in classes]


def read_cost_table(path: str) -> Dict[str, float]:
    """The machine-readable line of a cost-table summary ("step_ms = {...}")."""
    import json
    for line in open(path):
        if line.startswith("step_ms = "):
            return json.loads(line[len("step_ms = "):])
    raise ValueError(f"no step_ms line in {path}")
