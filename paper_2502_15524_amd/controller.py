"""Cold-start controller arithmetic: TTFT / TPOT prediction (section 4.1,
Eq. 1 and 2; Eq. 5 of section 5.2), resource allocation (section 4.1) and
network-contention-aware placement (section 4.2, Eq. 3 and 4), calibrated
with this engine's measured prefill, decode and host-link figures. Pure host code; nothing here touches the GPU.

Notation follows the paper: t_c container creation + runtime initialisation,
t_n network transfer between pipeline workers, t_p prefill and t_d decode
time of the whole model on one worker, M the model size, s the pipeline
parallelism size, w the number of full-memory workers (0 <= w <= s), b_i and
p_i the network and PCIe bandwidth of server i. Times in seconds, sizes in
bytes, bandwidths in bytes per second.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Sequence, Tuple


@dataclasses.dataclass(frozen=True)
class History:
    """Historical time costs of a model (section 4.1). t_cc, t_cu, t_l split
    t_c for the overlapped prediction of section 5.2 (container creation,
    GPU context initialisation, library loading)."""
    t_c: float
    t_n: float
    t_p: float
    t_d: float
    t_cc: float = 0.0
    t_cu: float = 0.0
    t_l: float = 0.0


@dataclasses.dataclass(frozen=True)
class Server:
    """A GPU server as the allocator sees it: network bandwidth b, PCIe
    bandwidth p, free GPU memory for one more worker, and the number of
    workers already running on its GPU (0 = a free GPU)."""
    name: str
    b: float
    p: float
    free_mem: float
    workers: int = 0

    @property
    def ratio(self) -> float:
        """Fetch-and-load seconds per byte, 1/b + 1/p."""
        return 1.0 / self.b + 1.0 / self.p


def prefill_factor(s: int, w: int) -> float:
    """Prefill (or decode) time of the group in units of the single-worker
    time: a full-memory worker computes its 1/s of the model at full speed,
    a low-memory worker shares its GPU and takes as long as the whole model."""
    if not (1 <= s and 0 <= w <= s):
        raise ValueError("need s >= 1 and 0 <= w <= s")
    return (s - w) + w / s


def predict_ttft(h: History, M: float, s: int, w: int, servers: Sequence[Server]) -> float:
    """Equation 1: runtime initialisation, fetching and loading 1/s of the
    model at the slowest selected server's rate, prefill, and s network
    transfers."""
    if len(servers) != s:
        raise ValueError("one server per pipeline worker")
    max_ratio = max(x.ratio for x in servers)
    return h.t_c + M / s * max_ratio + h.t_p * prefill_factor(s, w) + h.t_n * s


def predict_tpot(h: History, s: int, w: int) -> float:
    """Equation 2."""
    return h.t_d * prefill_factor(s, w) + h.t_n * s


def predict_ttft_overlapped(h: History, M: float, s: int, w: int,
                            servers: Sequence[Server]) -> float:
    """Equation 5 (worker-level overlapping): fetching overlaps container
    creation, loading overlaps library loading; the slowest worker decides."""
    if len(servers) != s:
        raise ValueError("one server per pipeline worker")
    part = M / s
    start = max(max(h.t_cc + h.t_cu + max(part / x.p, h.t_l), part / x.b) for x in servers)
    return start + h.t_p * prefill_factor(s, w) + h.t_n * s


@dataclasses.dataclass(frozen=True)
class Choice:
    s: int
    w: int
    servers: Tuple[Server, ...]
    ttft: float
    tpot: float

    @property
    def memory(self) -> float:
        """GPU memory reserved, in units of the model size."""
        return self.w + (self.s - self.w) / self.s

    @property
    def sharing(self) -> int:
        """Workers placed on GPUs that already run other workers."""
        return sum(1 for x in self.servers if x.workers > 0)


def _placement(servers: Sequence[Server], M: float, s: int, w: int):
    """The server group for s workers of which w hold the whole model.

    TTFT (Eq. 1) depends on the group only through its slowest fetch-and-load
    rate, so the group is a bottleneck choice: the smallest rate limit r such
    that, among the servers with ratio <= r, at least w can hold the model
    (M) and at least s can hold a 1/s part of it (every server that holds M
    holds M/s too). Under that limit, the fewest busy GPUs: the w
    whole-model slots take free GPUs first, then the remaining s - w slots
    do; within each, the faster server first. Returns None if no group
    exists."""
    part = M / s
    fits_full = [x for x in servers if x.free_mem >= M]
    fits_part = [x for x in servers if x.free_mem >= part]
    if len(fits_full) < w or len(fits_part) < s:
        return None
    for r in sorted({x.ratio for x in fits_part}):
        full = [x for x in fits_full if x.ratio <= r]
        usable = [x for x in fits_part if x.ratio <= r]
        if len(full) >= w and len(usable) >= s:
            break
    else:
        return None
    prefer = lambda x: (x.workers > 0, x.ratio)   # noqa: E731  free GPU, then faster
    chosen = sorted(full, key=prefer)[:w]
    rest = sorted((x for x in usable if x not in chosen), key=prefer)[:s - w]
    return tuple(chosen) + tuple(rest)


def enumerate_choices(h: History, M: float, servers: Sequence[Server],
                      max_s: int = 4) -> List[Choice]:
    """Every deployment choice with its TTFT and TPOT predictions (Eq. 1 and
    2): pipeline sizes s = 1 .. max_s (the paper caps it at 4), w = 0 .. s
    whole-model workers, each with the group `_placement` picks; choices
    without a feasible group are left out."""
    out = []
    for s in range(1, max_s + 1):
        for w in range(s + 1):
            g = _placement(servers, M, s, w)
            if g is not None:
                out.append(Choice(s, w, g, predict_ttft(h, M, s, w, g), predict_tpot(h, s, w)))
    return out


def allocate(h: History, M: float, servers: Sequence[Server], slo_ttft: float,
             slo_tpot: float, max_s: int = 4) -> Choice:
    """Resource allocation (section 4.1): among the choices whose predicted
    TTFT and TPOT meet the SLOs, the one with the fewest workers on busy GPUs
    (the paper prefers free GPUs), then the least GPU memory reserved, then
    the smallest pipeline. If none meets them, one worker holding the whole
    model on the server that fetches and loads it fastest."""
    ok = [c for c in enumerate_choices(h, M, servers, max_s)
          if c.ttft <= slo_ttft and c.tpot <= slo_tpot]
    if ok:
        return min(ok, key=lambda c: (c.sharing, c.memory, c.s))
    g = _placement(servers, M, 1, 1)
    if g is None:
        raise ValueError("no server fits the whole model")
    return Choice(1, 1, g, predict_ttft(h, M, 1, 1, g), predict_tpot(h, 1, 1))


class ServerBandwidth:
    """Network-contention-aware placement bookkeeping of one server (section
    4.2): its cold-start workers share bandwidth B equally; each has a
    fetching deadline D_i and a pending model size S_i."""

    def __init__(self, B: float):
        self.B = B
        self.workers: Dict[str, List[float]] = {}   # name -> [S_i, D_i]
        self.t_last = 0.0

    def _advance(self, T: float) -> None:
        """Equation 4: every pending size shrinks by B/N (T - T')."""
        n = len(self.workers)
        if n:
            for name in list(self.workers):
                self.workers[name][0] -= self.B / n * (T - self.t_last)
                if self.workers[name][0] < 0:          # fetched: leave the list
                    del self.workers[name]
        self.t_last = T

    def admits(self, T: float, size: float, deadline: float) -> bool:
        """Equation 3 for every worker, the newcomer included, with N + 1
        workers sharing B from time T."""
        self._advance(T)
        n1 = len(self.workers) + 1
        cand = list(self.workers.values()) + [[size, deadline]]
        return all(S <= self.B / n1 * (D - T) for S, D in cand)

    def add(self, name: str, T: float, size: float, deadline: float) -> bool:
        if not self.admits(T, size, deadline):
            return False
        self.workers[name] = [size, deadline]
        return True

    def finish(self, name: str, T: float) -> None:
        self._advance(T)
        self.workers.pop(name, None)


def calibrate(prefill_s: float, decode_s: float, t_c: float = 0.0, t_n: float = 0.0,
              **overlap) -> History:
    """A History from this engine's measured whole-model prefill and decode
    times (bench.py), plus assumed initialisation and network costs."""
    return History(t_c=t_c, t_n=t_n, t_p=prefill_s, t_d=decode_s, **overlap)
