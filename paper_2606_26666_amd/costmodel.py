"""Route cost model (Sec. 3.5), fitted to this GPU.

For one decode step over lengths N_i, route r is priced as

    T_r = sum_j KV_j / beta * max(1, C_min / C_j) * (1 - gamma [pairs])
          + L_r * lambda + Merge_r / beta + T_0 + T_f(r)

where the sum runs over the route's split launches j (one for the workqueue routes and
the rectangular grid, one per group for the length buckets), KV_j is the K/V bytes launch
j streams, C_j its split workgroups per compute unit, L_r the launches per step, Merge_r
the partial-state bytes written and read back, beta the streaming-read bandwidth and
lambda the device time per launch. The first three terms are the paper's model. Added
here, because on MI355X they are not small against a step:
  T_0     a fixed chain of memory round trips every step pays (lengths, page ids, first
          pages, state store, completion counter, merge), roughly 10 us;
  T_f(r)  a fixed term per route family (`FAMILY`: the one-launch route, whose planner
          runs inside the launch; the routes behind a planner kernel; the rectangular
          grids, which plan nothing), relative to the one-launch route;
  gamma   the faster KV stream of the one-launch route when it runs KV-head pairs (each
          workgroup then reads two heads' slices of every token, which evens out the
          per-head and per-XCD read rates).
lambda is measured by a probe; C_min, T_0, T_f, gamma and the effective beta (the KV
stream of a step runs below the probe's streaming-read rate, which is kept beside it) are
fitted to measured steps (`fit`).

Everything here is host arithmetic over the planner's counts (`pkv_plan_host`); it
launches nothing.
"""
from __future__ import annotations

import dataclasses
import json
import math

import numpy as np

from . import _binding as _b

ROUTES = ("one-launch", "plan+fused", "two-kernel", "rect", "exact-buckets", "coarse-buckets")
# route families that share a fixed per-step term T_f
FAMILY = {"one-launch": "one-launch", "plan+fused": "planner kernel", "two-kernel": "planner kernel",
          "rect": "rectangular", "exact-buckets": "rectangular", "coarse-buckets": "rectangular"}
CUS = 256                 # compute units of an MI355X
SPLITS_PER_ROW_HEAD = 4   # splits per KV head per active row the task target leaves room for
LAUNCHES = {"one-launch": 1, "plan+fused": 2, "two-kernel": 3}
MAX_BUCKET_ROWS = 64   # rows one rectangular launch can name
COARSE_BUCKET_TOKENS = 16384


@dataclasses.dataclass
class Calibration:
    beta_gbs: float          # effective KV streaming bandwidth of a step, GB/s
    launch_us: float         # device time per back-to-back launch, us
    c_min: float = 1.0       # occupancy (split workgroups per CU) below which KV streams slower
    fixed_us: float = 0.0    # per-step fixed latency T_0, us
    cus: int = 256           # compute units
    probe_beta_gbs: float = 0.0  # streaming-read bandwidth of the probe (a 1 GiB read), GB/s
    route_fixed_us: dict = dataclasses.field(default_factory=dict)  # T_f per FAMILY entry, us
    pair_gain: float = 0.0   # gamma: fraction of KV streaming time KV-head pairs save
    note: str = ""

    def save(self, path: str) -> None:
        with open(path, "w") as f:
            json.dump(dataclasses.asdict(self), f, indent=2, sort_keys=True)
            f.write("\n")

    @classmethod
    def load(cls, path: str) -> "Calibration":
        with open(path) as f:
            d = json.load(f)
        names = [fld.name for fld in dataclasses.fields(cls)]
        return cls(**{k: d[k] for k in names if k in d})


@dataclasses.dataclass
class RouteShape:
    """What a route does in one step: per split launch (KV bytes, split workgroups), the
    launch count and the partial-state bytes written and read."""
    launches: list            # [(kv_bytes, workgroups)] per split launch
    launch_count: int
    merge_bytes: int
    merge_launches: int
    route: str = "one-launch"
    pairs: bool = False       # the one-launch route runs KV-head pairs

    @property
    def workgroups(self) -> int:
        return int(sum(w for _, w in self.launches))


def slot_bytes(G: int, d: int = 128) -> int:
    """Partial-state slot: fp32 acc[G][d], m[G], l[G], padded to 16 bytes."""
    return 4 * (G * d + ((2 * G + 3) // 4) * 4)


def head_pairs(hq: int, hkv: int) -> bool:
    """Whether the one-launch route runs KV heads g and g + 1 in one workgroup: G = 4
    (the matrix-core task body; at G = 8 a pair's merge needs two rounds of loads and
    pairs measured 11% slower on the B8 traces) with an even KV-head count. The library
    does so when the task target is at least two tasks per resident workgroup."""
    return hkv > 0 and hq % hkv == 0 and hq // hkv == 4 and hkv % 2 == 0


PAIR_MAX_SPLITS = 24  # splits per (row, KV head) up to which KV-head pairs pay


def default_target(lens, hkv: int, cus: int = CUS, per_row: int = SPLITS_PER_ROW_HEAD, hq: int = 32) -> int:
    """Task target of the workqueue planner (Sec. 3.5's split choice) for a step over the
    lengths `lens`: one task per compute unit, raised so that each KV head has room for
    `per_row` splits per active row. With many KV heads a fixed target of one task per
    compute unit leaves a ragged batch one or two splits per row and head, and the longest
    row's task sets the step (measured on MI355X: B8 traces at Hkv = 32 run 24-47% faster
    at 1024 tasks than at 256).

    Two tasks per compute unit where KV-head pairs apply and, at that target, the longest
    row would get at most 24 splits per KV head (its share of the step's tokens times the
    2 * cus / Hkv splits per head): each workgroup then streams two heads' slices of every
    token, which evens out the per-head read rates, and a pair's last arriver merges both
    heads' few states in one round of loads. Measured at Hkv = 8: the B8 traces (longest
    row 20-35% of the tokens, at most 21 splits) run 3-6% faster than at 256 tasks; B4
    bimodal (31-35 splits) and B1 (64 splits) run 5% and 11% slower, the pair merges
    outgrowing the balance gain."""
    lens = np.asarray(lens, dtype=np.int64).reshape(-1)
    active = int(np.count_nonzero(lens))
    base = max(cus, per_row * hkv * max(1, active))
    total = int(lens.sum())
    if head_pairs(hq, hkv) and total > 0 and 2 * cus * int(lens.max()) <= PAIR_MAX_SPLITS * hkv * total:
        return max(base, 2 * cus)
    return base


def rect_split_count(n_rows: int, hkv: int, params) -> int:
    """One split count for a rectangular launch over n_rows rows (the batch rule)."""
    s = -(-params.target_tasks // (max(1, n_rows) * hkv))
    return int(min(max(s, params.split_min), params.split_max))


def bucket_groups(lens, exact: bool, bucket_tokens: int = COARSE_BUCKET_TOKENS):
    """Row groups of the bucket routes, as pkv_decode_buckets forms them: rows keyed by
    exact length or by ceil(length / bucket_tokens) (empty rows form their own group,
    launched so that their output is written as zeros), each key split into launches of
    at most 64 rows. Returns a list of row-index arrays."""
    lens = np.asarray(lens, dtype=np.int64)
    keys = np.where(lens == 0, -1, lens if exact else -(-lens // bucket_tokens))
    groups = []
    for k in sorted(set(keys.tolist())):
        rows = np.nonzero(keys == k)[0]
        for c in range(0, rows.size, MAX_BUCKET_ROWS):
            groups.append(rows[c:c + MAX_BUCKET_ROWS])
    return groups


def route_shape(route: str, lens, params, hq: int = 32, d: int = 128,
                max_pages_per_row: int | None = None) -> RouteShape:
    """Counts of one step of `route` over lengths `lens` with planner parameters `params`."""
    lens = np.asarray(lens, dtype=np.int64)
    hkv = params.num_kv_heads
    G = hq // hkv
    kv_tok = 2 * hkv * d * 2
    sb = slot_bytes(G, d)
    kv = int(lens.sum()) * kv_tok
    if route in LAUNCHES:
        maxp = max_pages_per_row or int(lens.max(initial=0)) // 16 + 1
        _, _, n = _b.pkv_plan_host(lens, params, maxp, with_tasks=False)
        pairs = route == "one-launch" and head_pairs(hq, hkv) and params.target_tasks >= 2 * CUS
        return RouteShape([(kv, n)], LAUNCHES[route], 2 * n * sb, 1 if route == "two-kernel" else 0, route, pairs)
    if route == "rect":
        active = int(np.count_nonzero(lens))
        slots = lens.size * hkv * rect_split_count(active, hkv, params)
        return RouteShape([(kv, slots)], 2, 2 * slots * sb, 1, route)
    if route in ("exact-buckets", "coarse-buckets"):
        launches, slots = [], 0
        groups = bucket_groups(lens, route == "exact-buckets")
        for rows in groups:
            s = rows.size * hkv * rect_split_count(rows.size, hkv, params)
            launches.append((int(lens[rows].sum()) * kv_tok, s))
            slots += s
        return RouteShape(launches, 2 * len(groups), 2 * slots * sb, len(groups), route)
    raise ValueError(f"unknown route {route}")


def estimate_us(shape: RouteShape, cal: Calibration) -> float:
    """T_r of the module docstring, in microseconds."""
    bw = cal.beta_gbs * 1e3  # bytes per microsecond
    t = 0.0
    for kv, wgs in shape.launches:
        c = wgs / cal.cus
        t += kv / bw * max(1.0, cal.c_min / c) if c > 0 else 0.0
    if shape.pairs:
        t *= 1.0 - cal.pair_gain
    return (t + shape.launch_count * cal.launch_us + shape.merge_bytes / bw + cal.fixed_us
            + cal.route_fixed_us.get(FAMILY[shape.route], 0.0))


def choose_route(lens, params, cal: Calibration, routes=ROUTES, **kw):
    """(cheapest route, {route: estimated us}) for one step."""
    est = {r: estimate_us(route_shape(r, lens, params, **kw), cal) for r in routes}
    return min(est, key=est.get), est


def fit(samples, probe_beta_gbs: float, launch_us: float, cus: int = 256,
        c_grid=None, beta_scales=None, gamma_grid=None) -> Calibration:
    """Fit the effective beta, C_min, gamma, T_0 and the per-family T_f to measured
    steps, lambda fixed by its probe.

    samples: [(RouteShape, measured_us)]. On a grid of (beta, C_min, gamma) the best
    intercepts are the mean residual of each route family (least squares in T_0 + T_f);
    the grid point with the smallest squared error wins. T_0 is the one-launch family's
    intercept (or the first family's, without one-launch samples) and T_f the other
    families' offsets from it. beta is searched as a fraction of the probe's
    streaming-read bandwidth.
    """
    if not samples:
        raise ValueError("no samples")
    if c_grid is None:
        c_grid = np.round(np.arange(0.1, 4.0001, 0.1), 4)
    if beta_scales is None:
        beta_scales = np.round(np.arange(0.60, 1.1001, 0.01), 4)
    if gamma_grid is None:
        gamma_grid = np.round(np.arange(0.0, 0.2001, 0.01), 4)
    fams = [FAMILY[sh.route] for sh, _ in samples]
    names = sorted(set(fams), key=lambda f: (f != "one-launch", f))
    meas = np.array([m for _, m in samples], dtype=np.float64)
    # per sample: KV bytes and workgroups per CU of each split launch, the fixed bytes and launches
    lsum = np.array([sh.launch_count * launch_us for sh, _ in samples])
    merge = np.array([sh.merge_bytes for sh, _ in samples], dtype=np.float64)
    pairs = np.array([sh.pairs for sh, _ in samples])
    best = None
    for c in c_grid:
        # KV bytes weighted by the occupancy factor, per sample
        kvw = np.array([sum(kv * max(1.0, c / (w / cus)) for kv, w in sh.launches if w > 0) for sh, _ in samples])
        for g in gamma_grid:
            kvg = np.where(pairs, kvw * (1.0 - g), kvw)
            for bs in beta_scales:
                bw = probe_beta_gbs * float(bs) * 1e3
                resid = meas - (kvg / bw + lsum + merge / bw)
                err = 0.0
                icpt = {}
                for f in names:
                    sel = np.array([x == f for x in fams])
                    icpt[f] = float(resid[sel].mean())
                    err += float(((resid[sel] - icpt[f]) ** 2).sum())
                if best is None or err < best[0] - 1e-9:
                    best = (err, float(bs), float(c), float(g), icpt)
    err, bs, c, g, icpt = best
    t0 = icpt[names[0]]
    rms = math.sqrt(err / len(samples))
    return Calibration(probe_beta_gbs * bs, launch_us, c, t0, cus, probe_beta_gbs,
                       route_fixed_us={f: icpt[f] - t0 for f in names}, pair_gain=g,
                       note=f"fit over {len(samples)} steps, rms {rms:.2f} us")
