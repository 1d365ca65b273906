"""Request traces for the continuous-batching harness (Sec. 3.7-3.8): each request has an
arrival step, a prompt length and a decode length. The families follow the paper's
synthetic traces; external traces come from CSV or JSON files with the fields
prompt_len, decode_len and optionally arrival_step.

bucketed     prompt lengths cycle through 8K, 16K, 32K, 64K
homogeneous  every prompt 32K
bimodal      one long prompt U[16384,32768] for every three short U[256,2048]
uniform      prompts U[1024,32768]
zipf         prompts min(32768, 256 k), k ~ Zipf(1.2)

Decode lengths are U[decode_min, decode_max]; arrivals are every `arrival_gap` steps
(0: all at step 0). Everything is seeded; no attention arithmetic lives here.
"""
from __future__ import annotations

import csv
import dataclasses
import json
import os

import numpy as np

FAMILIES = ("bucketed", "homogeneous", "bimodal", "uniform", "zipf")


@dataclasses.dataclass(frozen=True)
class Request:
    rid: int
    arrival_step: int
    prompt_len: int
    decode_len: int


def request_trace(family: str, n: int, seed: int = 20260622, decode_min: int = 64, decode_max: int = 256,
                  arrival_gap: int = 0) -> list:
    if n < 1:
        raise ValueError("n must be positive")
    r = np.random.Generator(np.random.PCG64(seed))
    if family == "bucketed":
        prompts = np.array([8192, 16384, 32768, 65536])[np.arange(n) % 4]
    elif family == "homogeneous":
        prompts = np.full(n, 32768)
    elif family == "bimodal":
        long = (np.arange(n) % 4) == 3          # one long request for every three short
        prompts = np.where(long, r.integers(16384, 32768 + 1, size=n), r.integers(256, 2048 + 1, size=n))
    elif family == "uniform":
        prompts = r.integers(1024, 32768 + 1, size=n)
    elif family == "zipf":
        prompts = np.minimum(32768, 256 * r.zipf(1.2, size=n))
    else:
        raise KeyError(family)
    decode = r.integers(decode_min, decode_max + 1, size=n)
    return [Request(i, i * arrival_gap, int(p), int(d)) for i, (p, d) in enumerate(zip(prompts, decode))]


def save_trace(trace, path: str) -> None:
    rows = [{"prompt_len": q.prompt_len, "decode_len": q.decode_len, "arrival_step": q.arrival_step}
            for q in trace]
    if path.endswith(".json"):
        with open(path, "w") as f:
            json.dump(rows, f, indent=1)
    else:
        with open(path, "w", newline="") as f:
            w = csv.DictWriter(f, fieldnames=["prompt_len", "decode_len", "arrival_step"])
            w.writeheader()
            w.writerows(rows)


def load_trace(path: str) -> list:
    """CSV (header row) or JSON list of objects; arrival_step defaults to 0."""
    if not os.path.exists(path):
        raise FileNotFoundError(path)
    if path.endswith(".json"):
        with open(path) as f:
            rows = json.load(f)
    else:
        with open(path, newline="") as f:
            rows = list(csv.DictReader(f))
    out = []
    for i, row in enumerate(rows):
        p, d = int(row["prompt_len"]), int(row["decode_len"])
        a = int(row.get("arrival_step") or 0)
        if p < 0 or d < 1 or a < 0:
            raise ValueError(f"bad request {i}: {row}")
        out.append(Request(i, a, p, d))
    return out
