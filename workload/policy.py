"""Seeded stand-in for the offline calibration of the paper (Alg. 1) and the
binary policy-blob format.

The paper calibrates, per bucket q = (tag, layer group), a task-error
sensitivity envelope V-bar (Eq. 5), a protection floor (Eq. 6), distortion
D(q, a) (Eq. 4) and adjacent upgrade scores rho_D (Eq. 7), then walks a
greedy upgrade path from the floors and freezes the selected policy, its
floors and the scores into a table Lambda.  Model trajectories and benchmark
data are not available, so V-bar and D are synthesised from seeded priors (a
criticality prior per tag, a depth prior per layer group); the floor rule,
the upgrade score and the greedy walk are then applied as the paper states,
stopping at a target expected KV budget beta instead of a development-set
reliability gate.  Only the frozen table is consumed by the hot path.

Blob layout (little-endian), version 1:
  0  char[4]  magic "PASK"
  4  u16      version (1)
  6  u16      header bytes (32)
  8  u32      n_tags
  12 u32      n_groups
  16 u32      n_layers
  20 u32      n_sink          (leading positions of every sequence kept HIGH)
  24 u32      recent_window   (protected recent window W, Section 3.1)
  28 u32      payload bytes
  32 u8       group_of_layer[n_layers]
     u8       action[n_tags][n_groups]   selected action a0
     u8       floor[n_tags][n_groups]    protection floor a-
     u8       zero padding to a multiple of 4
     f32      rho_up[n_tags][n_groups][2]  (R->L, L->H)
  end u32     FNV-1a 32-bit hash of all preceding bytes
Version 2 appends, after rho_up, the state of the online budget controller
(Eq. 9-10, Alg. 2):
     u32      n_states        (parser states s)
     u32      beta_q          target budget beta in units of 1/65536
     u32      reserve_q[n_states]  Gamma(s) in units of 1/16 of the bytes one token
                                  persists at RETAIN-HIGH in every layer
     u8       crit[n_states]  Crit(s): critical or lookahead-critical state
     u8       zero padding to a multiple of 4
Actions: 0 = DROP (release), 1 = RETAIN-LOW, 2 = RETAIN-HIGH.
"""

from __future__ import annotations

import struct
from dataclasses import dataclass, field

import numpy as np

from .tensors import sub_seed

DROP, LOW, HIGH = 0, 1, 2
# Stored bytes of one RETAIN-LOW entry relative to RETAIN-HIGH: int4 codes plus
# one fp16 scale per 32 elements, against bf16: (D/2 + 2*D/32) / (2*D).
LOW_COST_RATIO = 0.28125

CRITICALITY = {  # prior kappa_z per tag id (decode tags 0-5, prompt labels 6-11)
    0: 0.9, 1: 0.8, 2: 0.5, 3: 0.6, 4: 0.2, 5: 0.1,
    6: 0.9, 7: 0.85, 8: 0.8, 9: 0.6, 10: 0.3, 11: 0.15,
}
TAU_LOW, TAU_HIGH = 0.005, 0.01  # threshold pair selected in Section 4.5


@dataclass
class PolicyTable:
    n_tags: int
    n_groups: int
    n_layers: int
    group_of_layer: np.ndarray   # uint8 [n_layers]
    action: np.ndarray           # uint8 [n_tags, n_groups]
    floor: np.ndarray            # uint8 [n_tags, n_groups]
    rho_up: np.ndarray           # float32 [n_tags, n_groups, 2]
    n_sink: int = 0
    recent_window: int = 0
    beta: float = float("nan")
    expected_cost: float = float("nan")
    tag_probs: np.ndarray = field(default=None)
    # Online budget controller (blob version 2); n_states == 0: static lookup only.
    n_states: int = 0
    beta_q: int = 0
    reserve_q: np.ndarray = field(default=None)   # uint32 [n_states]
    crit: np.ndarray = field(default=None)        # uint8 [n_states]


def contiguous_groups(n_layers: int, n_groups: int) -> np.ndarray:
    """Layer l belongs to group l // (n_layers / n_groups) (equal contiguous groups)."""
    per = n_layers // n_groups
    assert per * n_groups == n_layers
    return (np.arange(n_layers) // per).astype(np.uint8)


def _expected_cost(act, p, w):
    cost = np.array([0.0, LOW_COST_RATIO, 1.0])
    num = (p[:, None] * w[None, :] * cost[act]).sum()
    den = (p[:, None] * w[None, :]).sum()
    return float(num / den)


def make_policy(n_tags: int, n_groups: int, n_layers: int, beta: float, seed: int,
                tag_probs: np.ndarray | None = None, n_sink: int = 0) -> PolicyTable:
    rng = np.random.default_rng(sub_seed(seed, "policy", n_tags, n_groups, int(beta * 1e6)))
    gol = contiguous_groups(n_layers, n_groups)
    w = np.bincount(gol, minlength=n_groups).astype(np.float64)      # layers per group
    p = (np.full(n_tags, 1.0 / n_tags) if tag_probs is None
         else np.asarray(tag_probs, dtype=np.float64))
    kappa = np.array([CRITICALITY[z] for z in range(n_tags)])
    depth = 0.6 + 0.8 * np.arange(n_groups) / max(1, n_groups - 1)  # rises with depth

    # Synthetic task-error sensitivities; V-bar(L) <= V-bar(R) (monotone envelope, Eq. 5).
    v_r = kappa[:, None] * depth[None, :] * rng.uniform(0, 0.03, size=(n_tags, n_groups))
    v_l = v_r * rng.uniform(0, 0.6, size=(n_tags, n_groups))
    # Protection floor (Eq. 6).
    floor = np.where(v_l > TAU_HIGH, HIGH, np.where(v_r > TAU_LOW, LOW, DROP)).astype(np.uint8)
    # Synthetic distortion, D(H) = 0 <= D(L) <= D(R).
    d_r = kappa[:, None] * depth[None, :] * rng.uniform(0.2, 1.0, size=(n_tags, n_groups))
    d_l = d_r * rng.uniform(0.05, 0.5, size=(n_tags, n_groups))
    m = np.array([0.0, LOW_COST_RATIO, 1.0])[None, None, :] * w[None, :, None]
    rho = np.zeros((n_tags, n_groups, 2), dtype=np.float64)
    rho[..., 0] = np.maximum(d_r - d_l, 0.0) / (m[..., 1] - m[..., 0])   # Eq. 7, R -> L
    rho[..., 1] = np.maximum(d_l - 0.0, 0.0) / (m[..., 2] - m[..., 1])   # Eq. 7, L -> H
    rho = rho.astype(np.float32)

    # Greedy path from the floors: take the eligible adjacent upgrade with the
    # largest score; an upgrade that would exceed the budget closes its bucket.
    act = floor.copy()
    closed = np.zeros((n_tags, n_groups), dtype=bool)
    if _expected_cost(act, p, w) <= beta:
        while True:
            best, best_key = None, None
            for z in range(n_tags):
                for c in range(n_groups):
                    a = act[z, c]
                    if a == HIGH or closed[z, c]:
                        continue
                    key = (float(rho[z, c, a]), -z, -c)
                    if best_key is None or key > best_key:
                        best, best_key = (z, c), key
            if best is None:
                break
            z, c = best
            trial = act.copy()
            trial[z, c] += 1
            if _expected_cost(trial, p, w) <= beta + 1e-12:
                act = trial
            else:
                closed[z, c] = True
    pol = PolicyTable(n_tags=n_tags, n_groups=n_groups, n_layers=n_layers, group_of_layer=gol,
                      action=act.astype(np.uint8), floor=floor, rho_up=rho, n_sink=n_sink,
                      beta=beta, tag_probs=p)
    pol.expected_cost = _expected_cost(np.maximum(act, floor), p, w)
    return pol


def floor_cost(pol: PolicyTable, tags) -> np.ndarray:
    """Bytes the floors alone persist for each token, in units of one token at
    RETAIN-HIGH in every layer: sum over groups of (layers of the group) x
    m(floor) / m(HIGH), with m(LOW) / m(HIGH) = 0.28125."""
    w = np.bincount(np.asarray(pol.group_of_layer), minlength=pol.n_groups).astype(np.float64)
    m = np.array([0.0, LOW_COST_RATIO, 1.0])
    per_tag = (m[np.asarray(pol.floor)] * w[None, :]).sum(axis=1) / w.sum()
    return per_tag[np.asarray(tags, dtype=np.int64)]


def with_budget_controller(pol: PolicyTable, traces, n_states: int, critical, beta: float | None = None,
                           quantile: float = 0.5) -> PolicyTable:
    """Adds the online controller's state to a table.

    traces: calibration (tags, states) pairs.  Gamma(s) follows Eq. 9: the
    empirical quantile, over every position u of every trace whose state is s,
    of the floor cost of the positions after u (the protected history still to
    come); it is stored in sixteenths of a full-precision token.  A state that
    never occurs reserves nothing."""
    samples = [[] for _ in range(n_states)]
    for tags, states in traces:
        f = floor_cost(pol, tags)
        future = np.concatenate([np.cumsum(f[::-1])[::-1][1:], [0.0]])   # floor cost after u
        for st in range(n_states):
            sel = np.asarray(states) == st
            if sel.any():
                samples[st].append(future[sel])
    reserve = np.zeros(n_states, dtype=np.uint32)
    for st in range(n_states):
        if samples[st]:
            reserve[st] = int(round(16.0 * float(np.quantile(np.concatenate(samples[st]), quantile))))
    crit = np.zeros(n_states, dtype=np.uint8)
    crit[list(critical)] = 1
    b = pol.beta if beta is None else beta
    out = PolicyTable(**{k: getattr(pol, k) for k in pol.__dataclass_fields__})
    out.n_states, out.beta_q, out.reserve_q, out.crit = n_states, int(round(b * 65536)), reserve, crit
    return out


def uniform_policy(n_tags: int, n_groups: int, n_layers: int, a: int, n_sink: int = 0) -> PolicyTable:
    """Every bucket selects action a, with floor DROP (special-case tables for tests)."""
    return PolicyTable(
        n_tags=n_tags, n_groups=n_groups, n_layers=n_layers,
        group_of_layer=contiguous_groups(n_layers, n_groups),
        action=np.full((n_tags, n_groups), a, dtype=np.uint8),
        floor=np.zeros((n_tags, n_groups), dtype=np.uint8),
        rho_up=np.zeros((n_tags, n_groups, 2), dtype=np.float32), n_sink=n_sink)


def fnv1a32(data: bytes) -> int:
    h = 0x811C9DC5
    for b in data:
        h ^= b
        h = (h * 0x01000193) & 0xFFFFFFFF
    return h


def pack_blob(pol: PolicyTable, version: int | None = None) -> bytes:
    """Version 1 for a static table, 2 when the table carries the controller."""
    if version is None:
        version = 2 if pol.n_states else 1
    gol = np.asarray(pol.group_of_layer, dtype=np.uint8).tobytes()
    act = np.asarray(pol.action, dtype=np.uint8).tobytes()
    flo = np.asarray(pol.floor, dtype=np.uint8).tobytes()
    body = gol + act + flo
    body += b"\0" * ((-len(body)) % 4)
    body += np.asarray(pol.rho_up, dtype="<f4").tobytes()
    if version == 2:
        body += struct.pack("<II", pol.n_states, pol.beta_q)
        body += np.asarray(pol.reserve_q, dtype="<u4").tobytes()
        body += np.asarray(pol.crit, dtype=np.uint8).tobytes()
        body += b"\0" * ((-len(body)) % 4)
    head = struct.pack("<4sHHIIIIII", b"PASK", version, 32, pol.n_tags, pol.n_groups,
                       pol.n_layers, pol.n_sink, pol.recent_window, len(body))
    data = head + body
    return data + struct.pack("<I", fnv1a32(data))
