"""Seeded synthetic workloads for one GPU's share of the EP MoE block.

This module only *generates inputs*: routing ids and weights, the placement of
logical experts on local slots, the per-batch split plan, activations and
expert weights (bf16 bits, or OCP e4m3 bytes with fp32 block scales).  It holds
none of the method's arithmetic and is used alike by the tests (to feed both
the oracle and the HIP library) and by the benchmark.

Recipe (the paper's synthetic arm routes with Zipf popularity, Sec. 2.4 and
Sec. 3.2):

* popularity p_r proportional to (r+1)^-s over ranks r = 0..E-1; expert id = rank;
* logits z[t,e] = sigma * N(0,1) + ln p_e, sigma = 1.5; top-K by descending z
  (ties to the lower id); routing weights = softmax over the K chosen logits,
  evaluated in fp64 and stored fp32;
* placement "local-hot": every slot's expert is homed here, the hottest
  experts get extra local replica slots; placement "remote-hot": this GPU is
  GPU 7 of an EP8 group whose experts are homed round-robin (id mod 8), so
  it homes the coldest residue class, and its extra slots hold replicas of
  the hottest experts (ids 0, 1, ...) homed on GPUs 0, 1, ...;
* plans: uniform (weight 1 per replica), replica-minimising (all weight on the
  home replica), token-balancing (a two-bin water-fill per replicated expert
  against the EP8 per-GPU loads of the same batch);
* activations x ~ N(0,1); expert weights ~ N(0, 0.02); replica slots hold
  copies of their expert's weights;
* bf16 = round-to-nearest-even of the fp32 sample; fp8 = e4m3 (RNE,
  saturating at 448) with fp32 scales amax/448: 1 x 128 blocks along the
  hidden dimension for x, 128 x 128 blocks for weights; fp8mx = the same
  with every scale rounded up to a power of two (UE8M0).

Independent streams: numpy SeedSequence([seed, stream]) with stream 0 for
logits, 1 for activations and 2 + e for the weights of logical expert e.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

SIGMA = 1.5
EP_GROUP = 8


# --------------------------------------------------------------------------
# number encodings (input preparation only)
# --------------------------------------------------------------------------

def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest even (finite
    inputs: the rounding increment cannot carry out of 32 bits)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = (u >> 16) & np.uint32(1)
    r += np.uint32(0x7FFF)
    r += u
    r >>= 16
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32)


def to_e4m3_codes(v: np.ndarray) -> np.ndarray:
    """fp32 values -> OCP e4m3 codes, round to nearest even, magnitudes
    saturated at 448.  Normal range: round the fp32 significand to 3 bits
    (the carry runs into the exponent field); subnormal range (|v| < 2^-6):
    the nearest multiple of 2^-9, ties to even."""
    f = np.ascontiguousarray(v, dtype=np.float32)
    a = np.minimum(np.abs(f), np.float32(448.0))
    ab = a.view(np.uint32)
    r = (ab >> 20) & np.uint32(1)
    r += np.uint32(0x7FFFF)
    r += ab
    r >>= 20
    normal = a >= np.float32(2.0 ** -6)
    # code = rounded (exponent, 3-bit mantissa) rebased from bias 127 to bias 7
    code = np.where(normal, r.view(np.int32) - np.int32((127 - 7) << 3),
                    np.rint(a * np.float32(512.0)).astype(np.int32))
    sign = (f.view(np.uint32) >> 24).astype(np.uint8) & np.uint8(0x80)
    return code.astype(np.uint8) | sign


def _pow2_ceil(v: np.ndarray) -> np.ndarray:
    """Smallest power of two >= v (fp32, v > 0): UE8M0 scales."""
    m, e = np.frexp(v.astype(np.float64))
    return np.ldexp(1.0, np.where(m == 0.5, e - 1, e)).astype(np.float32)


def quant_rows_1x128(x: np.ndarray, pow2: bool = False):
    """[R, C] fp32 -> (e4m3 codes [R, C], fp32 scales [R, C/128]); pow2:
    scales rounded up to powers of two."""
    R, C = x.shape
    xb = x.reshape(R, C // 128, 128).astype(np.float32)
    amax = np.abs(xb).max(axis=2)
    sc = np.where(amax > 0, amax / np.float32(448.0), np.float32(1.0)).astype(np.float32)
    if pow2:
        sc = _pow2_ceil(sc)
    q = to_e4m3_codes(xb / sc[:, :, None])
    return q.reshape(R, C), sc


def quant_blocks_128x128(w: np.ndarray, pow2: bool = False):
    """[R, C] fp32 -> (e4m3 codes [R, C], fp32 scales [R/128, C/128]); pow2:
    scales rounded up to powers of two."""
    R, C = w.shape
    wb = w.reshape(R // 128, 128, C // 128, 128).astype(np.float32)
    amax = np.abs(wb).max(axis=3).max(axis=1)
    sc = np.where(amax > 0, amax / np.float32(448.0), np.float32(1.0)).astype(np.float32)
    if pow2:
        sc = _pow2_ceil(sc)
    q = to_e4m3_codes(wb / sc[:, None, :, None])
    return q.reshape(R, C), sc


# --------------------------------------------------------------------------
# routing, placement, plans
# --------------------------------------------------------------------------

def zipf_popularity(E: int, s: float) -> np.ndarray:
    p = (np.arange(E, dtype=np.float64) + 1.0) ** (-s)
    return p / p.sum()


def routing(T: int, K: int, E: int, s: float, seed: int, sigma: float = SIGMA):
    """Top-K ids [T,K] int32 and softmax weights [T,K] fp32."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0])))
    z = sigma * rng.standard_normal((T, E)) + np.log(zipf_popularity(E, s))[None, :]
    # descending z, ties to the lower id: stable sort of -z
    order = np.argsort(-z, axis=1, kind="stable")[:, :K]
    zk = np.take_along_axis(z, order, axis=1)
    ez = np.exp(zk - zk.max(axis=1, keepdims=True))
    w = ez / ez.sum(axis=1, keepdims=True)
    return order.astype(np.int32), w.astype(np.float32)


@dataclass
class Placement:
    slot_expert: np.ndarray  # [S] int32
    home: np.ndarray  # [E] int32: home GPU of each expert in the EP group
    replica_gpus: list = field(default_factory=list)  # [E] list of GPUs holding a replica (incl. home)
    gpu: int = 0  # index of this GPU in the EP group


def placement_local_hot(E: int, n_local: int, n_extra: int) -> Placement:
    """All slots homed here: experts 0..n_local-1, plus second slots for the
    n_extra hottest (ids 0..n_extra-1), appended after the home slots."""
    se = list(range(n_local)) + list(range(n_extra))
    home = np.zeros(E, np.int32)
    reps = [[0] * (2 if e < n_extra else 1) for e in range(E)]
    return Placement(np.array(se, np.int32), home, reps)


def placement_local_hot_strided(E: int, n_local: int, n_extra: int, stride: int = EP_GROUP) -> Placement:
    """Home experts id = 0 mod stride (this GPU of an EP group); the extra
    slots copy the n_extra hottest *local* experts."""
    home_ids = [e for e in range(E) if e % stride == 0][:n_local]
    se = home_ids + home_ids[:n_extra]
    home = (np.arange(E) % stride).astype(np.int32)
    reps = [[int(home[e])] for e in range(E)]
    for e in home_ids[:n_extra]:
        reps[e].append(0)
    return Placement(np.array(se, np.int32), home, reps)


def placement_remote_hot(E: int, n_extra: int, stride: int = EP_GROUP) -> Placement:
    """GPU g = stride-1 of an EP group homes experts id = g mod stride; its
    n_extra extra slots hold replicas of the hottest experts homed elsewhere
    (ids 0..n_extra-1), each shared with its home GPU."""
    g = stride - 1
    home_ids = [e for e in range(E) if e % stride == g]
    extra = [e for e in range(E) if e % stride != g][:n_extra]
    se = home_ids + extra
    home = (np.arange(E) % stride).astype(np.int32)
    reps = [[int(home[e])] for e in range(E)]
    for e in extra:
        reps[e].append(g)
    return Placement(np.array(se, np.int32), home, reps, gpu=g)


@dataclass
class Plan:
    slot_weight: np.ndarray  # [S] uint32
    remote_weight: np.ndarray  # [E] uint32
    remote_replicas: np.ndarray  # [E] int32
    name: str = ""


def _remote_replicas(pl: Placement, E: int) -> np.ndarray:
    rr = np.zeros(E, np.int32)
    for e in range(E):
        rr[e] = sum(1 for g in pl.replica_gpus[e] if g != pl.gpu)
    return rr


def plan_uniform(pl: Placement, E: int) -> Plan:
    """Equal share per replica (the EPLB default split)."""
    S = len(pl.slot_expert)
    rr = _remote_replicas(pl, E)
    return Plan(np.ones(S, np.uint32), rr.astype(np.uint32), rr, "uniform")


def plan_replica_min(pl: Placement, E: int) -> Plan:
    """Whole expert on its home replica: weight 1 on the first local slot of a
    locally-homed expert, all weight remote for experts homed elsewhere."""
    S = len(pl.slot_expert)
    rr = _remote_replicas(pl, E)
    sw = np.zeros(S, np.uint32)
    rw = np.zeros(E, np.uint32)
    seen = set()
    for s, e in enumerate(pl.slot_expert.tolist()):
        if pl.home[e] == pl.gpu and e not in seen:
            sw[s] = 1
            seen.add(e)
    for e in range(E):
        if pl.home[e] != pl.gpu:
            rw[e] = 1
    return Plan(sw, rw, rr, "replica_min")


def plan_token_balancing(pl: Placement, E: int, topk_ids: np.ndarray, T_valid: int) -> Plan:
    """Two-bin water-fill per replicated expert: the local share x* moves this
    GPU's token load towards the home GPU's (EP8 loads of the same batch,
    replicated experts processed in descending count).  Weights are exact
    integers (x*, n_e - x*)."""
    S = len(pl.slot_expert)
    rr = _remote_replicas(pl, E)
    ids = topk_ids[:T_valid].reshape(-1)
    n = np.bincount(ids[ids >= 0], minlength=E).astype(np.int64)
    load = np.zeros(EP_GROUP, np.int64)
    replicated = [e for e in range(E) if len(pl.replica_gpus[e]) > 1]
    for e in range(E):
        if e not in replicated:
            load[pl.home[e]] += n[e]
    sw = np.zeros(S, np.uint32)
    rw = np.zeros(E, np.uint32)
    slot_of = {}
    for s, e in enumerate(pl.slot_expert.tolist()):
        slot_of.setdefault(e, []).append(s)
    me = pl.gpu
    for e in sorted(replicated, key=lambda e: (-n[e], e)):
        other = [g for g in pl.replica_gpus[e] if g != me]
        if not other:
            # all replicas local: split evenly
            for s in slot_of[e]:
                sw[s] = 1
            load[me] += n[e]
            continue
        g1 = other[0]
        x = int(np.clip((load[g1] + n[e] - load[me]) // 2, 0, n[e]))
        load[me] += x
        load[g1] += n[e] - x
        loc = slot_of.get(e, [])
        if loc:
            sw[loc[0]] = np.uint32(x)
        rw[e] = np.uint32(n[e] - x)
    for e in range(E):
        if e not in replicated:
            for s in slot_of.get(e, []):
                sw[s] = 1
            if pl.home[e] != me:
                rw[e] = 1
    return Plan(sw, rw, rr, "token_balancing")


# --------------------------------------------------------------------------
# activations and weights
# --------------------------------------------------------------------------

def _rng(seed, stream):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream])))


def activations(T: int, H: int, seed: int, dtype: str):
    x = _rng(seed, 1).standard_normal((T, H), dtype=np.float32)
    if dtype == "bf16":
        return to_bf16_bits(x), None
    return quant_rows_1x128(x, pow2=dtype == "fp8mx")


def expert_weights(e: int, H: int, I: int, seed: int, dtype: str, std: float = 0.02):
    """Weights of logical expert e: w13 [2I, H] (gate rows, then up rows) and
    w2 [H, I], plus 128 x 128 block scales for fp8."""
    r = _rng(seed, 2 + e)
    w13 = r.standard_normal((2 * I, H), dtype=np.float32) * np.float32(std)
    w2 = r.standard_normal((H, I), dtype=np.float32) * np.float32(std)
    if dtype == "bf16":
        return to_bf16_bits(w13), None, to_bf16_bits(w2), None
    q13, s13 = quant_blocks_128x128(w13, pow2=dtype == "fp8mx")
    q2, s2 = quant_blocks_128x128(w2, pow2=dtype == "fp8mx")
    return q13, s13, q2, s2


def slot_weights(slot_expert: np.ndarray, H: int, I: int, seed: int, dtype: str):
    """Per-slot weight tensors [S, 2I, H], [S, H, I] (+ scales), each replica
    slot holding its own copy of the expert's weights."""
    S = len(slot_expert)
    edt = np.uint16 if dtype == "bf16" else np.uint8
    w13 = np.empty((S, 2 * I, H), edt)
    w2 = np.empty((S, H, I), edt)
    s13 = s2 = None
    if dtype != "bf16":
        s13 = np.empty((S, 2 * I // 128, H // 128), np.float32)
        s2 = np.empty((S, H // 128, I // 128), np.float32)
    from concurrent.futures import ThreadPoolExecutor

    uniq = sorted(set(slot_expert.tolist()))
    with ThreadPoolExecutor(max_workers=min(8, len(uniq))) as ex:
        cache = dict(zip(uniq, ex.map(lambda e: expert_weights(e, H, I, seed, dtype), uniq)))
    for s, e in enumerate(slot_expert.tolist()):
        a, sa, b, sb = cache[e]
        w13[s] = a
        w2[s] = b
        if dtype != "bf16":
            s13[s] = sa
            s2[s] = sb
    return w13, s13, w2, s2


# --------------------------------------------------------------------------
# named workloads
# --------------------------------------------------------------------------

@dataclass
class Workload:
    name: str
    dtype: str
    T: int
    T_valid: int
    K: int
    E: int
    H: int
    I: int
    zipf: float
    placement: Placement
    plans: dict
    topk_ids: np.ndarray
    topk_w: np.ndarray
    seed: int

    @property
    def S(self):
        return len(self.placement.slot_expert)


WORKLOADS = {
    # name: (dtype, T, K, E, H, I, zipf, placement kind, extras, plans)
    "tiny": ("bf16", 96, 2, 6, 256, 512, 1.2, ("local_hot", 6, 2), ("uniform",)),
    "tiny_fp8": ("fp8", 96, 2, 6, 256, 512, 1.2, ("local_hot", 6, 2), ("uniform",)),
    "qwen3_decode_bf16": ("bf16", 512, 8, 128, 4096, 1536, 1.0, ("remote_hot", 2), ("token_balancing",)),
    "qwen3_decode_fp8": ("fp8", 1024, 8, 128, 4096, 1536, 1.2, ("local_hot_strided", 16, 2),
                         ("uniform", "replica_min")),
    "dsv3_decode_fp8": ("fp8", 256, 8, 256, 7168, 2048, 0.8, ("remote_hot", 4), ("uniform",)),
    "qwen3_prefill_bf16": ("bf16", 8192, 8, 128, 4096, 1536, 1.0, ("remote_hot", 2), ("uniform",)),
    "qwen3_prefill_fp8": ("fp8", 8192, 8, 128, 4096, 1536, 1.0, ("remote_hot", 2), ("uniform",)),
    # fp8 with power-of-two (UE8M0) scales
    "tiny_fp8mx": ("fp8mx", 96, 2, 6, 256, 512, 1.2, ("local_hot", 6, 2), ("uniform",)),
    "qwen3_decode_fp8mx": ("fp8mx", 1024, 8, 128, 4096, 1536, 1.2, ("local_hot_strided", 16, 2), ("uniform",)),
    "qwen3_prefill_fp8mx": ("fp8mx", 8192, 8, 128, 4096, 1536, 1.0, ("remote_hot", 2), ("uniform",)),
}


def make_workload(name: str, seed: int = 0, T: int | None = None) -> Workload:
    """Routing, placement and plans of a named workload (weights and
    activations are generated separately, they are large)."""
    dtype, T0, K, E, H, I, s, pk, plans = WORKLOADS[name]
    T = T0 if T is None else T
    ids, w = routing(T, K, E, s, seed)
    if pk[0] == "local_hot":
        pl = placement_local_hot(E, pk[1], pk[2])
    elif pk[0] == "local_hot_strided":
        pl = placement_local_hot_strided(E, pk[1], pk[2])
    else:
        pl = placement_remote_hot(E, pk[1])
    P = {}
    for p in plans:
        if p == "uniform":
            P[p] = plan_uniform(pl, E)
        elif p == "replica_min":
            P[p] = plan_replica_min(pl, E)
        else:
            P[p] = plan_token_balancing(pl, E, ids, T)
    return Workload(name, dtype, T, T, K, E, H, I, s, pl, P, ids, w, seed)


def describe(name: str, plan: str | None = None) -> str:
    """One-line description of a named workload."""
    dtype, T, K, E, H, I, s, pk, plans = WORKLOADS[name]
    S = {"local_hot": lambda: pk[1] + pk[2], "local_hot_strided": lambda: pk[1] + pk[2],
         "remote_hot": lambda: E // EP_GROUP + pk[1]}[pk[0]]()
    return (f"{S} local slots ({pk[0]} placement), H {H}, I {I}, {dtype}, {T} tokens, top-{K} of {E} experts, "
            f"Zipf({s}) popularity, Gaussian logits sigma {SIGMA}, plan {plan or plans[0]}")
