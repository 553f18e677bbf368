"""Seeded synthetic inputs for decode-instance selection.

This module only *draws* inputs: cluster topology, per-link telemetry, decode
instance state, requests with block-hash runs, and the block-hash sets resident
on each decode instance.  It contains none of the selection method's arithmetic
(no bandwidth derating, no prefix matching, no scoring, no argmin).  Both the
CPU oracle under ``oracle/`` and the HIP library consume exactly the arrays
produced here, so the two sides see byte-identical inputs.

Where the inputs come from in the paper:
  * fat-tree with four locality tiers (same node / same leaf / same pod /
    cross-pod), each with a static bandwidth and base latency -- Sec. III-A;
  * KV bytes per token from Eq. (1); block-level prefix hashes -- Sec. III-B;
  * decode state m_d, q_d, beta_d and the iteration-time line a + b*beta --
    Sec. III-C;
  * the operator's maps tier_map / tier_bandwidth / tier_latency /
    congestion -- Sec. III-E (network cost oracle interface).

The paper drives its simulator with production traces that are not available
here; the workload recipes below (lognormal lengths, Zipf-shared prefixes,
Poisson queues, uniform link utilisation) are synthetic stand-ins whose shapes
follow the configurations listed in ``CONFIGS``.

Block hashes of the shared prefix chains are the splitmix64 output finaliser
(Steele, Lea, Flood, "Fast splittable pseudorandom number generators",
OOPSLA 2014) -- a bijection on 64-bit words -- applied to a distinct
structured counter (domain, prefix id, block index) xor-ed with a per-seed
key, so the same block of the same prefix has the same hash in every request
and every cache, and distinct chain blocks never collide.  Request-private
blocks and decode-private resident blocks are independent uniform 64-bit
draws.  Hash value 0 is reserved as the empty-slot marker of the device
tables and is never produced.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Optional

import numpy as np

GB = 1e9  # bandwidth and memory use decimal gigabytes

_M64 = np.uint64(0xFFFFFFFFFFFFFFFF)

# hash domains (top byte of the counter fed to the finaliser)
_DOM_CHAIN = 1      # shared prefix chain k, block i
_DOM_SYSTEM = 2     # long system prefix k, block i (long-context workload)


def mix64(x: np.ndarray) -> np.ndarray:
    """splitmix64 output finaliser, vectorised over uint64 (wrapping)."""
    z = np.asarray(x, dtype=np.uint64).copy()
    with np.errstate(over="ignore"):
        z ^= z >> np.uint64(30)
        z *= np.uint64(0xBF58476D1CE4E5B9)
        z ^= z >> np.uint64(27)
        z *= np.uint64(0x94D049BB133111EB)
        z ^= z >> np.uint64(31)
    return z


def _seed_key(seed: int) -> np.uint64:
    return mix64(np.array([(seed * 0x9E3779B97F4A7C15 + 0x1234567) & 0xFFFFFFFFFFFFFFFF],
                          dtype=np.uint64))[0]


def block_hash(seed: int, domain: int, owner: np.ndarray, idx: np.ndarray) -> np.ndarray:
    """Distinct 64-bit block hashes for (domain, owner, idx) counters.

    owner < 2**32 and idx < 2**24 keep the counters distinct, so the
    bijective finaliser keeps the hashes distinct.
    """
    owner = np.asarray(owner, dtype=np.uint64)
    idx = np.asarray(idx, dtype=np.uint64)
    ctr = (np.uint64(domain) << np.uint64(56)) | (owner << np.uint64(24)) | idx
    h = mix64(ctr ^ _seed_key(seed))
    h[h == 0] = np.uint64(1)
    return h


def _rng(seed: int, *stream: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, *stream]))


# --------------------------------------------------------------------------
# configurations
# --------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Cluster:
    """Fat-tree shape: GPUs per node, nodes per leaf, leaves per pod, pods.

    GPU g is a prefill GPU iff g % prefill_every == 0 (two prefill and six
    decode GPUs per 8-GPU node, so every tier is reachable from every
    prefill instance).
    """
    gpus_per_node: int
    nodes_per_leaf: int
    leaves_per_pod: int
    pods: int
    prefill_every: int = 4

    @property
    def n_gpus(self) -> int:
        return self.gpus_per_node * self.nodes_per_leaf * self.leaves_per_pod * self.pods

    @property
    def n_nodes(self) -> int:
        return self.n_gpus // self.gpus_per_node

    @property
    def n_leaves(self) -> int:
        return self.n_nodes // self.nodes_per_leaf

    def coords(self):
        g = np.arange(self.n_gpus)
        node = g // self.gpus_per_node
        leaf = node // self.nodes_per_leaf
        pod = leaf // self.leaves_per_pod
        return node, leaf, pod

    def prefill_gpus(self) -> np.ndarray:
        g = np.arange(self.n_gpus)
        return g[g % self.prefill_every == 0]

    def decode_gpus(self) -> np.ndarray:
        g = np.arange(self.n_gpus)
        return g[g % self.prefill_every != 0]


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    cluster: Cluster
    n_requests: int                     # requests per selection call
    kv_bytes_per_token: int             # per prefill/decode GPU pair
    block_tokens: int = 512
    cache_per_decode: int = 4096        # resident block hashes per decode
    tier_bw: tuple = (900 * GB, 50 * GB, 25 * GB, 12.5 * GB)   # bytes/s
    tier_lat: tuple = (2e-6, 5e-6, 10e-6, 20e-6)               # seconds
    util_range: tuple = ((0.0, 0.9),) * 4   # per-tier link utilisation law
    length_law: str = "lognormal"       # or "uniform_long"
    len_median: float = 8000.0
    len_sigma: float = 1.0
    len_clip: tuple = (128, 131072)
    n_prefixes: int = 2000
    zipf_s: float = 1.1
    queue_mean: float = 4.0
    beta_range: tuple = (56, 64)
    beta_max: int = 64
    t_iter_a: float = 0.050
    t_iter_b: float = 0.0
    alpha: float = 1.0
    m_min: int = 1 << 30
    free_mem_gb: tuple = (20, 200)
    # long-context workload (shared long system prefixes)
    system_prefixes: int = 0
    system_share: float = 0.0
    system_blocks: tuple = (64, 128)
    system_resident_p: float = 0.75
    # streaming workload
    n_batches: int = 1
    ar1_rho: float = 0.9
    ar1_sigma: float = 0.05
    # ranking sweep
    n_scenarios: int = 0
    noise_sigmas: tuple = ()

    @property
    def n_prefill(self) -> int:
        return len(self.cluster.prefill_gpus())

    @property
    def n_decode(self) -> int:
        return len(self.cluster.decode_gpus())


KV_LLAMA3_70B = 2 * 80 * 8 * 128 * 2          # Eq. (1): 327,680 B/token
CLUSTER_64 = Cluster(8, 4, 2, 1)                # 64 GPUs, 8 nodes, 2 leaves, 1 pod
CLUSTER_4096 = Cluster(8, 8, 8, 8)              # 4096 GPUs, 512 nodes, 64 leaves, 8 pods

CONFIGS: Dict[str, Config] = {
    # 64-GPU tiny case, one snapshot
    "c0": Config("c0-64gpu-tiny", CLUSTER_64, 4096, KV_LLAMA3_70B),
    # 64 GPUs at TP=4 sizing: 16 batches of 65,536 with host updates in between
    "c1": Config("c1-64gpu-tp4-stream", CLUSTER_64, 65536, KV_LLAMA3_70B // 4, n_batches=16),
    # 4,096-GPU scale, one snapshot of 1,048,576 requests
    "c2": Config("c2-4096gpu-scoring", CLUSTER_4096, 1 << 20, KV_LLAMA3_70B,
                 cache_per_decode=65536),
    # stale-telemetry ranking sweep
    "c3": Config("c3-64gpu-rank-sweep", CLUSTER_64, 16384, KV_LLAMA3_70B,
                 n_scenarios=1024, noise_sigmas=(0.05, 0.1, 0.2, 0.4)),
    # long-context, cache-heavy
    "c4": Config("c4-4096gpu-long-context", CLUSTER_4096, 262144, KV_LLAMA3_70B,
                 cache_per_decode=262144, length_law="uniform_long",
                 util_range=((0.0, 0.9), (0.0, 0.9), (0.0, 0.9), (0.6, 0.95)),
                 system_prefixes=64, system_share=0.8),
}


def scaled(cfg: Config, **kw) -> Config:
    """A copy of ``cfg`` with some fields replaced (smaller test cases)."""
    return dataclasses.replace(cfg, **kw)


# --------------------------------------------------------------------------
# topology and telemetry (the operator's side of the interface)
# --------------------------------------------------------------------------

def pair_tiers(cluster: Cluster) -> np.ndarray:
    """tier_map[p][d] in {0,1,2,3}: same node / leaf / pod / cross-pod."""
    node, leaf, pod = cluster.coords()
    pg, dg = cluster.prefill_gpus(), cluster.decode_gpus()
    t = np.full((len(pg), len(dg)), 3, dtype=np.uint8)
    t[pod[pg][:, None] == pod[dg][None, :]] = 2
    t[leaf[pg][:, None] == leaf[dg][None, :]] = 1
    t[node[pg][:, None] == node[dg][None, :]] = 0
    return t


def draw_links(cfg: Config, seed: int) -> Dict[str, np.ndarray]:
    """Per-link utilisation: u0 per node (intra-node fabric), u1 per node
    (NIC uplink to the leaf), u2 per leaf (leaf-spine uplink), u3 per pod
    (pod-core uplink)."""
    cl = cfg.cluster
    rng = _rng(seed, 11)
    sizes = (cl.n_nodes, cl.n_nodes, cl.n_leaves, cl.pods)
    out = {}
    for t, n in enumerate(sizes):
        lo, hi = cfg.util_range[t]
        out[f"u{t}"] = rng.uniform(lo, hi, n)
    return out


def pair_util(cluster: Cluster, links: Dict[str, np.ndarray]) -> np.ndarray:
    """Collapse per-link utilisation to one congestion value per (p, d) pair.

    The pair's tier selects which links it crosses; its value is the larger
    utilisation of the two tier-level links at either end (for tier 0 both
    ends are the same node).  Constant per-tier utilisation gives back the
    paper's per-tier congestion c_tau exactly.
    """
    node, leaf, pod = cluster.coords()
    pg, dg = cluster.prefill_gpus(), cluster.decode_gpus()
    tiers = pair_tiers(cluster)
    dom = (node, node, leaf, pod)
    u = np.zeros(tiers.shape, dtype=np.float64)
    for t in range(4):
        lk = np.asarray(links[f"u{t}"], dtype=np.float64)
        v = np.maximum(lk[dom[t][pg]][:, None], lk[dom[t][dg]][None, :])
        u = np.where(tiers == t, v, u)
    return u.astype(np.float32)


def params_of(cfg: Config) -> Dict[str, object]:
    return dict(
        tier_bw=np.array(cfg.tier_bw, dtype=np.float64),
        tier_lat=np.array(cfg.tier_lat, dtype=np.float64),
        t_iter_a=float(cfg.t_iter_a), t_iter_b=float(cfg.t_iter_b),
        beta_max=int(cfg.beta_max), alpha=float(cfg.alpha), m_min=int(cfg.m_min),
        kv_bytes_per_token=int(cfg.kv_bytes_per_token), block_tokens=int(cfg.block_tokens),
    )


def make_snapshot(cfg: Config, seed: int = 0, inflight: str = "zero",
                  links: Optional[Dict[str, np.ndarray]] = None) -> Dict[str, object]:
    """One telemetry snapshot plus scheduler-visible decode state.

    inflight: "zero" (no transfers in flight) or "random" (0..16 per tier and
    prefill instance, to exercise the self-contention term).
    """
    cl = cfg.cluster
    P, D = cfg.n_prefill, cfg.n_decode
    if links is None:
        links = draw_links(cfg, seed)
    rng = _rng(seed, 12)
    lo, hi = cfg.free_mem_gb
    snap = dict(params_of(cfg))
    snap.update(
        n_prefill=P, n_decode=D,
        tier_map=np.ascontiguousarray(pair_tiers(cl).reshape(-1)),
        util=np.ascontiguousarray(pair_util(cl, links).reshape(-1)),
        links=links,
        free_mem=rng.integers(int(lo * GB), int(hi * GB), D, endpoint=True).astype(np.uint64),
        queue_depth=rng.poisson(cfg.queue_mean, D).astype(np.uint32),
        batch_size=rng.integers(cfg.beta_range[0], cfg.beta_range[1], D,
                                endpoint=True).astype(np.uint32),
    )
    if inflight == "zero":
        snap["n_inflight"] = np.zeros(4 * P, dtype=np.uint16)
    elif inflight == "random":
        snap["n_inflight"] = _rng(seed, 13).integers(0, 16, 4 * P, endpoint=True).astype(np.uint16)
    else:
        raise ValueError(inflight)
    return snap


# --------------------------------------------------------------------------
# prefix chains, requests and resident caches
# --------------------------------------------------------------------------

def _lengths(cfg: Config, rng: np.random.Generator, n: int) -> np.ndarray:
    if cfg.length_law == "lognormal":
        x = np.exp(math.log(cfg.len_median) + cfg.len_sigma * rng.standard_normal(n))
        return np.clip(np.rint(x), cfg.len_clip[0], cfg.len_clip[1]).astype(np.uint32)
    if cfg.length_law == "uniform_long":
        return rng.integers(65536, 131072, n, endpoint=True).astype(np.uint32)
    raise ValueError(cfg.length_law)


def zipf_weights(n: int, s: float) -> np.ndarray:
    w = np.arange(1, n + 1, dtype=np.float64) ** (-s)
    return w / w.sum()


def prefix_chains(cfg: Config, seed: int) -> Dict[str, np.ndarray]:
    """Lengths (in blocks) of the shared prefixes and their popularity."""
    rng = _rng(seed, 21)
    if cfg.system_prefixes:
        k = cfg.system_prefixes
        lo, hi = cfg.system_blocks
        return dict(domain=_DOM_SYSTEM,
                    blocks=rng.integers(lo, hi, k, endpoint=True).astype(np.int64),
                    weights=np.full(k, 1.0 / k))
    lens = _lengths(cfg, rng, cfg.n_prefixes).astype(np.int64)
    return dict(domain=_DOM_CHAIN, blocks=lens // cfg.block_tokens,
                weights=zipf_weights(cfg.n_prefixes, cfg.zipf_s))


def _ragged_index(counts: np.ndarray):
    """(row, position-within-row) for a ragged array with the given counts."""
    counts = np.asarray(counts, dtype=np.int64)
    total = int(counts.sum())
    rows = np.repeat(np.arange(len(counts)), counts)
    starts = np.cumsum(counts) - counts
    pos = np.arange(total, dtype=np.int64) - np.repeat(starts, counts)
    return rows, pos


def make_requests(cfg: Config, seed: int = 0, n_req: Optional[int] = None,
                  batch: int = 0, chains: Optional[Dict[str, np.ndarray]] = None
                  ) -> Dict[str, np.ndarray]:
    """Requests as CSR: prefill instance, input length, block-hash run.

    A request uses min(n_r, S_k) leading blocks of its shared prefix k, then
    request-private blocks; n_r = floor(len / block_tokens).
    """
    n_req = cfg.n_requests if n_req is None else n_req
    chains = prefix_chains(cfg, seed) if chains is None else chains
    rng = _rng(seed, 31, batch)
    prefill = rng.integers(0, cfg.n_prefill, n_req).astype(np.uint32)
    length = _lengths(cfg, rng, n_req)
    nblk = (length // np.uint32(cfg.block_tokens)).astype(np.int64)
    K = len(chains["blocks"])
    cdf = np.cumsum(chains["weights"])
    k = np.minimum(np.searchsorted(cdf, rng.random(n_req), side="right"), K - 1)
    shared = np.minimum(nblk, chains["blocks"][k])
    if cfg.system_prefixes:
        shared = np.where(rng.random(n_req) < cfg.system_share, shared, 0)
    off = np.zeros(n_req + 1, dtype=np.uint64)
    off[1:] = np.cumsum(nblk)
    # request-private blocks: independent uniform nonzero 64-bit values
    hashes = _rng(seed, 32, batch).integers(1, (1 << 64) - 1, int(off[-1]), dtype=np.uint64,
                                            endpoint=True)
    # shared blocks: leading blocks of the request's prefix chain
    sr, sp = _ragged_index(shared)
    hashes[off[:-1][sr].astype(np.int64) + sp] = block_hash(seed, int(chains["domain"]), k[sr], sp)
    return dict(n_req=n_req, prefill=prefill, len_tokens=length,
                hash_off=off, hashes=hashes.astype(np.uint64), prefix_id=k,
                shared_blocks=shared)


def make_caches(cfg: Config, seed: int = 0, chains: Optional[Dict[str, np.ndarray]] = None,
                n_decode: Optional[int] = None, per_decode: Optional[int] = None
                ) -> Dict[str, np.ndarray]:
    """Resident block-hash sets, one list per decode instance (CSR).

    Each decode holds leading segments (uniform random depth) of some shared
    prefix chains -- chosen with a popularity-weighted inclusion probability
    so that about half the capacity is chain blocks -- and fills the rest
    with decode-private blocks that no request carries.
    """
    D = cfg.n_decode if n_decode is None else n_decode
    cap = cfg.cache_per_decode if per_decode is None else per_decode
    chains = prefix_chains(cfg, seed) if chains is None else chains
    S = chains["blocks"]
    w = chains["weights"]
    K = len(S)
    rng = _rng(seed, 41)
    if cfg.system_prefixes:
        pi = np.full(K, cfg.system_resident_p)
    else:
        target = cap / 2.0
        ed = (S + 1) / 2.0
        lo, hi = 0.0, 1e9
        for _ in range(200):
            g = 0.5 * (lo + hi)
            if (np.minimum(1.0, g * w) * ed).sum() < target:
                lo = g
            else:
                hi = g
        pi = np.minimum(1.0, hi * w)
    off = np.arange(D + 1, dtype=np.uint64) * np.uint64(cap)
    out = np.empty(D * cap, dtype=np.uint64)
    n_chain = np.zeros(D, dtype=np.int64)
    rng_fill = _rng(seed, 42)
    step = max(1, (1 << 24) // max(cap, 1))
    for d0 in range(0, D, step):
        d1 = min(D, d0 + step)
        nd = d1 - d0
        inc = rng.random((nd, K)) < pi[None, :]
        depth = 1 + np.floor(rng.random((nd, K)) * S[None, :]).astype(np.int64)
        depth = np.where(inc & (S[None, :] > 0), np.minimum(depth, S[None, :]), 0)
        # keep the most popular chains when a decode would overflow
        csum = np.cumsum(depth, axis=1)
        depth = np.where(csum <= cap, depth, 0)
        nch = depth.sum(axis=1)
        n_chain[d0:d1] = nch
        dd, kk = np.nonzero(depth)
        cnt = depth[dd, kk]
        rows, pos = _ragged_index(cnt)
        ch = block_hash(seed, int(chains["domain"]), kk[rows], pos)
        # destination: decode-major (np.nonzero is row-major), chain blocks first
        seg_start = np.cumsum(cnt) - cnt
        dec_start = np.cumsum(nch) - nch
        local = seg_start[rows] - dec_start[dd[rows]] + pos
        # decode-private filler: independent uniform nonzero 64-bit values
        block = out[d0 * cap:d1 * cap].reshape(nd, cap)
        block[:] = rng_fill.integers(1, (1 << 64) - 1, (nd, cap), dtype=np.uint64, endpoint=True)
        block[dd[rows], local] = ch
    return dict(n_decode=D, hash_off=off, hashes=out, n_chain=n_chain)


# --------------------------------------------------------------------------
# telemetry dynamics: AR(1) drift (streaming) and noisy scenarios (sweep)
# --------------------------------------------------------------------------

def ar1_links(cfg: Config, seed: int, links0: Dict[str, np.ndarray], n_batches: int):
    """Link utilisation per batch: u_{t+1} = clamp(ubar + rho (u_t - ubar)
    + sigma eps, 0, 0.99), ubar = the initial draw."""
    rng = _rng(seed, 51)
    seq = [dict(links0)]
    cur = {k: np.asarray(v, dtype=np.float64).copy() for k, v in links0.items()}
    for _ in range(1, n_batches):
        nxt = {}
        for key in sorted(cur):
            ubar = np.asarray(links0[key], dtype=np.float64)
            eps = rng.standard_normal(len(ubar))
            nxt[key] = np.clip(ubar + cfg.ar1_rho * (cur[key] - ubar) + cfg.ar1_sigma * eps, 0.0, 0.99)
        cur = nxt
        seq.append(nxt)
    return seq


def scenario_utils(cfg: Config, seed: int, links: Dict[str, np.ndarray],
                   n_scen: Optional[int] = None, sigmas: Optional[tuple] = None):
    """Noisy telemetry scenarios: every link utilisation multiplied by
    exp(sigma * Z) (median 1), capped at 0.99.  Scenarios are split evenly
    across the sigma values.  Returns (util [S][P*D] float32, sigma per
    scenario)."""
    n_scen = cfg.n_scenarios if n_scen is None else n_scen
    sigmas = cfg.noise_sigmas if sigmas is None else sigmas
    rng = _rng(seed, 61)
    per = max(1, n_scen // len(sigmas))
    P, D = cfg.n_prefill, cfg.n_decode
    out = np.empty((n_scen, P * D), dtype=np.float32)
    sig = np.empty(n_scen)
    for s in range(n_scen):
        sg = sigmas[min(s // per, len(sigmas) - 1)]
        sig[s] = sg
        noisy = {}
        for key in sorted(links):
            u = np.asarray(links[key], dtype=np.float64)
            noisy[key] = np.minimum(u * np.exp(sg * rng.standard_normal(len(u))), 0.99)
        out[s] = pair_util(cfg.cluster, noisy).reshape(-1)
    return out, sig


# --------------------------------------------------------------------------
# staged (two-hop) routes
# --------------------------------------------------------------------------

def make_routes(cfg: Config, seed: int) -> Dict[str, np.ndarray]:
    """A staged route p -> staging store -> d for every pair, as maps of the
    snapshot's shape [P*D]: the first hop (prefill to a host-memory or SSD
    store) on a leaf, pod or cross-pod link (tier 1..3), the second (store
    to decode) on a same-node or same-leaf link (tier 0..1), and each hop's
    congestion uniform on [0, 0.9).  Staged routes then beat congested
    direct ones on the slow tiers and lose on the fast ones."""
    rng = _rng(seed, 71)
    n = cfg.n_prefill * cfg.n_decode
    return dict(route_tier1=rng.integers(1, 4, n).astype(np.uint8),
                route_util1=rng.uniform(0.0, 0.9, n).astype(np.float32),
                route_tier2=rng.integers(0, 2, n).astype(np.uint8),
                route_util2=rng.uniform(0.0, 0.9, n).astype(np.float32))


# --------------------------------------------------------------------------
# fat-tree links and KV-transfer flows (the transfer simulation's input)
# --------------------------------------------------------------------------

def fat_tree_links(cfg: Config, links: Dict[str, np.ndarray], spines: int = 4, cores: int = 4):
    """The cluster's links for the flow-level transfer simulation, with
    capacities after background load (bytes/s): per GPU an egress and an
    ingress port on its node's fabric (tier-0 bandwidth, the node's u0) and
    a NIC uplink and downlink (tier 1, the node's u1); per leaf `spines`
    uplinks and downlinks (tier 2, the leaf's u2); per pod `cores` uplinks
    and downlinks (tier 3, the pod's u3).  A flow alone on a path of tier tau
    with no background load moves at exactly B_tau.  Returns (cap [L],
    layout dict of the index bases)."""
    cl = cfg.cluster
    G, NL, NP = cl.n_gpus, cl.n_leaves, cl.pods
    node, leaf, pod = cl.coords()
    bw = np.asarray(cfg.tier_bw, dtype=np.float64)
    u = {t: np.asarray(links[f"u{t}"], dtype=np.float64) for t in range(4)}
    lay = dict(node_out=0, node_in=G, nic_up=2 * G, nic_down=3 * G, leaf_up=4 * G,
               leaf_down=4 * G + NL * spines, pod_up=4 * G + 2 * NL * spines,
               pod_down=4 * G + 2 * NL * spines + NP * cores, spines=spines, cores=cores)
    L = 4 * G + 2 * NL * spines + 2 * NP * cores
    cap = np.empty(L, dtype=np.float64)
    g = np.arange(G)
    cap[lay["node_out"] + g] = bw[0] * (1.0 - u[0][node])
    cap[lay["node_in"] + g] = bw[0] * (1.0 - u[0][node])
    cap[lay["nic_up"] + g] = bw[1] * (1.0 - u[1][node])
    cap[lay["nic_down"] + g] = bw[1] * (1.0 - u[1][node])
    lf = np.repeat(np.arange(NL), spines)
    cap[lay["leaf_up"]:lay["leaf_up"] + NL * spines] = bw[2] * (1.0 - u[2][lf])
    cap[lay["leaf_down"]:lay["leaf_down"] + NL * spines] = bw[2] * (1.0 - u[2][lf])
    pd = np.repeat(np.arange(NP), cores)
    cap[lay["pod_up"]:lay["pod_up"] + NP * cores] = bw[3] * (1.0 - u[3][pd])
    cap[lay["pod_down"]:lay["pod_down"] + NP * cores] = bw[3] * (1.0 - u[3][pd])
    return cap, lay


def transfer_paths(cfg: Config, seed: int, p_inst: np.ndarray, d_inst: np.ndarray, lay: Dict[str, int]):
    """The path of the KV transfer from prefill instance p_inst[i] to decode
    instance d_inst[i]: same node, the two fabric ports; same leaf, the two
    NICs; same pod, NIC, a leaf uplink, the matching downlink of the other
    leaf, NIC; across pods, NIC, a leaf uplink, a pod uplink, the matching
    pod downlink, a leaf downlink, NIC.  ECMP picks the spine and core
    uniformly at random per flow (seeded).  Returns (path_off [N+1] u64,
    path u32)."""
    cl = cfg.cluster
    node, leaf, pod = cl.coords()
    a = cl.prefill_gpus()[np.asarray(p_inst, dtype=np.int64)]
    b = cl.decode_gpus()[np.asarray(d_inst, dtype=np.int64)]
    rng = _rng(seed, 81)
    S, Cc = lay["spines"], lay["cores"]
    n = len(a)
    s1 = rng.integers(0, S, n)
    s2 = rng.integers(0, S, n)
    cc = rng.integers(0, Cc, n)
    tier = np.where(node[a] == node[b], 0, np.where(leaf[a] == leaf[b], 1, np.where(pod[a] == pod[b], 2, 3)))
    plen = np.array([2, 2, 4, 6])[tier]
    off = np.zeros(n + 1, dtype=np.uint64)
    off[1:] = np.cumsum(plen)
    cols = np.full((n, 6), -1, dtype=np.int64)
    t0, t1, t2, t3 = (tier == 0), (tier == 1), (tier == 2), (tier == 3)
    cols[t0, 0] = lay["node_out"] + a[t0]
    cols[t0, 1] = lay["node_in"] + b[t0]
    cols[t1, 0] = lay["nic_up"] + a[t1]
    cols[t1, 1] = lay["nic_down"] + b[t1]
    cols[t2, 0] = lay["nic_up"] + a[t2]
    cols[t2, 1] = lay["leaf_up"] + leaf[a[t2]] * S + s1[t2]
    cols[t2, 2] = lay["leaf_down"] + leaf[b[t2]] * S + s1[t2]
    cols[t2, 3] = lay["nic_down"] + b[t2]
    cols[t3, 0] = lay["nic_up"] + a[t3]
    cols[t3, 1] = lay["leaf_up"] + leaf[a[t3]] * S + s1[t3]
    cols[t3, 2] = lay["pod_up"] + pod[a[t3]] * Cc + cc[t3]
    cols[t3, 3] = lay["pod_down"] + pod[b[t3]] * Cc + cc[t3]
    cols[t3, 4] = lay["leaf_down"] + leaf[b[t3]] * S + s2[t3]
    cols[t3, 5] = lay["nic_down"] + b[t3]
    path = cols[cols >= 0].astype(np.uint32)   # row-major: each flow's links in order
    return off, path


def transfer_starts(seed: int, n: int, window: float = 0.05) -> np.ndarray:
    """Arrival times of n transfers (the moments their prefills complete),
    uniform over a window of `window` seconds."""
    return np.sort(_rng(seed, 91).uniform(0.0, window, n))
