"""Seeded synthetic inputs standing in for the paper's workloads.

The paper evaluates on a 5-node "student" network with textbook CPTs
(Sec. 5.1) and on a 334-variable network learned from the DLM assessment data
(Sec. 5.2, Sec. 6).  Neither the CPTs nor the data are available, so every
workload here is synthetic and seeded:

=====  ========================================================================
cfg    structure / values
=====  ========================================================================
1      student network (I, D, S, G, L; G ternary), rows ~ Dir(1), 2,000 columns,
       50% of entries hidden i.i.d., m = 1
2      same network, 100,000 columns, 50% hidden, m = 10
3      100-node random DAG, 0-3 parents among earlier nodes, K in {2,3,4},
       rows ~ Dir(0.5), 1,000,000 columns, 30% hidden, m = 5
4      30 latent binary concepts (never observed) + 300 binary items with 1-2
       concept parents, rows ~ Dir(1), 4,000 columns, 90% of item entries
       hidden, m = 20
5      1000-node random DAG, 0-4 parents, K in {2..8}, rows ~ Dir(0.5),
       2,000,000 columns in 250,000-column minibatches, 40% hidden, m = 10
=====  ========================================================================

Data are drawn by forward (ancestral) sampling from the true CPTs and entries
are hidden at random (Sec. 5.1).  The sampler starts from CPT rows ~ Dir(1)
(the paper initialises randomly, Sec. 5.2) and from uniform latent states;
observed entries are copied into every SAME replica.

Structure and CPT values come from numpy generators seeded with
``SeedSequence([151106416, cfg, purpose])``; the column-sized arrays come from
torch generators seeded from the same sequences, on the device that will hold
them (so a CPU-made and a GPU-made workload of the same config hold different
draws; both sides of every comparison receive the same arrays).
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence

import numpy as np
import torch

BASE_SEED = 151106416

# purposes for the seed sequences
_P_DAG, _P_TRUE, _P_DATA, _P_MASK, _P_INIT_THETA, _P_INIT_STATES, _P_HOLDOUT = range(7)

CONFIGS = {
    1: dict(name="student-2k", graph="student", n_cols=2_000, hidden=0.5, m=1, sweeps=20,
            alpha_true=1.0, nb=None),
    2: dict(name="student-100k", graph="student", n_cols=100_000, hidden=0.5, m=10, sweeps=50,
            alpha_true=1.0, nb=None),
    3: dict(name="random100-1m", graph=("random", 100, 3, 2, 4), n_cols=1_000_000, hidden=0.3,
            m=5, sweeps=20, alpha_true=0.5, nb=None),
    4: dict(name="concepts30-items300-4k", graph=("two_layer", 30, 300), n_cols=4_000,
            hidden=0.9, m=20, sweeps=200, alpha_true=1.0, nb=None),
    5: dict(name="random1000-2m", graph=("random", 1000, 4, 2, 8), n_cols=2_000_000,
            hidden=0.4, m=10, sweeps=10, alpha_true=0.5, nb=250_000),
}

PRIOR_ALPHA = 1.0


def sampler_seed(cfg_id: int) -> int:
    """The 64-bit key of the sampler's Philox stream for a config."""
    return BASE_SEED + int(cfg_id)


def _rng(cfg_id: int, purpose: int, extra: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([BASE_SEED, cfg_id, purpose, extra]))


def _torch_gen(cfg_id: int, purpose: int, extra: int, device) -> torch.Generator:
    seed = int(np.random.SeedSequence([BASE_SEED, cfg_id, purpose, extra]).generate_state(
        1, dtype=np.uint64)[0] & ((1 << 63) - 1))
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


@dataclasses.dataclass
class Network:
    """A discrete Bayesian network: ordered parent lists and cardinalities."""

    name: str
    parents: List[List[int]]
    card: np.ndarray

    @property
    def n(self) -> int:
        return len(self.parents)

    def csr(self):
        pptr = np.zeros(self.n + 1, dtype=np.int32)
        for i, ps in enumerate(self.parents):
            pptr[i + 1] = pptr[i] + len(ps)
        pidx = np.array([p for ps in self.parents for p in ps], dtype=np.int32)
        return pptr, pidx, np.ascontiguousarray(self.card, dtype=np.int32)


def cpt_layout(net: Network):
    """Offsets [n+1], rows [n] and per-node parent strides (last parent fastest)."""
    off = np.zeros(net.n + 1, dtype=np.int64)
    rows = np.zeros(net.n, dtype=np.int64)
    strides = []
    for i, ps in enumerate(net.parents):
        st = [0] * len(ps)
        r = 1
        for j in range(len(ps) - 1, -1, -1):
            st[j] = r
            r *= int(net.card[ps[j]])
        strides.append(st)
        rows[i] = r
        off[i + 1] = off[i] + r * int(net.card[i])
    return off, rows, strides


def koller() -> Network:
    """The 5-node student network of Sec. 5.1: X0=I, X1=D, X2=S, X3=G, X4=L with
    edges I->S, I->G, D->G, G->L; G ternary, the rest binary."""
    return Network("student", [[], [], [0], [0, 1], [3]], np.array([2, 2, 2, 3, 2], np.int32))


def _random_dag(cfg_id, n, max_par, kmin, kmax) -> Network:
    rng = _rng(cfg_id, _P_DAG)
    parents = []
    card = rng.integers(kmin, kmax + 1, size=n).astype(np.int32)
    for i in range(n):
        k = int(rng.integers(0, max_par + 1))
        k = min(k, i)
        ps = sorted(int(p) for p in rng.choice(i, size=k, replace=False)) if k else []
        parents.append(ps)
    return Network("random%d" % n, parents, card)


def _two_layer(cfg_id, n_concepts, n_items) -> Network:
    rng = _rng(cfg_id, _P_DAG)
    parents = [[] for _ in range(n_concepts)]
    for _ in range(n_items):
        k = int(rng.integers(1, 3))
        parents.append(sorted(int(p) for p in rng.choice(n_concepts, size=k, replace=False)))
    card = np.full(n_concepts + n_items, 2, dtype=np.int32)
    return Network("two_layer", parents, card)


def make_network(cfg_id: int) -> Network:
    g = CONFIGS[cfg_id]["graph"]
    if g == "student":
        return koller()
    if g[0] == "random":
        return _random_dag(cfg_id, g[1], g[2], g[3], g[4])
    if g[0] == "two_layer":
        return _two_layer(cfg_id, g[1], g[2])
    raise ValueError(g)


def dirichlet_rows(net: Network, alpha: float, rng: np.random.Generator) -> np.ndarray:
    off, rows, _ = cpt_layout(net)
    out = np.zeros(int(off[-1]), dtype=np.float64)
    for i in range(net.n):
        K = int(net.card[i])
        out[off[i]:off[i + 1]] = rng.dirichlet(np.full(K, alpha), size=int(rows[i])).reshape(-1)
    return out


def topo_order(net: Network) -> List[int]:
    indeg = [len(p) for p in net.parents]
    children = [[] for _ in range(net.n)]
    for h, ps in enumerate(net.parents):
        for p in ps:
            children[p].append(h)
    order, ready = [], sorted(i for i in range(net.n) if indeg[i] == 0)
    while ready:
        v = ready.pop(0)
        order.append(v)
        for h in children[v]:
            indeg[h] -= 1
            if indeg[h] == 0:
                ready.append(h)
                ready.sort()
    return order


def forward_sample(net: Network, theta: np.ndarray, n_cols: int, gen: torch.Generator,
                   device, dtype=torch.int8) -> torch.Tensor:
    """Ancestral sampling of n_cols complete cases: x[n][n_cols] (Sec. 5.1)."""
    off, rows, strides = cpt_layout(net)
    x = torch.zeros((net.n, n_cols), dtype=dtype, device=device)
    th = torch.as_tensor(theta, dtype=torch.float64, device=device)
    for i in topo_order(net):
        K = int(net.card[i])
        row = torch.zeros(n_cols, dtype=torch.int64, device=device)
        for p, s in zip(net.parents[i], strides[i]):
            row += x[p].to(torch.int64) * s
        cdf = torch.cumsum(th[off[i]:off[i + 1]].view(int(rows[i]), K), dim=1)
        u = torch.rand(n_cols, generator=gen, device=device, dtype=torch.float64)
        xi = (u[:, None] >= cdf[row, : K - 1]).sum(dim=1)
        x[i] = xi.clamp_(max=K - 1).to(dtype)
    return x


@dataclasses.dataclass
class Workload:
    cfg_id: int
    name: str
    net: Network
    true_theta: np.ndarray          # fp64 [cpt_total], generating CPTs
    init_theta: np.ndarray          # fp32 [cpt_total], sampler's starting CPTs
    n_cols: int                     # N, total columns
    nb: int                         # columns per minibatch
    M: int                          # number of minibatches
    ld: int                         # leading dimension of a minibatch row
    m: int                          # SAME replicas
    hidden: float
    sweeps: int
    alpha: float                    # Dirichlet prior of the resample
    seed: int                       # Philox key of the sampler
    states: List[torch.Tensor]      # per minibatch [n][m][ld] int8/int16
    obs: List[torch.Tensor]         # per minibatch [n][ld] uint8 (1 = observed)
    data: Optional[List[torch.Tensor]] = None  # per minibatch [n][nb] complete data

    def mb_cols(self, b: int) -> int:
        return min(self.nb, self.n_cols - b * self.nb)


def make_workload(cfg_id: int, n_cols: Optional[int] = None, m: Optional[int] = None,
                  nb: Optional[int] = None, device="cpu", ld_align: int = 1024,
                  keep_data: bool = False, minibatches: Optional[Sequence[int]] = None,
                  hidden: Optional[float] = None) -> Workload:
    """Generate a config's inputs (optionally at a reduced size) on ``device``.

    ``minibatches`` restricts generation to a subset of minibatch indices (the
    others are left as empty tensors); minibatch b always holds the same draws.
    """
    spec = CONFIGS[cfg_id]
    net = make_network(cfg_id)
    N = int(n_cols if n_cols is not None else spec["n_cols"])
    m = int(m if m is not None else spec["m"])
    nb_spec = spec["nb"] if spec["nb"] is not None else N
    nb = int(nb if nb is not None else min(nb_spec, N))
    M = (N + nb - 1) // nb
    ld = ((nb + ld_align - 1) // ld_align) * ld_align
    hid = float(hidden if hidden is not None else spec["hidden"])
    true_theta = dirichlet_rows(net, spec["alpha_true"], _rng(cfg_id, _P_TRUE))
    init_theta = dirichlet_rows(net, 1.0, _rng(cfg_id, _P_INIT_THETA)).astype(np.float32)
    sdt = torch.int8 if int(net.card.max()) <= 127 else torch.int16
    two_layer = isinstance(spec["graph"], tuple) and spec["graph"][0] == "two_layer"
    n_concepts = spec["graph"][1] if two_layer else 0
    states, obs, datas = [], [], []
    todo = set(range(M)) if minibatches is None else set(minibatches)
    for b in range(M):
        if b not in todo:
            states.append(torch.empty(0, dtype=sdt, device=device))
            obs.append(torch.empty(0, dtype=torch.uint8, device=device))
            datas.append(None)
            continue
        cols = min(nb, N - b * nb)
        g_data = _torch_gen(cfg_id, _P_DATA, b, device)
        g_mask = _torch_gen(cfg_id, _P_MASK, b, device)
        g_init = _torch_gen(cfg_id, _P_INIT_STATES, b, device)
        x = forward_sample(net, true_theta, cols, g_data, device, sdt)
        st = torch.zeros((net.n, m, ld), dtype=sdt, device=device)
        ob = torch.ones((net.n, ld), dtype=torch.uint8, device=device)
        for i in range(net.n):
            u = torch.rand(cols, generator=g_mask, device=device)
            if two_layer and i < n_concepts:
                o = torch.zeros(cols, dtype=torch.bool, device=device)
            else:
                o = u >= hid
            ob[i, :cols] = o.to(torch.uint8)
            lat = torch.randint(0, int(net.card[i]), (m, cols), generator=g_init, device=device,
                                dtype=torch.int64).to(sdt)
            st[i, :, :cols] = torch.where(o[None, :], x[i][None, :], lat)
        states.append(st)
        obs.append(ob)
        datas.append(x if keep_data else None)
    return Workload(cfg_id=cfg_id, name=spec["name"], net=net, true_theta=true_theta,
                    init_theta=init_theta, n_cols=N, nb=nb, M=M, ld=ld, m=m, hidden=hid,
                    sweeps=spec["sweeps"], alpha=PRIOR_ALPHA, seed=sampler_seed(cfg_id),
                    states=states, obs=obs, data=datas if keep_data else None)


def holdout(w: "Workload", b: int = 0, frac: float = 0.2):
    """Held-out split of minibatch b (Sec. 6: 80% of the known entries train,
    the rest test): each known entry of the real columns is a test entry with
    probability frac (numpy generator seeded for purpose 6).  Returns
    (obs_train, target): obs_train is obs with the test entries hidden;
    target [n][ld] holds the true value of every test entry and -1 elsewhere
    (numpy arrays, the states' dtype for target)."""
    obs = w.obs[b].cpu().numpy()
    st = w.states[b].cpu().numpy()
    n_cols = w.mb_cols(b)
    rng = _rng(w.cfg_id, _P_HOLDOUT, b)
    pick = (rng.random(obs.shape) < frac) & (obs == 1)
    pick[:, n_cols:] = False
    obs_train = obs.copy()
    obs_train[pick] = 0
    target = np.full(obs.shape, -1, dtype=st.dtype)
    target[pick] = st[:, 0, :][pick]
    return obs_train, target
