"""Seeded synthetic inputs for the RheoSampling hot path.

This module is the only code the oracle and the HIP path both consume.  It
defines the workloads (shapes, dtypes, temperatures) and generates draft /
target logit rows; it holds none of the method's arithmetic.

The paper's draft and target models (EAGLE-3 heads on Llama-3.1-8B, Vicuna-13B,
DeepSeek-R1-Distill-Llama-8B; Sec. 5.1) and its six datasets are not
available here, so every logit row is a deterministic function of the key of
the tree node it belongs to (the node's path key: the prefix key extended
token by token).  The same prefix therefore always sees the same logits.

Row recipes (all fp32 arithmetic, one torch op per rounding, so CPU and GPU
produce bit-identical rows; bf16 rows are the round-to-nearest-even of the
fp32 row):
  gauss   l_v = 2 * N_v                      (i.i.d. per node and token)
  zipf    l_v = -s * ln(1 + pi(v)) + sigma * N_v   with pi a keyed affine
          permutation of the vocabulary (a Zipf(s) log-prior over a seeded
          token order) and s = 1.1
  zipf_t3 as zipf with Student-t(3) noise; 5% of nodes get +12 on one keyed
          token (near one-hot peaks)
  flat    all logits 0 (uniform distributions; every comparison a tie)
  quantum > 0 rounds every logit to a multiple of it (massive ties)
  near_ties > 0 shifts the row's maximum to 0.125 and puts the next fp32
          values below it on low token ids (distinct logits whose integer
          weights coincide)
  mask > 0 sets each token to -inf with probability `mask` (a keyed 16-bit
          hash of (node key, token) below mask * 2^16): a masked vocabulary
  mask_tail > 0 sets the last mask_tail token ids of every row to -inf (a
          padded vocabulary)
  target  = draft row of the same node + sigma_t * N'_v (an independent
          noise stream of the same node key), rounded like the draft; a
          masked draft token stays -inf, and mask_target > 0 masks a further
          keyed fraction of the target's tokens (tokens the draft proposes
          and the target forbids)
Noise variates come from 65536-entry quantile tables indexed by a 16-bit
hash of (node key, token): a discretised N(0,1) or t(3).
"""

from dataclasses import dataclass, field
import math

import numpy as np
import torch

M32 = 0xFFFFFFFF
M64 = (1 << 64) - 1
GOLD = 0x9E3779B97F4A7C15


def splitmix64(x):
    """SplitMix64 finaliser (Steele, Lea, Flood, OOPSLA'14)."""
    x = (x + GOLD) & M64
    z = x
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def child_key(key, token):
    """Path key of the child reached from ``key`` by ``token``."""
    return splitmix64(key ^ (((token + 1) * GOLD) & M64))


@dataclass
class Workload:
    name: str
    B: int
    V: int
    K: int
    m: int
    depth: int
    R: int
    T: float
    dtype: str                  # "f32" or "bf16"
    support: int                # sparse top-S (0 = full vocabulary)
    recipe: str                 # gauss | zipf | zipf_t3
    sigma: float = 1.5          # draft noise scale (zipf recipes)
    sigma_t: float = 0.7        # target divergence (fixed)
    sigma_t_range: tuple = None  # per-sequence U(lo, hi) divergence
    quantum: float = 0.0        # > 0: logits rounded to multiples of it (ties)
    near_ties: int = 0          # > 0: the row is shifted so its maximum is 0.125
                                # and tokens 1, 4, 7, ... get the next values
                                # below it, one fp32 ulp apart
    seed: int = 0x5EED0000
    n_expand: int = None
    construct_tempered: bool = False
    construct_full: bool = False
    method: str = "rheo"        # "rheo" (Algorithm 1), "rrsw" (leads-first
                                # baseline, App. D.2) or "topk" (no sampled slot)
    eps_m0: float = 2.0 ** -40
    steps: int = 1              # steps the workload description asks for
    mask: float = 0.0           # fraction of tokens masked to -inf (keyed per row)
    mask_tail: int = 0          # last token ids masked to -inf in every row
    mask_target: float = 0.0    # fraction of tokens masked in target rows only

    def __post_init__(self):
        if self.n_expand is None:
            self.n_expand = self.K

    @property
    def n_nodes(self):
        """Unpruned nodes per sequence per step: K + (D-1) * n_expand * K."""
        return self.K + (self.depth - 1) * self.n_expand * self.K

    @property
    def n_expanded(self):
        """Expanded rows per sequence per step: 1 + (D-1) * n_expand."""
        return 1 + (self.depth - 1) * self.n_expand

    @property
    def elem_bytes(self):
        return 2 if self.dtype == "bf16" else 4

    def with_(self, **kw):
        d = dict(self.__dict__)
        d.update(kw)
        return Workload(**d)


# The five workloads of the build's target (shapes from the paper's settings:
# V = 32000 Vicuna, 128256 Llama-3.1 / DSL-8B; tree 60, depth 8 (Sec. 5.1);
# support 128 (App. B); T = 1.0 default (Sec. 5.1)), plus the headline
# batched shape.  K counts the sampled slot (Sec. 3.2).
WORKLOADS = {
    "tiny": Workload("tiny", B=1, V=32, K=3, m=1, depth=3, R=8, T=1.0,
                     dtype="f32", support=128, recipe="gauss", sigma_t=0.5,
                     seed=0x5EED0001, steps=10000),
    "llama2": Workload("llama2", B=1, V=32000, K=8, m=1, depth=6, R=60, T=1.0,
                       dtype="f32", support=128, recipe="zipf", sigma=1.5,
                       sigma_t=0.7, seed=0x5EED0002, steps=200),
    "llama3": Workload("llama3", B=1, V=128256, K=8, m=1, depth=7, R=60, T=1.0,
                       dtype="bf16", support=128, recipe="zipf", sigma=1.5,
                       sigma_t=1.0, seed=0x5EED0003, steps=100),
    "batched": Workload("batched", B=64, V=128256, K=10, m=1, depth=8, R=64,
                        T=1.0, dtype="bf16", support=128, recipe="zipf",
                        sigma=1.5, sigma_t_range=(0.3, 1.5), seed=0x5EED0004,
                        steps=20),
    "large": Workload("large", B=128, V=151936, K=10, m=1, depth=8, R=80, T=0.8,
                      dtype="bf16", support=128, recipe="zipf_t3", sigma=1.0,
                      sigma_t=1.0, seed=0x5EED0005, steps=10),
    "headline": Workload("headline", B=64, V=128256, K=8, m=1, depth=7, R=60,
                         T=1.0, dtype="bf16", support=128, recipe="zipf",
                         sigma=1.5, sigma_t_range=(0.3, 1.5), seed=0x5EED0006,
                         steps=20),
    # the headline shape with the full-vocabulary (dense) distributions
    "headline_dense": Workload("headline_dense", B=64, V=128256, K=8, m=1, depth=7, R=60,
                               T=1.0, dtype="bf16", support=0, recipe="zipf",
                               sigma=1.5, sigma_t_range=(0.3, 1.5), seed=0x5EED0007,
                               steps=20),
}


def seq_seed(w, b):
    return splitmix64(w.seed ^ (((b + 1) * 0xD1B54A32D192ED03) & M64))


def root_key(w, b, step):
    """Prefix key of sequence ``b`` at decoding step ``step``."""
    return splitmix64(seq_seed(w, b) ^ (((step + 1) * 0x8CB92BA72F3D8DD7) & M64))


def step_rng_key(w, step):
    """The rng key handed to the method's calls for one step."""
    return splitmix64(w.seed ^ 0x243F6A8885A308D3 ^ ((step * GOLD) & M64))


def seq_sigma_t(w, b):
    """Target divergence of sequence ``b`` (per-sequence when a range is set)."""
    if w.sigma_t_range is None:
        return float(w.sigma_t)
    lo, hi = w.sigma_t_range
    u = (splitmix64(seq_seed(w, b) ^ 0x5151) >> 11) / float(1 << 53)
    return float(np.float32(lo + (hi - lo) * u))


# ---------------------------------------------------------------------------
# row generation
# ---------------------------------------------------------------------------

_TABLES = {}


def _tables(device):
    key = str(device)
    if key not in _TABLES:
        from scipy import special, stats
        u = (np.arange(65536, dtype=np.float64) + 0.5) / 65536.0
        normal = special.ndtri(u).astype(np.float32)
        t3 = stats.t.ppf(u, 3).astype(np.float32)
        _TABLES[key] = (torch.from_numpy(normal).to(device),
                        torch.from_numpy(t3).to(device))
    return _TABLES[key]


_LNR = {}


def _log_rank(V, device):
    key = (V, str(device))
    if key not in _LNR:
        lnr = np.log1p(np.arange(V, dtype=np.float64)).astype(np.float32)
        _LNR[key] = torch.from_numpy(lnr).to(device)
    return _LNR[key]


def _mix32(x):
    """A 32-bit integer mixer on int64 tensors holding values < 2**32
    (multipliers < 2**31 so no product leaves int64)."""
    x = x ^ (x >> 16)
    x = (x * 0x7FEB352D) & M32
    x = x ^ (x >> 15)
    x = (x * 0x5BD1E995) & M32
    x = x ^ (x >> 16)
    return x


def _noise_index(keys_lo, keys_hi, v):
    h = _mix32(v ^ keys_lo)
    h = _mix32(h ^ keys_hi)
    return h >> 16


def _key_words(keys, salt, device):
    ks = [splitmix64(k ^ salt) for k in keys]
    lo = torch.tensor([k & M32 for k in ks], dtype=torch.int64, device=device)
    hi = torch.tensor([k >> 32 for k in ks], dtype=torch.int64, device=device)
    return lo.view(-1, 1), hi.view(-1, 1)


def _perm_params(keys, V):
    a_s, c_s = [], []
    for k in keys:
        h = splitmix64(k ^ 0x7A11)
        a = 1 + (h % (V - 1))
        while math.gcd(a, V) != 1:
            a += 1
        a_s.append(a)
        c_s.append((h >> 32) % V)
    return a_s, c_s


def _quantise(w, rows):
    if w.quantum:
        q = float(w.quantum)
        return torch.round(rows * (1.0 / q)) * q
    return rows


def _draft_fp32(w, keys, device):
    """fp32 draft rows for node keys (before dtype rounding)."""
    return _masked(w, keys, _draft_unmasked(w, keys, device), device)


def _mask_hashed(w, keys, row, frac, salt, device):
    """Tokens whose keyed 16-bit hash lies below frac * 2^16 set to -inf."""
    v = torch.arange(w.V, dtype=torch.int64, device=device).view(1, -1)
    lo, hi = _key_words(keys, salt, device)
    thr = int(round(float(frac) * 65536))
    return torch.where(_noise_index(lo, hi, v) < thr,
                       torch.tensor(-np.inf, dtype=torch.float32, device=device), row)


def _masked(w, keys, row, device):
    """Masked vocabulary: tokens set to -inf by a keyed hash, and the last
    ``mask_tail`` ids of every row."""
    if w.mask > 0:
        row = _mask_hashed(w, keys, row, w.mask, 0x3333, device)
    if w.mask_tail > 0:
        row = row.clone()
        row[:, w.V - w.mask_tail:] = -np.inf
    return row


def _draft_unmasked(w, keys, device):
    normal, t3 = _tables(device)
    V = w.V
    if w.recipe == "flat":
        return torch.zeros((len(keys), V), dtype=torch.float32, device=device)
    v = torch.arange(V, dtype=torch.int64, device=device).view(1, -1)
    lo, hi = _key_words(keys, 0x1111, device)
    idx = _noise_index(lo, hi, v)
    if w.recipe == "gauss":
        return normal[idx] * np.float32(2.0)
    table = t3 if w.recipe == "zipf_t3" else normal
    noise = table[idx] * np.float32(w.sigma)
    a_s, c_s = _perm_params(keys, V)
    a = torch.tensor(a_s, dtype=torch.int64, device=device).view(-1, 1)
    c = torch.tensor(c_s, dtype=torch.int64, device=device).view(-1, 1)
    pi = (a * v + c) % V
    prior = _log_rank(V, device)[pi] * np.float32(-1.1)
    row = prior + noise
    if w.recipe == "zipf_t3":
        peak = [peaked(w, k) for k in keys]
        if any(peak):
            tok = [splitmix64(k ^ 0x70C) % V for k in keys]
            for i, (pk, t) in enumerate(zip(peak, tok)):
                if pk:
                    row[i, t] = row[i, t] + np.float32(12.0)
    if w.near_ties:
        mx = row.max(dim=1, keepdim=True).values
        row = (row - mx) + np.float32(0.125)
        x = torch.full_like(mx, 0.125)
        for j in range(w.near_ties):
            x = torch.nextafter(x, torch.full_like(x, -np.inf))
            row[:, 1 + 3 * j] = x[:, 0]
    return row


def peaked(w, key):
    """Whether the node with path key ``key`` gets the near one-hot peak
    (+12 on one keyed token; 5 % of the nodes of the zipf_t3 recipe)."""
    return w.recipe == "zipf_t3" and (splitmix64(key ^ 0x9EA4) & 0xFFFF) < 3277


def _round(w, rows):
    if w.dtype == "bf16":
        return rows.to(torch.bfloat16)
    return rows


def draft_rows(w, keys, device="cpu", chunk=256):
    """Draft logits [len(keys), V] for the given node keys."""
    out = []
    for i in range(0, len(keys), chunk):
        out.append(_round(w, _quantise(w, _draft_fp32(w, keys[i:i + chunk], device))))
    return torch.cat(out, 0) if out else torch.empty(
        (0, w.V), dtype=torch.bfloat16 if w.dtype == "bf16" else torch.float32,
        device=device)


def target_rows(w, keys, sigmas, device="cpu", chunk=256):
    """Target logits [len(keys), V]: the node's draft row plus an independent
    N(0, sigma_t^2) stream (``sigmas`` gives sigma_t per row)."""
    normal, _ = _tables(device)
    out = []
    v = torch.arange(w.V, dtype=torch.int64, device=device).view(1, -1)
    for i in range(0, len(keys), chunk):
        ks = keys[i:i + chunk]
        base = _draft_fp32(w, ks, device)
        lo, hi = _key_words(ks, 0x2222, device)
        idx = _noise_index(lo, hi, v)
        sg = torch.tensor([np.float32(s) for s in sigmas[i:i + chunk]],
                          dtype=torch.float32, device=device).view(-1, 1)
        row = base if w.recipe == "flat" else _quantise(w, base + normal[idx] * sg)
        if w.mask_target > 0:
            row = _mask_hashed(w, ks, row, w.mask_target, 0x4444, device)
        out.append(_round(w, row))
    return torch.cat(out, 0)


def as_fp32_numpy(rows):
    """fp32 numpy view of generated rows (bf16 widens exactly)."""
    return rows.float().cpu().numpy()
