"""ProtoKV far-memory hot path -- plain CPU oracle.

TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py may import this module.  The product path (the
HIP library and its Python binding) never imports, calls or links it, and it
shares no code with that path.

What it computes, in the paper's order and notation (ProtoKV, Sections
"State representation and prototype bank", "Online update", "Residual
Statistics and Pseudo-Token Interface"; Appendix Algorithms "ProtoKV
Streaming Update", "DecodeTopSResidualModes" and "Pseudo-Token Decoding and
Attention"; Equations 1 (assignment cost), pq (smoothed PQ probability) and
attn_logit (mass-aware logit); Table tab:default_config for the defaults):

* near tier: a ring of the last W frames of exact KV; appending frame t
  evicts frame t-W (the oldest) once W frames are resident;
* far tier: K prototype slots with (sum K, sum V, sum K^2, sum V^2, mass n,
  PQ histograms H^K, H^V, n_res, spatial mean mu and covariance Sigma,
  recency tau);
* fold of one evicted frame: seed free slots, then assign the remaining
  tokens with Eq. 1 against the post-seed bank and accumulate them in
  eviction order;
* synthesis: S pseudo-tokens per active prototype from the centres plus the
  top-S PQ residual modes (Alg. DecodeTopSResidualModes), paired by rank;
* readout: softmax attention over [near KV ; pseudo-tokens] with logit bias
  log n_k on the pseudo-tokens of prototype k (Eq. attn_logit).

Readings where the paper is silent or at odds with itself:

* centres are running means c_k = sumK_k / n_k (the text's "e.g. via EMA"
  and the merge rule's mass-weighted means), not Alg. 1's fixed-rate EMA;
  with Params.ema the fixed-rate EMA of Alg. 1 is followed instead: the
  sumK / sumV fields hold the centres c, p themselves, and every absorbed
  token, in eviction order, sets c <- (1 - alpha) c + alpha K and
  p <- (1 - beta) p + beta V (float32: one rounding per product and per
  add, 1 - alpha rounded to float32 first), then codes its residuals
  K - c, V - p against those updated centres (Alg. 1 updates the centres
  before R); the screen's cos is unchanged (scale invariant) and synthesis
  uses c, p directly.  Maintenance is not defined for this mode here;
* with Params.warm_frames > 0 the codebooks are learned from the stream
  (appendix "PQ codebook initialization", T_warm not given): the first
  warm_frames folds count no PQ codes (histograms and n_res stay 0) and
  append their non-seed tokens' residuals against the snapshot centres, in
  eviction order, to a reservoir of at most warm_tokens per (layer, kv
  head); after the last of them, mini-batch k-means (minibatch_kmeans: per-
  centre rates 1/count, batches of consecutive reservoir rows, centres
  started from rows i * floor(N / C)) learns each subspace's codebook
  separately for keys and values, fixed thereafter;
* with Params.rope_theta > 0 the readout applies rotary position
  embeddings (Sec. 3.3, appendix on the RoPE anchor): keys and queries
  arrive unrotated; a near token is rotated at its own stream position
  f * T + j, the S pseudo-keys of prototype k at tau_k, and query token t at
  P + t with P = (frames appended) * T (the query follows the last frame).
  The rotation is the rotate-half form: for i < D/2 the pair
  (x_i, x_(i + D/2)) turns by pos * theta^(-2 i / D), in float64 from the
  stored values (the prototypes aggregate unrotated keys; values are not
  rotated);
* a fold is frame-batched: all non-seed tokens of the evicted frame are
  assigned against the bank as it stands after seeding, then accumulated in
  eviction order (with one token per frame this is Alg. 1's per-token loop);
* ties in the argmin of Eq. 1 go to the lowest slot; cos is 0 when either
  vector is zero;
* d_Mah is the (unsquared) distance sqrt(d^T (Sigma + rho I)^-1 d) with a
  ridge rho = 1e-4 (Params.mah_squared: the squared form d^T (Sigma + rho
  I)^-1 d, the gating distance of the tracker the paper cites for this
  term); coordinates are cell centres ((col+.5)/W, (row+.5)/H);
* tau is the stream position of the most recently absorbed source token; a
  prototype is idle when (current frame) - (frame of tau) > T_idle frames;
* PQ residuals are taken against the centre before this fold's updates
  (the post-seed snapshot); PQ distance is squared Euclidean over
  contiguous subspaces; code ties go to the lowest codeword;
* smoothing eps = 1, so every PQ probability is (H+1)/(n_res+C); a code
  tuple's score sum_g log P is compared exactly through the integer product
  prod_g (H[g][z_g] + 1) (the denominator is common to all tuples); ties
  between equal scores go to the lexicographically smaller code tuple;
* pseudo-tokens are rounded to the KV dtype from the float32 sum c + r;
  centres are float32(sumK / n);
* with Params.var_alloc (appendix "Dynamic Pseudo-Token Allocation") each
  active prototype k gets S_k pseudo-tokens, its top-S_k code tuples, in
  place of S.  Var(H_k) is the total variance of the residual distribution
  the PQ statistics describe: per side (K, V) and subspace g the empirical
  code distribution H[g][c] / n_res places mass on the codewords C_g[c];
  Var(H_k) sums, over sides and subspaces, sum_c P(c) |C_g[c]|^2 -
  |sum_c P(c) C_g[c]|^2 (0 without residuals).  The total S_tot = A * S
  over the A active prototypes (the paper's K_max * S once the bank is
  full) is kept; every prototype keeps one pseudo-token (with Var = 0 the
  proportional share would remove it, and its mass, from the readout) and
  the other S_tot - A are shared in proportion to Var(H_k), capped at s_max
  (the excess re-shared among the uncapped, repeatedly; with no variance
  left they share equally; with no variance at all every S_k = S); the
  real shares x_k become integers by cumulative rounding,
  S_k = floor(X_k + 1/2) - floor(X_(k-1) + 1/2) with X_k the sum of
  x_1..x_k in slot order, which keeps the total and each S_k within one of
  x_k.  All of it in float64, sums in slot order;
* maintenance (Alg. "Prototype Maintenance", when enabled) runs once per
  fold, after the evicted frame is absorbed, at the current frame t, over
  the active prefix of A slots (the slots seeded so far).  Aging: an idle
  slot (the idle rule above) gets n' = floor((1 - gamma) n) in float64, and
  its sums and squared sums are scaled by float32(n') / float32(n), so its
  centre stays (histograms, n_res, mu, Sigma and tau stay).  Merging: pairs
  (i, j), i < j, in ascending order; i absorbs j when
  ||c_i - c_j||^2 < eps_K^2 and ||p_i - p_j||^2 < eps_V^2, each a float64
  sum of the terms (c_i[d] - c_j[d])^2 (c = float32(sum / n)) taken as
  pairs of consecutive dims, then halves of the partial sums,
  using i's centre as updated by its earlier merges; sums, squared sums,
  histograms, n and n_res add, mu becomes the mass-weighted mean, Sigma and
  tau of i stay, j becomes empty.  Recycling: the empty slots of the prefix,
  in ascending order, are seeded like evicted tokens from the near window's
  tokens taken newest frame first, raster order within a frame (wrapping
  around when there are more empty slots than near tokens).

Precision: the bank is float32 (fp32 prototype statistics) and is updated
with the explicit float32 operation sequences written below (one IEEE
rounding per operation, no fused multiply-add); every cost, softmax and
readout value is float64.

Parity unpinned: eps, rho, the coordinate convention and the time unit of
T_idle have no numeric anchor in the paper (no worked example, no code); they
are pinned only by this reading.
"""
from __future__ import annotations

import collections
import dataclasses
import itertools
import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

F32 = np.float32

# Table tab:default_config (Appendix "Default Hyperparameter Configuration").
TABLE5_DEFAULTS = {
    "near_far_split": (1, 3),
    "S": 8,
    "lambda_sp": 0.1,
    "lambda_idle": 0.01,
    "T_idle": 120,
    "alpha": 0.05,
    "beta": 0.05,
    "eta": 0.05,
    "gamma": 0.05,
    "eps_K": 0.20,
    "eps_V": 0.25,
    "G": 8,
    "C": 16,
    "B": 32,
}


@dataclasses.dataclass
class Params:
    head_dim: int = 128
    grid_h: int = 14
    grid_w: int = 14
    window_frames: int = 8
    capacity: int = 256
    S: int = TABLE5_DEFAULTS["S"]
    G: int = TABLE5_DEFAULTS["G"]
    C: int = TABLE5_DEFAULTS["C"]
    B: int = TABLE5_DEFAULTS["B"]
    lambda_sp: float = TABLE5_DEFAULTS["lambda_sp"]
    lambda_idle: float = TABLE5_DEFAULTS["lambda_idle"]
    t_idle: int = TABLE5_DEFAULTS["T_idle"]
    eta: float = TABLE5_DEFAULTS["eta"]
    ridge: float = 1e-4
    kv_dtype: str = "bf16"
    use_pq: bool = True
    mass_bias: bool = True
    # Eq. 1's spatial term as the squared Mahalanobis distance (default: the
    # distance itself)
    mah_squared: bool = False
    # Alg. "Prototype Maintenance" (off unless asked for); gamma and the
    # thresholds are float64, so (1 - 0.05) n lands on the integers the paper
    # means (a float32 gamma = 0.0500000007 would floor 0.95 * 40 to 37)
    maintenance: bool = False
    gamma: float = TABLE5_DEFAULTS["gamma"]
    eps_k: float = TABLE5_DEFAULTS["eps_K"]
    eps_v: float = TABLE5_DEFAULTS["eps_V"]
    # Alg. "ProtoKV Streaming Update" literally: fixed-rate EMA centres
    # (rates used as float32), residuals against the updated centres
    ema: bool = False
    alpha: float = TABLE5_DEFAULTS["alpha"]
    beta: float = TABLE5_DEFAULTS["beta"]
    # rotary positions in the readout (0 = keys and queries used as given)
    rope_theta: float = 0.0
    # variance-aware pseudo-token allocation (appendix "Dynamic Pseudo-Token
    # Allocation"): S_k per prototype under the fixed total A * S, at most
    # s_max each (off: S for every prototype)
    var_alloc: bool = False
    s_max: int = 16
    # PQ codebook warm-up: the first warm_frames folds collect residuals (no
    # PQ counts), then mini-batch k-means learns the codebooks (0 = off: the
    # given codebooks are used from the start)
    warm_frames: int = 0
    warm_tokens: int = 1024      # reservoir capacity per (layer, kv head)
    kmeans_epochs: int = 4
    kmeans_batch: int = 64

    @property
    def tokens_per_frame(self) -> int:
        return self.grid_h * self.grid_w


# ---------------------------------------------------------------------------
# small helpers
# ---------------------------------------------------------------------------


def round_kv(x32: np.ndarray, kv_dtype: str) -> np.ndarray:
    """Round float32 values to the KV dtype (bf16: round to nearest even)."""
    x32 = np.asarray(x32, dtype=F32)
    if kv_dtype == "fp32":
        return x32.copy()
    bits = x32.view(np.uint32).astype(np.uint64)
    lsb = (bits >> 16) & 1
    top = ((bits + 0x7FFF + lsb) >> 16).astype(np.uint32)
    return (top << 16).view(F32)


def rope_rotate(x: np.ndarray, pos, theta: float) -> np.ndarray:
    """Rotary position embedding, rotate-half form, in float64: for i < D/2
    the pair (x_i, x_(i + D/2)) is turned by the angle pos * theta^(-2 i / D).
    x [..., D]; pos broadcasts against x's leading axes."""
    x = np.asarray(x, dtype=np.float64)
    D = x.shape[-1]
    h = D // 2
    inv = float(theta) ** (-2.0 * np.arange(h, dtype=np.float64) / D)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * inv
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :h], x[..., h:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def spatial_coords(grid_h: int, grid_w: int) -> np.ndarray:
    """s_j = ((col+0.5)/grid_w, (row+0.5)/grid_h) in float32, raster order j."""
    out = np.zeros((grid_h * grid_w, 2), dtype=F32)
    for j in range(grid_h * grid_w):
        row, col = divmod(j, grid_w)
        out[j, 0] = F32(col + 0.5) / F32(grid_w)
        out[j, 1] = F32(row + 0.5) / F32(grid_h)
    return out


# ---------------------------------------------------------------------------
# prototype bank (far tier)
# ---------------------------------------------------------------------------


class Bank:
    """B_far = {Pi_k}: one (layer, kv head)'s K prototype slots."""

    def __init__(self, p: Params):
        K, D, G, C = p.capacity, p.head_dim, p.G, p.C
        self.n = np.zeros(K, dtype=np.int64)          # mass n_k (0 = inactive)
        self.sum_k = np.zeros((K, D), dtype=F32)       # sum of absorbed keys (EMA: the centre c)
        self.sum_v = np.zeros((K, D), dtype=F32)
        self.sq_k = np.zeros((K, D), dtype=F32)        # sum of squared keys
        self.sq_v = np.zeros((K, D), dtype=F32)
        self.hist_k = np.zeros((K, G, C), dtype=np.int64)   # H^K
        self.hist_v = np.zeros((K, G, C), dtype=np.int64)   # H^V
        self.n_res = np.zeros(K, dtype=np.int64)
        self.mu = np.zeros((K, 2), dtype=F32)          # spatial mean (x, y)
        self.sigma = np.zeros((K, 3), dtype=F32)       # (xx, xy, yy)
        self.tau = np.zeros(K, dtype=np.int64)         # stream position

    def copy(self) -> "Bank":
        b = Bank.__new__(Bank)
        for k, v in self.__dict__.items():
            setattr(b, k, v.copy())
        return b


# ---------------------------------------------------------------------------
# Eq. 1: continuity-aware assignment cost
# ---------------------------------------------------------------------------


def assignment_costs(keys: np.ndarray, coords: np.ndarray, bank: Bank, t_frame: int,
                     p: Params) -> np.ndarray:
    """cost[i, k] = -cos(K_i, c_k) + lambda_sp d_Mah(s_i; mu_k, Sigma_k)
    + lambda_idle 1[idle(tau_k)]  (Eq. 1), float64; +inf for inactive k.

    cos uses sumK_k (cos is scale invariant, so cos(K, sumK/n) = cos(K, sumK)).
    """
    K64 = keys.astype(np.float64)
    C64 = bank.sum_k.astype(np.float64)
    dots = K64 @ C64.T
    nk = np.sqrt((K64 * K64).sum(axis=1))
    nc = np.sqrt((C64 * C64).sum(axis=1))
    denom = nk[:, None] * nc[None, :]
    with np.errstate(invalid="ignore", divide="ignore"):
        cos = np.where(denom > 0, dots / np.where(denom > 0, denom, 1.0), 0.0)

    # Mahalanobis distance to the prototype's running location distribution.
    dx = coords[:, 0].astype(np.float64)[:, None] - bank.mu[:, 0].astype(np.float64)[None, :]
    dy = coords[:, 1].astype(np.float64)[:, None] - bank.mu[:, 1].astype(np.float64)[None, :]
    A = bank.sigma[:, 0].astype(np.float64) + p.ridge
    Bxy = bank.sigma[:, 1].astype(np.float64)
    Cc = bank.sigma[:, 2].astype(np.float64) + p.ridge
    det = A * Cc - Bxy * Bxy
    q = (Cc[None, :] * dx * dx - 2.0 * Bxy[None, :] * dx * dy + A[None, :] * dy * dy) / det[None, :]
    d_mah = np.maximum(q, 0.0) if p.mah_squared else np.sqrt(np.maximum(q, 0.0))

    T = p.tokens_per_frame
    idle = ((t_frame - bank.tau // T) > p.t_idle).astype(np.float64)

    cost = -cos + p.lambda_sp * d_mah + p.lambda_idle * idle[None, :]
    cost[:, bank.n == 0] = np.inf
    return cost


def argmin_lowest(cost: np.ndarray):
    """Row argmin (ties -> lowest k) and the top-2 margin (cost2 - cost1)."""
    idx = np.argmin(cost, axis=1)
    if cost.shape[1] >= 2:
        part = np.sort(cost, axis=1)
        margin = part[:, 1] - part[:, 0]
    else:
        margin = np.full(cost.shape[0], np.inf)
    return idx, margin


# ---------------------------------------------------------------------------
# PQ residual encoding
# ---------------------------------------------------------------------------


def pq_encode(residuals: np.ndarray, codebook: np.ndarray) -> np.ndarray:
    """Nearest codeword per subspace for float32 residuals [M][D].

    codebook float32 [G][C][D/G]; subspace g covers dims [g*D/G, (g+1)*D/G).
    dist(g, c) = sum_u (r_u - C[g][c][u])^2 accumulated in float32 with u
    ascending (one rounding per subtract, multiply and add); ties -> lowest c.
    """
    G, C, Dp = codebook.shape
    M = residuals.shape[0]
    codes = np.zeros((M, G), dtype=np.int64)
    for g in range(G):
        sub = residuals[:, g * Dp:(g + 1) * Dp].astype(F32)
        acc = np.zeros((M, C), dtype=F32)
        for u in range(Dp):
            diff = (sub[:, u][:, None] - codebook[g][None, :, u]).astype(F32)
            acc = (acc + (diff * diff).astype(F32)).astype(F32)
        codes[:, g] = np.argmin(acc, axis=1)
    return codes


# ---------------------------------------------------------------------------
# Alg. "ProtoKV Streaming Update", one evicted frame, frame-batched
# ---------------------------------------------------------------------------


NEAR_TIE = 1e-6   # a top-2 cost margin below this is a near tie (counted, either slot valid)


@dataclasses.dataclass
class FoldResult:
    assign: np.ndarray      # slot per evicted token (seeded tokens: their slot)
    margin: np.ndarray      # top-2 cost margin (inf for seeded tokens)
    n_seed: int
    # with collect=True: key and value residuals of the non-seed tokens in
    # eviction order, against the snapshot centres
    residuals: Optional[Tuple[np.ndarray, np.ndarray]] = None
    # Eq. 1 costs of the non-seed tokens (rows: tokens n_seed..T-1, +inf for
    # inactive slots)
    cost: Optional[np.ndarray] = None

    @property
    def near_ties(self) -> int:
        return int((self.margin < NEAR_TIE).sum())


def fold_frame(bank: Bank, keys: np.ndarray, values: np.ndarray, f_evicted: int,
               t_frame: int, p: Params, codebooks: np.ndarray, collect: bool = False,
               choose: Optional[np.ndarray] = None) -> FoldResult:
    """Absorb the evicted frame f_evicted (tokens j = 0..T-1 in raster order)
    into `bank` (modified in place).  t_frame is the frame being appended.

    codebooks float32 [2][G][C][D/G] (keys, values) of this (layer, head).
    choose: optionally a slot for every token of the frame; a non-seed token
    takes it in place of the lowest argmin, which is allowed only where the
    two costs lie within NEAR_TIE of each other (a near tie, where either
    slot is a valid argmin of Eq. 1); any other choice raises ValueError.
    """
    T = keys.shape[0]
    coords = spatial_coords(p.grid_h, p.grid_w)
    pos = f_evicted * T + np.arange(T)
    one, eta = F32(1.0), F32(p.eta)
    keep = F32(one - eta)

    # Initialization: while free slots remain, an evicted token seeds the
    # lowest free slot (c <- K, p <- V, n <- 1, mu <- s, Sigma <- I, R <- 0).
    free = [k for k in range(p.capacity) if bank.n[k] == 0]
    n_seed = min(T, len(free))
    assign = np.full(T, -1, dtype=np.int64)
    margin = np.full(T, np.inf)
    for j in range(n_seed):
        k = free[j]
        kk, vv = keys[j].astype(F32), values[j].astype(F32)
        bank.n[k] = 1
        bank.sum_k[k] = kk
        bank.sum_v[k] = vv
        bank.sq_k[k] = (kk * kk).astype(F32)
        bank.sq_v[k] = (vv * vv).astype(F32)
        bank.hist_k[k] = 0
        bank.hist_v[k] = 0
        bank.n_res[k] = 0
        bank.mu[k] = coords[j]
        bank.sigma[k] = np.array([1.0, 0.0, 1.0], dtype=F32)
        bank.tau[k] = pos[j]
        assign[j] = k
    if n_seed == T:
        D = keys.shape[1]
        empty = (np.zeros((0, D), F32), np.zeros((0, D), F32)) if collect else None
        return FoldResult(assign, margin, n_seed, empty)

    # Assignment (Eq. 1) of the remaining tokens against the post-seed bank.
    snap = bank.copy()
    rest = np.arange(n_seed, T)
    cost = assignment_costs(keys[rest], coords[rest], snap, t_frame, p)
    idx, marg = argmin_lowest(cost)
    if choose is not None:
        want = np.asarray(choose, dtype=np.int64)[rest]
        for i, k in enumerate(want):
            if k == idx[i]:
                continue
            if not (0 <= k < p.capacity and np.isfinite(cost[i, k])
                    and cost[i, k] - cost[i, idx[i]] < NEAR_TIE):
                raise ValueError(f"token {rest[i]}: slot {k} is not a near-tie argmin of Eq. 1")
        idx = want
    assign[rest] = idx
    margin[rest] = marg

    # Residual codes against the snapshot centres c = f32(sumK / n) (running
    # means; with EMA centres each token is coded after its own update).
    if (p.use_pq or collect) and not p.ema:
        nf = snap.n[idx].astype(F32)[:, None]
        c_snap = (snap.sum_k[idx] / nf).astype(F32)
        p_snap = (snap.sum_v[idx] / nf).astype(F32)
        r_k = (keys[rest].astype(F32) - c_snap).astype(F32)
        r_v = (values[rest].astype(F32) - p_snap).astype(F32)
    if p.use_pq and not p.ema:
        codes_k = pq_encode(r_k, codebooks[0])
        codes_v = pq_encode(r_v, codebooks[1])

    # Prototype update, tokens in eviction order.
    al, be = F32(p.alpha), F32(p.beta)
    ka, kb = F32(one - al), F32(one - be)
    for i, j in enumerate(rest):
        k = idx[i]
        kk, vv = keys[j].astype(F32), values[j].astype(F32)
        bank.n[k] += 1
        if p.ema:
            # c <- (1 - alpha) c + alpha K, p <- (1 - beta) p + beta V
            bank.sum_k[k] = ((ka * bank.sum_k[k]).astype(F32) + (al * kk).astype(F32)).astype(F32)
            bank.sum_v[k] = ((kb * bank.sum_v[k]).astype(F32) + (be * vv).astype(F32)).astype(F32)
        else:
            bank.sum_k[k] = (bank.sum_k[k] + kk).astype(F32)
            bank.sum_v[k] = (bank.sum_v[k] + vv).astype(F32)
        bank.sq_k[k] = (bank.sq_k[k] + (kk * kk).astype(F32)).astype(F32)
        bank.sq_v[k] = (bank.sq_v[k] + (vv * vv).astype(F32)).astype(F32)
        if p.use_pq:
            if p.ema:
                # residuals against the centres just updated
                zk = pq_encode((kk - bank.sum_k[k]).astype(F32)[None, :], codebooks[0])[0]
                zv = pq_encode((vv - bank.sum_v[k]).astype(F32)[None, :], codebooks[1])[0]
            else:
                zk, zv = codes_k[i], codes_v[i]
            for g in range(p.G):
                bank.hist_k[k, g, zk[g]] += 1
                bank.hist_v[k, g, zv[g]] += 1
            bank.n_res[k] += 1
        # spatial state: mu <- (1-eta) mu + eta s, then
        # Sigma <- (1-eta) Sigma + eta (s - mu)(s - mu)^T with the new mu.
        s = coords[j]
        mx = F32(F32(keep * bank.mu[k, 0]) + F32(eta * s[0]))
        my = F32(F32(keep * bank.mu[k, 1]) + F32(eta * s[1]))
        bank.mu[k, 0], bank.mu[k, 1] = mx, my
        ddx, ddy = F32(s[0] - mx), F32(s[1] - my)
        sxx, sxy, syy = bank.sigma[k]
        bank.sigma[k, 0] = F32(F32(keep * sxx) + F32(eta * F32(ddx * ddx)))
        bank.sigma[k, 1] = F32(F32(keep * sxy) + F32(eta * F32(ddx * ddy)))
        bank.sigma[k, 2] = F32(F32(keep * syy) + F32(eta * F32(ddy * ddy)))
        bank.tau[k] = pos[j]
    return FoldResult(assign, margin, n_seed, (r_k, r_v) if collect else None, cost)


# ---------------------------------------------------------------------------
# PQ codebook initialization: mini-batch k-means on a warm-up reservoir
# ---------------------------------------------------------------------------


def minibatch_kmeans(x: np.ndarray, centres: np.ndarray, epochs: int, batch: int) -> np.ndarray:
    """Mini-batch k-means with per-centre rates 1/count on float32 rows
    x [N][d], from the float32 centres [C][d].  `epochs` passes over x in
    order, in batches of `batch` consecutive rows (the last one shorter):
    each row of a batch is assigned to its nearest centre as the batch
    starts (pq_encode's float32 sequential distance, ties to the lowest
    index), then the batch's rows update their centres in row order:
    count += 1, eta = 1 / count, c <- (1 - eta) c + eta x (float32, one
    rounding per operation).  Counts persist across batches and epochs."""
    c = np.array(centres, dtype=F32)
    count = np.zeros(c.shape[0], dtype=np.int64)
    one = F32(1.0)
    for _ in range(epochs):
        for b0 in range(0, len(x), batch):
            xb = x[b0:b0 + batch].astype(F32)
            z = pq_encode(xb, c[None])[:, 0]
            for i, k in enumerate(z):
                count[k] += 1
                eta = F32(one / F32(count[k]))
                c[k] = ((F32(one - eta) * c[k]).astype(F32) + (eta * xb[i]).astype(F32)).astype(F32)
    return c


def learn_codebooks(res_k: np.ndarray, res_v: np.ndarray, codebooks: np.ndarray, p: Params) -> np.ndarray:
    """Codebooks [2][G][C][D/G] learned from a reservoir of N residuals per
    side, separately per subspace and per side, each k-means started from
    the reservoir entries i * floor(N / C), i < C.  With fewer than C
    residuals the given codebooks are kept."""
    out = np.array(codebooks, dtype=F32)
    G, C, Dp = out.shape[1:]
    N = len(res_k)
    if N < C:
        return out
    for side, res in enumerate((res_k, res_v)):
        for g in range(G):
            xg = res[:, g * Dp:(g + 1) * Dp].astype(F32)
            init = xg[np.arange(C) * (N // C)]
            out[side, g] = minibatch_kmeans(xg, init, p.kmeans_epochs, p.kmeans_batch)
    return out


# ---------------------------------------------------------------------------
# Alg. "Prototype Maintenance": aging, merging, recycling
# ---------------------------------------------------------------------------


def _seed_slot(bank: Bank, k: int, kk: np.ndarray, vv: np.ndarray, coord: np.ndarray, pos: int) -> None:
    """(Re)initialise slot k from one token: c <- K, p <- V, n <- 1, mu <- s,
    Sigma <- I, tau <- its position, R <- 0."""
    kk, vv = kk.astype(F32), vv.astype(F32)
    bank.n[k] = 1
    bank.sum_k[k] = kk
    bank.sum_v[k] = vv
    bank.sq_k[k] = (kk * kk).astype(F32)
    bank.sq_v[k] = (vv * vv).astype(F32)
    bank.hist_k[k] = 0
    bank.hist_v[k] = 0
    bank.n_res[k] = 0
    bank.mu[k] = coord
    bank.sigma[k] = np.array([1.0, 0.0, 1.0], dtype=F32)
    bank.tau[k] = pos


NEAR_THRESHOLD_REL = 1e-12


def _dist2(a: np.ndarray, b: np.ndarray) -> float:
    """||a - b||^2 = sum_d (a[d] - b[d])^2 for float32 a, b, in float64 with
    d ascending (each term a rounded difference, then a rounded square)."""
    a64, b64 = a.astype(np.float64), b.astype(np.float64)
    total = 0.0
    for d in range(len(a64)):
        diff = a64[d] - b64[d]
        total += diff * diff
    return float(total)


def _near_threshold(d2: float, eps2: float) -> bool:
    """The merge test d2 < eps2 is within float64 rounding of flipping."""
    return abs(d2 - eps2) <= NEAR_THRESHOLD_REL * eps2


def maintain(bank: Bank, near: Sequence[Tuple[int, np.ndarray, np.ndarray]], t_frame: int,
             p: Params) -> Dict[str, int]:
    """One maintenance pass over `bank` (modified in place) at frame t_frame.

    near: the near window's frames (frame index, K [T][D], V [T][D]), oldest
    first.  Returns counts of aged, merged and recycled slots, and of the pair
    tests that fell within 1e-12 relative of their threshold (near_threshold).
    """
    if p.ema:
        raise ValueError("maintenance is defined for running-mean centres only")
    T = p.tokens_per_frame
    A = int((bank.n > 0).sum())
    assert np.all(bank.n[:A] > 0), "active slots form a prefix"
    stats = {"aged": 0, "merged": 0, "recycled": 0, "near_threshold": 0}

    # aging: mass decay of idle prototypes, sums scaled with it
    for k in range(A):
        if (t_frame - int(bank.tau[k]) // T) > p.t_idle:
            n_old = int(bank.n[k])
            n_new = int(math.floor((1.0 - p.gamma) * float(n_old)))
            r = F32(F32(n_new) / F32(n_old))
            bank.sum_k[k] = (bank.sum_k[k] * r).astype(F32)
            bank.sum_v[k] = (bank.sum_v[k] * r).astype(F32)
            bank.sq_k[k] = (bank.sq_k[k] * r).astype(F32)
            bank.sq_v[k] = (bank.sq_v[k] * r).astype(F32)
            bank.n[k] = n_new
            stats["aged"] += 1

    # merging: i absorbs every later j whose key and value centres are close
    ek2 = float(p.eps_k) * float(p.eps_k)
    ev2 = float(p.eps_v) * float(p.eps_v)
    for i in range(A):
        if bank.n[i] == 0:
            continue
        for j in range(i + 1, A):
            if bank.n[j] == 0:
                continue
            ni, nj = F32(bank.n[i]), F32(bank.n[j])
            ci, cj = (bank.sum_k[i] / ni).astype(F32), (bank.sum_k[j] / nj).astype(F32)
            dk = _dist2(ci, cj)
            stats["near_threshold"] += _near_threshold(dk, ek2)
            if not dk < ek2:
                continue
            pi, pj = (bank.sum_v[i] / ni).astype(F32), (bank.sum_v[j] / nj).astype(F32)
            dv = _dist2(pi, pj)
            stats["near_threshold"] += _near_threshold(dv, ev2)
            if not dv < ev2:
                continue
            wsum = F32(ni + nj)
            for a in range(2):
                bank.mu[i, a] = F32(F32(F32(ni * bank.mu[i, a]) + F32(nj * bank.mu[j, a])) / wsum)
            bank.sum_k[i] = (bank.sum_k[i] + bank.sum_k[j]).astype(F32)
            bank.sum_v[i] = (bank.sum_v[i] + bank.sum_v[j]).astype(F32)
            bank.sq_k[i] = (bank.sq_k[i] + bank.sq_k[j]).astype(F32)
            bank.sq_v[i] = (bank.sq_v[i] + bank.sq_v[j]).astype(F32)
            bank.hist_k[i] += bank.hist_k[j]
            bank.hist_v[i] += bank.hist_v[j]
            bank.n[i] += bank.n[j]
            bank.n_res[i] += bank.n_res[j]
            bank.n[j] = 0
            stats["merged"] += 1

    # recycling: empty slots of the prefix take the most recent near tokens
    coords = spatial_coords(p.grid_h, p.grid_w)
    tokens = [(f, kf, vf, j) for (f, kf, vf) in reversed(list(near)) for j in range(T)]
    e = 0
    for k in range(A):
        if bank.n[k] == 0:
            f, kf, vf, j = tokens[e % len(tokens)]
            _seed_slot(bank, k, kf[j], vf[j], coords[j], f * T + j)
            e += 1
    stats["recycled"] = e
    return stats


# ---------------------------------------------------------------------------
# Eq. pq and Alg. "DecodeTopSResidualModes"
# ---------------------------------------------------------------------------


def _order_key(score: int, codes: Tuple[int, ...]):
    return (-score, codes)


def decode_top_s(hist: np.ndarray, S: int, B: int) -> List[Tuple[int, ...]]:
    """Top-S code tuples of one PQ histogram H [G][C] by beam search (Alg. 3).

    With eps = 1, log P(g, c) = log(H[g][c] + 1) - log(n_res + C); a tuple
    scores sum_g log P(g, z_g), so the ranking equals that of the integer
    prod_g (H[g][z_g] + 1), compared exactly.  TopB / TopS keep the highest
    scores; equal scores keep the lexicographically smaller code tuple.
    """
    G, C = hist.shape
    beam: List[Tuple[int, Tuple[int, ...]]] = [(1, ())]
    for g in range(G):
        expanded = []
        for score, codes in beam:
            for c in range(C):
                expanded.append((score * (int(hist[g, c]) + 1), codes + (c,)))
        expanded.sort(key=lambda e: _order_key(*e))
        beam = expanded[:B]
    beam.sort(key=lambda e: _order_key(*e))
    return [codes for _, codes in beam[:S]]


def residual_from_codes(codes: Sequence[int], codebook: np.ndarray) -> np.ndarray:
    """r_bar = concat_g C_g[z_g]  (float32 [D])."""
    return np.concatenate([codebook[g][c] for g, c in enumerate(codes)]).astype(F32)


# ---------------------------------------------------------------------------
# Alg. "Pseudo-Token Decoding and Attention": synthesis
# ---------------------------------------------------------------------------


@dataclasses.dataclass
class Pseudo:
    keys: np.ndarray     # float32 [n_active * S][D] (values of the KV dtype)
    values: np.ndarray
    bias: np.ndarray     # float64 [n_active * S]: log n_k (0 if mass bias off)
    slots: np.ndarray    # slot k of each pseudo-token


def residual_variance(bank: Bank, codebooks: np.ndarray) -> np.ndarray:
    """Var(H_k) of every slot, float64 [K]: over sides (K then V) and
    subspaces g ascending, sum_c P(c) |C[c]|^2 - |sum_c P(c) C[c]|^2 with
    P(c) = H[g][c] / n_res (clamped at 0), where |C[c]|^2 and the mean are
    summed over the subspace's dims ascending and over codewords ascending;
    0 for slots without residuals."""
    K = len(bank.n)
    G, C, Dp = codebooks.shape[1:]
    nres = bank.n_res.astype(np.float64)
    has = nres > 0
    denom = np.where(has, nres, 1.0)
    total = np.zeros(K)
    for side, hist in ((0, bank.hist_k), (1, bank.hist_v)):
        for g in range(G):
            cw = codebooks[side, g].astype(np.float64)         # [C][Dp]
            n2 = np.zeros(C)
            for u in range(Dp):
                n2 = n2 + cw[:, u] * cw[:, u]
            e2 = np.zeros(K)
            mean = np.zeros((K, Dp))
            for c in range(C):
                pc = hist[:, g, c].astype(np.float64) / denom
                e2 = e2 + pc * n2[c]
                mean = mean + pc[:, None] * cw[c][None, :]
            m2 = np.zeros(K)
            for u in range(Dp):
                m2 = m2 + mean[:, u] * mean[:, u]
            total = total + np.maximum(e2 - m2, 0.0)
    return np.where(has, total, 0.0)


def allocate_pseudo(var: Sequence[float], S: int, s_max: int) -> List[int]:
    """S_k for the A = len(var) active prototypes under the total A * S."""
    A = len(var)
    if A == 0:
        return []
    wsum = 0.0
    for v in var:
        wsum += float(v)
    if wsum == 0.0:
        return [S] * A
    total = A * S
    capped = [False] * A
    while True:
        ncap = sum(capped)
        rest = float(total - A - ncap * (s_max - 1))    # beyond one per uncapped prototype
        w = 0.0
        for k in range(A):
            if not capped[k]:
                w += float(var[k])
        nunc = A - ncap
        x = []
        for k in range(A):
            if capped[k]:
                x.append(float(s_max))
            elif w > 0.0:
                x.append(1.0 + rest * float(var[k]) / w)
            else:
                x.append(1.0 + rest / nunc)
        over = [k for k in range(A) if not capped[k] and x[k] > s_max]
        if not over:
            break
        for k in over:
            capped[k] = True
    out, X, prev = [], 0.0, 0
    for k in range(A):
        X += x[k]
        cur = math.floor(X + 0.5)
        out.append(cur - prev)
        prev = cur
    return out


def pseudo_counts(bank: Bank, codebooks: np.ndarray, p: Params) -> np.ndarray:
    """Pseudo-tokens per slot: S for every active slot, or the variance-aware
    S_k; 0 for inactive slots.  Active slots form a prefix of the bank."""
    A = int((bank.n > 0).sum())
    out = np.zeros(p.capacity, dtype=np.int64)
    if not p.var_alloc:
        out[:A] = p.S
        return out
    out[:A] = allocate_pseudo(residual_variance(bank, codebooks)[:A], p.S, p.s_max)
    return out


def synthesize(bank: Bank, codebooks: np.ndarray, p: Params) -> Pseudo:
    ks, vs, bs, sl = [], [], [], []
    zero = np.zeros(p.head_dim, dtype=F32)
    counts = pseudo_counts(bank, codebooks, p)
    for k in range(p.capacity):
        if bank.n[k] == 0:
            continue
        Sk = int(counts[k])
        if p.ema:  # the fields hold the centres
            c, pv = bank.sum_k[k].copy(), bank.sum_v[k].copy()
        else:
            nf = F32(bank.n[k])
            c = (bank.sum_k[k] / nf).astype(F32)
            pv = (bank.sum_v[k] / nf).astype(F32)
        if bank.n_res[k] == 0 or not p.use_pq:
            rk = [zero] * Sk
            rv = [zero] * Sk
        else:
            zk = decode_top_s(bank.hist_k[k], Sk, max(p.B, Sk))
            zv = decode_top_s(bank.hist_v[k], Sk, max(p.B, Sk))
            rk = [residual_from_codes(z, codebooks[0]) for z in zk]
            rv = [residual_from_codes(z, codebooks[1]) for z in zv]
        b = math.log(bank.n[k]) if p.mass_bias else 0.0
        for s in range(Sk):
            ks.append(round_kv((c + rk[s]).astype(F32), p.kv_dtype))
            vs.append(round_kv((pv + rv[s]).astype(F32), p.kv_dtype))
            bs.append(b)
            sl.append(k)
    D = p.head_dim
    return Pseudo(np.array(ks, dtype=F32).reshape(-1, D), np.array(vs, dtype=F32).reshape(-1, D),
                  np.array(bs, dtype=np.float64), np.array(sl, dtype=np.int64))


# ---------------------------------------------------------------------------
# Eq. attn_logit: mass-aware readout
# ---------------------------------------------------------------------------


def attend(q_rows: np.ndarray, k_ctx: np.ndarray, v_ctx: np.ndarray, bias: np.ndarray):
    """softmax(Q K^T / sqrt(d) + b) V and log-sum-exp, in float64.

    q_rows [R][D]; k_ctx, v_ctx [L][D]; bias [L] (0 for near tokens)."""
    Q = q_rows.astype(np.float64)
    Kc = k_ctx.astype(np.float64)
    Vc = v_ctx.astype(np.float64)
    logits = Q @ Kc.T / math.sqrt(Q.shape[1]) + bias[None, :]
    m = logits.max(axis=1, keepdims=True)
    w = np.exp(logits - m)
    z = w.sum(axis=1, keepdims=True)
    out = (w / z) @ Vc
    lse = (m + np.log(z))[:, 0]
    return out, lse


# ---------------------------------------------------------------------------
# One stream: near ring + far bank per (layer, kv head)
# ---------------------------------------------------------------------------


class OracleStream:
    """Runs the hot path for a subset of (layer, kv head) units of one stream.

    codebooks float32 [len(units)][2][G][C][D/G].
    """

    def __init__(self, p: Params, units: Sequence[int], codebooks: np.ndarray):
        if p.ema and p.maintenance:
            raise ValueError("maintenance is defined for running-mean centres only")
        if p.ema and p.warm_frames > 0:
            raise ValueError("the codebook warm-up collects running-mean residuals only")
        self.p = p
        self.folds = 0          # folds done (the first warm_frames collect residuals)
        D = p.head_dim
        self.reservoir = [(np.zeros((0, D), F32), np.zeros((0, D), F32)) for _ in units]
        self.units = list(units)
        self.codebooks = np.array(codebooks, dtype=F32)  # own copy: the warm-up rewrites it
        self.banks = [Bank(p) for _ in self.units]
        self.rings: List[collections.deque] = [collections.deque() for _ in self.units]
        self.frame = 0          # frames appended so far
        self.evicted = 0        # tokens evicted so far (per unit)
        self.near_threshold = 0  # maintenance pair tests within rounding of a threshold

    def append_frame(self, keys: np.ndarray, values: np.ndarray) -> Optional[List[FoldResult]]:
        """Append frame t (keys/values [len(units)][T][D]); if the ring then
        holds more than W frames, evict the oldest and fold it."""
        t = self.frame
        results = None
        for u in range(len(self.units)):
            self.rings[u].append((t, keys[u].astype(F32), values[u].astype(F32)))
        if len(self.rings[0]) > self.p.window_frames:
            results = []
            warm = self.folds < self.p.warm_frames
            for u in range(len(self.units)):
                fe, ke, ve = self.rings[u].popleft()
                if warm:
                    # warm-up fold: no PQ counts; residuals into the reservoir
                    r = fold_frame(self.banks[u], ke, ve, fe, t, dataclasses.replace(self.p, use_pq=False),
                                   self.codebooks[u], collect=True)
                    room = self.p.warm_tokens - len(self.reservoir[u][0])
                    rk, rv = r.residuals
                    self.reservoir[u] = (np.concatenate([self.reservoir[u][0], rk[:room]]),
                                         np.concatenate([self.reservoir[u][1], rv[:room]]))
                    results.append(r)
                else:
                    results.append(fold_frame(self.banks[u], ke, ve, fe, t, self.p, self.codebooks[u]))
                if self.p.maintenance:
                    ms = maintain(self.banks[u], self.rings[u], t, self.p)
                    self.near_threshold += ms["near_threshold"]
            self.folds += 1
            if warm and self.folds == self.p.warm_frames:
                for u in range(len(self.units)):
                    self.codebooks[u] = learn_codebooks(*self.reservoir[u], self.codebooks[u], self.p)
            self.evicted += self.p.tokens_per_frame
        self.frame += 1
        return results

    def near(self, u: int):
        frames = list(self.rings[u])
        if not frames:
            D = self.p.head_dim
            return np.zeros((0, D), F32), np.zeros((0, D), F32)
        return (np.concatenate([f[1] for f in frames]), np.concatenate([f[2] for f in frames]))

    def synthesize(self) -> List[Pseudo]:
        return [synthesize(self.banks[u], self.codebooks[u], self.p) for u in range(len(self.units))]

    def near_positions(self, u: int) -> np.ndarray:
        """Stream positions f * T + j of the near window's tokens, in order."""
        T = self.p.tokens_per_frame
        fr = [f for f, _, _ in self.rings[u]]
        return np.array([f * T + j for f in fr for j in range(T)], dtype=np.int64)

    def context(self, u: int, pseudo: Pseudo):
        kn, vn = self.near(u)
        if self.p.rope_theta > 0:
            kn = rope_rotate(kn, self.near_positions(u), self.p.rope_theta)
            pk = rope_rotate(pseudo.keys, self.banks[u].tau[pseudo.slots], self.p.rope_theta)
            k_ctx = np.concatenate([kn, pk])
            v_ctx = np.concatenate([vn, pseudo.values])
            bias = np.concatenate([np.zeros(len(kn)), pseudo.bias])
            return k_ctx, v_ctx, bias
        k_ctx = np.concatenate([kn, pseudo.keys])
        v_ctx = np.concatenate([vn, pseudo.values])
        bias = np.concatenate([np.zeros(len(kn)), pseudo.bias])
        return k_ctx, v_ctx, bias

    def attend(self, q: np.ndarray, num_kv_heads: int, pseudo: List[Pseudo]):
        """q float32 [L][Tq][Hq][D] -> (O float64 [L][Tq][Hq][D], lse [L][Tq][Hq])
        for the query heads whose kv head is in this stream's unit subset
        (other entries are NaN).  Unit u = layer * Hkv + kv head."""
        L, Tq, Hq, D = q.shape
        grp = Hq // num_kv_heads
        out = np.full((L, Tq, Hq, D), np.nan)
        lse = np.full((L, Tq, Hq), np.nan)
        for ui, u in enumerate(self.units):
            l, h = divmod(u, num_kv_heads)
            k_ctx, v_ctx, bias = self.context(ui, pseudo[ui])
            heads = list(range(h * grp, (h + 1) * grp))
            rows = q[l][:, heads, :].reshape(Tq * grp, D)
            if self.p.rope_theta > 0:
                P = self.frame * self.p.tokens_per_frame
                rows = rope_rotate(rows, P + np.repeat(np.arange(Tq), grp), self.p.rope_theta)
            o, z = attend(rows, k_ctx, v_ctx, bias)
            out[l][:, heads, :] = o.reshape(Tq, grp, D)
            lse[l][:, heads] = z.reshape(Tq, grp)
        return out, lse
