"""Runs the HIP path (through the C-ABI binding) and the CPU oracle side by
side on the same seeded bytes and compares them to the parity bar:

* assignments bit-exact, except near ties: a token whose exact top-2 cost
  margin is below 1e-6 may take another slot only if the oracle's Eq. 1 cost
  of that slot is within 1e-6 of the row minimum; near ties are counted, and
  the device's near-tie counter must equal the oracle's count where the
  oracle follows every unit;
* prototype statistics: mass, n_res, histograms, recency exact; sums and
  sums of squares within relative 1e-4 per row (||a-b|| <= 1e-4 ||b||), and
  bitwise where the test asks for it; spatial mean/covariance within 1e-6;
* pseudo-tokens exact (same bank -> same codes -> same rounding);
* readout within absolute 2e-2 of the oracle's float64 output.

Two modes.  `Pair` runs the oracle free over the whole stream on sampled
units and is authoritative: after a fold in which the device took another
valid slot for a near tie, the device's state of those units is replaced by
the oracle's (protokv_set_state), so the divergence cannot propagate.
`Resync` checks single folds at full size: the device's pre-fold state is
read (protokv_get_state), the oracle folds the same evicted frame from it,
and the device's fold must match; where the device took another valid slot
for a near tie, the oracle folds again with that choice and the banks are
still compared bit for bit.
"""
from __future__ import annotations

import math
import sys
from typing import List, Optional, Sequence

import numpy as np

from oracle import protokv_oracle as O
from paper_2606_26762_amd import protokv as pk
from paper_2606_26762_amd import workloads as W

READOUT_ATOL = 2e-2
LSE_ATOL = 2e-3
STAT_RTOL = 1e-4


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def oracle_params(wl: W.Workload, **kw) -> O.Params:
    p = O.Params(head_dim=wl.head_dim, grid_h=wl.grid_h, grid_w=wl.grid_w,
                 window_frames=wl.window_frames, capacity=wl.capacity, kv_dtype=wl.kv_dtype)
    for k, v in kw.items():
        setattr(p, k, v)
    return p


def gpu_config(wl: W.Workload, p: O.Params, streams: int = 1, max_query_tokens=None) -> pk.Config:
    flags = ((pk.FLAG_PQ if p.use_pq else 0) | (pk.FLAG_MASS_BIAS if p.mass_bias else 0)
             | (pk.FLAG_MAINTENANCE if p.maintenance else 0) | (pk.FLAG_EMA_CENTRES if p.ema else 0)
             | (pk.FLAG_MAH_SQUARED if p.mah_squared else 0) | (pk.FLAG_VAR_ALLOC if p.var_alloc else 0))
    return pk.default_config(
        num_streams=streams, num_layers=wl.num_layers, num_kv_heads=wl.num_kv_heads,
        num_q_heads=wl.num_q_heads, head_dim=wl.head_dim, grid_h=wl.grid_h, grid_w=wl.grid_w,
        window_frames=wl.window_frames, capacity=wl.capacity, pseudo_per_proto=p.S,
        pq_codewords=p.C, beam=max(p.B, p.S), t_idle=p.t_idle,
        max_query_tokens=max_query_tokens or wl.query_tokens,
        kv_dtype=pk.KV_FP32 if wl.kv_dtype == "fp32" else pk.KV_BF16, flags=flags,
        eta=p.eta, lambda_sp=p.lambda_sp, lambda_idle=p.lambda_idle, ridge=p.ridge,
        gamma=p.gamma, eps_k=p.eps_k, eps_v=p.eps_v, alpha=p.alpha, beta=p.beta, rope_theta=p.rope_theta,
        warm_frames=p.warm_frames, warm_tokens=p.warm_tokens, kmeans_epochs=p.kmeans_epochs,
        kmeans_batch=p.kmeans_batch, pseudo_max=p.s_max)


def assert_bank_equal(gb, u: int, ob: O.Bank, C: int, where: str, bitwise: bool):
    """GPU bank rows of unit u (decoded dict) against an oracle Bank."""
    assert np.array_equal(gb["n"][u].astype(np.int64), ob.n), where + " mass"
    assert np.array_equal(gb["n_res"][u].astype(np.int64), ob.n_res), where + " n_res"
    assert np.array_equal(gb["hist_k"][u][:, :, :C].astype(np.int64), ob.hist_k), where + " H^K"
    assert np.array_equal(gb["hist_v"][u][:, :, :C].astype(np.int64), ob.hist_v), where + " H^V"
    assert not gb["hist_k"][u][:, :, C:].any()
    act = ob.n > 0
    assert np.array_equal(gb["tau"][u][act].astype(np.int64), ob.tau[act]), where + " tau"
    for name in ("sum_k", "sum_v", "sq_k", "sq_v"):
        g = gb[name][u][act].astype(np.float64)
        o = getattr(ob, name)[act].astype(np.float64)
        err = np.linalg.norm(g - o, axis=1)
        ref = np.linalg.norm(o, axis=1)
        assert np.all(err <= STAT_RTOL * ref + 1e-30), f"{where} {name} rel {np.max(err / (ref + 1e-30))}"
        if bitwise:
            assert np.array_equal(g, o), f"{where} {name} not bitwise equal"
    assert np.allclose(gb["mu"][u][act], ob.mu[act], atol=1e-6, rtol=0), where + " mu"
    assert np.allclose(gb["sigma"][u][act], ob.sigma[act], atol=1e-6, rtol=1e-6), where + " sigma"
    if bitwise:
        assert np.array_equal(gb["mu"][u][act], ob.mu[act]) and \
            np.array_equal(gb["sigma"][u][act], ob.sigma[act]), where + " spatial not bitwise"


def bank_from_rows(gb, u: int, p: O.Params) -> O.Bank:
    """Oracle Bank holding the decoded rows of unit u of a device state."""
    b = O.Bank(p)
    b.n = gb["n"][u].astype(np.int64)
    b.n_res = gb["n_res"][u].astype(np.int64)
    for name in ("sum_k", "sum_v", "sq_k", "sq_v"):
        setattr(b, name, gb[name][u].astype(np.float32).copy())
    b.hist_k = gb["hist_k"][u][:, :, :p.C].astype(np.int64)
    b.hist_v = gb["hist_v"][u][:, :, :p.C].astype(np.int64)
    b.mu = gb["mu"][u].astype(np.float32).copy()
    b.sigma = gb["sigma"][u].astype(np.float32).copy()
    b.tau = gb["tau"][u].astype(np.int64)
    return b


def rows_from_bank(ob: O.Bank) -> np.ndarray:
    """The documented row layout (uint8) of an oracle Bank, for protokv_set_state."""
    K = len(ob.n)
    d = {"sum_k": ob.sum_k[None], "sum_v": ob.sum_v[None], "sq_k": ob.sq_k[None], "sq_v": ob.sq_v[None],
         "hist_k": ob.hist_k[None], "hist_v": ob.hist_v[None], "n": ob.n[None], "n_res": ob.n_res[None],
         "mu": ob.mu[None], "sigma": ob.sigma[None], "tau": ob.tau[None]}
    return pk.encode_bank(d, 1, K)


def check_assignments(ga: np.ndarray, res: "O.FoldResult", where: str) -> np.ndarray:
    """Assignments equal except near ties, where the device's slot must be a
    valid argmin within 1e-6 of the oracle's minimum cost.  Returns the
    indices of the tokens where the device took another valid slot."""
    bad = np.nonzero(ga != res.assign)[0]
    if len(bad):
        tie = res.margin[bad] < O.NEAR_TIE
        assert np.all(tie), (
            f"{where}: assignment mismatch at tokens {bad[:8].tolist()} gpu {ga[bad[:8]].tolist()} "
            f"oracle {res.assign[bad[:8]].tolist()} margins {res.margin[bad[:8]].tolist()}")
        for j in bad:
            row = res.cost[j - res.n_seed]
            k = int(ga[j])
            assert 0 <= k < len(row) and np.isfinite(row[k]) and row[k] - row.min() < O.NEAR_TIE, (
                f"{where}: token {j}: device slot {k} costs {row[k] if 0 <= k < len(row) else None}, "
                f"{row[k] - row.min() if 0 <= k < len(row) else None} above the minimum")
    return bad


def check_bank_invariants(gb, units: Sequence[int], evicted: int, active: int, C: int, where: str):
    """What holds for every unit at any size without maintenance: the masses
    add up to the tokens evicted, every histogram row sums to n_res, and the
    residual counts add up to the tokens that were not seeds."""
    for u in units:
        n = gb["n"][u].astype(np.int64)
        assert int(n.sum()) == evicted, f"{where} unit {u}: sum n {int(n.sum())} != evicted {evicted}"
        assert int((n > 0).sum()) == active and np.all(n[:active] > 0), f"{where} unit {u}: active prefix"
        nres = gb["n_res"][u].astype(np.int64)
        for name in ("hist_k", "hist_v"):
            h = gb[name][u].astype(np.int64)
            assert not h[:, :, C:].any()
            assert np.array_equal(h.sum(axis=2), np.repeat(nres[:, None], 8, axis=1)), f"{where} unit {u} {name}"
        assert int(nres.sum()) == evicted - active, f"{where} unit {u}: sum n_res"


class Resync:
    """Full-size run: every unit of every stream on the GPU, frames drawn on
    the device.  At chosen frames the device's pre-fold state is read, the
    oracle folds the sampled (stream, unit) pairs from it with the evicted
    frame's bytes, and the device's fold must match: assignments except near
    ties (each a valid argmin), rows bitwise (after an excused near tie the
    oracle folds again with the device's valid choice).  The readout check
    synthesizes from the device's bank in the oracle and attends over the
    sampled units' near window."""

    def __init__(self, wl: W.Workload, sample: Sequence, streams: int = 1, seed: int = 5,
                 cb_samples: int = 1024, **pkw):
        import collections
        import torch
        self.torch = torch
        self.wl = wl
        self.p = oracle_params(wl, **pkw)
        self.streams = streams
        self.sample = [tuple(x) for x in sample]          # (stream, unit)
        self.cb = W.make_codebooks_device(wl, n_streams=streams, samples=cb_samples, iters=8)
        self.cfg = gpu_config(wl, self.p, streams)
        self.gpu = pk.ProtoKV(self.cfg, self.cb.reshape(-1, *self.cb.shape[2:]))
        self.dev = W.DeviceStream(wl, n_streams=streams, seed=seed)
        self.ring = collections.deque(maxlen=wl.window_frames + 1)
        self.t = 0
        self.folds_checked = 0
        self.near_ties = 0
        self.excused = 0
        self._sidx = torch.tensor([s for s, _ in self.sample], device="cuda")
        self._uidx = torch.tensor([u for _, u in self.sample], device="cuda")

    def _sampled(self, x):
        wl = self.wl
        xf = x.view(self.streams, wl.units, wl.tokens_per_frame, wl.head_dim)
        return xf[self._sidx, self._uidx].float().cpu().numpy()

    def step(self, check: bool = False):
        wl = self.wl
        k, v = self.dev.next_frame()
        self.ring.append((self.t, self._sampled(k), self._sampled(v)))
        evict = self.t >= wl.window_frames
        streams = sorted({s for s, _ in self.sample})
        if check and evict:
            before = {s: self.gpu.get_state(s).bank() for s in streams}
        self.gpu.append_frame(list(range(self.streams)), k, v)
        self.gpu.fold()
        if check and evict:
            fe, ke, ve = self.ring[0]
            assert fe == self.t - wl.window_frames
            after = {s: self.gpu.read_bank(s) for s in streams}
            assign = {s: self.gpu.read_assignments(s) for s in streams}
            for i, (s, u) in enumerate(self.sample):
                where = f"frame {self.t} stream {s} unit {u}"
                ob = bank_from_rows(before[s], u, self.p)
                res = O.fold_frame(ob, ke[i], ve[i], fe, self.t, self.p, self.cb[s][u])
                excused = check_assignments(assign[s][u], res, where)
                self.near_ties += res.near_ties
                if len(excused):
                    self.excused += len(excused)
                    ob = bank_from_rows(before[s], u, self.p)
                    O.fold_frame(ob, ke[i], ve[i], fe, self.t, self.p, self.cb[s][u], choose=assign[s][u])
                assert_bank_equal(after[s], u, ob, self.p.C, where, bitwise=True)
                self.folds_checked += 1
        self.t += 1

    def check_invariants(self):
        """Mass, histogram and residual-count identities on every unit of every stream."""
        wl = self.wl
        for s in range(self.streams):
            info = self.gpu.stream_info(s)
            gb = self.gpu.read_bank(s)
            check_bank_invariants(gb, range(wl.units), int(info.evicted_tokens), int(info.active_slots),
                                  self.p.C, f"stream {s}")

    def check_readout(self, stream: int):
        """Synthesis (exact rows) and attention (abs 2e-2) of the sampled units of `stream`."""
        torch, wl = self.torch, self.wl
        self.gpu.synthesize(stream)
        gb = self.gpu.read_bank(stream)
        q = self.dev.query()
        # first readout before the rows are read back (bf16, S >= 5: rows
        # formed inside the readout), second one over the written rows
        outs = []
        for _ in range(2):
            o, lse = self.gpu.attend(stream, q)
            torch.cuda.synchronize()
            outs.append((o.float().cpu().numpy(), lse.cpu().numpy()))
            if len(outs) == 1:
                gk, gv, gbias = self.gpu.read_pseudo()
        qh = q.float().cpu().numpy()
        grp = wl.num_q_heads // wl.num_kv_heads
        near = list(self.ring)[-min(self.t, wl.window_frames):]
        worst = 0.0
        for i, (s, u) in enumerate(self.sample):
            if s != stream:
                continue
            ob = bank_from_rows(gb, u, self.p)
            ps = O.synthesize(ob, self.cb[s][u], self.p)
            n = len(ps.keys)
            assert n == int((ob.n > 0).sum()) * self.p.S
            assert np.array_equal(gk[u][:n], ps.keys), f"stream {s} unit {u}: pseudo keys differ"
            assert np.array_equal(gv[u][:n], ps.values), f"stream {s} unit {u}: pseudo values differ"
            slots, first = np.unique(ps.slots, return_index=True)
            assert np.allclose(gbias[u][slots], ps.bias[first], rtol=1e-6, atol=1e-6)
            kn = np.concatenate([f[1][i] for f in near])
            vn = np.concatenate([f[2][i] for f in near])
            k_ctx = np.concatenate([kn, ps.keys])
            v_ctx = np.concatenate([vn, ps.values])
            bias = np.concatenate([np.zeros(len(kn)), ps.bias])
            l, h = divmod(u, wl.num_kv_heads)
            heads = list(range(h * grp, (h + 1) * grp))
            rows = qh[l][:, heads, :].reshape(-1, wl.head_dim)
            oo, ol = O.attend(rows, k_ctx, v_ctx, bias)
            for which, (go, gl) in zip(("formed rows", "written rows"), outs):
                d = np.abs(go[l][:, heads].reshape(-1, wl.head_dim) - oo).max()
                dl = np.abs(gl[l][:, heads].reshape(-1) - ol).max()
                assert d <= READOUT_ATOL, f"stream {s} unit {u} ({which}): readout abs err {d}"
                assert dl <= LSE_ATOL, f"stream {s} unit {u} ({which}): lse abs err {dl}"
                worst = max(worst, float(d))
        return worst


class Pair:
    """GPU handle over all units of `streams` streams + a free-running oracle
    over the sampled units of the streams in `oracle_streams` (default all)."""

    def __init__(self, wl: W.Workload, sample: Optional[Sequence[int]] = None, streams: int = 1,
                 cb_samples: int = 1024, cb_iters: int = 8, max_query_tokens=None,
                 oracle_streams: Optional[Sequence[int]] = None, **pkw):
        import torch
        self.torch = torch
        self.wl = wl
        self.p = oracle_params(wl, **pkw)
        self.streams = streams
        self.sample = list(range(wl.units)) if sample is None else list(sample)
        self.tracked = list(range(streams)) if oracle_streams is None else list(oracle_streams)
        if streams * wl.units > 1024 and self.p.C == 16:
            # many units: the same Lloyd recipe, batched on the device
            self.cb = W.make_codebooks_device(wl, n_streams=streams, samples=cb_samples, iters=cb_iters)
        else:
            self.cb = np.stack([W.make_codebooks(wl, stream=s, samples=cb_samples, iters=cb_iters,
                                                 C=self.p.C) for s in range(streams)])
        self.cfg = gpu_config(wl, self.p, streams, max_query_tokens)
        self.gpu = pk.ProtoKV(self.cfg, self.cb)
        self.host = {s: W.HostStream(wl, stream=s, units=self.sample) for s in self.tracked}
        self.oracle = {s: O.OracleStream(self.p, self.sample, self.cb[s][self.sample]) for s in self.tracked}
        full = len(self.sample) == wl.units and len(self.tracked) == streams
        self.dev = None if full else W.DeviceStream(wl, n_streams=streams, seed=99)
        self.dtype = torch.float32 if wl.kv_dtype == "fp32" else torch.bfloat16
        self.near_ties = 0          # oracle near ties over every checked fold
        self.excused = 0            # tokens where the device took another valid slot
        self.resyncs = 0            # device states replaced by the oracle's after an excused token
        self.assign_checked = 0
        self.frames = [0] * streams
        self._rows_pending = None
        self._idx = torch.tensor(self.sample, device="cuda")

    # -- input -------------------------------------------------------------
    def _frames(self, streams: Sequence[int]):
        """One frame of each listed stream as device tensors [n][L][Hkv][T][D]
        (device-drawn, the tracked streams' sampled units overwritten with
        host bytes) and the host bytes of the tracked streams."""
        torch, wl = self.torch, self.wl
        shape = (len(streams), wl.num_layers, wl.num_kv_heads, wl.tokens_per_frame, wl.head_dim)
        if self.dev is not None:
            ka, va = self.dev.next_frame()
            if list(streams) != list(range(self.streams)):
                sel = torch.tensor(list(streams), device="cuda")
                ka, va = ka.index_select(0, sel).contiguous(), va.index_select(0, sel).contiguous()
        else:
            ka = torch.empty(shape, dtype=self.dtype, device="cuda")
            va = torch.empty_like(ka)
        host = {}
        for i, s in enumerate(streams):
            if s not in self.oracle:
                continue
            kh, vh = self.host[s].next_frame()
            host[s] = (kh, vh)
            kf = ka[i].view(wl.units, wl.tokens_per_frame, wl.head_dim)
            vf = va[i].view(wl.units, wl.tokens_per_frame, wl.head_dim)
            kf[self._idx] = torch.from_numpy(kh).to("cuda", self.dtype)
            vf[self._idx] = torch.from_numpy(vh).to("cuda", self.dtype)
        return ka, va, host

    # -- stepping ------------------------------------------------------------
    def step(self, streams: Optional[Sequence[int]] = None, check_assign: bool = True):
        """Append one frame to each listed stream (one batched call), fold,
        and compare the assignments of the sampled units of the tracked
        streams.  A device choice that differs from the oracle's is accepted
        only for a near tie (a valid argmin), and then the oracle's state of
        the sampled units is written back to the device."""
        streams = list(range(self.streams)) if streams is None else list(streams)
        K, V, host = self._frames(streams)
        results = {s: self.oracle[s].append_frame(*host[s]) for s in host}
        self.gpu.append_frame(streams, K, V)
        self.gpu.fold()
        for s in streams:
            self.frames[s] += 1
            res = results.get(s)
            if res is None:
                continue
            if self.p.maintenance:
                assert self.oracle[s].near_threshold == 0, (
                    f"stream {s} frame {self.frames[s] - 1}: a maintenance pair test fell within rounding "
                    f"of its threshold (the device may decide it the other way)")
            self.near_ties += sum(r.near_ties for r in res)
            if not check_assign:
                continue
            ga = self.gpu.read_assignments(s)
            excused = 0
            for i, u in enumerate(self.sample):
                bad = check_assignments(ga[u], res[i], f"stream {s} frame {self.frames[s] - 1} unit {u}")
                excused += len(bad)
                self.assign_checked += len(res[i].assign)
            if excused:
                self.excused += excused
                self.resync(s)

    def resync(self, stream: int):
        """Write the oracle's banks of the sampled units into the device's state."""
        st = self.gpu.get_state(stream)
        for i, u in enumerate(self.sample):
            st.set_bank_rows(u, rows_from_bank(self.oracle[stream].banks[i]))
        self.gpu.set_state(stream, st)
        self.resyncs += 1

    def check_near_tie_counter(self):
        """With every unit of every stream followed, the device's near-tie
        counter equals the oracle's count."""
        if len(self.sample) == self.wl.units and len(self.tracked) == self.streams:
            c = self.gpu.counters()
            assert int(c.near_ties) == self.near_ties, (int(c.near_ties), self.near_ties)

    # -- checks --------------------------------------------------------------
    def check_bank(self, stream: int = 0, bitwise: bool = False):
        gb = self.gpu.read_bank(stream)
        for i, u in enumerate(self.sample):
            assert_bank_equal(gb, u, self.oracle[stream].banks[i], self.p.C,
                              f"stream {stream} unit {u}", bitwise)
        return gb

    def synthesize(self, stream: int = 0, check: bool = True):
        """GPU and oracle synthesis.  The GPU's rows are compared after the
        next attend of this stream: for bf16 KV with S >= 5 that attend forms
        the rows itself, and reading them back first would hand it written
        rows instead."""
        self.gpu.synthesize(stream)
        pseudo = self.oracle[stream].synthesize()
        self._rows_pending = (stream, pseudo) if check else None
        return pseudo

    def check_rows(self):
        """Pseudo-token rows and biases read back (written on demand) against the oracle's."""
        if self._rows_pending is None:
            return
        stream, pseudo = self._rows_pending
        self._rows_pending = None
        gk, gv, gbias = self.gpu.read_pseudo()
        gcounts = self.gpu.read_pseudo_counts() if self.p.var_alloc else None
        S = self.p.S
        for i, u in enumerate(self.sample):
            ps = pseudo[i]
            n = len(ps.keys)
            assert n == int((self.oracle[stream].banks[i].n > 0).sum()) * S
            if self.p.rope_theta > 0:
                # keys rotated at tau_k: float32 on the GPU, float64 in the
                # oracle, so within one unit of the KV dtype's last place
                # (plus cancellation inside a rotated pair)
                tau = self.oracle[stream].banks[i].tau[ps.slots]
                want = O.round_kv(O.rope_rotate(ps.keys, tau, self.p.rope_theta).astype(np.float32),
                                  self.p.kv_dtype).astype(np.float64)
                ulp = 2.0 ** -7 if self.p.kv_dtype == "bf16" else 2.0 ** -22
                tol = ulp * np.abs(want) + 2.0 ** -20 * np.linalg.norm(want, axis=1, keepdims=True)
                err = np.abs(gk[u][:n].astype(np.float64) - want)
                assert np.all(err <= tol), f"unit {u}: rotated pseudo keys differ by {np.max(err - tol)} beyond tol"
            else:
                assert np.array_equal(gk[u][:n], ps.keys), f"unit {u}: pseudo keys differ"
            assert np.array_equal(gv[u][:n], ps.values), f"unit {u}: pseudo values differ"
            slots, first = np.unique(ps.slots, return_index=True)
            assert np.allclose(gbias[u][slots], ps.bias[first], rtol=1e-6, atol=1e-6)
            if self.p.var_alloc:
                want = O.pseudo_counts(self.oracle[stream].banks[i], self.oracle[stream].codebooks[i], self.p)
                assert np.array_equal(gcounts[u].astype(np.int64), want), f"unit {u}: pseudo-token counts differ"

    def query(self, rng: np.random.Generator, tq: Optional[int] = None) -> np.ndarray:
        wl = self.wl
        tq = tq or wl.query_tokens
        q = rng.standard_normal((wl.num_layers, tq, wl.num_q_heads, wl.head_dim))
        # a third of the rows look for a sampled key direction, for peaked attention
        q[:, ::3] *= 3.0
        return W.quantize(q, wl.kv_dtype)

    def attend(self, q: np.ndarray, pseudo, stream: int = 0):
        torch, wl = self.torch, self.wl
        qd = torch.from_numpy(q).to("cuda", self.dtype).contiguous()
        o, lse = self.gpu.attend(stream, qd)
        torch.cuda.synchronize()
        go = o.float().cpu().numpy()
        gl = lse.cpu().numpy()
        oo, ol = self.oracle[stream].attend(q, wl.num_kv_heads, pseudo)
        grp = wl.num_q_heads // wl.num_kv_heads
        worst = 0.0
        for u in self.sample:
            l, h = divmod(u, wl.num_kv_heads)
            heads = list(range(h * grp, (h + 1) * grp))
            d = np.abs(go[l][:, heads] - oo[l][:, heads]).max()
            worst = max(worst, float(d))
            assert d <= READOUT_ATOL, f"unit {u}: readout abs err {d}"
            dl = np.abs(gl[l][:, heads] - ol[l][:, heads]).max()
            assert dl <= LSE_ATOL, f"unit {u}: lse abs err {dl}"
        if self._rows_pending is not None and self._rows_pending[0] == stream:
            self.check_rows()
        return worst, go, gl
