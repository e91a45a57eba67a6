"""GPU: the stream state calls (protokv_get_state / protokv_set_state).

A stream's state is the near tier, the prototype bank, its codebooks and its
position (Alg. "ProtoKV Streaming Update" carries B_near and B_far from one
token to the next).  Checked here: a state built on the host from the
oracle's bank, loaded into the device, gives a device fold equal to the
oracle's (bitwise); a state read from one handle and loaded into a fresh
handle continues identically; malformed blobs are refused on the host; and
the eviction limit of the exact decode is enforced at append.  Each test
prints its case before any GPU step.
"""
import numpy as np
import pytest

from paper_2606_26762_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_26762_amd import protokv as pk
    pk.lib()
    yield


def H():
    from tests import gpu_harness
    return gpu_harness


def _small():
    return W.WORKLOADS["7b"].with_(num_layers=1, num_kv_heads=2, num_q_heads=4, grid_h=7, grid_w=7,
                                   frames=14, window_frames=2, capacity=64, query_tokens=6)


def test_oracle_state_loaded_into_the_device_folds_like_the_oracle():
    """The oracle runs a stream alone; the device receives its bank and ring
    through protokv_set_state and folds the next frames; every fold's
    assignments and bank equal the oracle's, then the readout."""
    import torch
    from oracle import protokv_oracle as O
    h = H()
    wl = _small()
    h.log("case: oracle state -> device, T=49 K=64 W=2")
    p = h.oracle_params(wl)
    cb = W.make_codebooks(wl, samples=512, iters=6)
    gen = W.HostStream(wl)
    ora = O.OracleStream(p, list(range(wl.units)), cb)
    frames = [gen.next_frame() for _ in range(wl.frames)]
    for k, v in frames[:8]:
        ora.append_frame(k, v)
    gpu = h.pk.ProtoKV(h.gpu_config(wl, p), cb)
    st = gpu.get_state(0)
    hd = st.header
    assert (hd.frames, hd.evicted_tokens, hd.active_slots) == (0, 0, 0)
    # the oracle's position, ring (slot f mod (W + 1)) and banks
    T = wl.tokens_per_frame
    hd.frames = 8
    hd.evicted_tokens = (8 - wl.window_frames) * T
    hd.folds = 8 - wl.window_frames
    hd.active_slots = int((ora.banks[0].n > 0).sum())
    st.blob[:128] = np.frombuffer(bytes(hd), dtype=np.uint8)
    es = 2
    ring_k = st.blob[hd.off_ring_k:hd.off_ring_k + wl.units * (wl.window_frames + 1) * T * 128 * es].view(np.uint16)
    ring_v = st.blob[hd.off_ring_v:hd.off_ring_v + wl.units * (wl.window_frames + 1) * T * 128 * es].view(np.uint16)
    ring_k = ring_k.reshape(wl.units, wl.window_frames + 1, T, 128)
    ring_v = ring_v.reshape(wl.units, wl.window_frames + 1, T, 128)
    for f in range(8 - wl.window_frames - 1, 8):
        k, v = frames[f]
        ring_k[:, f % (wl.window_frames + 1)] = W.to_bf16_bits(k)
        ring_v[:, f % (wl.window_frames + 1)] = W.to_bf16_bits(v)
    for u in range(wl.units):
        st.set_bank_rows(u, h.rows_from_bank(ora.banks[u]))
    gpu.set_state(0, st)
    info = gpu.stream_info(0)
    assert (info.frames, info.active_slots, info.pending) == (8, hd.active_slots, 0)
    back = gpu.read_bank(0)
    for u in range(wl.units):
        h.assert_bank_equal(back, u, ora.banks[u], p.C, f"loaded unit {u}", bitwise=True)
    for f in range(8, wl.frames):
        k, v = frames[f]
        res = ora.append_frame(k, v)
        kd = torch.from_numpy(k).to("cuda", torch.bfloat16).view(1, 1, 2, T, 128).contiguous()
        vd = torch.from_numpy(v).to("cuda", torch.bfloat16).view(1, 1, 2, T, 128).contiguous()
        gpu.append_frame([0], kd, vd)
        gpu.fold()
        ga = gpu.read_assignments(0)
        gb = gpu.read_bank(0)
        for u in range(wl.units):
            assert not len(h.check_assignments(ga[u], res[u], f"frame {f} unit {u}"))
            h.assert_bank_equal(gb, u, ora.banks[u], p.C, f"frame {f} unit {u}", bitwise=True)
    gpu.synthesize(0)
    pseudo = ora.synthesize()
    q = W.quantize(np.random.default_rng(8).standard_normal((1, wl.query_tokens, 4, 128)), "bf16")
    o, _ = gpu.attend(0, torch.from_numpy(q).to("cuda", torch.bfloat16).contiguous())
    torch.cuda.synchronize()
    oo, _ = ora.attend(q, wl.num_kv_heads, pseudo)
    err = float(np.abs(o.float().cpu().numpy() - oo).max())
    h.log(f"readout err {err:.2e}")
    assert err <= h.READOUT_ATOL


@pytest.mark.parametrize("rope", [False, True])
def test_state_round_trip_continues_identically(rope):
    """get_state of a running stream, set_state into stream 1 of another
    handle: both continue over the same frames with identical assignments,
    banks and readouts (with rotary positions the rotated ring travels too)."""
    import torch
    h = H()
    wl = _small()
    h.log(f"case: state round trip rope={rope}")
    kw = dict(rope_theta=1e4) if rope else {}
    a = h.Pair(wl, **kw)
    for _ in range(7):
        a.step()
    st = a.gpu.get_state(0)
    cfg2 = h.gpu_config(wl, a.p, streams=2)
    b = h.pk.ProtoKV(cfg2, np.concatenate([a.cb, a.cb]))
    b.set_state(1, st)
    st2 = b.get_state(1)
    assert np.array_equal(st.blob, st2.blob)
    rng = np.random.default_rng(9)
    for f in range(5):
        k = torch.from_numpy(W.quantize(rng.standard_normal((1, 1, 2, 49, 128)), "bf16")).to("cuda", torch.bfloat16)
        v = torch.from_numpy(W.quantize(rng.standard_normal((1, 1, 2, 49, 128)), "bf16")).to("cuda", torch.bfloat16)
        a.gpu.append_frame([0], k, v)
        a.gpu.fold()
        b.append_frame([1], k, v)
        b.fold()
        assert np.array_equal(a.gpu.read_assignments(0), b.read_assignments(1))
    ba, bb = a.gpu.get_state(0), b.get_state(1)
    assert np.array_equal(ba.blob, bb.blob)
    q = torch.from_numpy(W.quantize(rng.standard_normal((1, 6, 4, 128)), "bf16")).to("cuda", torch.bfloat16)
    a.gpu.synthesize(0)
    oa, la = a.gpu.attend(0, q)
    b.synthesize(1)
    ob, lb = b.attend(1, q)
    torch.cuda.synchronize()
    assert torch.equal(oa, ob) and torch.equal(la, lb)


def test_malformed_states_are_refused_and_the_eviction_limit_holds():
    """Host-side checks of set_state (nothing is copied on a refusal), the
    state machine around it, and the exact decode's eviction limit: a stream
    positioned just below it may append until the next eviction would pass it."""
    import torch
    h = H()
    pk = h.pk
    wl = W.WORKLOADS["7b"].with_(num_layers=1, num_kv_heads=1, num_q_heads=1, grid_h=2, grid_w=2,
                                 frames=4, window_frames=1, capacity=4, query_tokens=2)
    h.log("case: malformed states and the eviction limit")
    pair = h.Pair(wl)
    for _ in range(3):
        pair.step()
    g = pair.gpu
    good = g.get_state(0)

    def refused(mutate, status=1):
        st = pk.State(good.blob.copy(), "bf16")
        mutate(st)
        with pytest.raises(pk.ProtoKVError) as e:
            g.set_state(0, st)
        assert e.value.status == status

    def hdr(**kw):
        def m(st):
            for k2, v2 in kw.items():
                setattr(st.header, k2, v2)
            st.blob[:128] = np.frombuffer(bytes(st.header), dtype=np.uint8)
        return m
    refused(hdr(magic=0))
    refused(hdr(capacity=8))
    refused(hdr(frames=5))                        # evicted / folds no longer follow from frames
    refused(hdr(active_slots=3))                  # n > 0 beyond the active prefix
    bank = good.bank()

    def bad_hist(st):
        b2 = {k2: v2.copy() for k2, v2 in bank.items()}
        b2["hist_k"][0, 0, 3, 0] += 1             # a histogram row no longer sums to n_res
        st.set_bank_rows(0, pk.encode_bank({k2: v2[:1] for k2, v2 in b2.items()}, 1, 4))
    refused(bad_hist)
    with pytest.raises(pk.ProtoKVError) as e:
        g.set_state(0, good.blob[:-256])
    assert e.value.status == 1
    # pending eviction: state calls refused
    k = torch.zeros((1, 1, 1, 4, 128), dtype=torch.bfloat16, device="cuda")
    g.append_frame([0], k, k)
    with pytest.raises(pk.ProtoKVError) as e:
        g.get_state(0)
    assert e.value.status == 4
    g.fold()
    # the eviction limit: T = 4, W = 1; a stream with (frames - 1) * 4 evicted
    # tokens may append while the total stays <= PROTOKV_MAX_EVICTED_TOKENS
    st = g.get_state(0)
    lim = pk.MAX_EVICTED_TOKENS
    frames = lim // 4 + 1            # evicted = (frames - 1) * 4 = 16777212 <= lim
    hdr(frames=frames, evicted_tokens=(frames - 1) * 4, folds=frames - 1)(st)
    g.set_state(0, st)
    info = g.stream_info(0)
    assert info.evicted_tokens == (frames - 1) * 4 and info.evicted_tokens + 4 > lim
    with pytest.raises(pk.ProtoKVError) as e:
        g.append_frame([0], k, k)
    assert e.value.status == 2
    assert g.stream_info(0).frames == frames and g.stream_info(0).pending == 0


@pytest.mark.parametrize("S", [8, 5])
def test_decode_on_crafted_histograms(S):
    """The decode (exact top-S residual tuples, Alg. "DecodeTopSResidualModes")
    on histograms made for ties, loaded through protokv_set_state: every
    codeword with the same count (all products equal: the packed tuple
    decides), one count vector permuted per subspace (products collide
    across tuples), random counts up to 3, and counts whose top products
    pass 2^64 (the 128-bit merge).  Pseudo-token rows bitwise against the
    oracle's, and the readout."""
    import torch
    from oracle import protokv_oracle as O
    h = H()
    wl = _small()
    h.log(f"case: crafted histograms, S={S}, T=49 K=64 W=2")
    p = h.oracle_params(wl, S=S)
    cb = W.make_codebooks(wl, samples=512, iters=6)
    gen = W.HostStream(wl)
    ora = O.OracleStream(p, list(range(wl.units)), cb)
    frames = [gen.next_frame() for _ in range(8)]
    for k, v in frames:
        ora.append_frame(k, v)
    rng = np.random.default_rng(90 + S)
    C, G = p.C, 8
    for u in range(wl.units):
        b = ora.banks[u]
        for k in np.nonzero(b.n > 0)[0]:
            kind = k % 4
            for hist in (b.hist_k, b.hist_v):
                if kind == 0:
                    nres = 3 * C
                    hist[k] = 3
                elif kind == 1:
                    base = np.array([6, 4, 4, 3, 3, 2, 2, 1, 1, 1, 1, 0, 0, 0, 0, 0], dtype=np.int64)[:C]
                    nres = int(base.sum())
                    for g in range(G):
                        hist[k, g] = base[rng.permutation(C)]
                elif kind == 2:
                    nres = 20
                    for g in range(G):
                        hist[k, g] = rng.multinomial(nres, np.full(C, 1.0 / C))
                else:
                    nres = 60000
                    for g in range(G):
                        hist[k, g] = rng.multinomial(nres, rng.dirichlet(np.full(C, 0.5)))
            b.n_res[k] = nres
            b.n[k] = max(int(b.n[k]), nres + 1)
    gpu = h.pk.ProtoKV(h.gpu_config(wl, p), cb)
    st = gpu.get_state(0)
    hd = st.header
    T, Wf = wl.tokens_per_frame, wl.window_frames
    hd.frames = 1300   # enough evicted tokens for n_res = 60000
    hd.folds = hd.frames - Wf
    hd.evicted_tokens = hd.folds * T
    hd.active_slots = int((ora.banks[0].n > 0).sum())
    assert all(int((b.n > 0).sum()) == hd.active_slots for b in ora.banks)
    st.blob[:128] = np.frombuffer(bytes(hd), dtype=np.uint8)
    ring = wl.units * (Wf + 1) * T * 128 * 2
    ring_k = st.blob[hd.off_ring_k:hd.off_ring_k + ring].view(np.uint16).reshape(wl.units, Wf + 1, T, 128)
    ring_v = st.blob[hd.off_ring_v:hd.off_ring_v + ring].view(np.uint16).reshape(wl.units, Wf + 1, T, 128)
    # the oracle's near window (its last W frames) as the device's last W frames
    for i, f in enumerate(range(hd.frames - Wf, hd.frames)):
        k, v = frames[8 - Wf + i]
        ring_k[:, f % (Wf + 1)] = W.to_bf16_bits(k)
        ring_v[:, f % (Wf + 1)] = W.to_bf16_bits(v)
    for u in range(wl.units):
        st.set_bank_rows(u, h.rows_from_bank(ora.banks[u]))
    gpu.set_state(0, st)
    gpu.synthesize(0)
    pseudo = ora.synthesize()
    q = W.quantize(np.random.default_rng(9).standard_normal((1, wl.query_tokens, 4, 128)), "bf16")
    o, _ = gpu.attend(0, torch.from_numpy(q).to("cuda", torch.bfloat16).contiguous())  # rows formed in LDS
    torch.cuda.synchronize()
    oo, _ = ora.attend(q, wl.num_kv_heads, pseudo)
    err = float(np.abs(o.float().cpu().numpy() - oo).max())
    gk, gv, gbias = gpu.read_pseudo()
    for u in range(wl.units):
        ps = pseudo[u]
        n = len(ps.keys)
        assert np.array_equal(gk[u][:n], ps.keys), f"unit {u}: pseudo keys differ"
        assert np.array_equal(gv[u][:n], ps.values), f"unit {u}: pseudo values differ"
    h.log(f"readout err {err:.2e}, rows bitwise")
    assert err <= h.READOUT_ATOL
